"""Tolerance helpers shared by the GPU parity tests.

Floating point tensors pass iff max_i |x_i - y_i| / (|y_i| + RMS(y)) <= rtol,
with y the fp64 oracle: relative where values are large, relative to the
tensor's RMS where a sum cancels to near zero.  Norms and clip factors are
positive and use plain relative error.  Integer results compare exactly.
"""
import numpy as np

# bf16-input workloads: the oracle reads the very bf16 values the kernels
# read and every product of two bf16 values is exact in fp32, so the only
# differences are fp32 rounding of the sums, as for fp32 inputs; the tests
# hold them to the fp32 bound (the contract's bf16 bound is 2e-2).
RTOL = {"f32": 1e-4, "bf16": 1e-4}


def g12_error(x, y) -> float:
    x = np.asarray(x, dtype=np.float64).reshape(-1)
    y = np.asarray(y, dtype=np.float64).reshape(-1)
    assert x.shape == y.shape, (x.shape, y.shape)
    if y.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(y * y)))
    den = np.abs(y) + rms
    den[den == 0] = 1.0
    return float(np.max(np.abs(x - y) / den))


def assert_g12(x, y, rtol, what=""):
    err = g12_error(x, y)
    assert err <= rtol, "%s: error %.3g > %.3g" % (what, err, rtol)
    return err


def assert_rel(x, y, rtol, what=""):
    x = np.asarray(x, dtype=np.float64).reshape(-1)
    y = np.asarray(y, dtype=np.float64).reshape(-1)
    with np.errstate(divide="ignore", invalid="ignore"):
        err = np.max(np.abs(x - y) / np.maximum(np.abs(y), 1e-30)) if y.size else 0.0
    assert err <= rtol, "%s: relative error %.3g > %.3g" % (what, err, rtol)
    return err
