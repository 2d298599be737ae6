"""Oracle for the DP-SGD gradient step -- TEST INFRASTRUCTURE ONLY.

Plain double-precision CPU reference (``dp_oracle.c``) of what the HIP library
computes.  Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import it; the product path never does.  It shares no
code with the HIP library; both are fed from ``paper_2109_12298_amd.workloads``,
which draws numbers only.

The Python layer marshals numpy arrays (everything widened to float64; ids
int64) into the C functions and strings the steps together in the order of
the DP-SGD step (section 1 and figure 1 of the paper): per-sample gradients,
per-sample l2 norms over all parameters, clip factors, clipped sum, noise,
division.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dp_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_d = ctypes.POINTER(ctypes.c_double)
_i64 = ctypes.POINTER(ctypes.c_int64)
_u32 = ctypes.POINTER(ctypes.c_uint32)
_L = ctypes.c_long


def build(force: bool = True) -> str:
    """Compile dp_oracle.c into liboracle.so with gcc (IEEE fp64, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
               "-ffp-contract=off", "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        L = ctypes.CDLL(_LIB)
        L.dpo_linear.argtypes = [_d, _d, _L, _L, _L, _L, ctypes.c_double, _d, _d]
        L.dpo_conv2d.argtypes = [_d, _d] + [_L] * 13 + [ctypes.c_double, _d, _d]
        L.dpo_embedding.argtypes = [_i64, _d, _L, _L, _L, _L, ctypes.c_double, _i64, _i64, _d, _L]
        L.dpo_embedding.restype = _L
        L.dpo_layernorm.argtypes = [_d, _d, _L, _L, _L, ctypes.c_double, _d, _d]
        L.dpo_groupnorm.argtypes = [_d, _d, _L, _L, _L, ctypes.c_double, _d, _d]
        L.dpo_lstm_forward.argtypes = [_d, _d, _d, _d, _d, _L, _L, _L, _L, _d, _d, _d]
        L.dpo_lstm_backward.argtypes = [_d, _d, _d, _d, _d, _L, _L, _L, _d]
        L.dpo_sqnorm_accumulate.argtypes = [_d, _L, _L, _d]
        L.dpo_norms.argtypes = [_d, _L, _d]
        L.dpo_clip_factors.argtypes = [_d, _L, ctypes.c_double, _d]
        L.dpo_clip_sum.argtypes = [_d, _d, _L, _L, _d]
        L.dpo_clip_sum_embedding.argtypes = [_i64, _i64, _d, _d, _L, _L, _L, _d]
        L.dpo_philox4x32_10.argtypes = [_u32, _u32, _u32]
        L.dpo_philox_normals.argtypes = [_L, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32, _u32, _d]
        L.dpo_num_threads.restype = ctypes.c_int
        L.dpo_set_num_threads.argtypes = [ctypes.c_int]
        L.dpo_add_noise.argtypes = [_d, _L, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32,
                                    ctypes.c_double, ctypes.c_double, ctypes.c_double, _d]
        _lib = L
    return _lib


def num_threads() -> int:
    return int(lib().dpo_num_threads())


def set_num_threads(n: int) -> None:
    """OpenMP threads for the parallel loops (timing only; results do not depend on it)."""
    lib().dpo_set_num_threads(int(n))


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a: np.ndarray, t=_d):
    return a.ctypes.data_as(t)


# --------------------------------------------------------------------------
# per-sample gradients
# --------------------------------------------------------------------------

def linear_grad(A, B, scale: float = 1.0, bias: bool = True):
    """Per-sample Linear grads (appendix "Vectorized Computation").

    A [N, T, d_in] or [N, d_in]; B [N, T, d_out] or [N, d_out].
    Returns gW [N, d_out, d_in] and gb [N, d_out] (None without bias)."""
    A = _f64(A); B = _f64(B)
    if A.ndim == 2:
        A = A[:, None, :]; B = B[:, None, :]
    N, T, din = A.shape
    dout = B.shape[2]
    gW = np.empty((N, dout, din)); gb = np.empty((N, dout)) if bias else None
    lib().dpo_linear(_p(A), _p(B), N, T, din, dout, float(scale), _p(gW),
                     _p(gb) if bias else None)
    return gW, gb


def conv2d_grad(X, GY, k, stride=(1, 1), pad=(0, 0), scale: float = 1.0, bias: bool = True):
    """Per-sample Conv2d weight/bias grads by direct loops (groups=1, dilation=1)."""
    X = _f64(X); GY = _f64(GY)
    N, Cin, H, W = X.shape
    Cout, Ho, Wo = GY.shape[1:]
    kh, kw = k
    gW = np.empty((N, Cout, Cin, kh, kw)); gb = np.empty((N, Cout)) if bias else None
    lib().dpo_conv2d(_p(X), _p(GY), N, Cin, H, W, Cout, Ho, Wo, kh, kw, stride[0], stride[1],
                     pad[0], pad[1], float(scale), _p(gW), _p(gb) if bias else None)
    return gW, gb


def embedding_grad(ids, B, V: int, scale: float = 1.0, cap: Optional[int] = None):
    """Per-sample Embedding grads in CSR form: (row_ptr [N+1], uniq [nnz], rows [nnz, D])."""
    ids = np.ascontiguousarray(ids, dtype=np.int64); B = _f64(B)
    N, T = ids.shape
    D = B.shape[2]
    cap = N * T if cap is None else int(cap)
    row_ptr = np.zeros(N + 1, dtype=np.int64)
    uniq = np.zeros(max(cap, 1), dtype=np.int64)
    rows = np.zeros((max(cap, 1), D))
    nnz = lib().dpo_embedding(_p(ids, _i64), _p(B), N, T, V, D, float(scale), _p(row_ptr, _i64),
                              _p(uniq, _i64), _p(rows), cap)
    if nnz == -2:
        raise ValueError("token id outside [0, V)")
    if nnz == -1:
        raise ValueError("CSR capacity exceeded")
    return row_ptr, uniq[:nnz].copy(), rows[:nnz].copy()


def layernorm_grad(xhat, B, scale: float = 1.0):
    """Per-sample LayerNorm affine grads: (ggamma [N, D], gbeta [N, D])."""
    xhat = _f64(xhat); B = _f64(B)
    N, T, D = B.shape
    gg = np.empty((N, D)); gbt = np.empty((N, D))
    lib().dpo_layernorm(_p(xhat), _p(B), N, T, D, float(scale), _p(gg), _p(gbt))
    return gg, gbt


def _opt(a):
    return None if a is None else _f64(a)


def _popt(a):
    return None if a is None else _p(a)


def lstm_forward(x, W_ih, W_hh, b_ih=None, b_hh=None):
    """LSTM forward (gate order i, f, g, o; zero initial state): returns
    (gates [N, T, 4H] after their nonlinearities, c [N, T, H], h [N, T, H])."""
    x = _f64(x); W_ih = _f64(W_ih); W_hh = _f64(W_hh)
    b_ih = _opt(b_ih); b_hh = _opt(b_hh)
    N, T, D = x.shape
    H = W_hh.shape[1]
    gates = np.empty((N, T, 4 * H)); c = np.empty((N, T, H)); h = np.empty((N, T, H))
    lib().dpo_lstm_forward(_p(x), _p(W_ih), _p(W_hh), _popt(b_ih), _popt(b_hh), N, T, D, H, _p(gates), _p(c), _p(h))
    return gates, c, h


def lstm_backward(gates, c, W_hh, dh_out=None, dh_last=None):
    """Backward through time of the LSTM: the gradient of each sample's loss
    with respect to the gate pre-activations, delta [N, T, 4H], from the
    stored gates and cell states and the loss gradient at the hidden states
    (dh_out [N, T, H] at every step and/or dh_last [N, H] at the last)."""
    gates = _f64(gates); c = _f64(c); W_hh = _f64(W_hh)
    dh_out = _opt(dh_out); dh_last = _opt(dh_last)
    N, T, H = c.shape
    delta = np.empty((N, T, 4 * H))
    lib().dpo_lstm_backward(_p(gates), _p(c), _p(W_hh), _popt(dh_out), _popt(dh_last), N, T, H, _p(delta))
    return delta


def groupnorm_grad(xhat, B, scale: float = 1.0):
    """Per-sample GroupNorm / InstanceNorm affine grads from the normalized
    input: (ggamma [N, C], gbeta [N, C]); xhat and B are [N, C, *spatial]."""
    xhat = _f64(xhat); B = _f64(B)
    N, C = B.shape[0], B.shape[1]
    P = int(np.prod(B.shape[2:])) if B.ndim > 2 else 1
    xhat = np.ascontiguousarray(xhat.reshape(N, C, P)); B = np.ascontiguousarray(B.reshape(N, C, P))
    gg = np.empty((N, C)); gbt = np.empty((N, C))
    lib().dpo_groupnorm(_p(xhat), _p(B), N, C, P, float(scale), _p(gg), _p(gbt))
    return gg, gbt


# --------------------------------------------------------------------------
# norms, clip, sum, noise
# --------------------------------------------------------------------------

def sqnorm_accumulate(G, sq: np.ndarray) -> np.ndarray:
    G = _f64(G)
    N = G.shape[0]
    G2 = G.reshape(N, int(np.prod(G.shape[1:])))
    lib().dpo_sqnorm_accumulate(_p(G2), N, G2.shape[1], _p(sq))
    return sq


def norms(sq) -> np.ndarray:
    sq = _f64(sq)
    out = np.empty_like(sq)
    lib().dpo_norms(_p(sq), sq.shape[0], _p(out))
    return out


def clip_factors(norm, C: float) -> np.ndarray:
    norm = _f64(norm)
    out = np.empty_like(norm)
    lib().dpo_clip_factors(_p(norm), norm.shape[0], float(C), _p(out))
    return out


def clip_sum(G, c) -> np.ndarray:
    G = _f64(G); c = _f64(c)
    N = G.shape[0]
    G2 = G.reshape(N, int(np.prod(G.shape[1:])))
    S = np.empty(G2.shape[1])
    lib().dpo_clip_sum(_p(G2), _p(c), N, G2.shape[1], _p(S))
    return S.reshape(G.shape[1:])


def clip_sum_embedding(row_ptr, uniq, rows, c, V: int) -> np.ndarray:
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int64)
    uniq = np.ascontiguousarray(uniq, dtype=np.int64)
    rows = _f64(rows); c = _f64(c)
    N = row_ptr.shape[0] - 1
    D = rows.shape[1] if rows.ndim == 2 else 1
    S = np.empty((V, D))
    lib().dpo_clip_sum_embedding(_p(row_ptr, _i64), _p(uniq, _i64), _p(rows), _p(c), N, V, D, _p(S))
    return S


def philox4x32_10(ctr: Sequence[int], key: Sequence[int]) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().dpo_philox4x32_10(_p(c, _u32), _p(k, _u32), _p(out, _u32))
    return out


def philox_normals(numel: int, seed: int, step: int, param_index: int):
    """(raw uint32 words, fp64 normals) of one parameter tensor's noise stream."""
    raw = np.zeros(max(numel, 1), dtype=np.uint32)
    z = np.zeros(max(numel, 1))
    lib().dpo_philox_normals(numel, seed, step, param_index, _p(raw, _u32), _p(z))
    return raw[:numel], z[:numel]


def add_noise(S, seed: int, step: int, param_index: int, sigma: float, C: float, denom: float):
    S = _f64(S)
    flat = S.reshape(-1)
    out = np.empty_like(flat)
    lib().dpo_add_noise(_p(flat), flat.shape[0], seed, step, param_index, float(sigma), float(C),
                        float(denom), _p(out))
    return out.reshape(S.shape)


# --------------------------------------------------------------------------
# the whole step over a workload's layers
# --------------------------------------------------------------------------

def layer_grads(layer, li, scale: float) -> Dict[str, object]:
    """Per-sample grads of one layer from its drawn inputs (values as the device sees them)."""
    from paper_2109_12298_amd import workloads as W
    if isinstance(layer, W.Linear):
        gW, gb = linear_grad(li.A, li.B, scale, layer.bias)
        return {"weight": gW, "bias": gb} if layer.bias else {"weight": gW}
    if isinstance(layer, W.Conv2d):
        gW, gb = conv2d_grad(li.A, li.B, layer.k, layer.stride, layer.pad, scale, layer.bias)
        return {"weight": gW, "bias": gb} if layer.bias else {"weight": gW}
    if isinstance(layer, W.Embedding):
        rp, uq, rows = embedding_grad(li.ids, li.B, layer.V, scale)
        return {"csr": (rp, uq, rows)}
    if isinstance(layer, W.LayerNorm):
        gg, gbt = layernorm_grad(li.A, li.B, scale)
        return {"weight": gg, "bias": gbt}
    if isinstance(layer, W.GroupNorm):
        gg, gbt = groupnorm_grad(li.A, li.B, scale)
        return {"weight": gg, "bias": gbt}
    raise TypeError(layer)


def dp_step(wl, inputs, step: int = 0, C: Optional[float] = None, sigma: Optional[float] = None,
            denom: Optional[float] = None, scale: Optional[float] = None,
            noise: bool = True) -> Dict[str, object]:
    """One DP-SGD gradient step over ``inputs`` (from ``workloads.make_inputs``).

    Inputs are taken as the device sees them (bf16 workloads are rounded first).
    Returns per-layer per-sample grads, per-layer squared norms, norm, c, the
    clipped sums S (name -> array) and the final grads out (name -> array)."""
    from paper_2109_12298_amd import workloads as W
    C = wl.C if C is None else C
    sigma = wl.sigma if sigma is None else sigma
    scale = wl.scale if scale is None else scale
    N = inputs[0].B.shape[0]
    denom = float(N) if denom is None else denom
    grads: List[Dict[str, object]] = []
    sq_layers = []
    derived: Dict[str, np.ndarray] = {}
    for li in inputs:
        layer = li.layer
        if isinstance(layer, W.LSTMRecurrence):
            # the gate backprop of the LSTM's weights, by the backward through
            # time; the recurrence has no parameters of its own
            a = li.aux
            derived[layer.name] = lstm_backward(a["gates"], a["c"], a["W_hh"], dh_last=a["dh_last"])
            grads.append({})
            sq_layers.append(np.zeros(N))
            continue
        B = derived[layer.bsource] if getattr(layer, "bsource", None) else li.B
        dev = W.LayerInputs(layer, A=W.rounded_like_device(wl, li.A),
                            B=W.rounded_like_device(wl, B), ids=li.ids)
        g = layer_grads(layer, dev, scale)
        sq = np.zeros(N)
        if "csr" in g:
            rp, uq, rows = g["csr"]
            for n in range(N):
                sq[n] += float(np.sum(rows[rp[n]:rp[n + 1]] ** 2))
        else:
            for key in ("weight", "bias"):
                if key in g:
                    sqnorm_accumulate(g[key], sq)
        grads.append(g)
        sq_layers.append(sq)
    sq_total = np.zeros(N)
    for sq in sq_layers:
        sq_total += sq
    norm = norms(sq_total)
    c = clip_factors(norm, C)
    S: Dict[str, np.ndarray] = {}
    for li, g in zip(inputs, grads):
        layer = li.layer
        if "csr" in g:
            S[layer.name + ".weight"] = clip_sum_embedding(*g["csr"], c, layer.V)
        else:
            for key in ("weight", "bias"):
                if key in g:
                    S[layer.name + "." + key] = clip_sum(g[key], c)
    out: Dict[str, np.ndarray] = {}
    if noise:
        for pidx, (pname, shape) in enumerate(wl.param_tensors()):
            out[pname] = add_noise(S[pname], wl.seed, step, pidx, sigma, C, denom)
    return {"grads": grads, "sq_layers": np.stack(sq_layers), "norm": norm, "c": c, "S": S,
            "out": out, "derived": derived}
