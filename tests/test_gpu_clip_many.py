"""GPU parity of the grouped fused clipped sum of Linear layers
(dp_clip_accumulate_linear_many) against the fp64 oracle's clipped sum of the
per-sample gradients, through the C ABI."""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from compare import assert_g12
from paper_2109_12298_amd import binding as dp

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


# (T, d_in, d_out, bias, dtype): the grouped bf16 kernel takes T % 32 == 0 and
# feature sizes that are multiples of 8; the others go through the single-layer
# kernels inside the same call
LAYERS = [(32, 256, 128, True, "bf16"),      # exactly one tile
          (64, 264, 136, True, "bf16"),      # ragged in j and i: 2 x 2 tiles
          (96, 8, 8, False, "bf16"),         # tiny
          (128, 768, 200, True, "bf16"),     # the transformer's T, ragged i
          (33, 64, 40, True, "bf16"),        # T not a multiple of 32: single-layer path
          (32, 12, 20, True, "bf16")]        # features not multiples of 8: single-layer path


def make_layer(rng, N, T, din, dout, dtype):
    A = rng.standard_normal((N, T, din)).astype(np.float32)
    B = (rng.standard_normal((N, T, dout)) / 8).astype(np.float32)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    At = torch.from_numpy(A).to(tdt).to(DEV)
    Bt = torch.from_numpy(B).to(tdt).to(DEV)
    return At, Bt


def run_many(layers, N, norm, C, scale, dt, seed=0):
    rng = np.random.default_rng(seed)
    ops, outs, ents = [], [], []
    for (T, din, dout, bias, _) in layers:
        At, Bt = make_layer(rng, N, T, din, dout, "bf16" if dt == dp.DP_BF16 else "f32")
        sW = torch.full((dout, din), 7.0, device=DEV)
        sb = torch.full((dout,), 7.0, device=DEV) if bias else None
        ops.append((At, Bt))
        outs.append((sW, sb))
        ents.append((At, Bt, T, din, dout, scale, sW, sb))
    items = dp.make_linear_clips(ents)
    need = dp.dp_clip_accumulate_linear_many_workspace_bytes(items, len(ents), dt, N)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=DEV)
    normt = torch.from_numpy(np.asarray(norm, dtype=np.float32)).to(DEV)
    dp.dp_clip_accumulate_linear_many(items, len(ents), dt, N, normt, C, None, ws)
    torch.cuda.synchronize()
    return ops, outs


def oracle_sums(At, Bt, norm, C, scale):
    A = At.float().cpu().numpy().astype(np.float64)
    B = Bt.float().cpu().numpy().astype(np.float64)
    rW, rb = oracle.linear_grad(A, B, scale)
    c = oracle.clip_factors(np.asarray(norm, dtype=np.float32).astype(np.float64), C)
    return oracle.clip_sum(rW, c), oracle.clip_sum(rb, c)


@pytest.mark.parametrize("N", [1, 3, 8])
def test_grouped_clip_sum_matches_oracle(N):
    say("clip_many N=", N)
    rng = np.random.default_rng(100 + N)
    norm = rng.uniform(0.2, 3.0, N)
    C = float(np.median(norm))
    ops, outs = run_many(LAYERS, N, norm, C, 0.7, dp.DP_BF16, seed=N)
    for (At, Bt), (sW, sb), L in zip(ops, outs, LAYERS):
        rW, rb = oracle_sums(At, Bt, norm, C, 0.7)
        assert_g12(sW.cpu().numpy(), rW, 1e-4, "sumW %s" % (L,))
        if sb is not None:
            assert_g12(sb.cpu().numpy(), rb, 1e-4, "sumb %s" % (L,))


def test_grouped_clip_sum_is_deterministic_and_matches_single_calls():
    N = 4
    say("clip_many determinism")
    norm = np.array([0.5, 2.0, 1.0, 4.0])
    ops1, outs1 = run_many(LAYERS[:4], N, norm, 1.0, 1.0, dp.DP_BF16, seed=9)
    ops2, outs2 = run_many(LAYERS[:4], N, norm, 1.0, 1.0, dp.DP_BF16, seed=9)
    normt = torch.from_numpy(norm.astype(np.float32)).to(DEV)
    for (At, Bt), (sW1, sb1), (sW2, sb2), (T, din, dout, bias, _) in zip(ops1, outs1, outs2, LAYERS):
        np.testing.assert_array_equal(sW1.cpu().numpy(), sW2.cpu().numpy())
        # the single-layer entry point on the same inputs agrees to rounding
        sW = torch.empty((dout, din), device=DEV)
        sb = torch.empty(dout, device=DEV) if bias else None
        ws = torch.empty(max(dp.dp_clip_accumulate_linear_workspace_bytes(N, T, din, dout, dp.DP_BF16), 1),
                         dtype=torch.uint8, device=DEV)
        dp.dp_clip_accumulate_linear(At, Bt, dp.DP_BF16, N, T, din, dout, 1.0, normt, 1.0, sW, sb, None, ws)
        assert_g12(sW1.cpu().numpy(), sW.cpu().numpy(), 1e-5, "grouped vs single W")
        if bias:
            assert_g12(sb1.cpu().numpy(), sb.cpu().numpy(), 1e-5, "grouped vs single b")


def test_grouped_clip_sum_special_factors():
    """A sample whose clip factor underflows to 0 adds nothing; a non-finite
    norm turns every sum to NaN (never passes unclipped)."""
    N = 3
    say("clip_many special factors")
    layers = [LAYERS[0], LAYERS[1]]
    # C = 1e-30: c = 1e-30 / (norm + 1e-6) is tiny but nonzero for norms ~ 1
    # and underflows to exactly 0 in fp32 for norm 1e20
    norm = np.array([1.0, 1e20, 0.5])
    ops, outs = run_many(layers, N, norm, 1e-30, 1.0, dp.DP_BF16, seed=3)
    for (At, Bt), (sW, sb) in zip(ops, outs):
        A = At.float().cpu().numpy().astype(np.float64)
        B = Bt.float().cpu().numpy().astype(np.float64)
        rW, rb = oracle.linear_grad(A, B, 1.0)
        c = np.array([1e-30 / (1.0 + 1e-6), 0.0, 1e-30 / (0.5 + 1e-6)])
        assert_g12(sW.cpu().numpy(), oracle.clip_sum(rW, c), 1e-4, "underflow W")
        assert_g12(sb.cpu().numpy(), oracle.clip_sum(rb, c), 1e-4, "underflow b")
    norm = np.array([1.0, math.inf, 0.5])
    ops, outs = run_many(layers, N, norm, 1.0, 1.0, dp.DP_BF16, seed=4)
    for sW, sb in outs:
        assert np.isnan(sW.cpu().numpy()).all()
        assert np.isnan(sb.cpu().numpy()).all()


def test_grouped_clip_sum_fp32_and_empty():
    """fp32 layers and N = 0 go through the single-layer kernels' rules."""
    say("clip_many fp32 / empty")
    N = 3
    norm = np.array([0.3, 1.7, 0.9])
    layers = [(32, 64, 16, True, "f32"), (5, 7, 9, False, "f32")]
    ops, outs = run_many(layers, N, norm, 1.0, 1.0, dp.DP_F32, seed=5)
    for (At, Bt), (sW, sb) in zip(ops, outs):
        rW, rb = oracle_sums(At, Bt, norm, 1.0, 1.0)
        assert_g12(sW.cpu().numpy(), rW, 1e-4, "f32 W")
        if sb is not None:
            assert_g12(sb.cpu().numpy(), rb, 1e-4, "f32 b")
    ops, outs = run_many(LAYERS[:2], 0, [], 1.0, 1.0, dp.DP_BF16, seed=6)
    for sW, sb in outs:
        assert not sW.cpu().numpy().any()
        assert not sb.cpu().numpy().any()


def test_grouped_clip_sum_more_samples_than_one_launch():
    """Batches above the per-launch sample count run as several launches, each
    adding to the stored sums."""
    N = 4003
    say("clip_many N=", N)
    layers = [(32, 8, 8, True, "bf16"), (64, 16, 24, True, "bf16")]
    rng = np.random.default_rng(77)
    norm = rng.uniform(0.2, 3.0, N)
    C = float(np.median(norm))
    ops, outs = run_many(layers, N, norm, C, 1.3, dp.DP_BF16, seed=11)
    for (At, Bt), (sW, sb), L in zip(ops, outs, layers):
        rW, rb = oracle_sums(At, Bt, norm, C, 1.3)
        assert_g12(sW.cpu().numpy(), rW, 1e-4, "sumW %s" % (L,))
        assert_g12(sb.cpu().numpy(), rb, 1e-4, "sumb %s" % (L,))
