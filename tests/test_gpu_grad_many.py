"""GPU parity of the grouped per-sample-gradient call (dp_grad_sample_many)
against the fp64 oracle, and against the single-layer entry points on the
same inputs, through the C ABI."""
import sys

import numpy as np
import pytest
import torch

import oracle
from compare import assert_g12, assert_rel
from paper_2109_12298_amd import binding as dp

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


# ("lin", d_in, d_out, T, bias) or ("conv", Cin, H, W, Cout, kh, kw, sh, sw, ph, pw, bias)
MNIST = [("conv", 1, 28, 28, 16, 8, 8, 2, 2, 3, 3, True), ("conv", 16, 13, 13, 32, 4, 4, 2, 2, 0, 0, True),
         ("lin", 512, 32, 1, True), ("lin", 32, 10, 1, True)]
RAGGED = [("conv", 3, 7, 9, 5, 3, 3, 2, 2, 1, 1, True),        # 27 weight columns: one ragged block
          ("conv", 5, 9, 4, 66, 2, 3, 1, 2, 1, 0, False),      # 4 blocks per wave, no bias
          ("conv", 3, 12, 12, 32, 4, 4, 2, 2, 1, 1, True),     # 6 blocks: 2 per wave
          ("lin", 7, 9, 1, True),                              # d_in % 4 != 0: scalar outer product
          ("lin", 3000, 5, 1, False),                          # 2 rows per block, several blocks per sample
          ("lin", 64, 16, 8, True),                            # T > 1: runs alone inside the call
          ("conv", 2, 130, 130, 4, 3, 3, 1, 1, 1, 1, True)]    # too large for one workgroup: runs alone


def make(spec, N, rng, tdt):
    if spec[0] == "lin":
        _, din, dout, T, bias = spec
        A = rng.standard_normal((N, T, din) if T > 1 else (N, din)).astype(np.float32)
        B = (rng.standard_normal((N, T, dout) if T > 1 else (N, dout)) / 4).astype(np.float32)
        gW = torch.full((N, dout, din), 7.0, device=DEV)
        gb = torch.full((N, dout), 7.0, device=DEV) if bias else None
    else:
        _, Cin, H, Wd, Cout, kh, kw, sh, sw, ph, pw, bias = spec
        Ho, Wo = (H + 2 * ph - kh) // sh + 1, (Wd + 2 * pw - kw) // sw + 1
        A = rng.standard_normal((N, Cin, H, Wd)).astype(np.float32)
        B = (rng.standard_normal((N, Cout, Ho, Wo)) / 4).astype(np.float32)
        gW = torch.full((N, Cout, Cin, kh, kw), 7.0, device=DEV)
        gb = torch.full((N, Cout), 7.0, device=DEV) if bias else None
    At = torch.from_numpy(A).to(tdt).to(DEV)
    Bt = torch.from_numpy(B).to(tdt).to(DEV)
    sq = torch.full((N,), 7.0, device=DEV)
    return At, Bt, gW, gb, sq


def item(spec, At, Bt, gW, gb, sq, scale):
    if spec[0] == "lin":
        _, din, dout, T, _ = spec
        return dp.linear_grad_item(At, Bt, T, din, dout, scale, gW, gb, sq)
    _, Cin, H, Wd, Cout, kh, kw, sh, sw, ph, pw, _ = spec
    Ho, Wo = (H + 2 * ph - kh) // sh + 1, (Wd + 2 * pw - kw) // sw + 1
    return dp.conv2d_grad_item(At, Bt, Cin, H, Wd, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw, scale, gW, gb, sq)


def run_many(specs, N, dt, scale, seed):
    rng = np.random.default_rng(seed)
    tdt = torch.bfloat16 if dt == dp.DP_BF16 else torch.float32
    bufs = [make(s, N, rng, tdt) for s in specs]
    items = dp.make_layer_grads([item(s, *b, scale) for s, b in zip(specs, bufs)])
    ws = torch.empty(max(dp.dp_grad_sample_many_workspace_bytes(items, len(specs), dt, N), 1), dtype=torch.uint8,
                     device=DEV)
    dp.dp_grad_sample_many(items, len(specs), dt, N, None, ws)
    torch.cuda.synchronize()
    return bufs, items


def oracle_layer(spec, At, Bt, scale):
    A = At.float().cpu().numpy().astype(np.float64)
    B = Bt.float().cpu().numpy().astype(np.float64)
    if spec[0] == "lin":
        rW, rb = oracle.linear_grad(A, B, scale)
    else:
        _, Cin, H, Wd, Cout, kh, kw, sh, sw, ph, pw, _ = spec
        rW, rb = oracle.conv2d_grad(A, B, (kh, kw), (sh, sw), (ph, pw), scale)
    rsq = np.zeros(A.shape[0])
    oracle.sqnorm_accumulate(rW, rsq)
    if spec[-1]:
        oracle.sqnorm_accumulate(rb, rsq)
    return rW, rb, rsq


def check_oracle(specs, bufs, scale, what):
    for spec, (At, Bt, gW, gb, sq) in zip(specs, bufs):
        rW, rb, rsq = oracle_layer(spec, At, Bt, scale)
        assert_g12(gW.cpu().numpy(), rW, 1e-4, "%s gW %s" % (what, spec))
        if gb is not None:
            assert_g12(gb.cpu().numpy(), rb, 1e-4, "%s gb %s" % (what, spec))
        assert_rel(sq.cpu().numpy(), rsq, 1e-4, "%s sqnorm %s" % (what, spec))


@pytest.mark.parametrize("N", [1, 5, 256])
def test_grouped_mnist_layers_match_oracle(N):
    say("grad_many mnist N=", N)
    specs = MNIST
    bufs, items = run_many(specs, N, dp.DP_F32, 0.8, seed=N)
    assert all(dp.dp_grad_sample_many_grouped(items, k, dp.DP_F32, N) for k in range(len(specs)))
    check_oracle(specs, bufs, 0.8, "mnist")


@pytest.mark.parametrize("dt", [dp.DP_F32, dp.DP_BF16])
def test_grouped_ragged_and_mixed_layers_match_oracle(dt):
    say("grad_many ragged dt=", dt)
    bufs, items = run_many(RAGGED, 3, dt, 1.3, seed=11 + dt)
    got = [dp.dp_grad_sample_many_grouped(items, k, dt, 3) for k in range(len(RAGGED))]
    assert got == [True, True, True, True, True, False, False]
    check_oracle(RAGGED, bufs, 1.3, "ragged")


def test_grouped_equals_single_layer_calls_bitwise():
    """The grouped launch runs the single-layer kernels' workgroup bodies, so
    the results are the same bits."""
    say("grad_many vs single")
    N = 6
    specs = MNIST + RAGGED[:5]
    bufs, _ = run_many(specs, N, dp.DP_F32, 1.1, seed=5)
    for spec, (At, Bt, gW, gb, sq) in zip(specs, bufs):
        gW2, gb2, sq2 = torch.empty_like(gW), (torch.empty_like(gb) if gb is not None else None), torch.empty_like(sq)
        if spec[0] == "lin":
            _, din, dout, T, _ = spec
            dp.dp_grad_sample_linear(At, Bt, dp.DP_F32, N, T, din, dout, 1.1, gW2, gb2, sq2)
        else:
            _, Cin, H, Wd, Cout, kh, kw, sh, sw, ph, pw, _ = spec
            Ho, Wo = (H + 2 * ph - kh) // sh + 1, (Wd + 2 * pw - kw) // sw + 1
            ws = torch.empty(max(dp.dp_grad_sample_conv2d_workspace_bytes(N, Cin, H, Wd, Cout, kh, kw, sh, sw, ph,
                                                                           pw), 1), dtype=torch.uint8, device=DEV)
            dp.dp_grad_sample_conv2d(At, Bt, dp.DP_F32, N, Cin, H, Wd, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw, 1, 1, 1,
                                     1.1, gW2, gb2, sq2, None, ws)
        torch.cuda.synchronize()
        assert torch.equal(gW, gW2), spec
        if gb is not None:
            assert torch.equal(gb, gb2), spec
        assert torch.equal(sq, sq2), spec


def test_grouped_more_layers_than_one_launch():
    """More than eight grouped layers run as several launches."""
    say("grad_many 11 layers")
    specs = MNIST + RAGGED[:5] + MNIST[:2]
    bufs, _ = run_many(specs, 2, dp.DP_F32, 1.0, seed=21)
    check_oracle(specs, bufs, 1.0, "eleven")


# bf16 Linear layers over a sequence: the staged grouped launch (runs of
# samples per tile, balanced over every layer), and one that is not staged
SEQ = [("lin", 768, 768, 128, True), ("lin", 768, 3072, 128, True), ("lin", 3072, 768, 128, True),
       ("lin", 264, 392, 64, False),                         # ragged tiles, no bias
       ("lin", 64, 16, 8, True)]                             # T % 32 != 0: the single-layer path


@pytest.mark.parametrize("N", [1, 5, 37])
def test_grouped_bf16_sequence_layers_match_oracle_and_single_calls(N):
    say("grad_many bf16 sequence layers N=", N)
    specs = SEQ if N < 37 else SEQ[3:]
    bufs, items = run_many(specs, N, dp.DP_BF16, 0.9, seed=40 + N)
    got = [dp.dp_grad_sample_many_grouped(items, k, dp.DP_BF16, N) for k in range(len(specs))]
    assert got == [s[3] % 32 == 0 for s in specs]
    check_oracle(specs, bufs, 0.9, "bf16 seq")
    for spec, (At, Bt, gW, gb, sq) in zip(specs, bufs):
        _, din, dout, T, _ = spec
        gW2, gb2, sq2 = torch.empty_like(gW), (torch.empty_like(gb) if gb is not None else None), torch.empty_like(sq)
        ws = torch.empty(max(dp.dp_grad_sample_linear_workspace_bytes(N, T, din, dout, dp.DP_BF16), 1),
                         dtype=torch.uint8, device=DEV)
        dp.dp_grad_sample_linear(At, Bt, dp.DP_BF16, N, T, din, dout, 0.9, gW2, gb2, sq2, None, ws)
        torch.cuda.synchronize()
        assert torch.equal(gW, gW2), spec
        if gb is not None:
            assert torch.equal(gb, gb2), spec
        assert torch.equal(sq, sq2), spec


def test_grouped_bf16_more_layers_than_one_launch():
    """Eighteen staged layers: two grouped launches, each with its own partials."""
    say("grad_many 18 bf16 sequence layers")
    specs = [("lin", 64 + 8 * (k % 3), 128 + 8 * (k % 5), 32 * (1 + k % 2), k % 4 != 1) for k in range(18)]
    bufs, items = run_many(specs, 3, dp.DP_BF16, 1.2, seed=77)
    assert all(dp.dp_grad_sample_many_grouped(items, k, dp.DP_BF16, 3) for k in range(len(specs)))
    check_oracle(specs, bufs, 1.2, "eighteen bf16")


# fp32 Linear layers over a sequence: the staged grouped launch (a sample's
# tiles of all layers together); the first two read the same B, as an LSTM's
# W_ih and W_hh do
SEQ32 = [("lin", 100, 400, 256, True), ("lin", 100, 400, 256, True),
         ("lin", 36, 52, 48, False),                         # ragged tiles, no bias
         ("lin", 64, 16, 8, True),                           # T % 16 != 0: the single-layer path
         ("lin", 7, 9, 1, True)]                             # T = 1: the small-layer launch


@pytest.mark.parametrize("N", [1, 5, 37])
def test_grouped_fp32_sequence_layers_match_oracle_and_single_calls(N):
    say("grad_many fp32 sequence layers N=", N)
    specs = SEQ32 if N < 37 else [("lin", 100, 400, 64, True), ("lin", 100, 400, 64, True)] + SEQ32[2:]
    rng = np.random.default_rng(60 + N)
    bufs = [make(s, N, rng, torch.float32) for s in specs]
    bufs[1] = (bufs[1][0], bufs[0][1]) + tuple(bufs[1][2:])
    items = dp.make_layer_grads([item(s, *b, 0.7) for s, b in zip(specs, bufs)])
    ws = torch.empty(max(dp.dp_grad_sample_many_workspace_bytes(items, len(specs), dp.DP_F32, N), 1),
                     dtype=torch.uint8, device=DEV)
    dp.dp_grad_sample_many(items, len(specs), dp.DP_F32, N, None, ws)
    torch.cuda.synchronize()
    got = [dp.dp_grad_sample_many_grouped(items, k, dp.DP_F32, N) for k in range(len(specs))]
    assert got == [True, True, True, False, True]
    check_oracle(specs, bufs, 0.7, "fp32 seq")
    for spec, (At, Bt, gW, gb, sq) in zip(specs, bufs):
        _, din, dout, T, _ = spec
        gW2, gb2, sq2 = torch.empty_like(gW), (torch.empty_like(gb) if gb is not None else None), torch.empty_like(sq)
        ws1 = torch.empty(max(dp.dp_grad_sample_linear_workspace_bytes(N, T, din, dout, dp.DP_F32), 1),
                          dtype=torch.uint8, device=DEV)
        dp.dp_grad_sample_linear(At, Bt, dp.DP_F32, N, T, din, dout, 0.7, gW2, gb2, sq2, None, ws1)
        torch.cuda.synchronize()
        assert torch.equal(gW, gW2), spec
        if gb is not None:
            assert torch.equal(gb, gb2), spec
        assert torch.equal(sq, sq2), spec


def test_grouped_fp32_more_layers_than_one_launch():
    """Eighteen staged fp32 layers: two grouped launches, each with its own partials."""
    say("grad_many 18 fp32 sequence layers")
    specs = [("lin", 16 + 4 * (k % 3), 20 + 4 * (k % 5), 16 * (1 + k % 2), k % 4 != 1) for k in range(18)]
    bufs, items = run_many(specs, 3, dp.DP_F32, 1.2, seed=78)
    assert all(dp.dp_grad_sample_many_grouped(items, k, dp.DP_F32, 3) for k in range(len(specs)))
    check_oracle(specs, bufs, 1.2, "eighteen fp32")
