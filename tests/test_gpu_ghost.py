"""GPU parity of the ghost norm (dp_ghost_norm_linear): each sample's squared
gradient norm from the Gram matrices, against the fp64 oracle's norm of the
materialized per-sample gradient (its definition), through the C ABI."""
import sys

import numpy as np
import pytest
import torch

import oracle
from compare import assert_rel
from paper_2109_12298_amd import binding as dp

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def inputs(rng, N, T, din, dout, dtype):
    A = rng.standard_normal((N, T, din)).astype(np.float32)
    B = (rng.standard_normal((N, T, dout)) / 8).astype(np.float32)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    return torch.from_numpy(A).to(tdt).to(DEV), torch.from_numpy(B).to(tdt).to(DEV)


def ghost(At, Bt, dt, N, T, din, dout, scale, bias):
    sq = torch.full((max(N, 1),), 7.0, device=DEV)[:N]
    ws = torch.empty(max(dp.dp_ghost_norm_linear_workspace_bytes(N, T, din, dout), 1), dtype=torch.uint8, device=DEV)
    dp.dp_ghost_norm_linear(At, Bt, dt, N, T, din, dout, scale, bias, sq, None, ws)
    torch.cuda.synchronize()
    return sq.cpu().numpy()


def oracle_sq(At, Bt, scale, bias, samples=None):
    A = At.float().cpu().numpy().astype(np.float64)
    B = Bt.float().cpu().numpy().astype(np.float64)
    if samples is not None:
        A, B = A[samples], B[samples]
    rW, rb = oracle.linear_grad(A, B, scale, bias=bias)
    rsq = np.zeros(A.shape[0])
    oracle.sqnorm_accumulate(rW, rsq)
    if bias:
        oracle.sqnorm_accumulate(rb, rsq)
    return rsq


# (N, T, d_in, d_out, bias, dtype)
SHAPES = [(3, 1, 5, 7, True, "f32"),            # one position: the rank-one closed form
          (2, 64, 768, 768, True, "bf16"),      # one 64 x 64 tile pair, 16-byte loads
          (3, 128, 264, 136, True, "bf16"),     # three tile pairs, ragged feature stages
          (2, 130, 12, 20, False, "bf16"),      # ragged T (six pairs), element loads, no bias
          (2, 256, 100, 400, True, "f32"),      # the LSTM's shape, fp32 MFMA
          (1, 33, 7, 9, True, "f32"),           # element loads, fp32
          (4, 200, 33, 64, True, "bf16")]       # d_in not a multiple of 8


@pytest.mark.parametrize("shape", SHAPES)
def test_ghost_norm_matches_oracle(shape):
    N, T, din, dout, bias, dtype = shape
    say("ghost", shape)
    rng = np.random.default_rng(T + din)
    At, Bt = inputs(rng, N, T, din, dout, dtype)
    dt = dp.DP_BF16 if dtype == "bf16" else dp.DP_F32
    got = ghost(At, Bt, dt, N, T, din, dout, 0.9, bias)
    assert_rel(got, oracle_sq(At, Bt, 0.9, bias), 1e-4, "ghost sqnorm %s" % (shape,))
    # the materializing entry point's norm on the same inputs
    gW = torch.empty((N, dout, din), device=DEV)
    gb = torch.empty((N, dout), device=DEV) if bias else None
    sq = torch.empty(N, device=DEV)
    ws = torch.empty(max(dp.dp_grad_sample_linear_workspace_bytes(N, T, din, dout, dt), 1), dtype=torch.uint8,
                     device=DEV)
    dp.dp_grad_sample_linear(At, Bt, dt, N, T, din, dout, 0.9, gW, gb, sq, None, ws)
    torch.cuda.synchronize()
    assert_rel(got, sq.cpu().numpy(), 1e-4, "ghost vs materialized")


def test_ghost_norm_edges():
    say("ghost edges")
    rng = np.random.default_rng(5)
    At, Bt = inputs(rng, 3, 0, 8, 8, "f32")
    assert not ghost(At, Bt, dp.DP_F32, 3, 0, 8, 8, 1.0, True).any()       # T = 0: zero norms
    At, Bt = inputs(rng, 0, 16, 8, 8, "bf16")
    assert ghost(At, Bt, dp.DP_BF16, 0, 16, 8, 8, 1.0, True).size == 0
    # a zero backprop gives a zero norm; a repeated position doubles the Gram entries exactly
    At, Bt = inputs(rng, 2, 64, 32, 16, "f32")
    Bt.zero_()
    assert not ghost(At, Bt, dp.DP_F32, 2, 64, 32, 16, 1.0, True).any()
    a = torch.from_numpy(rng.standard_normal((1, 1, 32)).astype(np.float32)).to(DEV)
    b = torch.from_numpy(rng.standard_normal((1, 1, 16)).astype(np.float32)).to(DEV)
    one = ghost(a, b, dp.DP_F32, 1, 1, 32, 16, 1.0, False)
    two = ghost(a.repeat(1, 2, 1).contiguous(), b.repeat(1, 2, 1).contiguous(), dp.DP_F32, 1, 2, 32, 16, 1.0, False)
    np.testing.assert_allclose(two, 4 * one, rtol=1e-6)      # |2 b a^T|^2 = 4 |b a^T|^2


def test_ghost_norm_transformer_ffn_full_size_sampled():
    """The transformer block's ffn1 at full size (N = 32, T = 128, 768 -> 3072,
    bf16): every sample on the GPU, four of them through the oracle."""
    N, T, din, dout = 32, 128, 768, 3072
    say("ghost ffn1 full size")
    rng = np.random.default_rng(77)
    At, Bt = inputs(rng, N, T, din, dout, "bf16")
    got = ghost(At, Bt, dp.DP_BF16, N, T, din, dout, 1.0, True)
    picks = [0, 7, 19, 31]
    assert_rel(got[picks], oracle_sq(At, Bt, 1.0, True, samples=picks), 1e-4, "ffn1 sampled")


def ghost_many(layers, dt, N, scale=0.9):
    """dp_ghost_norm_linear_many over (A, B, T, d_in, d_out, bias) layers: each layer's sqnorm."""
    outs = [torch.full((max(N, 1),), 7.0, device=DEV)[:N] for _ in layers]
    items = dp.make_ghost_layers([(A, B, T, din, dout, scale, bias, sq)
                                  for (A, B, T, din, dout, bias), sq in zip(layers, outs)])
    ws = torch.empty(max(dp.dp_ghost_norm_linear_many_workspace_bytes(items, len(layers), N), 1),
                     dtype=torch.uint8, device=DEV)
    dp.dp_ghost_norm_linear_many(items, len(layers), dt, N, None, ws)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in outs]


# (T, d_in, d_out, bias) per layer; one call per list
MANY_BF16 = [(128, 264, 136, True),     # three pairs, ragged feature stages
             (130, 16, 24, False),      # ragged T: six pairs
             (64, 768, 768, True),      # one pair
             (200, 33, 64, True),       # d_in not a multiple of 8: the element-load launch
             (0, 8, 8, True),           # no positions: zero norms
             (96, 40, 3000, True)]      # d_out much larger than d_in


@pytest.mark.parametrize("N", [1, 3])
def test_ghost_norm_many_matches_oracle(N):
    """A few samples: the units do not fill the GPU, so each pair is split
    into feature chunks and a second launch adds them."""
    say("ghost many bf16 N", N)
    rng = np.random.default_rng(40 + N)
    layers = []
    for T, din, dout, bias in MANY_BF16:
        A, B = inputs(rng, N, T, din, dout, "bf16")
        layers.append((A, B, T, din, dout, bias))
    got = ghost_many(layers, dp.DP_BF16, N)
    for (A, B, T, din, dout, bias), g in zip(layers, got):
        assert_rel(g, oracle_sq(A, B, 0.9, bias), 1e-4, "many T=%d %dx%d" % (T, din, dout))
        alone = ghost(A, B, dp.DP_BF16, N, T, din, dout, 0.9, bias)
        assert_rel(g, alone, 1e-5, "many vs alone T=%d %dx%d" % (T, din, dout))


def test_ghost_norm_many_one_chunk_matches_oracle_and_single_calls():
    """64 samples of T = 256 (ten tile pairs each): enough units for one chunk
    per pair, the Gram tiles' product formed in registers; each layer alone
    has enough units too, so the grouped call equals the single calls bit for
    bit.  fp32 and bf16, with an element-load layer."""
    N = 64
    for dtype, shapes in (("f32", [(256, 40, 24, True), (256, 16, 48, False)]),
                          ("bf16", [(256, 40, 24, True), (256, 16, 48, False), (250, 20, 12, True)])):
        say("ghost many one chunk", dtype)
        rng = np.random.default_rng(9)
        dt = dp.DP_BF16 if dtype == "bf16" else dp.DP_F32
        layers = []
        for T, din, dout, bias in shapes:
            A, B = inputs(rng, N, T, din, dout, dtype)
            layers.append((A, B, T, din, dout, bias))
        got = ghost_many(layers, dt, N)
        for (A, B, T, din, dout, bias), g in zip(layers, got):
            assert_rel(g, oracle_sq(A, B, 0.9, bias), 1e-4, "one chunk %s T=%d %dx%d" % (dtype, T, din, dout))
            alone = ghost(A, B, dt, N, T, din, dout, 0.9, bias)
            np.testing.assert_array_equal(g, alone)


def test_ghost_norm_many_transformer_full_size_sampled():
    """The transformer block's six Linear layers (N = 32, T = 128, bf16) in one
    grouped call, the benchmark's launch: every sample on the GPU, two per
    layer through the oracle, and every sample against the layer's own call
    (which splits its 96 units into feature chunks)."""
    N, T = 32, 128
    say("ghost many transformer full size")
    rng = np.random.default_rng(78)
    shapes = [(768, 768)] * 4 + [(768, 3072), (3072, 768)]
    layers = []
    for din, dout in shapes:
        A, B = inputs(rng, N, T, din, dout, "bf16")
        layers.append((A, B, T, din, dout, True))
    got = ghost_many(layers, dp.DP_BF16, N, scale=1.0)
    for k, ((A, B, _, din, dout, bias), g) in enumerate(zip(layers, got)):
        picks = [k, 31 - 2 * k]
        assert_rel(g[picks], oracle_sq(A, B, 1.0, bias, samples=picks), 1e-4, "layer %d sampled" % k)
        alone = ghost(A, B, dp.DP_BF16, N, T, din, dout, 1.0, bias)
        assert_rel(g, alone, 1e-5, "layer %d vs alone" % k)


def test_ghost_norm_many_more_layers_than_one_launch_table():
    """18 layers: the Gram launch, the pair sums and (few units) the chunk
    combine each run as two launches of up to 16 layers; every layer against
    its own single call."""
    N = 2
    say("ghost many, 18 layers")
    rng = np.random.default_rng(21)
    layers = []
    for k in range(18):
        T, din, dout = 64 + 17 * (k % 3), 16 + 8 * (k % 5), 24 + 8 * (k % 4)
        A, B = inputs(rng, N, T, din, dout, "bf16")
        layers.append((A, B, T, din, dout, k % 2 == 0))
    got = ghost_many(layers, dp.DP_BF16, N)
    for (A, B, T, din, dout, bias), g in zip(layers, got):
        alone = ghost(A, B, dp.DP_BF16, N, T, din, dout, 0.9, bias)
        assert_rel(g, alone, 1e-5, "18 layers T=%d %dx%d" % (T, din, dout))
    picks = [0, 17]
    for k in picks:
        A, B, T, din, dout, bias = layers[k]
        assert_rel(got[k], oracle_sq(A, B, 0.9, bias), 1e-4, "18 layers oracle %d" % k)
