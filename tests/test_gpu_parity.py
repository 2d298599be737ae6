"""GPU parity: every step of the HIP path against the fp64 oracle on the same
seeded inputs, through the C ABI.  Sizes keep the oracle to seconds while
still spanning several tiles and ragged tails."""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from compare import RTOL, assert_g12, assert_rel
from paper_2109_12298_amd import binding as dp
from paper_2109_12298_amd import workloads as W
from paper_2109_12298_amd.step import DPStep

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def compare_step(wl, inputs, got, ref, rtol, what):
    for li, g, r in zip(inputs, got["grads"], ref["grads"]):
        name = li.layer.name
        if not g:
            continue                # ghost norm: the layer's per-sample gradient is never formed
        if "csr" in r:
            rp, uq, rows = g["csr"]
            rrp, ruq, rrows = r["csr"]
            np.testing.assert_array_equal(rp, rrp, err_msg=what + " row_ptr " + name)
            np.testing.assert_array_equal(uq, ruq, err_msg=what + " uniq " + name)
            assert_g12(rows, rrows, rtol, what + " rows " + name)
        else:
            for k in r:
                assert_g12(g[k], r[k], rtol, "%s grad %s.%s" % (what, name, k))
    for name, d in ref.get("derived", {}).items():
        # a derived backprop decays back through time: each sample against its own scale
        for n in range(d.shape[0]):
            assert_g12(got["derived"][name][n], d[n], rtol, "%s derived %s n=%d" % (what, name, n))
    assert_rel(got["sq_layers"], ref["sq_layers"], rtol, what + " sqnorm")
    assert_rel(got["norm"], ref["norm"], rtol, what + " norm")
    for k in ref["S"]:
        assert_g12(got["S"][k], ref["S"][k], rtol, what + " S " + k)
    for k in ref["out"]:
        assert_g12(got["out"][k], ref["out"][k], rtol, what + " out " + k)
    assert got["status"] == 0


SMALL = [("linear_tiny", None), ("mnist_cnn", None), ("cifar_cnn", 3), ("text_lstm", 5),
         ("transformer_block", 2), ("cifar_gn", 3), ("text_lstm_bptt", 5)]


@pytest.mark.parametrize("name,n", SMALL)
@pytest.mark.parametrize("mode", ["auto", "fused", "colreduce"])
def test_workload_step_matches_oracle(name, n, mode):
    wl = W.get(name)
    if mode != "auto" and not any(isinstance(l, W.Linear) for l in wl.layers):
        pytest.skip("no Linear layer")
    say(name, "n=", n, "mode=", mode)
    inputs = W.make_inputs(wl, n=n)
    st = DPStep(wl, inputs, DEV, clip_mode=mode)
    st.run(step=3)
    got = st.results()
    ref = oracle.dp_step(wl, inputs, step=3)
    compare_step(wl, inputs, got, ref, RTOL[wl.dtype], name)


@pytest.mark.parametrize("name,n,mode", [("transformer_block", 2, "fused"), ("text_lstm", 5, "fused"),
                                         ("linear_tiny", None, "fused"), ("cifar_cnn", 3, "fused")])
def test_workload_step_with_ghost_norms_matches_oracle(name, n, mode):
    """Ghost norms for the fused Linear layers where 2 T^2 < d_in d_out: the
    norms, clipped sums and outputs still match the oracle's step, which
    forms every per-sample gradient."""
    wl = W.get(name)
    say(name, "n=", n, "ghost norms, clip mode", mode)
    inputs = W.make_inputs(wl, n=n)
    st = DPStep(wl, inputs, DEV, clip_mode=mode, norm_mode="ghost")
    ghosts = [lb.layer.name for lb in st.layers if lb.ghost]
    if name == "transformer_block":
        assert ghosts == ["wq", "wk", "wv", "wo", "ffn1", "ffn2"]
    if name == "text_lstm":
        assert ghosts == ["fc"]           # T = 256 is too long for the LSTM weights (2 T^2 > d_in d_out)
    st.run(step=3)
    got = st.results()
    ref = oracle.dp_step(wl, inputs, step=3)
    compare_step(wl, inputs, got, ref, RTOL[wl.dtype], name + " ghost")


def split_batches(inputs, K):
    """K physical batches of a logical batch's inputs (along the sample axis)."""
    N = next(li.B.shape[0] for li in inputs if li.B is not None)
    n = N // K
    return [W.take_samples(inputs, slice(k * n, (k + 1) * n)) for k in range(K)]


@pytest.mark.parametrize("name,n,mode", [("mnist_cnn", 4, "auto"), ("linear_tiny", 5, "fused"),
                                         ("text_lstm", 2, "auto"), ("transformer_block", 2, "fused"),
                                         ("transformer_block", 2, "colreduce"), ("text_lstm_bptt", 2, "auto")])
def test_virtual_steps_match_one_logical_step(name, n, mode):
    """Virtual steps: three physical batches of n samples, their clipped sums
    added up and noised once, equal the oracle's step over the 3n samples
    (clipping is per sample, so the grouping into physical batches does not
    change the result beyond summation order)."""
    K = 3
    wl = W.get(name)
    say(name, "virtual steps", K, "x", n, "mode", mode)
    inputs = W.make_inputs(wl, n=K * n)
    batches = split_batches(inputs, K)
    st = DPStep(wl, batches[0], DEV, clip_mode=mode, virtual_batches=K)
    st.run_virtual(batches, step=3)
    got = st.results()
    ref = oracle.dp_step(wl, inputs, step=3)
    rtol = RTOL[wl.dtype]
    for k in ref["S"]:
        assert_g12(got["acc"][k], ref["S"][k], rtol, "running sum " + k)
        assert_g12(got["out"][k], ref["out"][k], rtol, "out " + k)
    assert got["status"] == 0
    # a second logical step starts again from zero
    st.run_virtual(batches, step=3)
    again = st.results()
    for k in ref["out"]:
        np.testing.assert_array_equal(again["out"][k], got["out"][k])


def test_virtual_steps_in_a_graph_match_eager():
    """A captured graph of virtual steps (two physical batches per logical
    step, here the resident inputs twice) replays what eager calls compute."""
    wl = W.get("mnist_cnn")
    inputs = W.make_inputs(wl, n=6)
    say("virtual steps graph")
    st = DPStep(wl, inputs, DEV, virtual_batches=2)
    st.capture(first_step=5, parallel=False, steps_per_replay=2)
    st.replay()
    got = st.results()
    eager = DPStep(wl, inputs, DEV, virtual_batches=2)
    eager.run_virtual([inputs, inputs], step=6)
    ref = eager.results()
    for k in ref["out"]:
        np.testing.assert_array_equal(got["out"][k], ref["out"][k], err_msg=k)
        np.testing.assert_array_equal(got["acc"][k], ref["acc"][k], err_msg=k)


def test_runs_are_bitwise_deterministic():
    wl = W.get("text_lstm")
    inputs = W.make_inputs(wl, n=7)
    st = DPStep(wl, inputs, DEV)
    say("determinism text_lstm")
    st.run(step=1)
    a = st.results()
    st.run(step=1)
    b = st.results()
    for k in a["out"]:
        np.testing.assert_array_equal(a["out"][k], b["out"][k])
        np.testing.assert_array_equal(a["S"][k], b["S"][k])
    np.testing.assert_array_equal(a["norm"], b["norm"])


def test_noise_stream_bits_and_values():
    for numel, seed, step, pidx in [(1, 0, 0, 0), (7, 3, 5, 2), (1000003, 0, 0, 1), (4096, 2**63 + 11, 2**40 + 3, 9)]:
        say("philox", numel, seed, step, pidx)
        z = torch.empty(numel, dtype=torch.float32, device=DEV)
        raw = torch.empty(numel, dtype=torch.int32, device=DEV)
        dp.dp_philox_normals(z, raw, numel, seed, step, pidx)
        torch.cuda.synchronize()
        rraw, rz = oracle.philox_normals(numel, seed, step, pidx)
        np.testing.assert_array_equal(raw.cpu().numpy().view(np.uint32), rraw)
        zg = z.cpu().numpy().astype(np.float64)
        assert np.max(np.abs(zg - rz) / (1 + np.abs(rz))) < 2e-6


def test_add_noise_matches_oracle_and_is_resumable():
    r = np.random.default_rng(0)
    S = r.standard_normal(12345).astype(np.float32)
    St = torch.from_numpy(S).to(DEV)
    outs = []
    for step in range(3):
        say("add_noise step", step)
        o = torch.empty_like(St)
        dp.dp_add_noise(St, o, S.size, 42, step, 7, 0.8, 1.5, 32.0)
        outs.append(o.cpu().numpy())
        ref = oracle.add_noise(S.astype(np.float64), 42, step, 7, 0.8, 1.5, 32.0)
        assert_g12(outs[-1], ref, 1e-5, "add_noise")
    # resume: a fresh call for step 1 reproduces it exactly; in place is allowed
    o = St.clone()
    dp.dp_add_noise(o, o, S.size, 42, 1, 7, 0.8, 1.5, 32.0)
    np.testing.assert_array_equal(o.cpu().numpy(), outs[1])
    # sigma = 0 with C = inf: plain division
    o = torch.empty_like(St)
    dp.dp_add_noise(St, o, S.size, 42, 0, 7, 0.0, math.inf, 4.0)
    np.testing.assert_array_equal(o.cpu().numpy(), S / np.float32(4.0))


LINEAR_SHAPES = [(1, 1, 1, 1), (3, 1, 37, 13), (2, 2, 5, 3), (4, 5, 37, 13), (3, 33, 65, 70),
                 (2, 70, 130, 64), (5, 1, 4096, 10), (2, 17, 3, 129),
                 # feature sizes that are multiples of 8: the bf16 MFMA path for bf16 inputs
                 (1, 2, 8, 8), (3, 33, 136, 72), (2, 130, 264, 392), (2, 64, 128, 128), (9, 16, 256, 24),
                 # multiples of 4 but not 8: 16-byte fp32 / 8-byte bf16 loads on the fp32-MFMA path
                 (3, 40, 100, 20), (2, 256, 100, 400),
                 # T a multiple of 32: the staged bf16 kernel (ragged tiles; one sample per workgroup;
                 # runs of several samples are covered by test_bf16_staged_sample_runs_with_a_tail)
                 (1, 32, 8, 8), (3, 32, 136, 72), (2, 64, 264, 392), (5, 96, 128, 256), (181, 32, 512, 384),
                 # fp32 with T a multiple of 16 and features multiples of 4 (several of the above too): the
                 # fp32 kernel staged straight into LDS, at its narrowest and with mostly clamped chunks
                 (4, 16, 4, 4), (3, 48, 12, 68)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,T,din,dout", LINEAR_SHAPES)
def test_linear_ragged_shapes(dtype, N, T, din, dout):
    say("linear", dtype, N, T, din, dout)
    r = np.random.default_rng(N * 1000 + T)
    A = r.standard_normal((N, T, din)).astype(np.float32)
    B = (r.standard_normal((N, T, dout)) / 8).astype(np.float32)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    At = torch.from_numpy(A).to(tdt).to(DEV)
    Bt = torch.from_numpy(B).to(tdt).to(DEV)
    dt = dp.DP_BF16 if dtype == "bf16" else dp.DP_F32
    gW = torch.empty((N, dout, din), device=DEV)
    gb = torch.empty((N, dout), device=DEV)
    sq = torch.empty(N, device=DEV)
    ws = torch.empty(max(dp.dp_grad_sample_linear_workspace_bytes(N, T, din, dout, dt), 1),
                     dtype=torch.uint8, device=DEV)
    dp.dp_grad_sample_linear(At, Bt, dt, N, T, din, dout, 0.7, gW, gb, sq, None, ws)
    Ad = At.float().cpu().numpy().astype(np.float64)
    Bd = Bt.float().cpu().numpy().astype(np.float64)
    rW, rb = oracle.linear_grad(Ad, Bd, 0.7)
    rsq = np.zeros(N)
    oracle.sqnorm_accumulate(rW, rsq); oracle.sqnorm_accumulate(rb, rsq)
    assert_g12(gW.cpu().numpy(), rW, 1e-4, "gW")
    assert_g12(gb.cpu().numpy(), rb, 1e-4, "gb")
    assert_rel(sq.cpu().numpy(), rsq, 1e-4, "sqnorm")
    # fused clipped sum against the oracle's clipped sum of the per-sample grads
    norm = np.sqrt(rsq)
    C = float(np.median(norm))
    c = oracle.clip_factors(norm, C)
    normt = torch.from_numpy(norm.astype(np.float32)).to(DEV)
    sW = torch.empty((dout, din), device=DEV)
    sb = torch.empty(dout, device=DEV)
    ws2 = torch.empty(max(dp.dp_clip_accumulate_linear_workspace_bytes(N, T, din, dout, dt), 1),
                      dtype=torch.uint8, device=DEV)
    dp.dp_clip_accumulate_linear(At, Bt, dt, N, T, din, dout, 0.7, normt, C, sW, sb, None, ws2)
    cf = oracle.clip_factors(norm.astype(np.float32).astype(np.float64), C)
    assert_g12(sW.cpu().numpy(), oracle.clip_sum(rW, cf), 1e-4, "fused sumW")
    assert_g12(sb.cpu().numpy(), oracle.clip_sum(rb, cf), 1e-4, "fused sumb")
    # column reduction over the stored per-sample grads
    s2 = torch.empty((dout, din), device=DEV)
    cout = torch.empty(N, device=DEV)
    ws3 = torch.empty(max(dp.dp_clip_accumulate_workspace_bytes(N, dout * din), 1), dtype=torch.uint8, device=DEV)
    dp.dp_clip_accumulate(gW, normt, C, N, dout * din, s2, cout, None, ws3)
    assert_g12(s2.cpu().numpy(), oracle.clip_sum(rW, cf), 1e-4, "colreduce sumW")
    assert_rel(cout.cpu().numpy(), cf, 1e-6, "c")


def staged_run_length(N, din, dout):
    """Samples per workgroup of the staged bf16 kernel: its 256 (d_in) x 128
    (d_out) tiles times N spread over about 1024 workgroups, between 1 and 8."""
    tiles = -(-din // 256) * -(-dout // 128)
    return min(max(tiles * N // 1024, 1), 8)


@pytest.mark.parametrize("N,T,din,dout,check", [
    (29, 32, 768, 3072, None),                     # runs of 2 samples, the 15th run a one-sample tail
    (181, 32, 512, 1536, [0, 3, 4, 7, 176, 179, 180])])   # runs of 4, the 46th a one-sample tail
def test_bf16_staged_sample_runs_with_a_tail(N, T, din, dout, check):
    """The staged bf16 kernel walks a run of consecutive samples per
    workgroup, storing each at its boundary while the next one's operands are
    already staged; a last run shorter than the others stops early.  Every
    sample (or the run-boundary samples and the tail) against the oracle, at
    the fp32 tolerance (the oracle reads the same bf16 bits)."""
    per = staged_run_length(N, din, dout)
    assert per >= 2 and N % per == 1, (per, N)
    say("bf16 staged runs", N, T, din, dout, "per", per)
    r = np.random.default_rng(N + din)
    A = torch.from_numpy(r.standard_normal((N, T, din)).astype(np.float32)).to(torch.bfloat16)
    B = torch.from_numpy((r.standard_normal((N, T, dout)) / 8).astype(np.float32)).to(torch.bfloat16)
    At, Bt = A.to(DEV), B.to(DEV)
    gW = torch.empty((N, dout, din), device=DEV)
    gb = torch.empty((N, dout), device=DEV)
    sq = torch.empty(N, device=DEV)
    ws = torch.empty(max(dp.dp_grad_sample_linear_workspace_bytes(N, T, din, dout, dp.DP_BF16), 1),
                     dtype=torch.uint8, device=DEV)
    dp.dp_grad_sample_linear(At, Bt, dp.DP_BF16, N, T, din, dout, 0.9, gW, gb, sq, None, ws)
    torch.cuda.synchronize()
    idx = list(range(N)) if check is None else check
    Ad = A.float().numpy().astype(np.float64)[idx]
    Bd = B.float().numpy().astype(np.float64)[idx]
    rW, rb = oracle.linear_grad(Ad, Bd, 0.9)
    rsq = np.zeros(len(idx))
    oracle.sqnorm_accumulate(rW, rsq); oracle.sqnorm_accumulate(rb, rsq)
    sel = torch.tensor(idx, device=DEV)
    assert_g12(gW[sel].cpu().numpy(), rW, 1e-4, "gW")
    assert_g12(gb[sel].cpu().numpy(), rb, 1e-4, "gb")
    assert_rel(sq[sel].cpu().numpy(), rsq, 1e-4, "sqnorm")


def test_sqnorm_from_grads_and_clip_factors_match_oracle():
    """dp_sqnorm_from_grads (squared norm of materialized per-sample
    gradients) and dp_clip_factors on a random batch whose norms straddle C,
    including a zero norm and norms at C and just below it."""
    r = np.random.default_rng(77)
    for N, numel in [(1, 1), (37, 1000), (300, 4099), (5, 262144)]:
        say("sqnorm_from_grads", N, numel)
        G = (r.standard_normal((N, numel)) * r.uniform(0.01, 3.0, (N, 1))).astype(np.float32)
        G[0] = 0.0
        sq = torch.empty(N, device=DEV)
        dp.dp_sqnorm_from_grads(torch.from_numpy(G).to(DEV), N, numel, sq)
        rsq = np.zeros(N)
        oracle.sqnorm_accumulate(G.astype(np.float64), rsq)
        got = sq.cpu().numpy()
        assert got[0] == 0.0
        assert_rel(got[1:], rsq[1:], 1e-5, "sqnorm_from_grads")
    N, C = 4096, 1.3
    norm = np.exp(r.normal(np.log(C), 1.0, N)).astype(np.float32)
    norm[:4] = [0.0, C, np.float32(C - 1e-6), np.float32(C + 1e-6)]
    c = torch.empty(N, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dp.dp_clip_factors(torch.from_numpy(norm).to(DEV), N, C, c, status)
    ref = oracle.clip_factors(norm.astype(np.float64), C)
    got = c.cpu().numpy()
    assert_rel(got, ref, 1e-6, "clip factors")
    assert np.all((got == 1.0) == (ref == 1.0)), "which samples are left unclipped"
    assert int(status.item()) == 0


CONV_SHAPES = [  # N, Cin, H, W, Cout, kh, kw, sh, sw, ph, pw
    (2, 3, 7, 9, 5, 3, 3, 2, 2, 1, 1), (3, 1, 28, 28, 16, 8, 8, 2, 2, 3, 3), (2, 16, 13, 13, 32, 4, 4, 2, 2, 0, 0),
    (2, 3, 32, 32, 32, 3, 3, 1, 1, 1, 1), (1, 70, 6, 5, 33, 1, 1, 1, 1, 0, 0), (2, 5, 9, 4, 66, 2, 3, 1, 2, 1, 0),
    (1, 130, 8, 8, 129, 3, 3, 1, 1, 1, 1),
    (2, 8, 10, 10, 32, 4, 4, 1, 1, 0, 0),      # 128 x 32 tile, two-way K split
    (1, 2, 130, 130, 4, 3, 3, 1, 1, 1, 1),     # input planes too large for LDS: gathered fallback
    (2, 32, 32, 32, 64, 3, 3, 1, 1, 1, 1), (2, 64, 16, 16, 64, 3, 3, 1, 1, 1, 1),
    (2, 64, 16, 16, 128, 3, 3, 1, 1, 1, 1), (2, 128, 8, 8, 128, 3, 3, 1, 1, 1, 1),
    (2, 128, 8, 8, 256, 3, 3, 1, 1, 1, 1),
    (3, 4, 8, 8, 20, 3, 3, 1, 1, 0, 0),        # unpadded, sizes multiples of 4: direct-to-LDS staging
    (2, 12, 9, 10, 24, 3, 2, 2, 2, 0, 0),      # the same with stride 2
    # row chunks with full nine-block tiles at stride 1 (the branch-free contraction):
    (2, 32, 16, 16, 20, 3, 3, 1, 1, 1, 1),     # one channel block, four wave rows
    (2, 62, 8, 8, 64, 3, 3, 1, 1, 1, 1),       # two column tiles, the last block past the weight's columns
    (3, 32, 12, 12, 96, 3, 3, 1, 1, 1, 1)]     # a second channel tile only half used


# One shape per tile configuration of the fast path and staging mode (whole
# sample in one load round trip, or position chunks); batch sizes above 512
# workgroups select the four-wave tiles, smaller grids the eight-wave ones.
CONV_CONFIG_SHAPES = [
    (520, 1, 20, 21, 5, 1, 1, 1, 1, 1, 1), (520, 1, 5, 6, 5, 1, 1, 2, 2, 0, 0),            # 32 x 32, 4 waves
    (520, 33, 13, 14, 5, 1, 1, 1, 1, 1, 1), (520, 33, 5, 6, 5, 1, 1, 2, 2, 0, 0),          # 64 x 32, 4 waves
    (1, 1, 13, 14, 33, 1, 1, 1, 1, 1, 1), (1, 1, 5, 6, 33, 1, 1, 2, 2, 0, 0),              # 32 x 64
    (1, 33, 11, 12, 33, 1, 1, 1, 1, 1, 1), (1, 33, 5, 6, 33, 1, 1, 2, 2, 0, 0),            # 64 x 64
    (520, 24, 20, 21, 5, 2, 2, 2, 2, 1, 1), (520, 8, 5, 6, 5, 3, 3, 2, 2, 1, 1),           # 128 x 32, 4 waves
    (520, 24, 20, 21, 5, 3, 3, 2, 2, 1, 1), (520, 20, 5, 6, 5, 3, 3, 2, 2, 1, 1),          # 256 x 32, 4 waves
    (260, 24, 20, 21, 33, 2, 2, 2, 2, 0, 0), (260, 8, 5, 6, 33, 3, 3, 2, 2, 1, 1),         # 128 x 64
    (130, 12, 20, 21, 128, 3, 3, 2, 2, 0, 0), (130, 12, 5, 6, 128, 3, 3, 2, 2, 1, 1),      # 128 x 128
    (1, 12, 20, 21, 128, 2, 2, 2, 2, 0, 0), (1, 64, 6, 7, 128, 1, 1, 2, 2, 1, 1),          # 64 x 128
    (1, 1, 20, 21, 5, 1, 1, 1, 1, 1, 1), (1, 1, 5, 6, 5, 1, 1, 2, 2, 0, 0),                # 32 x 32, 8 waves
    (1, 33, 13, 14, 5, 1, 1, 1, 1, 1, 1), (1, 33, 5, 6, 5, 1, 1, 2, 2, 0, 0),              # 64 x 32, 8 waves
    (1, 24, 20, 21, 5, 2, 2, 2, 2, 1, 1), (1, 8, 5, 6, 5, 3, 3, 2, 2, 1, 1),               # 128 x 32, 8 waves
    (1, 24, 20, 21, 5, 3, 3, 2, 2, 1, 1), (1, 20, 5, 6, 5, 3, 3, 2, 2, 1, 1)]              # 256 x 32, 8 waves


@pytest.fixture(params=["auto", "tiled", "rows"])
def conv_path(request):
    """Run a conv test with the automatic kernel choice (one workgroup per
    sample for samples that fit LDS, else output row chunks), and again with
    the tiled and the row-chunked kernels forced."""
    path = {"tiled": dp.DP_CONV_TILED, "rows": dp.DP_CONV_ROWS}.get(request.param, dp.DP_CONV_AUTO)
    prev = dp.dp_conv2d_set_path(path)
    yield request.param
    dp.dp_conv2d_set_path(prev)


@pytest.mark.parametrize("shape", CONV_SHAPES + CONV_CONFIG_SHAPES)
def test_conv_shapes(shape, conv_path):
    N, Cin, H, Wd, Cout, kh, kw, sh, sw, ph, pw = shape
    say("conv", conv_path, shape)
    Ho = (H + 2 * ph - kh) // sh + 1
    Wo = (Wd + 2 * pw - kw) // sw + 1
    r = np.random.default_rng(sum(shape))
    X = r.standard_normal((N, Cin, H, Wd)).astype(np.float32)
    GY = (r.standard_normal((N, Cout, Ho, Wo)) / 4).astype(np.float32)
    Xt, Gt = torch.from_numpy(X).to(DEV), torch.from_numpy(GY).to(DEV)
    gW = torch.empty((N, Cout, Cin, kh, kw), device=DEV)
    gb = torch.empty((N, Cout), device=DEV)
    sq = torch.empty(N, device=DEV)
    ws = torch.empty(max(dp.dp_grad_sample_conv2d_workspace_bytes(N, Cin, H, Wd, Cout, kh, kw, sh, sw, ph, pw), 1),
                     dtype=torch.uint8, device=DEV)
    dp.dp_grad_sample_conv2d(Xt, Gt, dp.DP_F32, N, Cin, H, Wd, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw, 1, 1, 1, 1.3,
                             gW, gb, sq, None, ws)
    rW, rb = oracle.conv2d_grad(X, GY, (kh, kw), (sh, sw), (ph, pw), 1.3)
    rsq = np.zeros(N)
    oracle.sqnorm_accumulate(rW, rsq); oracle.sqnorm_accumulate(rb, rsq)
    assert_g12(gW.cpu().numpy(), rW, 1e-4, "conv gW")
    assert_g12(gb.cpu().numpy(), rb, 1e-4, "conv gb")
    assert_rel(sq.cpu().numpy(), rsq, 1e-4, "conv sqnorm")


def run_conv_case(shape, dt, scale, seed):
    N, Cin, H, Wd, Cout, kh, kw, sh, sw, ph, pw = shape
    Ho = (H + 2 * ph - kh) // sh + 1
    Wo = (Wd + 2 * pw - kw) // sw + 1
    r = np.random.default_rng(seed)
    X = torch.from_numpy(r.standard_normal((N, Cin, H, Wd)).astype(np.float32))
    GY = torch.from_numpy((r.standard_normal((N, Cout, Ho, Wo)) / 4).astype(np.float32))
    if dt == dp.DP_BF16:
        X, GY = X.to(torch.bfloat16), GY.to(torch.bfloat16)
    gW = torch.empty((N, Cout, Cin, kh, kw), device=DEV)
    gb = torch.empty((N, Cout), device=DEV)
    sq = torch.empty(N, device=DEV)
    ws = torch.empty(max(dp.dp_grad_sample_conv2d_workspace_bytes(N, Cin, H, Wd, Cout, kh, kw, sh, sw, ph, pw), 1),
                     dtype=torch.uint8, device=DEV)
    dp.dp_grad_sample_conv2d(X.to(DEV), GY.to(DEV), dt, N, Cin, H, Wd, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw, 1, 1, 1,
                             scale, gW, gb, sq, None, ws)
    Xr, Gr = X.float().numpy().astype(np.float64), GY.float().numpy().astype(np.float64)
    rW, rb = oracle.conv2d_grad(Xr, Gr, (kh, kw), (sh, sw), (ph, pw), scale)
    rsq = np.zeros(N)
    oracle.sqnorm_accumulate(rW, rsq); oracle.sqnorm_accumulate(rb, rsq)
    assert_g12(gW.cpu().numpy(), rW, 1e-4, "conv gW")
    assert_g12(gb.cpu().numpy(), rb, 1e-4, "conv gb")
    assert_rel(sq.cpu().numpy(), rsq, 1e-4, "conv sqnorm")


@pytest.mark.parametrize("dt", [dp.DP_F32, dp.DP_BF16])
def test_conv_rows_many_units(dt):
    """The row-chunked kernel on more (sample, tile) workgroups than the CUs
    hold at once (100 samples x 16 tiles of the CIFAR c6 shape), every
    sample compared with the oracle."""
    prev = dp.dp_conv2d_set_path(dp.DP_CONV_ROWS)
    try:
        shape = (100, 128, 8, 8, 256, 3, 3, 1, 1, 1, 1)
        say("conv many units", dt, shape)
        run_conv_case(shape, dt, 0.7, seed=91 + dt)
    finally:
        dp.dp_conv2d_set_path(prev)


@pytest.mark.parametrize("shape", [CONV_SHAPES[1], CONV_SHAPES[2], CONV_SHAPES[3], CONV_SHAPES[5], CONV_SHAPES[-3],
                                   CONV_SHAPES[-2]])
def test_conv_shapes_bf16(shape, conv_path):
    """bf16 inputs (scalar staging loads) against the oracle on the rounded values."""
    N, Cin, H, Wd, Cout, kh, kw, sh, sw, ph, pw = shape
    say("conv bf16", conv_path, shape)
    Ho = (H + 2 * ph - kh) // sh + 1
    Wo = (Wd + 2 * pw - kw) // sw + 1
    r = np.random.default_rng(sum(shape) + 1)
    X = torch.from_numpy(r.standard_normal((N, Cin, H, Wd)).astype(np.float32)).to(torch.bfloat16)
    GY = torch.from_numpy((r.standard_normal((N, Cout, Ho, Wo)) / 4).astype(np.float32)).to(torch.bfloat16)
    gW = torch.empty((N, Cout, Cin, kh, kw), device=DEV)
    gb = torch.empty((N, Cout), device=DEV)
    sq = torch.empty(N, device=DEV)
    ws = torch.empty(max(dp.dp_grad_sample_conv2d_workspace_bytes(N, Cin, H, Wd, Cout, kh, kw, sh, sw, ph, pw), 1),
                     dtype=torch.uint8, device=DEV)
    dp.dp_grad_sample_conv2d(X.to(DEV), GY.to(DEV), dp.DP_BF16, N, Cin, H, Wd, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw,
                             1, 1, 1, 0.9, gW, gb, sq, None, ws)
    Xr, Gr = X.float().numpy().astype(np.float64), GY.float().numpy().astype(np.float64)
    rW, rb = oracle.conv2d_grad(Xr, Gr, (kh, kw), (sh, sw), (ph, pw), 0.9)
    rsq = np.zeros(N)
    oracle.sqnorm_accumulate(rW, rsq); oracle.sqnorm_accumulate(rb, rsq)
    assert_g12(gW.cpu().numpy(), rW, 1e-4, "conv bf16 gW")
    assert_g12(gb.cpu().numpy(), rb, 1e-4, "conv bf16 gb")
    assert_rel(sq.cpu().numpy(), rsq, 1e-4, "conv bf16 sqnorm")


def run_embedding(ids, B, V, cap=None, scale=1.0, dt=None):
    N, T = ids.shape
    D = B.shape[2]
    cap = N * T if cap is None else cap
    dt = dp.DP_F32 if dt is None else dt
    idt = torch.from_numpy(ids).to(DEV)
    Bt = torch.from_numpy(B.astype(np.float32)).to(DEV)
    if dt == dp.DP_BF16:
        Bt = Bt.to(torch.bfloat16)
    rp = torch.empty(N + 1, dtype=torch.int64, device=DEV)
    uq = torch.full((max(cap, 1),), -7, dtype=torch.int64, device=DEV)
    rows = torch.zeros((max(cap, 1), D), device=DEV)
    sq = torch.empty(N, device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = torch.empty(max(dp.dp_grad_sample_embedding_workspace_bytes(N, T), 1), dtype=torch.uint8, device=DEV)
    dp.dp_grad_sample_embedding(idt, Bt, dt, N, T, V, D, scale, rp, uq, rows, cap, sq, st, ws)
    torch.cuda.synchronize()
    return rp.cpu().numpy(), uq.cpu().numpy(), rows.cpu().numpy(), sq.cpu().numpy(), int(st.item())


@pytest.mark.parametrize("D", [37, 100, 300])
@pytest.mark.parametrize("case", ["zipf", "truncated", "all_equal", "all_distinct", "T1", "long", "batch130",
                                  "bf16", "T600", "N2100", "equal256", "half_equal"])
def test_embedding_cases(case, D):
    say("embedding", case, D)
    r = np.random.default_rng(11)
    V = 1000
    dt = dp.DP_F32
    if case == "zipf":
        ids = np.minimum(r.zipf(1.1, (9, 256)), V) - 1
    elif case == "truncated":
        wl = W.Workload(99, "t", 6, W.F32, 1.0, 1.0, (W.Embedding("e", V, D, 200, truncate=True),))
        ids = W.make_inputs(wl)[0].ids
    elif case == "all_equal":
        ids = np.full((3, 50), 17)
    elif case == "all_distinct":
        ids = np.stack([r.permutation(V)[:300] for _ in range(4)])
    elif case == "T1":
        ids = r.integers(0, V, (8, 1))
    elif case == "batch130":        # three 64-sample chunks in the clipped sum
        ids = np.minimum(r.zipf(1.1, (130, 64)), V) - 1
    elif case == "bf16":
        ids = np.minimum(r.zipf(1.1, (9, 100)), V) - 1
        dt = dp.DP_BF16
    elif case == "T600":            # past the rank sort: the bitonic network with padding
        ids = np.minimum(r.zipf(1.1, (3, 600)), V) - 1
    elif case == "N2100":           # more samples than the rows pass adds up itself: a scan launch
        ids = np.minimum(r.zipf(1.3, (2100, 6)), V) - 1
    elif case == "equal256":        # several rows-pass workgroups per sample; the first owns every position
        ids = np.full((3, 256), 17)
    elif case == "half_equal":      # one segment across the workgroups' nominal split points, then distinct ids
        ids = np.stack([np.concatenate([np.full(160, 3), 10 + r.permutation(900)[:96]]) for _ in range(5)])
    else:
        ids = r.integers(0, 40, (2, 4096))
    ids = ids.astype(np.int64)
    B = r.standard_normal(ids.shape + (D,))
    if dt == dp.DP_BF16:
        B32 = torch.from_numpy(B.astype(np.float32)).to(torch.bfloat16).float().numpy().astype(np.float64)
    else:
        B32 = B.astype(np.float32).astype(np.float64)
    rp, uq, rows, sq, st = run_embedding(ids, B, V, scale=0.5, dt=dt)
    rrp, ruq, rrows = oracle.embedding_grad(ids, B32, V, 0.5)
    assert st == 0
    np.testing.assert_array_equal(rp, rrp)
    np.testing.assert_array_equal(uq[:rp[-1]], ruq)
    assert_g12(rows[:rp[-1]], rrows, 1e-4, "rows")
    rsq = np.array([np.sum(rrows[rrp[n]:rrp[n + 1]] ** 2) for n in range(ids.shape[0])])
    assert_rel(sq, rsq, 1e-4, "sqnorm")
    # dense clipped sum
    norm = np.sqrt(rsq)
    C = float(np.median(norm))
    c = oracle.clip_factors(norm.astype(np.float32).astype(np.float64), C)
    S = torch.full((V, D), 7.0, device=DEV)
    N = ids.shape[0]
    wsc = torch.empty(dp.dp_clip_accumulate_embedding_workspace_bytes(N, V), dtype=torch.uint8, device=DEV)
    dp.dp_clip_accumulate_embedding(torch.from_numpy(rp).to(DEV), torch.from_numpy(uq).to(DEV),
                                    torch.from_numpy(rows).to(DEV), rows.shape[0],
                                    torch.from_numpy(norm.astype(np.float32)).to(DEV), C, N, V, D, S, None, wsc)
    assert_g12(S.cpu().numpy(), oracle.clip_sum_embedding(rrp, ruq, rrows, c, V), 1e-4, "dense S")


def test_embedding_two_pass_scan():
    """T > 512 takes the two-launch path; with N > 2048 it adds the distinct
    counts in a scan launch of its own."""
    r = np.random.default_rng(14)
    V, D = 1000, 4
    ids = (np.minimum(r.zipf(1.3, (2100, 520)), V) - 1).astype(np.int64)
    B = r.standard_normal(ids.shape + (D,))
    say("embedding two-pass scan")
    rp, uq, rows, sq, st = run_embedding(ids, B, V, scale=0.5)
    rrp, ruq, rrows = oracle.embedding_grad(ids, B.astype(np.float32).astype(np.float64), V, 0.5)
    assert st == 0
    np.testing.assert_array_equal(rp, rrp)
    np.testing.assert_array_equal(uq[:rp[-1]], ruq)
    assert_g12(rows[:rp[-1]], rrows, 1e-4, "rows")


@pytest.mark.parametrize("T", [20, 600])
def test_embedding_flags(T):
    r = np.random.default_rng(12)
    ids = r.integers(0, 50, (3, T)).astype(np.int64)
    B = r.standard_normal((3, T, 4))
    # capacity too small: flagged, true counts kept, nothing written past cap
    say("embedding cap")
    rp, uq, rows, sq, st = run_embedding(ids, B, 50, cap=10)
    assert st & dp.DP_FLAG_CAP
    rrp, _, _ = oracle.embedding_grad(ids, B, 50)
    np.testing.assert_array_equal(rp, rrp)
    # the clipped sum over the truncated CSR: flagged, and only the stored rows count
    say("embedding clip cap")
    S = torch.empty((50, 4), device=DEV)
    stt = torch.zeros(1, dtype=torch.int32, device=DEV)
    wsc = torch.empty(dp.dp_clip_accumulate_embedding_workspace_bytes(3, 50), dtype=torch.uint8, device=DEV)
    dp.dp_clip_accumulate_embedding(torch.from_numpy(rp).to(DEV), torch.from_numpy(uq).to(DEV),
                                    torch.from_numpy(rows).to(DEV), 10, torch.ones(3, device=DEV), 1e9, 3, 50, 4, S,
                                    stt, wsc)
    assert int(stt.item()) & dp.DP_FLAG_CAP
    ref = np.zeros((50, 4))
    for k in range(10):
        ref[uq[k]] += rows[k]
    assert_g12(S.cpu().numpy(), ref, 1e-5, "clip over capped CSR")
    # an id outside [0, V): flagged and left out
    say("embedding bad id")
    bad = ids.copy(); bad[1, 3] = 50; bad[2, 0] = -1
    rp, uq, rows, sq, st = run_embedding(bad, B, 50)
    assert st & dp.DP_FLAG_BAD_INDEX


GN_SHAPES = [(3, 5, 7), (4, 16, 64), (2, 40, 1024), (5, 17, 9), (1, 64, 4096), (2, 3, 0)]


@pytest.mark.parametrize("N,C,P", GN_SHAPES)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_groupnorm_affine_matches_oracle(N, C, P, dtype):
    """GroupNorm / InstanceNorm affine per-sample grads against the oracle,
    over ragged position counts (scalar path), multiples of 4 (16-byte
    loads), one and several channel blocks, P = 0 (zero sums); with and
    without the bias, norms and repeated runs bit for bit."""
    r = np.random.default_rng(17 + N * 7 + C + P)
    say("groupnorm", N, C, P, dtype)
    xh = torch.from_numpy(r.standard_normal((N, C, P)).astype(np.float32)).to(dtype)
    B = torch.from_numpy(r.standard_normal((N, C, P)).astype(np.float32)).to(dtype)
    dt = dp.DP_BF16 if dtype == torch.bfloat16 else dp.DP_F32
    g = torch.full((N, C), 7.0, device=DEV); b = torch.full((N, C), 7.0, device=DEV)
    sq = torch.full((N,), 7.0, device=DEV)
    ws = torch.empty(max(dp.dp_grad_sample_groupnorm_workspace_bytes(N, C, P), 1), dtype=torch.uint8, device=DEV)
    xd, Bd = xh.to(DEV), B.to(DEV)
    dp.dp_grad_sample_groupnorm(xd, Bd, dt, N, C, P, 1.25, g, b, sq, None, ws)
    rg, rb = oracle.groupnorm_grad(xh.float().numpy(), B.float().numpy(), 1.25)
    rtol = 1e-4        # the oracle reads the same bf16 values; only fp32 sums differ
    assert_g12(g.cpu().numpy(), rg, rtol, "ggamma")
    assert_g12(b.cpu().numpy(), rb, rtol, "gbeta")
    assert_rel(sq.cpu().numpy(), (rg ** 2).sum(1) + (rb ** 2).sum(1), rtol, "groupnorm sqnorm")
    g2 = torch.empty_like(g); sq2 = torch.empty_like(sq)
    dp.dp_grad_sample_groupnorm(xd, Bd, dt, N, C, P, 1.25, g2, None, sq2, None, ws)
    np.testing.assert_array_equal(g2.cpu().numpy(), g.cpu().numpy())
    assert_rel(sq2.cpu().numpy(), (rg ** 2).sum(1), rtol, "groupnorm sqnorm without bias")
    g3 = torch.empty_like(g)
    dp.dp_grad_sample_groupnorm(xd, Bd, dt, N, C, P, 1.25, g3, None, None, None, ws)
    np.testing.assert_array_equal(g3.cpu().numpy(), g.cpu().numpy())


def test_layernorm_and_empty_inputs():
    r = np.random.default_rng(13)
    N, T, D = 3, 37, 771
    xh = r.standard_normal((N, T, D)).astype(np.float32)
    B = r.standard_normal((N, T, D)).astype(np.float32)
    say("layernorm")
    g = torch.empty((N, D), device=DEV); b = torch.empty((N, D), device=DEV); sq = torch.empty(N, device=DEV)
    ws = torch.empty(dp.dp_grad_sample_layernorm_workspace_bytes(N, T, D), dtype=torch.uint8, device=DEV)
    dp.dp_grad_sample_layernorm(torch.from_numpy(xh).to(DEV), torch.from_numpy(B).to(DEV), dp.DP_F32, N, T, D, 2.0,
                                g, b, sq, None, ws)
    rg, rb = oracle.layernorm_grad(xh, B, 2.0)
    assert_g12(g.cpu().numpy(), rg, 1e-4, "ggamma")
    assert_g12(b.cpu().numpy(), rb, 1e-4, "gbeta")
    assert_rel(sq.cpu().numpy(), (rg ** 2).sum(1) + (rb ** 2).sum(1), 1e-4, "ln sqnorm")
    # the vector path (D % 4 == 0), bf16 and fp32, with a position count that is not a multiple of 4
    for dtype in (torch.float32, torch.bfloat16):
        N2, T2, D2 = 3, 41, 1028
        xh2 = torch.from_numpy(r.standard_normal((N2, T2, D2)).astype(np.float32)).to(dtype)
        B2 = torch.from_numpy(r.standard_normal((N2, T2, D2)).astype(np.float32)).to(dtype)
        g2 = torch.empty((N2, D2), device=DEV); b2 = torch.empty((N2, D2), device=DEV)
        ws2 = torch.empty(dp.dp_grad_sample_layernorm_workspace_bytes(N2, T2, D2), dtype=torch.uint8, device=DEV)
        dt2 = dp.DP_BF16 if dtype == torch.bfloat16 else dp.DP_F32
        dp.dp_grad_sample_layernorm(xh2.to(DEV), B2.to(DEV), dt2, N2, T2, D2, 1.0, g2, b2, None, None, ws2)
        rg2, rb2 = oracle.layernorm_grad(xh2.float().numpy(), B2.float().numpy(), 1.0)
        assert_g12(g2.cpu().numpy(), rg2, 1e-4, "ggamma vec")
        assert_g12(b2.cpu().numpy(), rb2, 1e-4, "gbeta vec")
    # T = 0: empty sums are zero
    say("linear T=0")
    gW = torch.full((2, 3, 4), 5.0, device=DEV); gbias = torch.full((2, 3), 5.0, device=DEV)
    sq = torch.full((2,), 5.0, device=DEV)
    dp.dp_grad_sample_linear(None, None, dp.DP_F32, 2, 0, 4, 3, 1.0, gW, gbias, sq, None, None)
    assert float(gW.abs().sum()) == 0 and float(gbias.abs().sum()) == 0 and float(sq.abs().sum()) == 0
    # N = 0: the clipped sum is zero
    say("clip N=0")
    S = torch.full((10,), 5.0, device=DEV)
    dp.dp_clip_accumulate(None, None, 1.0, 0, 10, S)
    assert float(S.abs().sum()) == 0


def test_layernorm_many_matches_oracle_and_single_calls():
    """dp_grad_sample_layernorm_many: 16-byte and element-load layers, a
    partial last chunk, one-chunk layers (squared norm written directly), no
    positions, a layer without sqnorm; against the oracle and the
    single-layer call."""
    r = np.random.default_rng(17)
    for dtype, shapes in ((torch.bfloat16, [(37, 771), (41, 1028), (128, 768), (0, 64), (5, 40), (33, 8)]),
                          (torch.float32, [(37, 771), (41, 1028), (200, 100), (3, 32)])):
        N = 5
        dt = dp.DP_BF16 if dtype == torch.bfloat16 else dp.DP_F32
        say("layernorm many", dtype)
        ents, outs, ins = [], [], []
        for k, (T, D) in enumerate(shapes):
            xh = torch.from_numpy(r.standard_normal((N, T, D)).astype(np.float32)).to(dtype).to(DEV)
            B = torch.from_numpy(r.standard_normal((N, T, D)).astype(np.float32)).to(dtype).to(DEV)
            g = torch.full((N, D), 7.0, device=DEV)
            b = torch.full((N, D), 7.0, device=DEV)
            sq = None if k == 1 else torch.full((N,), 7.0, device=DEV)
            ents.append((xh, B, T, D, 1.5, g, b, sq))
            outs.append((g, b, sq))
            ins.append((xh, B, T, D))
        items = dp.make_layernorm_layers(ents)
        ws = torch.empty(max(dp.dp_grad_sample_layernorm_many_workspace_bytes(items, len(ents), N, dt), 1),
                         dtype=torch.uint8, device=DEV)
        dp.dp_grad_sample_layernorm_many(items, len(ents), dt, N, None, ws)
        torch.cuda.synchronize()
        for (xh, B, T, D), (g, b, sq) in zip(ins, outs):
            rg, rb = oracle.layernorm_grad(xh.float().cpu().numpy().astype(np.float64),
                                           B.float().cpu().numpy().astype(np.float64), 1.5)
            assert_g12(g.cpu().numpy(), rg, 1e-4, "ggamma many T=%d D=%d" % (T, D))
            assert_g12(b.cpu().numpy(), rb, 1e-4, "gbeta many T=%d D=%d" % (T, D))
            if sq is not None:
                assert_rel(sq.cpu().numpy(), (rg ** 2).sum(1) + (rb ** 2).sum(1), 1e-4, "ln many sqnorm")
            g1 = torch.empty((N, D), device=DEV); b1 = torch.empty((N, D), device=DEV)
            ws1 = torch.empty(max(dp.dp_grad_sample_layernorm_workspace_bytes(N, T, D), 1), dtype=torch.uint8,
                              device=DEV)
            dp.dp_grad_sample_layernorm(xh, B, dt, N, T, D, 1.5, g1, b1, None, None, ws1)
            torch.cuda.synchronize()
            assert_g12(g.cpu().numpy(), g1.cpu().numpy(), 1e-5, "many vs single")
            assert_g12(b.cpu().numpy(), b1.cpu().numpy(), 1e-5, "many vs single")


def test_layernorm_many_more_layers_than_one_launch_table():
    """18 LayerNorm layers (two launches of up to 16), against single calls."""
    r = np.random.default_rng(18)
    N = 3
    say("layernorm many, 18 layers")
    ents, outs, ins = [], [], []
    for k in range(18):
        T, D = 5 + 7 * (k % 4), 64 * (1 + k % 3) + (4 if k % 5 == 0 else 0)
        xh = torch.from_numpy(r.standard_normal((N, T, D)).astype(np.float32)).to(DEV)
        B = torch.from_numpy(r.standard_normal((N, T, D)).astype(np.float32)).to(DEV)
        g = torch.empty((N, D), device=DEV); b = torch.empty((N, D), device=DEV); sq = torch.empty(N, device=DEV)
        ents.append((xh, B, T, D, 0.7, g, b, sq)); outs.append((g, b, sq)); ins.append((xh, B, T, D))
    items = dp.make_layernorm_layers(ents)
    ws = torch.empty(max(dp.dp_grad_sample_layernorm_many_workspace_bytes(items, 18, N, dp.DP_F32), 1),
                     dtype=torch.uint8, device=DEV)
    dp.dp_grad_sample_layernorm_many(items, 18, dp.DP_F32, N, None, ws)
    torch.cuda.synchronize()
    for (xh, B, T, D), (g, b, sq) in zip(ins, outs):
        g1 = torch.empty((N, D), device=DEV); b1 = torch.empty((N, D), device=DEV); sq1 = torch.empty(N, device=DEV)
        ws1 = torch.empty(max(dp.dp_grad_sample_layernorm_workspace_bytes(N, T, D), 1), dtype=torch.uint8,
                          device=DEV)
        dp.dp_grad_sample_layernorm(xh, B, dp.DP_F32, N, T, D, 0.7, g1, b1, sq1, None, ws1)
        torch.cuda.synchronize()
        assert_g12(g.cpu().numpy(), g1.cpu().numpy(), 1e-5, "18 layers ggamma")
        assert_g12(b.cpu().numpy(), b1.cpu().numpy(), 1e-5, "18 layers gbeta")
        assert_rel(sq.cpu().numpy(), sq1.cpu().numpy(), 1e-5, "18 layers sqnorm")


def test_nonfinite_sample_poisons_instead_of_passing():
    wl = W.get("linear_tiny")
    inputs = W.make_inputs(wl, n=8)
    inputs[0].B[3, 0] = np.nan
    say("nonfinite")
    st = DPStep(wl, inputs, DEV)
    st.run()
    got = st.results()
    assert got["status"] & dp.DP_FLAG_NONFINITE
    assert math.isnan(got["norm"][3])
    assert np.isnan(got["S"]["fc.weight"]).any()


def test_sigma0_Cinf_reproduces_the_mean_gradient():
    wl = W.get("mnist_cnn")
    inputs = W.make_inputs(wl, n=16)
    say("sigma0 Cinf")
    st = DPStep(wl, inputs, DEV, C=math.inf, sigma=0.0)
    st.run()
    got = st.results()
    ref = oracle.dp_step(wl, inputs, C=math.inf, sigma=0.0)
    for k in ref["out"]:
        assert_g12(got["out"][k], ref["out"][k], 1e-4, k)


def test_clip_noise_many_matches_the_single_tensor_calls():
    r = np.random.default_rng(21)
    for N in (0, 5, 300):
        say("clip_noise_many N=", N)
        shapes = [1, 7, 1024, 4099, 16, 33 * 3]
        norm = torch.from_numpy(r.uniform(0.1, 3.0, max(N, 1)).astype(np.float32)).to(DEV)
        entries, refs = [], []
        for i, numel in enumerate(shapes):
            G = torch.from_numpy(r.standard_normal((max(N, 1), numel)).astype(np.float32)).to(DEV)[:N]
            S = torch.full((numel,), 7.0, device=DEV)
            O = torch.empty(numel, device=DEV)
            if i % 3 == 2:      # sum given (fused route): only noise
                S = torch.from_numpy(r.standard_normal(numel).astype(np.float32)).to(DEV)
                entries.append((None, S, O, numel, i + 3))
            elif i % 3 == 1:    # clip only, no output
                entries.append((G, S, None, numel, i + 3))
            else:
                entries.append((G, S, O, numel, i + 3))
            refs.append((G, S.clone(), O))
        params = dp.make_params(entries)
        ws = torch.empty(max(dp.dp_clip_noise_many_workspace_bytes(params, len(entries), N), 1), dtype=torch.uint8,
                         device=DEV)
        dp.dp_clip_noise_many(params, len(entries), N, norm, 1.3, 5, 9, None, 0.7, 11.0, None, ws)
        for (g, s, o, numel, pidx), (G, S0, _) in zip(entries, refs):
            if g is not None:
                Sr = torch.empty(numel, device=DEV)
                ws2 = torch.empty(max(dp.dp_clip_accumulate_workspace_bytes(N, numel), 1), dtype=torch.uint8,
                                  device=DEV)
                dp.dp_clip_accumulate(G if N else None, norm if N else None, 1.3, N, numel, Sr, None, None, ws2)
                assert_g12(s.cpu().numpy(), Sr.cpu().numpy(), 1e-6, "sum")
            else:
                Sr = S0
            if o is not None:
                Or = torch.empty(numel, device=DEV)
                dp.dp_add_noise(Sr, Or, numel, 5, 9, pidx, 0.7, 1.3, 11.0)
                assert_g12(o.cpu().numpy(), Or.cpu().numpy(), 1e-6, "out")


def test_graph_replay_matches_eager_steps():
    wl = W.get("mnist_cnn")
    inputs = W.make_inputs(wl, n=20)
    st = DPStep(wl, inputs, DEV)
    say("graph capture mnist_cnn")
    st.capture(first_step=4)
    eager = DPStep(wl, inputs, DEV)
    for k in range(4):
        st.replay()
        got = st.results()
        eager.run(step=4 + k)                      # eager work between replays
        ref = eager.results()
        for name in ref["out"]:
            np.testing.assert_array_equal(got["out"][name], ref["out"][name], err_msg="replay %d %s" % (k, name))
            np.testing.assert_array_equal(got["S"][name], ref["S"][name])
        np.testing.assert_array_equal(got["norm"], ref["norm"])
    assert int(st.step_dev.item()) == 7     # the counter holds the last replayed step


@pytest.mark.parametrize("name,n,mode", [("text_lstm", 8, "materialize"), ("transformer_block", 4, "materialize"),
                                         ("transformer_block", 4, "ghost")])
def test_grouped_calls_replay_like_eager(name, n, mode):
    """Graph replays of the steps whose calls keep state between launches of
    one call (the embedding's ticket and per-sample states, cleared by a fill
    kernel) or group layers (LayerNorm, ghost norms): every replay, with eager
    work in between, equals the eager step bit for bit."""
    wl = W.get(name)
    inputs = W.make_inputs(wl, n=n)
    clip = "fused" if mode == "ghost" else "auto"          # ghost norms need the fused clipped sum
    st = DPStep(wl, inputs, DEV, clip_mode=clip, norm_mode=mode)
    if mode == "ghost":
        assert st.ghost
    say("graph capture", name, mode)
    st.capture(first_step=3)
    eager = DPStep(wl, inputs, DEV, clip_mode=clip, norm_mode=mode)
    for k in range(3):
        st.replay()
        got = st.results()
        eager.run(step=3 + k)
        ref = eager.results()
        np.testing.assert_array_equal(got["norm"], ref["norm"], err_msg="replay %d norm" % k)
        for key in ref["out"]:
            np.testing.assert_array_equal(got["out"][key], ref["out"][key], err_msg="replay %d %s" % (k, key))
    assert int(st.status.item()) == 0


@pytest.mark.parametrize("parallel", [False, True])
def test_graph_with_several_steps_per_replay(parallel):
    """A graph holding three steps: each replay runs steps s, s+1, s+2 (each
    with its own noise), leaving the last step's outputs."""
    wl = W.get("mnist_cnn")
    inputs = W.make_inputs(wl, n=20)
    st = DPStep(wl, inputs, DEV)
    if parallel:
        # branches take one step per replay (refused on the host before any capture)
        with pytest.raises(ValueError):
            st.capture(first_step=2, parallel=True, steps_per_replay=3)
        say("graph capture mnist_cnn, branches, 1 step per replay")
        st.capture(first_step=2, parallel=True)
        eager = DPStep(wl, inputs, DEV)
        for k in range(2):
            st.replay()
            got = st.results()
            eager.run(step=2 + k)
            ref = eager.results()
            for name in ref["out"]:
                np.testing.assert_array_equal(got["out"][name], ref["out"][name], err_msg="replay %d %s" % (k, name))
        return
    say("graph capture mnist_cnn, 3 steps per replay, parallel", parallel)
    st.capture(first_step=2, parallel=parallel, steps_per_replay=3)
    eager = DPStep(wl, inputs, DEV)
    for k in range(2):
        st.replay()
        got = st.results()
        eager.run(step=2 + 3 * k + 2)
        ref = eager.results()
        for name in ref["out"]:
            np.testing.assert_array_equal(got["out"][name], ref["out"][name], err_msg="replay %d %s" % (k, name))
        np.testing.assert_array_equal(got["norm"], ref["norm"])
    assert int(st.step_dev.item()) == 5     # the first step of the last replay (steps 5, 6, 7)


def test_noise_schedule_and_expected_batch_match_oracle():
    """A noise schedule (three entries, step t takes entry min(t, 2), one of
    them 0) and an expected-batch denominator (q times a pool of 40): each
    eager step matches the oracle's step with that step's sigma and the same
    denominator; a one-entry schedule equals the fixed sigma bit for bit."""
    wl = W.get("mnist_cnn")
    inputs = W.make_inputs(wl, n=12)
    sched = [1.3, 0.0, 0.6]
    denom = 0.25 * 40
    st = DPStep(wl, inputs, DEV, sigma_schedule=sched, denom=denom)
    for t in (0, 1, 2, 5):
        say("noise schedule, step", t)
        st.run(step=t)
        got = st.results()
        ref = oracle.dp_step(wl, inputs, step=t, sigma=sched[min(t, 2)], denom=denom)
        compare_step(wl, inputs, got, ref, RTOL[wl.dtype], "schedule step %d" % t)
    one = DPStep(wl, inputs, DEV, sigma_schedule=[0.7])
    fixed = DPStep(wl, inputs, DEV, sigma=0.7)
    one.run(step=4)
    fixed.run(step=4)
    a, b = one.results(), fixed.results()
    for k in b["out"]:
        np.testing.assert_array_equal(a["out"][k], b["out"][k], err_msg=k)


@pytest.mark.parametrize("parallel", [False, True])
def test_noise_schedule_in_a_graph_matches_eager(parallel):
    """A captured graph with three steps per replay follows the schedule
    from replay to replay (the step counter on the device picks the entry)."""
    wl = W.get("mnist_cnn")
    inputs = W.make_inputs(wl, n=20)
    sched = [0.5, 1.5, 0.0, 2.0, 0.25]
    st = DPStep(wl, inputs, DEV, sigma_schedule=sched)
    if parallel:
        with pytest.raises(ValueError):     # branches take one step per replay
            st.capture(first_step=1, parallel=True, steps_per_replay=3)
        return
    say("graph with a noise schedule, parallel", parallel)
    st.capture(first_step=1, parallel=parallel, steps_per_replay=3)
    eager = DPStep(wl, inputs, DEV, sigma_schedule=sched)
    for k in range(3):
        st.replay()
        got = st.results()
        eager.run(step=1 + 3 * k + 2)
        ref = eager.results()
        for name in ref["out"]:
            np.testing.assert_array_equal(got["out"][name], ref["out"][name], err_msg="replay %d %s" % (k, name))
    assert got["status"] == 0


def _prefix(inputs, n):
    return W.take_samples(inputs, slice(0, n))


@pytest.mark.parametrize("name,nmax", [("mnist_cnn", 20), ("text_lstm", 9), ("transformer_block", 5),
                                       ("text_lstm_bptt", 6)])
def test_variable_batch_in_a_graph_matches_eager(name, nmax):
    """A graph captured once on nmax rows follows the batch size set on the
    device before each replay (Poisson sampling's variable batch): its noised
    outputs match an eager step on just the active rows, the padding rows
    (random, nonzero) add nothing, their norms are -1, and an empty batch
    leaves every clipped sum zero.  Covers the norms folded into the clip
    launch (MNIST), the embedding's and the bf16 fused clipped sums (the LSTM
    and the transformer block take their norms first)."""
    wl = W.get(name)
    inputs = W.make_inputs(wl, n=nmax)
    denom = 0.8 * nmax                        # an expected batch size q * pool
    st = DPStep(wl, inputs, DEV, denom=denom, variable_batch=True)
    say("variable batch in a graph", name, nmax)
    st.capture(first_step=0, steps_per_replay=1)
    for k, na in enumerate([nmax, nmax // 2 + 1, 0, 1, nmax - 1]):
        st.set_active(na)
        st.replay()
        got = st.results()
        assert got["status"] == 0, (k, na)
        assert np.all(got["norm"][na:] == -1.0), (k, na)
        # the oracle's step over just the active rows, same step and divisor
        ref_o = oracle.dp_step(wl, _prefix(inputs, na), step=k, denom=denom)
        for pn in ref_o["out"]:
            assert_g12(got["out"][pn], ref_o["out"][pn], RTOL[wl.dtype], "oracle replay %d (batch %d) %s" % (k, na, pn))
            assert_g12(got["S"][pn], ref_o["S"][pn], RTOL[wl.dtype], "oracle S %d (batch %d) %s" % (k, na, pn))
        if na == 0:
            for pn, v in got["S"].items():
                assert np.all(v == 0.0), (k, pn)
            continue
        assert_rel(got["norm"][:na], ref_o["norm"], RTOL[wl.dtype], "oracle norms %d" % k)
        eager = DPStep(wl, _prefix(inputs, na), DEV, denom=denom)
        eager.run(step=k)
        ref = eager.results()
        np.testing.assert_allclose(got["norm"][:na], ref["norm"], rtol=1e-5, err_msg="norms %d" % k)
        for pn in ref["out"]:
            r = ref["out"][pn]
            np.testing.assert_allclose(got["out"][pn], r, rtol=2e-4, atol=2e-5 * float(np.abs(r).max() + 1e-30),
                                       err_msg="replay %d (batch %d) %s" % (k, na, pn))


def test_negative_norm_gives_a_zero_clip_factor():
    """The padding marker: dp_per_sample_norms_active writes -1 past the
    active size (clamped to N) without a flag, and dp_clip_factors maps a
    negative norm to 0 while a NaN norm still gives NaN and the flag."""
    r = np.random.default_rng(5)
    sq = torch.tensor(r.random((3, 10), dtype=np.float32), device=DEV)
    norm = torch.empty(10, dtype=torch.float32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    for na, want in [(4, 4), (0, 0), (25, 10), (-3, 0)]:
        nd = torch.tensor([na], dtype=torch.int64, device=DEV)
        dp.dp_per_sample_norms_active(sq, 3, 10, nd, norm, status)
        got = norm.cpu().numpy()
        ref = np.sqrt(sq.cpu().numpy().astype(np.float64).sum(axis=0))
        np.testing.assert_allclose(got[:want], ref[:want], rtol=1e-6)
        assert np.all(got[want:] == -1.0)
    assert int(status.item()) == 0
    nrm = torch.tensor([-1.0, 0.5, 4.0, float("nan")], device=DEV)
    c = torch.empty(4, dtype=torch.float32, device=DEV)
    dp.dp_clip_factors(nrm, 4, 1.0, c, status)
    cv = c.cpu().numpy()
    assert cv[0] == 0.0 and cv[1] == 1.0 and abs(cv[2] - 1.0 / (4.0 + 1e-6)) < 1e-7 and np.isnan(cv[3])
    assert int(status.item()) & dp.DP_FLAG_NONFINITE


def test_noise_schedule_bad_entry_raises_the_flag():
    """A negative schedule entry raises DP_FLAG_NONFINITE for that step and
    leaves NaN outputs; the steps before it are unaffected."""
    wl = W.get("linear_tiny")
    inputs = W.make_inputs(wl)
    st = DPStep(wl, inputs, DEV, sigma_schedule=[0.5, -1.0])
    st.run(step=0)
    ok = st.results()
    assert ok["status"] == 0
    st.run(step=1)
    bad = st.results()
    assert bad["status"] & dp.DP_FLAG_NONFINITE
    assert all(np.isnan(v).all() for v in bad["out"].values())


@pytest.mark.parametrize("numel,N", [(4 * 64 * 300, 37), (4 * 32 * 300, 70), (4 * 16 * 100, 33), (4099, 129)])
def test_norms_clip_noise_each_sample_group_count_matches_oracle(numel, N):
    """The one-launch clip takes 4, 8 or 16 sample groups per workgroup from
    the tensors' sizes (the first three shapes give 4, 8 and 16; the last is
    a scalar-column tensor): norms, clipped sum and noised output each
    against the oracle."""
    r = np.random.default_rng(numel + N)
    say("norms_clip_noise groups, numel", numel, "N", N)
    L, C, sigma, denom, seed, step = 2, 0.9, 0.7, 41.0, 23, 6
    sq_h = r.uniform(0.05, 2.0, (L, N)).astype(np.float32)
    G_h = r.standard_normal((N, numel)).astype(np.float32)
    sq = torch.from_numpy(sq_h).to(DEV)
    G = torch.from_numpy(G_h).to(DEV)
    S = torch.empty(numel, device=DEV)
    O = torch.empty(numel, device=DEV)
    norm = torch.empty(N, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    pa = dp.make_params([(G, S, O, numel, 3)])
    dp.dp_norms_clip_noise(sq, L, pa, 1, N, norm, C, seed, step, None, sigma, denom, status, None)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    nr = oracle.norms(sq_h.astype(np.float64).sum(axis=0))   # layers added, then the root
    assert_rel(norm.cpu().numpy(), nr, RTOL["f32"], "norms")
    ref_s = oracle.clip_sum(G_h, oracle.clip_factors(nr, C))
    assert_g12(S.cpu().numpy(), ref_s, RTOL["f32"], "clipped sum")
    ref_o = oracle.add_noise(ref_s, seed, step, 3, sigma, C, denom)
    assert_g12(O.cpu().numpy(), ref_o, RTOL["f32"], "noised output")


@pytest.mark.parametrize("N", [0, 5, 40, 300, 4100])
def test_norms_clip_noise_one_launch_matches_two_launch_path(N):
    """dp_norms_clip_noise (norms, column reduce and finish in one launch)
    matches dp_per_sample_norms + dp_clip_noise_many: norms bit for bit, sums
    and outputs to rounding (the two group the samples differently), and it is
    bitwise repeatable, also with more than 40 tensors and more samples than
    its LDS chunk of clip factors."""
    r = np.random.default_rng(31 + N)
    say("norms_clip_noise N=", N)
    shapes = [1, 7, 1024, 4099, 16, 33 * 3, 5000, 8] * 6      # 48 tensors: two groups
    if N > 1000:
        shapes = [1, 7, 64, 4099, 16, 33, 500, 8] * 6
    L = 3
    sq = torch.from_numpy(r.uniform(0.01, 1.5, (L, max(N, 1))).astype(np.float32)).to(DEV)[:, :N].contiguous()
    entries_a, entries_b = [], []
    for i, numel in enumerate(shapes):
        G = torch.from_numpy(r.standard_normal((max(N, 1), numel)).astype(np.float32)).to(DEV)[:N]
        Sa, Sb = torch.full((numel,), 7.0, device=DEV), torch.full((numel,), 7.0, device=DEV)
        Oa, Ob = torch.empty(numel, device=DEV), torch.empty(numel, device=DEV)
        if i % 5 == 2:      # sum given (fused route): only noise
            Sa.copy_(torch.from_numpy(r.standard_normal(numel).astype(np.float32)))
            Sb.copy_(Sa)
            entries_a.append((None, Sa, Oa, numel, i))
            entries_b.append((None, Sb, Ob, numel, i))
        elif i % 5 == 4:    # no output
            entries_a.append((G, Sa, None, numel, i))
            entries_b.append((G, Sb, None, numel, i))
        else:
            entries_a.append((G, Sa, Oa, numel, i))
            entries_b.append((G, Sb, Ob, numel, i))
    pa, pb = dp.make_params(entries_a), dp.make_params(entries_b)
    n = len(shapes)
    assert dp.dp_norms_clip_noise_workspace_bytes(pa, n, N) == 0
    ws_b = torch.empty(max(dp.dp_clip_noise_many_workspace_bytes(pb, n, N), 1), dtype=torch.uint8, device=DEV)
    norm_a = torch.full((max(N, 1),), -1.0, device=DEV)
    norm_b = torch.full((max(N, 1),), -1.0, device=DEV)
    first = None
    for step in (3, 3, 5):
        dp.dp_norms_clip_noise(sq, L, pa, n, N, norm_a, 1.1, 17, step, None, 0.9, 13.0, None, None)
        if N:
            dp.dp_per_sample_norms(sq, L, N, norm_b)
        dp.dp_clip_noise_many(pb, n, N, norm_b, 1.1, 17, step, None, 0.9, 13.0, None, ws_b)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(norm_a.cpu().numpy()[:N], norm_b.cpu().numpy()[:N])
        got = [(sa.cpu().numpy(), None if oa is None else oa.cpu().numpy()) for (_, sa, oa, _, _) in entries_a]
        for (ga, sa, oa, numel, _), (gb, sb, ob, _, _) in zip(entries_a, entries_b):
            assert_g12(sa.cpu().numpy(), sb.cpu().numpy(), 1e-5, "S numel %d" % numel)
            if oa is not None:
                assert_g12(oa.cpu().numpy(), ob.cpu().numpy(), 1e-5, "out numel %d" % numel)
        if first is None:
            first = got
        elif step == 3:
            for (s1, o1), (s2, o2) in zip(first, got):      # same step again: the same bits
                np.testing.assert_array_equal(s1, s2)
                if o1 is not None:
                    np.testing.assert_array_equal(o1, o2)
    # a given norm (sqnorm NULL) is read, not written
    if N:
        dp.dp_norms_clip_noise(None, 0, pa, n, N, norm_b, 1.1, 17, 6, None, 0.9, 13.0, None, None)
        dp.dp_clip_noise_many(pb, n, N, norm_b, 1.1, 17, 6, None, 0.9, 13.0, None, ws_b)
        torch.cuda.synchronize()
        for (ga, sa, oa, numel, _), (gb, sb, ob, _, _) in zip(entries_a, entries_b):
            assert_g12(sa.cpu().numpy(), sb.cpu().numpy(), 1e-5, "S numel %d" % numel)
