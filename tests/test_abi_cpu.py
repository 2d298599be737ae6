"""C-ABI contract on the CPU: the library loads, exports every declared symbol,
and rejects invalid arguments on the host before anything reaches HIP."""
import math
import os
import re

import pytest

from paper_2109_12298_amd import binding as dp
from paper_2109_12298_amd import step as stepmod
from paper_2109_12298_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    names = set()
    inc = os.path.join(ROOT, "include")
    for fn in os.listdir(inc):
        if fn.endswith(".h"):
            text = open(os.path.join(inc, fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(dp_[a-z0-9_]+)\s*\(", text))
    return names


def test_library_exports_every_declared_symbol():
    L = dp.lib()
    names = declared_symbols()
    assert len(names) >= 20
    for n in names:
        assert hasattr(L, n), n
    assert names == set(dp.SIGNATURES), names ^ set(dp.SIGNATURES)


def test_status_strings_and_version():
    assert dp.dp_abi_version() == 1
    for code in range(6):
        s = dp.dp_status_string(code)
        assert s.startswith(["DP_OK", "DP_EINVAL", "DP_EDTYPE", "DP_EUNSUPPORTED", "DP_ECAP", "DP_EHIP"][code])
    assert dp.dp_status_string(99) == "unknown dp_status"


def code_of(fn, *a, **k):
    try:
        fn(*a, **k)
    except dp.DPError as e:
        return e.code
    return dp.DP_OK


# Addresses below are never dereferenced: every call fails validation first.
FAKE = 0x1000


def test_linear_validation():
    f = dp.dp_grad_sample_linear
    assert code_of(f, FAKE, FAKE, 7, 2, 1, 3, 4, 1.0, FAKE, stream=0) == dp.DP_EDTYPE
    assert code_of(f, FAKE, FAKE, dp.DP_F32, -1, 1, 3, 4, 1.0, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 1, 0, 4, 1.0, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(f, None, FAKE, dp.DP_F32, 2, 1, 3, 4, 1.0, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 1, 3, 4, 1.0, None, stream=0) == dp.DP_EINVAL
    # T > 1 with a per-sample norm needs a workspace
    assert dp.dp_grad_sample_linear_workspace_bytes(2, 8, 3, 4, dp.DP_F32) > 0
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 8, 3, 4, 1.0, FAKE, None, FAKE, stream=0) == dp.DP_EINVAL
    assert dp.dp_grad_sample_linear_workspace_bytes(2, 1, 3, 4, dp.DP_F32) == 0


def test_conv_validation():
    f = dp.dp_grad_sample_conv2d
    # N, Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw, dh, dw, groups
    good = (2, 3, 8, 8, 4, 8, 8, 3, 3, 1, 1, 1, 1, 1, 1, 1)
    assert code_of(f, FAKE, FAKE, dp.DP_F32, *good[:15], 2, 1.0, FAKE, stream=0) == dp.DP_EUNSUPPORTED
    bad_dil = good[:13] + (2, 1, 1)
    assert code_of(f, FAKE, FAKE, dp.DP_F32, *bad_dil, 1.0, FAKE, stream=0) == dp.DP_EUNSUPPORTED
    bad_ho = good[:5] + (7,) + good[6:]
    assert code_of(f, FAKE, FAKE, dp.DP_F32, *bad_ho, 1.0, FAKE, stream=0) == dp.DP_EINVAL
    too_small = (2, 3, 2, 2, 4, 0, 0, 5, 5, 1, 1, 0, 0, 1, 1, 1)
    assert code_of(f, FAKE, FAKE, dp.DP_F32, *too_small, 1.0, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(f, FAKE, FAKE, 9, *good, 1.0, FAKE, stream=0) == dp.DP_EDTYPE


def test_noalloc_linear_validation():
    f = dp.dp_grad_sample_linear_noalloc
    assert dp.dp_grad_sample_linear_noalloc_max_bytes() == 8 << 20
    # a workspace beyond the fixed scratch array: refused before anything is enqueued
    assert dp.dp_grad_sample_linear_workspace_bytes(2**20, 2, 1024, 1024, dp.DP_F32) > 8 << 20
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2**20, 2, 1024, 1024, 1.0, FAKE, FAKE, FAKE, stream=0) == dp.DP_ECAP
    assert code_of(f, FAKE, FAKE, 7, 2, 2, 8, 8, 1.0, FAKE, stream=0) == dp.DP_EDTYPE
    assert code_of(f, None, FAKE, dp.DP_F32, 2, 2, 8, 8, 1.0, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 2, 8, 8, 1.0, None, stream=0) == dp.DP_EINVAL


def test_lstm_backward_validation():
    f = dp.dp_lstm_backward
    assert code_of(f, FAKE, FAKE, FAKE, None, FAKE, 2, 5, 129, FAKE, stream=0) == dp.DP_EUNSUPPORTED
    assert code_of(f, FAKE, FAKE, FAKE, None, FAKE, 2, 5, 0, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(f, None, FAKE, FAKE, None, FAKE, 2, 5, 100, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(f, FAKE, FAKE, FAKE, None, FAKE, 2, 5, 100, None, stream=0) == dp.DP_EINVAL
    assert code_of(f, FAKE, FAKE, FAKE, None, FAKE, -1, 5, 100, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(f, None, None, None, None, None, 0, 5, 100, None, stream=0) == dp.DP_OK   # nothing to do


def test_embedding_layernorm_validation():
    f = dp.dp_grad_sample_embedding
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 5000, 10, 4, 1.0, FAKE, FAKE, FAKE, 10, stream=0) == \
        dp.DP_EUNSUPPORTED
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 5, 2**31, 4, 1.0, FAKE, FAKE, FAKE, 10, stream=0) == dp.DP_EINVAL
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 5, 10, 4, 1.0, None, FAKE, FAKE, 10, stream=0) == dp.DP_EINVAL
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 5, 10, 4, 1.0, FAKE, FAKE, FAKE, 10, None, None, None,
                   stream=0) == dp.DP_EINVAL   # workspace required
    # N*T beyond 32-bit position indices is refused before anything is enqueued
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2**20, 4096, 10, 4, 1.0, FAKE, FAKE, FAKE, 10, stream=0) == \
        dp.DP_EUNSUPPORTED
    g = dp.dp_grad_sample_layernorm
    assert code_of(g, FAKE, FAKE, dp.DP_F32, 2, 5, 0, 1.0, FAKE, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(g, FAKE, FAKE, dp.DP_F32, 2, 5, 8, 1.0, FAKE, None, stream=0) == dp.DP_EINVAL


def test_clip_and_noise_validation():
    assert code_of(dp.dp_clip_factors, FAKE, 4, 0.0, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(dp.dp_clip_factors, FAKE, 4, -1.0, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(dp.dp_per_sample_norms, None, 2, 4, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(dp.dp_clip_accumulate, FAKE, FAKE, 1.0, 4, 10, None, stream=0) == dp.DP_EINVAL
    n = dp.dp_clip_accumulate_workspace_bytes(4096, 10)
    assert n > 0
    assert code_of(dp.dp_clip_accumulate, FAKE, FAKE, 1.0, 4096, 10, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(dp.dp_clip_accumulate_embedding, FAKE, FAKE, FAKE, 8, FAKE, 1.0, 2, 0, 4, FAKE,
                   stream=0) == dp.DP_EINVAL
    nb = dp.dp_clip_accumulate_embedding_workspace_bytes(2, 10)
    assert nb >= 10 * 64 * 4
    assert code_of(dp.dp_clip_accumulate_embedding, FAKE, FAKE, FAKE, 8, FAKE, 1.0, 2, 10, 4, FAKE,
                   stream=0) == dp.DP_EINVAL     # workspace missing
    f = dp.dp_add_noise
    assert code_of(f, FAKE, FAKE, 16, 0, 0, 0, 1.0, math.inf, 4.0, stream=0) == dp.DP_EINVAL  # sigma>0, C=inf
    assert code_of(f, FAKE, FAKE, 16, 0, 0, 0, -1.0, 1.0, 4.0, stream=0) == dp.DP_EINVAL
    assert code_of(f, FAKE, FAKE, 16, 0, 0, 0, 1.0, 1.0, 0.0, stream=0) == dp.DP_EINVAL
    assert code_of(f, None, FAKE, 16, 0, 0, 0, 1.0, 1.0, 1.0, stream=0) == dp.DP_EINVAL
    assert code_of(f, FAKE, FAKE, 2**34 + 4, 0, 0, 0, 1.0, 1.0, 1.0, stream=0) == dp.DP_EINVAL
    # empty inputs are valid no-ops that enqueue nothing
    assert code_of(f, None, None, 0, 0, 0, 0, 1.0, 1.0, 1.0, stream=0) == dp.DP_OK
    assert code_of(dp.dp_philox_normals, None, None, 0, 0, 0, 0, stream=0) == dp.DP_OK
    assert code_of(dp.dp_grad_sample_linear, None, None, dp.DP_F32, 0, 3, 4, 5, 1.0, None, stream=0) == dp.DP_OK


def test_groupnorm_validation_and_workspace():
    """dp_grad_sample_groupnorm: workspace only for several channel blocks;
    bad sizes, a missing output or workspace are refused before any launch."""
    assert dp.dp_grad_sample_groupnorm_workspace_bytes(4, 16, 64) == 0
    assert dp.dp_grad_sample_groupnorm_workspace_bytes(4, 17, 64) == 4 * 2 * 4
    assert dp.dp_grad_sample_groupnorm_workspace_bytes(0, 17, 64) == 0
    f = dp.dp_grad_sample_groupnorm
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 0, 8, 1.0, FAKE, stream=0) == dp.DP_EINVAL       # C = 0
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 3, -1, 1.0, FAKE, stream=0) == dp.DP_EINVAL      # P < 0
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 3, 8, 1.0, None, stream=0) == dp.DP_EINVAL       # no ggamma
    assert code_of(f, None, FAKE, dp.DP_F32, 2, 3, 8, 1.0, FAKE, stream=0) == dp.DP_EINVAL       # no xhat
    assert code_of(f, FAKE, FAKE, 7, 2, 3, 8, 1.0, FAKE, stream=0) == dp.DP_EDTYPE
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 40, 8, 1.0, FAKE, FAKE, FAKE, stream=0) == dp.DP_EINVAL  # ws


def test_noise_schedule_validation():
    """dp_norms_clip_noise_sched refuses a missing table, an empty one and an
    infinite C (a schedule may hold positive entries), and a zero
    denominator, before enqueueing anything."""
    f = dp.lib().dp_norms_clip_noise_sched
    # (sqnorm, L, params, count, N, norm, C, seed, step, step_dev, table, len, n_active, denom, status, ws,
    #  ws_bytes, stream)
    assert f(None, 0, None, 0, 0, None, 1.0, 0, 0, None, None, 1, None, 1.0, None, None, 0, None) == dp.DP_EINVAL
    assert f(None, 0, None, 0, 0, None, 1.0, 0, 0, None, FAKE, 0, None, 1.0, None, None, 0, None) == dp.DP_EINVAL
    assert f(None, 0, None, 0, 0, None, math.inf, 0, 0, None, FAKE, 3, FAKE, 1.0, None, None, 0,
             None) == dp.DP_EINVAL
    assert f(None, 0, None, 0, 0, None, 1.0, 0, 0, None, FAKE, 3, FAKE, 0.0, None, None, 0, None) == dp.DP_EINVAL


def test_active_norms_validation():
    """dp_per_sample_norms_active refuses a negative batch or layer count and
    missing buffers before enqueueing anything; N = 0 is a no-op."""
    f = dp.lib().dp_per_sample_norms_active
    # (sqnorm, L, N, n_active, norm, status, stream)
    assert f(FAKE, 2, -1, FAKE, FAKE, None, None) == dp.DP_EINVAL
    assert f(FAKE, -1, 4, FAKE, FAKE, None, None) == dp.DP_EINVAL
    assert f(FAKE, 2, 4, FAKE, None, None, None) == dp.DP_EINVAL
    assert f(None, 2, 4, FAKE, FAKE, None, None) == dp.DP_EINVAL
    assert f(None, 0, 0, None, None, None, None) == dp.DP_OK


def test_clip_sum_route_choice():
    # small T = 1 Linear: rereading 16.8 MB of grads in the shared grouped launch beats two extra launches
    assert stepmod.linear_clip_mode(W.Linear("fc1", 512, 32), 256, W.F32) == "colreduce"
    # a wide T = 1 Linear on a big batch: the fused GEMM reads N*(d_in+d_out) instead of N*P
    assert stepmod.linear_clip_mode(W.Linear("big", 4096, 1024), 4096, W.F32) == "fused"
    # LSTM weights (K = N*T = 16384, small outputs): rereading the grads is cheaper
    assert stepmod.linear_clip_mode(W.Linear("ih", 100, 400, T=256), 64, W.F32) == "colreduce"


def test_product_path_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2109_12298_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
                text = open(os.path.join(dirpath, fn)).read()
                assert "import oracle" not in text and "from oracle" not in text, fn
                assert "dp_oracle" not in text and "liboracle" not in text, fn


def test_conv2d_path_choice_round_trips():
    """The conv kernel choice is process-wide state: set returns the previous
    value and an unknown value is refused without changing it."""
    prev = dp.dp_conv2d_set_path(dp.DP_CONV_TILED)
    try:
        assert dp.dp_conv2d_set_path(dp.DP_CONV_AUTO) == dp.DP_CONV_TILED
        assert dp.dp_conv2d_set_path(dp.DP_CONV_ROWS) == dp.DP_CONV_AUTO
        assert dp.dp_conv2d_set_path(dp.DP_CONV_AUTO) == dp.DP_CONV_ROWS
        assert dp.lib().dp_conv2d_set_path(7) == -1
        assert dp.dp_conv2d_set_path(dp.DP_CONV_AUTO) == dp.DP_CONV_AUTO
    finally:
        dp.dp_conv2d_set_path(prev)


def test_conv2d_kernel_choice_follows_the_path():
    """Which conv kernel runs: the one-workgroup-per-sample kernel for a plane
    that fits LDS (MNIST's first layer), the row-chunked kernel for a wide
    32x32 plane with 288 weight columns, the tiled kernel when forced, and -1
    for a shape the call refuses."""
    prev = dp.dp_conv2d_set_path(dp.DP_CONV_AUTO)
    try:
        mnist_c1 = (256, 1, 28, 28, 16, 8, 8, 2, 2, 3, 3)
        cifar_c2 = (256, 32, 32, 32, 32, 3, 3, 1, 1, 1, 1)
        assert dp.dp_conv2d_kernel_choice(*mnist_c1) == dp.DP_CONV_KERNEL_SMALL
        assert dp.dp_conv2d_kernel_choice(*cifar_c2) == dp.DP_CONV_KERNEL_ROWS
        assert dp.dp_conv2d_kernel_choice(256, 1, 2, 2, 4, 3, 3, 1, 1, 0, 0) == -1
        dp.dp_conv2d_set_path(dp.DP_CONV_TILED)
        assert dp.dp_conv2d_kernel_choice(*mnist_c1) == dp.DP_CONV_KERNEL_TILED
        assert dp.dp_conv2d_kernel_choice(*cifar_c2) == dp.DP_CONV_KERNEL_TILED
        dp.dp_conv2d_set_path(dp.DP_CONV_ROWS)
        assert dp.dp_conv2d_kernel_choice(*cifar_c2) == dp.DP_CONV_KERNEL_ROWS
    finally:
        dp.dp_conv2d_set_path(prev)


def test_grad_sample_many_grouping_and_validation():
    """Which layers the grouped per-sample-gradient launch takes, and that an
    invalid layer anywhere in the list is refused before anything runs."""
    fc = dp.linear_grad_item(FAKE, FAKE, 1, 512, 32, 1.0, FAKE)
    seq = dp.linear_grad_item(FAKE, FAKE, 8, 64, 16, 1.0, FAKE)
    c1 = dp.conv2d_grad_item(FAKE, FAKE, 1, 28, 28, 16, 14, 14, 8, 8, 2, 2, 3, 3, 1.0, FAKE)
    big = dp.conv2d_grad_item(FAKE, FAKE, 64, 32, 32, 64, 32, 32, 3, 3, 1, 1, 1, 1, 1.0, FAKE)
    items = dp.make_layer_grads([fc, seq, c1, big])
    got = [dp.dp_grad_sample_many_grouped(items, k, dp.DP_F32, 256) for k in range(4)]
    assert got == [True, False, True, False]
    # the forced tiled conv kernel keeps convolutions out of the group
    prev = dp.dp_conv2d_set_path(dp.DP_CONV_TILED)
    try:
        assert not dp.dp_grad_sample_many_grouped(items, 2, dp.DP_F32, 256)
    finally:
        dp.dp_conv2d_set_path(prev)
    # workspace: the largest need of the layers outside the group
    need = dp.dp_grad_sample_many_workspace_bytes(items, 4, dp.DP_F32, 256)
    assert need == max(dp.dp_grad_sample_linear_workspace_bytes(256, 8, 64, 16, dp.DP_F32),
                       dp.dp_grad_sample_conv2d_workspace_bytes(256, 64, 32, 32, 64, 3, 3, 1, 1, 1, 1))
    f = dp.dp_grad_sample_many
    assert code_of(f, items, 2, 7, 256, stream=0) == dp.DP_EDTYPE
    assert code_of(f, items, 65, dp.DP_F32, 256, stream=0) == dp.DP_EINVAL
    bad_ho = dict(c1, Ho=13)
    assert code_of(f, dp.make_layer_grads([fc, bad_ho]), 2, dp.DP_F32, 256, stream=0) == dp.DP_EINVAL
    no_out = dict(fc, gW=None)
    assert code_of(f, dp.make_layer_grads([c1, no_out]), 2, dp.DP_F32, 256, stream=0) == dp.DP_EINVAL
    bad_kind = dict(fc, kind=5)
    assert code_of(f, dp.make_layer_grads([bad_kind]), 1, dp.DP_F32, 4, stream=0) == dp.DP_EINVAL
    # a missing workspace for the layers that run alone
    assert code_of(f, items, 4, dp.DP_F32, 256, stream=0) == dp.DP_EINVAL
    # empty batches and empty lists enqueue nothing
    assert code_of(f, items, 4, dp.DP_F32, 0, stream=0) == dp.DP_OK
    assert code_of(f, items, 0, dp.DP_F32, 256, stream=0) == dp.DP_OK


def test_ghost_norm_validation():
    f = dp.dp_ghost_norm_linear
    assert code_of(f, FAKE, FAKE, 7, 2, 8, 3, 4, 1.0, True, FAKE, stream=0) == dp.DP_EDTYPE
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 8, 0, 4, 1.0, True, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(f, None, FAKE, dp.DP_F32, 2, 8, 3, 4, 1.0, True, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 8, 3, 4, 1.0, True, None, stream=0) == dp.DP_EINVAL
    # one float per (sample, 64 x 64 tile pair) when there are several pairs
    # (padded to 256 bytes); the partial Gram tiles (2 x 16 KB per sample,
    # pair and feature chunk) only when the units are too few to fill the GPU
    ws = dp.dp_ghost_norm_linear_workspace_bytes
    assert ws(0, 64, 3, 4) == 0
    assert ws(5, 0, 3, 4) == 0
    assert ws(5, 64, 3, 4) == 0                     # one pair, one chunk: written into sqnorm
    assert ws(5, 65, 3, 4) == 256                   # three pairs; 7 features make one chunk
    assert ws(32, 128, 768, 3072) == 512 + 32 * 3 * 6 * 2 * 16384    # 96 units: six chunks each
    assert ws(200, 128, 768, 3072) == 200 * 3 * 4 + 160          # 600 units: one chunk
    assert code_of(f, FAKE, FAKE, dp.DP_F32, 2, 65, 3, 4, 1.0, True, FAKE, stream=0) == dp.DP_EINVAL
    assert code_of(f, None, None, dp.DP_F32, 0, 8, 3, 4, 1.0, True, None, stream=0) == dp.DP_OK


def test_layernorm_many_validation():
    f = dp.dp_grad_sample_layernorm_many
    FF = 1 << 20
    lay = lambda T, D, gg=FF: (FF, FF, T, D, 1.0, gg, FF, FF)
    items = dp.make_layernorm_layers([lay(128, 768), lay(128, 768), lay(7, 64)])
    ws = dp.dp_grad_sample_layernorm_many_workspace_bytes
    # one float per (sample, 128-byte feature chunk) of a layer with several chunks
    assert ws(items, 3, 32, dp.DP_BF16) == 2 * 32 * 12 * 4            # 12 chunks of 64; 64 features: one
    assert ws(items, 3, 32, dp.DP_F32) == 2 * 32 * 24 * 4 + 256       # 24 chunks of 32; 2 chunks (256-padded)
    assert ws(items, 3, 0, dp.DP_BF16) == 0 and ws(items, 0, 32, dp.DP_BF16) == 0
    assert code_of(f, items, 3, 7, 32, stream=0) == dp.DP_EDTYPE
    assert code_of(f, items, 65, dp.DP_BF16, 32, stream=0) == dp.DP_EINVAL
    assert code_of(f, items, 3, dp.DP_BF16, 32, stream=0) == dp.DP_EINVAL       # no workspace
    bad = dp.make_layernorm_layers([lay(128, 768), lay(128, 0)])
    assert code_of(f, bad, 2, dp.DP_BF16, 32, stream=0) == dp.DP_EINVAL
    nog = dp.make_layernorm_layers([lay(8, 64, None)])
    assert code_of(f, nog, 1, dp.DP_BF16, 32, stream=0) == dp.DP_EINVAL
    assert code_of(f, items, 3, dp.DP_BF16, 0, stream=0) == dp.DP_OK
    assert code_of(f, items, 0, dp.DP_BF16, 32, stream=0) == dp.DP_OK


def test_ghost_norm_many_validation():
    f = dp.dp_ghost_norm_linear_many
    FF = 1 << 20
    lay = lambda T, din, dout, sq=FF: (FF, FF, T, din, dout, 1.0, True, sq)
    transformer = [lay(128, 768, 768)] * 4 + [lay(128, 768, 3072), lay(128, 3072, 768)]
    items = dp.make_ghost_layers(transformer)
    # 6 layers x 32 samples x 3 pairs fill the GPU: one chunk, the pair values only
    assert dp.dp_ghost_norm_linear_many_workspace_bytes(items, 6, 32) == 6 * 512
    # alone, each layer's 96 units are split into feature chunks
    one = dp.make_ghost_layers(transformer[:1])
    assert dp.dp_ghost_norm_linear_many_workspace_bytes(one, 1, 32) == \
        dp.dp_ghost_norm_linear_workspace_bytes(32, 128, 768, 768)
    assert dp.dp_ghost_norm_linear_many_workspace_bytes(items, 0, 32) == 0
    assert code_of(f, items, 6, 7, 32, stream=0) == dp.DP_EDTYPE
    assert code_of(f, items, 65, dp.DP_BF16, 32, stream=0) == dp.DP_EINVAL
    assert code_of(f, items, 6, dp.DP_BF16, 32, stream=0) == dp.DP_EINVAL       # no workspace
    bad = dp.make_ghost_layers(transformer[:2] + [lay(128, 0, 768)])
    assert code_of(f, bad, 3, dp.DP_BF16, 32, stream=0) == dp.DP_EINVAL
    nosq = dp.make_ghost_layers([lay(128, 768, 768, None)])
    assert code_of(f, nosq, 1, dp.DP_BF16, 32, stream=0) == dp.DP_EINVAL
    huge = dp.make_ghost_layers([lay(1 << 12, 1 << 20, 8)])
    assert code_of(f, huge, 1, dp.DP_BF16, 1, stream=0) == dp.DP_EUNSUPPORTED
    # empty batches and empty lists enqueue nothing
    assert code_of(f, items, 6, dp.DP_BF16, 0, stream=0) == dp.DP_OK
    assert code_of(f, items, 0, dp.DP_BF16, 32, stream=0) == dp.DP_OK
