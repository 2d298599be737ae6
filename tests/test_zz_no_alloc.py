"""dp_grad_sample_linear_noalloc (scratch in a fixed device array inside the
library, no caller workspace) against dp_grad_sample_linear with a caller
workspace: identical kernels, so identical bits, on two calls in a row, the
second on a smaller input (the array keeps the first call's contents)."""
import sys

import numpy as np
import pytest
import torch

from paper_2109_12298_amd import binding as dp

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def run_both(dtype, N, T, din, dout, seed):
    r = np.random.default_rng(seed)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dt = dp.DP_BF16 if dtype == "bf16" else dp.DP_F32
    A = torch.from_numpy(r.standard_normal((N, T, din)).astype(np.float32)).to(tdt).to(DEV)
    B = torch.from_numpy((r.standard_normal((N, T, dout)) / 8).astype(np.float32)).to(tdt).to(DEV)
    need = dp.dp_grad_sample_linear_workspace_bytes(N, T, din, dout, dt)
    assert 0 < need <= dp.dp_grad_sample_linear_noalloc_max_bytes()
    out = []
    for noalloc in (True, False):
        gW = torch.full((N, dout, din), 7.0, device=DEV)
        gb = torch.full((N, dout), 7.0, device=DEV)
        sq = torch.full((N,), 7.0, device=DEV)
        st = torch.zeros(1, dtype=torch.int32, device=DEV)
        if noalloc:
            dp.dp_grad_sample_linear_noalloc(A, B, dt, N, T, din, dout, 0.8, gW, gb, sq, st)
        else:
            ws = torch.empty(need, dtype=torch.uint8, device=DEV)
            dp.dp_grad_sample_linear(A, B, dt, N, T, din, dout, 0.8, gW, gb, sq, st, ws)
        torch.cuda.synchronize()
        assert int(st.item()) == 0
        out.append((gW.cpu().numpy(), gb.cpu().numpy(), sq.cpu().numpy()))
    return out


@pytest.mark.parametrize("dtype,first,second", [
    ("bf16", (29, 32, 768, 3072), (5, 64, 264, 392)),      # staged bf16 kernel, then a ragged one
    ("f32", (7, 40, 100, 20), (3, 33, 65, 70))])           # fp32 MFMA kernel
def test_noalloc_linear_matches_the_workspace_entry_point(dtype, first, second):
    for k, shape in enumerate((first, second)):
        say("noalloc linear", dtype, shape)
        (gW0, gb0, sq0), (gW1, gb1, sq1) = run_both(dtype, *shape, seed=k + 3)
        np.testing.assert_array_equal(gW0, gW1)
        np.testing.assert_array_equal(gb0, gb1)
        np.testing.assert_array_equal(sq0, sq1)
        assert np.all(np.isfinite(sq0)) and np.all(sq0 > 0)
