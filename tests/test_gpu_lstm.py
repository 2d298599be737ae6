"""GPU parity of the LSTM's backward through time (dp_lstm_backward) against
the oracle, through the C ABI.  The stored activations come from the oracle's
forward with random weights (consistent gates and cell states), rounded to
fp32; both sides then read the same fp32 values."""
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


def lstm_case(N, T, D, H, per_step, last, seed):
    r = np.random.default_rng(seed)
    k = 1.0 / np.sqrt(H)
    x = r.standard_normal((N, T, D))
    W_ih, W_hh = r.uniform(-k, k, (4 * H, D)), r.uniform(-k, k, (4 * H, H))
    b_ih, b_hh = r.uniform(-k, k, 4 * H), r.uniform(-k, k, 4 * H)
    gates, c, _ = oracle.lstm_forward(x, W_ih, W_hh, b_ih, b_hh)
    f32 = lambda a: None if a is None else np.ascontiguousarray(a, dtype=np.float32)
    dh_out = f32(r.standard_normal((N, T, H))) if per_step else None
    dh_last = f32(r.standard_normal((N, H))) if last else None
    return f32(gates), f32(c), f32(W_hh), dh_out, dh_last


def run_device(gates, c, W_hh, dh_out, dh_last):
    N, T, H = c.shape
    dev = lambda a: None if a is None else torch.from_numpy(a).to(DEV)
    delta = torch.full((N, T, 4 * H), 7.0, device=DEV)
    dp.dp_lstm_backward(dev(gates), dev(c), dev(W_hh), dev(dh_out), dev(dh_last), N, T, H, delta)
    torch.cuda.synchronize()
    return delta.cpu().numpy()


@pytest.mark.parametrize("N,T,D,H,per_step,last", [
    (1, 1, 3, 4, False, True), (3, 7, 5, 4, True, True), (2, 13, 8, 37, True, True),   # ragged gate blocks
    (5, 33, 20, 100, False, True), (2, 257, 100, 100, True, False),                   # T not a multiple of the ring
    (2, 20, 16, 128, True, True), (3, 6, 4, 1, True, True), (64, 256, 100, 100, False, True)])
def test_lstm_backward_matches_oracle(N, T, D, H, per_step, last):
    say("lstm backward", N, T, D, H, per_step, last)
    gates, c, W_hh, dh_out, dh_last = lstm_case(N, T, D, H, per_step, last, seed=N * 100 + T)
    got = run_device(gates, c, W_hh, dh_out, dh_last)
    ref = oracle.lstm_backward(gates, c, W_hh, dh_out=dh_out, dh_last=dh_last)
    # per sample: the gradient decays backwards in time, so each sample's
    # values are judged against its own scale
    for n in range(N):
        assert_g12(got[n], ref[n], 1e-4, "delta n=%d" % n)
    again = run_device(gates, c, W_hh, dh_out, dh_last)
    np.testing.assert_array_equal(got, again)


def test_lstm_backward_without_upstream_gradient_is_zero():
    gates, c, W_hh, _, _ = lstm_case(2, 9, 4, 8, False, False, seed=3)
    got = run_device(gates, c, W_hh, None, None)
    assert np.all(got == 0.0)
