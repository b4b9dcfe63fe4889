"""Failure paths on the GPU, forced from the host so every kernel still ends.

  * RRS_DEBUG precondition checks: a non-finite input or a perm / block order
    that is not a permutation returns RRS_ERR_PRECONDITION before anything is
    enqueued (outputs keep their sentinel bytes); valid inputs pass, and
    without RRS_DEBUG the same calls are not checked.
  * The one-launch quantizers' bounded wait (the workgroups' group maxima
    exchanged within the launch, Eq. 1 taking the maximum over all tokens):
    the test hook makes the readers also wait for a row of maxima that no
    workgroup writes, so every wait runs out after a few polls; the kernel
    must end, mark the call as failed and write NaN into alpha and s_group,
    and the next ordinary call on the same workspace must be correct again.
"""
import ctypes
import os

import numpy as np
import pytest

import synth
from oracle import rrs_oracle as O
from tests._gpu_util import check_codes, to_gpu, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

PRECONDITION = -10


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2409_20361_amd as rrs
    rrs.lib()


def _rrs():
    import paper_2409_20361_amd as rrs
    return rrs


@pytest.fixture
def debug_env():
    old = os.environ.get("RRS_DEBUG")
    os.environ["RRS_DEBUG"] = "1"
    yield
    if old is None:
        del os.environ["RRS_DEBUG"]
    else:
        os.environ["RRS_DEBUG"] = old


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _quant_raw(X, g, perm, Xq, a, s, ws):
    rrs = _rrs()
    M, K = X.shape
    return rrs.lib().rrs_rotate_smooth_quant(
        X.data_ptr(), M, K, g, None if perm is None else perm.data_ptr(), Xq.data_ptr(),
        a.data_ptr(), s.data_ptr(), ws.data_ptr(), ws.numel(), _stream())


def _bufs(M, K, g):
    rrs = _rrs()
    Xq = torch.full((M, K // 2), 0xA5, dtype=torch.uint8, device="cuda")
    a = torch.full((M,), 3.0, dtype=torch.float32, device="cuda")
    s = torch.full((K // g,), 3.0, dtype=torch.float32, device="cuda")
    ws = torch.zeros((rrs.workspace_bytes(M, K, g),), dtype=torch.uint8, device="cuda")
    return Xq, a, s, ws


def _untouched(Xq, a, s):
    torch.cuda.synchronize()
    return bool((Xq == 0xA5).all()) and bool((a == 3.0).all()) and bool((s == 3.0).all())


@pytest.mark.parametrize("M", [5, 40])
def test_debug_rejects_bad_perm_and_nonfinite_x(debug_env, M):
    K, g = 1024, 128
    w = synth.custom("dbg", M, K, 16, g, 3, n_chan=4, n_spike=2)
    X = to_gpu(synth.activations(w))
    perm = synth.permutation(K, 9)
    print(f"[case] debug quant M={M}", flush=True)
    Xq, a, s, ws = _bufs(M, K, g)
    assert _quant_raw(X, g, to_gpu(perm), Xq, a, s, ws) == 0
    bad = perm.copy()
    bad[7] = bad[8]          # a repeated entry: not a permutation
    Xq, a, s, ws = _bufs(M, K, g)
    assert _quant_raw(X, g, to_gpu(bad), Xq, a, s, ws) == PRECONDITION
    assert _untouched(Xq, a, s)
    oob = perm.copy()
    oob[0] = K               # out of range
    assert _quant_raw(X, g, to_gpu(oob), Xq, a, s, ws) == PRECONDITION
    Xn = X.clone()
    Xn[M - 1, 17] = float("inf")
    assert _quant_raw(Xn, g, None, Xq, a, s, ws) == PRECONDITION
    Xn[M - 1, 17] = float("nan")
    assert _quant_raw(Xn, g, None, Xq, a, s, ws) == PRECONDITION
    assert _untouched(Xq, a, s)


def test_debug_off_does_not_check():
    assert not os.environ.get("RRS_DEBUG")
    K, g, M = 1024, 128, 5
    w = synth.custom("dbg", M, K, 16, g, 4, n_chan=4, n_spike=2)
    X = to_gpu(synth.activations(w))
    bad = synth.permutation(K, 9)
    bad[7] = bad[8]
    Xq, a, s, ws = _bufs(M, K, g)
    # undefined results, but no check and no error
    assert _quant_raw(X, g, to_gpu(bad), Xq, a, s, ws) == 0
    torch.cuda.synchronize()


def test_debug_rejects_bad_weight_and_scales(debug_env):
    rrs = _rrs()
    K, N, M, g = 512, 32, 4, 128
    w = synth.custom("dbgw", M, K, N, g, 5, n_chan=2)
    W = to_gpu(synth.weights(w))
    Wq = torch.full((N, K // 2), 0xA5, dtype=torch.uint8, device="cuda")
    beta = torch.full((N,), 3.0, dtype=torch.float32, device="cuda")
    lib = rrs.lib()
    print("[case] debug weights and scales", flush=True)
    assert lib.rrs_prepare_weight(W.data_ptr(), K, N, None, Wq.data_ptr(), beta.data_ptr(),
                                  _stream()) == 0
    Wn = W.clone()
    Wn[3, 5] = float("-inf")
    Wq2 = torch.full((N, K // 2), 0xA5, dtype=torch.uint8, device="cuda")
    assert lib.rrs_prepare_weight(Wn.data_ptr(), K, N, None, Wq2.data_ptr(), beta.data_ptr(),
                                  _stream()) == PRECONDITION
    torch.cuda.synchronize()
    assert bool((Wq2 == 0xA5).all())
    bad = to_gpu(np.zeros(K, np.int32))
    assert lib.rrs_prepare_weight(W.data_ptr(), K, N, bad.data_ptr(), Wq2.data_ptr(),
                                  beta.data_ptr(), _stream()) == PRECONDITION
    # GEMM: a NaN scale is rejected
    X = to_gpu(synth.activations(w))
    Xq, a, s = rrs.rotate_smooth_quant(X, g)
    Y = torch.zeros((M, N), dtype=torch.float16, device="cuda")
    beta_n = beta.clone()
    beta_n[4] = float("nan")
    assert lib.rrs_w4a4_gemm(Xq.data_ptr(), a.data_ptr(), s.data_ptr(), Wq.data_ptr(),
                             beta_n.data_ptr(), M, N, K, g, Y.data_ptr(), _stream()) == PRECONDITION
    s_n = s.clone()
    s_n[1] = float("inf")
    assert lib.rrs_w4a4_gemm(Xq.data_ptr(), a.data_ptr(), s_n.data_ptr(), Wq.data_ptr(),
                             beta.data_ptr(), M, N, K, g, Y.data_ptr(), _stream()) == PRECONDITION
    assert lib.rrs_w4a4_gemm(Xq.data_ptr(), a.data_ptr(), s.data_ptr(), Wq.data_ptr(),
                             beta.data_ptr(), M, N, K, g, Y.data_ptr(), _stream()) == 0
    # the layer: a bad perm, then a valid call
    ws = torch.zeros((rrs.linear_workspace_bytes(M, K, g),), dtype=torch.uint8, device="cuda")
    assert lib.rrs_linear(X.data_ptr(), Wq.data_ptr(), beta.data_ptr(), M, N, K, g,
                          bad.data_ptr(), Y.data_ptr(), ws.data_ptr(), ws.numel(),
                          _stream()) == PRECONDITION
    assert lib.rrs_linear(X.data_ptr(), Wq.data_ptr(), beta.data_ptr(), M, N, K, g, None,
                          Y.data_ptr(), ws.data_ptr(), ws.numel(), _stream()) == 0
    torch.cuda.synchronize()


def test_debug_rejects_bad_block_order(debug_env):
    rrs = _rrs()
    K, N, M, g = 1024, 32, 20, 128
    w = synth.custom("dbgo", M, K, N, g, 6, n_chan=3, n_spike=2)
    X = to_gpu(synth.activations(w))
    Wq, beta = rrs.prepare_weight(to_gpu(synth.weights(w)))
    Xq, a, s, order = rrs.rotate_smooth_quant_reorder(X, g)
    Y = torch.zeros((M, N), dtype=torch.float16, device="cuda")
    lib = rrs.lib()
    print("[case] debug block order", flush=True)
    args = lambda o: (Xq.data_ptr(), a.data_ptr(), s.data_ptr(), Wq.data_ptr(),  # noqa: E731
                      beta.data_ptr(), o.data_ptr(), M, N, K, g, 0, Y.data_ptr(), _stream())
    assert lib.rrs_w4a4_gemm_reorder(*args(order)) == 0
    bad = order.clone()
    bad[0] = bad[1]
    assert lib.rrs_w4a4_gemm_reorder(*args(bad)) == PRECONDITION
    torch.cuda.synchronize()


# ------------------------------------------------------------------ bounded wait

@pytest.mark.parametrize("M,K,g", [(2, 8192, 128), (8, 8192, 128), (15, 1024, 64),
                                   (300, 4096, 128), (2040, 4096, 128), (40, 1024, 64),
                                   (40, 8192, 128), (63, 8192, 256), (31, 8192, 64),
                                   (90, 1024, 64)])
def test_one_launch_wait_runs_out_loudly(M, K, g):
    # per-row kernel up to 16 tokens (up to 32 / 64 by g), fused kernel above
    # (K <= 4096)
    rrs = _rrs()
    w = synth.custom("qw", M, K, 16, g, M + K, n_chan=max(1, K // 100), n_spike=2,
                     spike_mag=(100, 500))
    Xh = synth.activations(w)
    X = to_gpu(Xh)
    ws = torch.zeros((rrs.workspace_bytes(M, K, g),), dtype=torch.uint8, device="cuda")
    print(f"[case] one-launch wait runs out M={M} K={K} g={g}", flush=True)
    Xq, a, s, failed = rrs.quant_rows_wait_hook(X, g, extra_rows=1, max_polls=8, workspace=ws)
    assert failed, "the exchange must report the waits that ran out"
    assert bool(torch.isnan(a).all()), "alpha must be NaN after a failed exchange"
    assert bool(torch.isnan(s).all()), "s_group must be NaN after a failed exchange"
    # the same kernel with nothing extra to wait for passes, and so does the
    # next ordinary call on the same workspace
    Xq, a, s, failed = rrs.quant_rows_wait_hook(X, g, extra_rows=0, max_polls=1 << 18,
                                                workspace=ws)
    assert not failed
    act = O.rotate_smooth_quant(Xh, g)
    np.testing.assert_array_equal(to_np(a), act.alpha)
    np.testing.assert_array_equal(to_np(s), act.s)
    check_codes(to_np(Xq), act, "hook, nothing extra")
    Xq, a, s = rrs.rotate_smooth_quant(X, g, workspace=ws)
    np.testing.assert_array_equal(to_np(a), act.alpha)
    np.testing.assert_array_equal(to_np(s), act.s)


@pytest.mark.parametrize("M,K,g", [(2, 8192, 128), (8, 8192, 64), (15, 1024, 256),
                                   (64, 4096, 128), (100, 4096, 128), (600, 1024, 256)])
def test_reorder_one_launch_wait_runs_out_loudly(M, K, g):
    # the runtime-reorder quantizer's one-launch forms: up to 16 rows, one
    # workgroup per row; more rows at K <= 4096, runs of 16 workgroups (at
    # 64 x 4096 the extra row opens a run with no workgroup to lead it, at
    # 100 x 4096 and 600 x 1024 the last run's leader waits for it)
    rrs = _rrs()
    w = synth.custom("rw", M, K, 16, g, M + K + 1, n_chan=max(1, K // 100), n_spike=2,
                     spike_mag=(100, 500))
    Xh = synth.activations(w)
    X = to_gpu(Xh)
    ws = torch.zeros((rrs.reorder_workspace_bytes(M, K, g),), dtype=torch.uint8, device="cuda")
    print(f"[case] reorder one-launch wait runs out M={M} K={K} g={g}", flush=True)
    Xq, a, s, order, failed = rrs.quant_reorder_wait_hook(X, g, extra_rows=1, max_polls=8,
                                                          workspace=ws)
    assert failed, "the exchange must report the waits that ran out"
    assert bool(torch.isnan(a).all()), "alpha must be NaN after a failed exchange"
    assert bool(torch.isnan(s).all()), "s_group must be NaN after a failed exchange"
    # nothing extra to wait for: the hook and the ordinary call on the same
    # workspace both match the oracle
    act, border, _ = O.rotate_smooth_quant_reorder(Xh, g, 32)
    Xq, a, s, order, failed = rrs.quant_reorder_wait_hook(X, g, extra_rows=0,
                                                          max_polls=1 << 18, workspace=ws)
    assert not failed
    np.testing.assert_array_equal(to_np(order), border)
    np.testing.assert_array_equal(to_np(a), act.alpha)
    np.testing.assert_array_equal(to_np(s), act.s)
    check_codes(to_np(Xq), act, "reorder hook, nothing extra")
    Xq, a, s, order = rrs.rotate_smooth_quant_reorder(X, g, workspace=ws)
    np.testing.assert_array_equal(to_np(order), border)
    np.testing.assert_array_equal(to_np(a), act.alpha)


def test_quant_rows_debug_reports_no_false_timeout(debug_env):
    rrs = _rrs()
    M, K, g = 8, 8192, 128
    w = synth.custom("qd", M, K, 16, g, 77, n_chan=80, n_spike=2)
    Xh = synth.activations(w)
    Xq, a, s = rrs.rotate_smooth_quant(to_gpu(Xh), g)   # raises on a non-zero status
    act = O.rotate_smooth_quant(Xh, g)
    np.testing.assert_array_equal(to_np(a), act.alpha)


@pytest.mark.parametrize("M,K", [(8, 8192), (300, 4096)])
def test_reorder_debug_reports_no_false_timeout(debug_env, M, K):
    # RRS_DEBUG checks the fail word after both one-launch reorder forms (per
    # row, and runs of workgroups); a completed exchange must not report one.
    rrs = _rrs()
    g = 128
    w = synth.custom("rd", M, K, 16, g, 78 + M, n_chan=80, n_spike=2)
    Xh = synth.activations(w)
    Xq, a, s, order = rrs.rotate_smooth_quant_reorder(to_gpu(Xh), g)  # raises on failure
    act, border, _ = O.rotate_smooth_quant_reorder(Xh, g, 32)
    np.testing.assert_array_equal(to_np(order), border)
    np.testing.assert_array_equal(to_np(a), act.alpha)


def test_quant_rows_hook_argument_checks():
    rrs = _rrs()
    lib = rrs.lib()
    X = torch.zeros((4, 1024), dtype=torch.float16, device="cuda")
    n = ctypes.c_int32(0)
    Xq, a, s, ws = _bufs(4, 1024, 128)
    call = lambda M, extra, polls: lib.rrs_test_quant_rows_wait(  # noqa: E731
        X.data_ptr(), M, 1024, 128, extra, polls, Xq.data_ptr(), a.data_ptr(), s.data_ptr(),
        ws.data_ptr(), ws.numel(), ctypes.byref(n), _stream())
    assert call(1, 1, 8) == -2       # one row: no one-launch exchange
    assert call(4, 61, 8) == -9      # more than 64 rows in all for the per-row kernel
    assert call(4, -1, 8) == -9
    assert call(4, 1, 0) == -9
    assert _untouched(Xq, a, s)
