"""The tiled Wq layout (RRS_WEIGHT_TILED) against the row-major default.

Weight preparation with the flag must write exactly the row-major codes moved
to the documented tiled positions (tests/_gpu_util.tile_wq, itself checked
against the byte formula of include/rrs.h in test_abi), with the same scales;
every GEMM entry point must then give bit-identical outputs from either layout
(same kernels, same arithmetic, only the weight addresses differ). The
row-major path itself is checked against the oracle in the other GPU tests."""
import numpy as np
import pytest

import synth
from tests._gpu_util import tile_wq, to_gpu, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2409_20361_amd as rrs
    rrs.lib()


def _rrs():
    import paper_2409_20361_amd as rrs
    return rrs


def _work(M, K, N, g, seed):
    return synth.custom("layout", M, K, N, g, seed, n_chan=max(1, K // 100),
                        chan_factor=(20, 100), n_spike=max(1, M * K // 2000), spike_mag=(100, 500))


def _both_weights(w, perm=None, flags=0):
    rrs = _rrs()
    W = to_gpu(synth.weights(w))
    p = None if perm is None else to_gpu(perm)
    Wr, br = rrs.prepare_weight(W, p, flags=flags)
    Wt, bt = rrs.prepare_weight(W, p, flags=flags | rrs.WEIGHT_TILED)
    return (Wr, br), (Wt, bt)


def _same(a, b, label):
    assert torch.equal(a, b), (
        f"{label}: {int((a != b).sum())} outputs differ between the two weight layouts")


@pytest.mark.parametrize("K,N,perm,flags", [
    (512, 48, False, 0), (4096, 256, True, 0), (8192, 112, False, 1), (16384, 32, True, 1)])
def test_tiled_prepare_is_the_row_major_codes_moved(K, N, perm, flags):
    print(f"[case] tiled prepare K={K} N={N} perm={perm} flags={flags}", flush=True)
    w = _work(1, K, N, 128, 11 + K + N)
    pm = synth.permutation(K, 4) if perm else None
    (Wr, br), (Wt, bt) = _both_weights(w, pm, flags)
    np.testing.assert_array_equal(to_np(Wt), tile_wq(to_np(Wr)))
    _same(br, bt, "beta")


def test_tiled_sub_channel_prepare():
    rrs = _rrs()
    K, N, g = 4096, 64, 128
    print(f"[case] tiled sub-channel prepare K={K} N={N} g={g}", flush=True)
    W = to_gpu(synth.weights(_work(1, K, N, g, 3)))
    Wr, sr = rrs.prepare_weight_sub_channel(W, g)
    Wt, st = rrs.prepare_weight_sub_channel(W, g, flags=rrs.WEIGHT_TILED)
    np.testing.assert_array_equal(to_np(Wt), tile_wq(to_np(Wr)))
    _same(sr, st, "w_sub")


# M = 1, 8 and 16 take one block of 16 tokens in the few-token kernel, 24 and
# 40 two and 64 four (row-major weights from M = 8 on: four column blocks per
# workgroup, so N = 208 and 336 leave a partial last workgroup); 65 and 300
# take the main kernel.
@pytest.mark.parametrize("M,K,N,g", [
    (1, 8192, 256, 128), (8, 4096, 512, 64), (16, 2048, 128, 512), (24, 4096, 512, 256),
    (64, 2048, 384, 512), (65, 4096, 512, 128), (300, 1024, 640, 128),
    (8, 4096, 208, 128), (40, 2048, 336, 64)])
def test_gemm_and_linear_agree_across_layouts(M, K, N, g):
    rrs = _rrs()
    print(f"[case] layouts gemm/linear M={M} K={K} N={N} g={g}", flush=True)
    w = _work(M, K, N, g, 100 + M)
    X = to_gpu(synth.activations(w))
    (Wr, br), (Wt, bt) = _both_weights(w)
    Xq, a, s = rrs.rotate_smooth_quant(X, g)
    _same(rrs.w4a4_gemm(Xq, a, s, Wr, br, g),
          rrs.w4a4_gemm(Xq, a, s, Wt, bt, g, flags=rrs.WEIGHT_TILED), "w4a4_gemm")
    _same(rrs.linear(X, Wr, br, g), rrs.linear(X, Wt, bt, g, flags=rrs.WEIGHT_TILED), "linear")


@pytest.mark.parametrize("M", [8, 200])
def test_ablations_and_baselines_agree_across_layouts(M):
    rrs = _rrs()
    K, N, g = 4096, 256, 128
    T = rrs.WEIGHT_TILED
    print(f"[case] layouts ablations/baselines M={M}", flush=True)
    w = _work(M, K, N, g, 300 + M)
    X = to_gpu(synth.activations(w))
    # without rotation
    (Wr, br), (Wt, bt) = _both_weights(w, flags=rrs.SKIP_ROTATION)
    f = rrs.SKIP_ROTATION
    _same(rrs.linear(X, Wr, br, g, flags=f), rrs.linear(X, Wt, bt, g, flags=f | T),
          "linear without rotation")
    # per-channel (QuaRot-style: no smoothing) on the main loop and the scheme skeleton
    (Wr, br), (Wt, bt) = _both_weights(w)
    Xq, a, s = rrs.rotate_smooth_quant(X, g, flags=rrs.SKIP_SMOOTHING)
    _same(rrs.w4a4_gemm_per_channel(Xq, a, Wr, br),
          rrs.w4a4_gemm_per_channel(Xq, a, Wt, bt, flags=T), "per-channel")
    Xq, a, s = rrs.rotate_smooth_quant(X, g)
    for scheme in (rrs.SCHEME_PER_CHANNEL, rrs.SCHEME_RUNTIME_SMOOTH):
        _same(rrs.w4a4_gemm_scheme(scheme, Xq, a, s, Wr, br, g),
              rrs.w4a4_gemm_scheme(scheme, Xq, a, s, Wt, bt, g, flags=T), f"scheme {scheme}")
    # sub-channel
    W = to_gpu(synth.weights(w))
    Wr, sr = rrs.prepare_weight_sub_channel(W, g)
    Wt, st = rrs.prepare_weight_sub_channel(W, g, flags=T)
    Xs, xs = rrs.quantize_sub_channel(X, g)
    _same(rrs.w4a4_gemm_scheme(rrs.SCHEME_SUB_CHANNEL, Xs, xs, None, Wr, sr, g),
          rrs.w4a4_gemm_scheme(rrs.SCHEME_SUB_CHANNEL, Xs, xs, None, Wt, st, g, flags=T),
          "sub-channel")


@pytest.mark.parametrize("M", [8, 16, 200])
def test_runtime_reorder_agrees_across_layouts(M):
    # M <= 16: the few-token gather kernel; above: the main kernel's gather loop.
    rrs = _rrs()
    K, N, g = 8192, 256, 128
    print(f"[case] layouts runtime reorder M={M}", flush=True)
    w = _work(M, K, N, g, 500 + M)
    X = to_gpu(synth.activations(w))
    (Wr, br), (Wt, bt) = _both_weights(w)
    _same(rrs.linear_reorder(X, Wr, br, g),
          rrs.linear_reorder(X, Wt, bt, g, flags=rrs.WEIGHT_TILED), "linear_reorder")
