"""GPU parity of the kernel-comparison baselines (Section 4.5, Fig. 6) against
the CPU oracle: sub-channel quantizers bit for bit; the per-channel, Runtime
Smooth and sub-channel GEMMs of the shared skeleton within the output
tolerance derived from their arithmetic."""
import numpy as np
import pytest

import synth
from oracle import rrs_oracle as O
from tests._gpu_util import check_codes, check_y, near_half_integer, to_gpu, to_np

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


def _case(M, K, N, g, seed):
    w = synth.custom("b", M, K, N, g, seed, n_chan=max(1, K // 100), n_spike=max(1, M * K // 4000),
                     spike_mag=(100, 500))
    return synth.activations(w), synth.weights(w)


def _check_sub_codes(gpu_packed, ref, label):
    gq = O.unpack_int4(gpu_packed)
    diff = gq != ref.q
    if diff.any():
        bad = diff & ~near_half_integer(ref.v)
        assert not bad.any(), f"{label}: {int(bad.sum())} code mismatches"


@pytest.mark.parametrize("M,K,g,flags", [
    (16, 512, 128, 0), (37, 1024, 64, 0), (300, 4096, 128, 0), (5, 8192, 512, 0),
    (3, 16384, 64, 0), (64, 2048, 256, 1), (1, 512, 512, 1),
])
def test_quantize_sub_channel(M, K, g, flags):
    rrs = _rrs()
    X, _ = _case(M, K, 16, g, 31 + M + K)
    print(f"[case] sub-channel quant M={M} K={K} g={g} flags={flags}", flush=True)
    ref = O.sub_channel_quant(X, g, rotate=not (flags & rrs.SKIP_ROTATION))
    Xq, a = rrs.quantize_sub_channel(to_gpu(X), g, flags=flags)
    np.testing.assert_array_equal(to_np(a), ref.scale.T)
    _check_sub_codes(to_np(Xq), ref, "sub-channel activations")


@pytest.mark.parametrize("K,N,g,flags", [(512, 48, 128, 0), (4096, 160, 64, 0),
                                          (16384, 32, 512, 0), (2048, 400, 128, 1)])
def test_prepare_weight_sub_channel(K, N, g, flags):
    rrs = _rrs()
    _, W = _case(4, K, N, g, 41 + K + N)
    print(f"[case] sub-channel weights K={K} N={N} g={g} flags={flags}", flush=True)
    ref = O.sub_channel_weight(W, g, rotate=not (flags & rrs.SKIP_ROTATION))
    Wq, ws = rrs.prepare_weight_sub_channel(to_gpu(W), g, flags=flags)
    np.testing.assert_array_equal(to_np(ws), ref.scale.T)
    _check_sub_codes(to_np(Wq), ref, "sub-channel weights")


SHAPES = [(16, 512, 512, 128), (130, 1024, 272, 64), (256, 4096, 384, 128), (33, 2048, 160, 256)]


@pytest.mark.parametrize("M,K,N,g", SHAPES)
def test_scheme_per_channel(M, K, N, g):
    rrs = _rrs()
    X, W = _case(M, K, N, g, 51 + M)
    print(f"[case] per-channel scheme M={M} K={K} N={N}", flush=True)
    act = O.rotate_smooth_quant(X, g, smooth=False)
    wq = O.prepare_weight(W)
    Xq, a, _ = rrs.rotate_smooth_quant(to_gpu(X), g, flags=rrs.SKIP_SMOOTHING)
    Wq, beta = rrs.prepare_weight(to_gpu(W))
    check_codes(to_np(Xq), act, "per-channel activations")
    Y = rrs.w4a4_gemm_scheme(rrs.SCHEME_PER_CHANNEL, Xq, a, None, Wq, beta, g)
    P = O.group_partials(act.q, wq.q, g)
    ones = np.ones(K // g, np.float32)
    Yref = O.output(P, ones, act.alpha, wq.beta, norm=K)
    check_y(to_np(Y), Yref, P, ones, act.alpha, wq.beta, K, "per-channel")


@pytest.mark.parametrize("M,K,N,g", SHAPES)
def test_scheme_runtime_smooth_matches_main_kernel(M, K, N, g):
    rrs = _rrs()
    X, W = _case(M, K, N, g, 61 + M)
    print(f"[case] RS scheme M={M} K={K} N={N} g={g}", flush=True)
    Xg = to_gpu(X)
    Xq, a, s = rrs.rotate_smooth_quant(Xg, g)
    Wq, beta = rrs.prepare_weight(to_gpu(W))
    Y = rrs.w4a4_gemm_scheme(rrs.SCHEME_RUNTIME_SMOOTH, Xq, a, s, Wq, beta, g)
    Yref, act, wq, P = O.linear(X, W, g)
    check_y(to_np(Y), Yref, P, act.s, act.alpha, wq.beta, K, "RS scheme")


@pytest.mark.parametrize("M,K,N,g", SHAPES)
@pytest.mark.parametrize("flags", [0, 1])
def test_scheme_sub_channel(M, K, N, g, flags):
    rrs = _rrs()
    X, W = _case(M, K, N, g, 71 + M + flags)
    print(f"[case] sub-channel scheme M={M} K={K} N={N} g={g} flags={flags}", flush=True)
    rot = not (flags & rrs.SKIP_ROTATION)
    ax = O.sub_channel_quant(X, g, rotate=rot)
    aw = O.sub_channel_weight(W, g, rotate=rot)
    Xq, a = rrs.quantize_sub_channel(to_gpu(X), g, flags=flags)
    Wq, ws = rrs.prepare_weight_sub_channel(to_gpu(W), g, flags=flags)
    Y = to_np(rrs.w4a4_gemm_scheme(rrs.SCHEME_SUB_CHANNEL, Xq, a, None, Wq, ws, g, flags=flags))
    P = O.group_partials(ax.q, aw.q.T, g)
    norm = K if rot else 1
    Yref = O.output_sub_channel(P, ax.scale, aw.scale, norm)
    T = O.output_sub_channel_abs_terms(P, ax.scale, aw.scale, norm)
    G = K // g
    # per term: fl(a_ib * w_nb) and one fused multiply-add, then the sum: (G + 4) eps T
    bound = 1e-2 * np.maximum(np.abs(Yref), 2.0 ** -14) + (G + 4) * 2.0 ** -24 * T
    err = np.abs(Y.astype(np.float64) - Yref)
    assert np.all(np.isfinite(Y))
    assert np.all(err <= bound), f"sub-channel: {int((err > bound).sum())} outputs out of tolerance"


@pytest.mark.parametrize("M,K,N,g", SHAPES + [(8, 8192, 64, 128), (300, 4096, 1040, 128)])
@pytest.mark.parametrize("flags", [0, 1])
def test_per_channel_tuned(M, K, N, g, flags):
    rrs = _rrs()
    X, W = _case(M, K, N, g, 81 + M + flags)
    print(f"[case] per-channel tuned M={M} K={K} N={N} flags={flags}", flush=True)
    rot = not (flags & rrs.SKIP_ROTATION)
    act = O.rotate_smooth_quant(X, g, smooth=False, rotate=rot)
    wq = O.prepare_weight(W, rotate=rot)
    Xq, a, _ = rrs.rotate_smooth_quant(to_gpu(X), g, flags=flags | rrs.SKIP_SMOOTHING)
    Wq, beta = rrs.prepare_weight(to_gpu(W), flags=flags)
    Y = rrs.w4a4_gemm_per_channel(Xq, a, Wq, beta, flags=flags)
    P = O.group_partials(act.q, wq.q, g)
    ones = np.ones(K // g, np.float32)
    norm = K if rot else 1
    Yref = O.output(P, ones, act.alpha, wq.beta, norm=norm)
    check_y(to_np(Y), Yref, P, ones, act.alpha, wq.beta, norm, "per-channel tuned")
