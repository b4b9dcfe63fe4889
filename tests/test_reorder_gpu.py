"""GPU parity of the runtime channel reorder (Fig. 4 step (1) taken at run time)
against the CPU oracle: block order, group scales, token scales and codes bit
for bit (a code may differ only at a flagged rounding boundary); the GEMM that
gathers weight blocks, and the whole layer, within the output tolerance of
tests/_gpu_util.check_y."""
import numpy as np
import pytest

import synth
from oracle import rrs_oracle as O
from tests._gpu_util import check_codes, check_y, to_gpu, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

BLOCK = 32


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2409_20361_amd as rrs
    rrs.lib()
    assert rrs.REORDER_BLOCK == BLOCK


def _rrs():
    import paper_2409_20361_amd as rrs
    return rrs


def _case(M, K, N, g, seed):
    w = synth.custom("r", M, K, N, g, seed, n_chan=max(1, K // 100), chan_factor=(20, 100),
                     n_spike=max(1, M * K // 10000), spike_mag=(100, 500))
    return w, synth.activations(w), synth.weights(w)


def _quant_case(X, g, flags, label):
    rrs = _rrs()
    rot = not (flags & rrs.SKIP_ROTATION)
    print(f"[case] reorder quant {label} M={X.shape[0]} K={X.shape[1]} g={g} flags={flags}",
          flush=True)
    act, order, perm = O.rotate_smooth_quant_reorder(X, g, BLOCK, rotate=rot)
    Xq, a, s, bo = rrs.rotate_smooth_quant_reorder(to_gpu(X), g, flags=flags)
    np.testing.assert_array_equal(to_np(bo), order, err_msg=f"{label}: block order")
    np.testing.assert_array_equal(to_np(s), act.s, err_msg=f"{label}: s_group")
    np.testing.assert_array_equal(to_np(a), act.alpha, err_msg=f"{label}: alpha")
    flips = check_codes(to_np(Xq), act, label)
    assert flips == 0 or flips < 1e-6 * X.size
    return act, order, (Xq, a, s, bo)


# One launch: the per-row kernel exchanging block maxima, up to 16 rows at
# K <= 8192 (including the decode shape); the one-row-per-wave kernel with its
# two-level exchange, more rows at K <= 4096 (four or eight waves, one or two
# rows per wave). Two launches: K = 8192 / 16384 with more than 16 rows, and
# more rows than the one-launch kernel holds.
@pytest.mark.parametrize("M,K,g,flags", [
    (16, 512, 128, 0), (1, 512, 64, 0), (100, 1024, 256, 0), (37, 2048, 64, 0),
    (700, 2048, 128, 0), (5, 4096, 512, 0), (300, 8192, 64, 0), (9, 16384, 128, 0),
    (64, 4096, 128, 1), (20, 8192, 256, 1), (513, 1024, 512, 1),
    (2, 1024, 64, 0), (8, 8192, 128, 0), (16, 8192, 64, 0), (3, 2048, 256, 1),
    (12, 4096, 128, 1), (2, 8192, 512, 0), (1, 8192, 128, 0), (17, 8192, 128, 0),
    (3000, 4096, 128, 0), (5000, 512, 64, 0), (9000, 1024, 128, 0), (4500, 4096, 256, 0),
])
def test_quant_reorder(M, K, g, flags):
    _, X, _ = _case(M, K, 16, g, 7 + M + K + g)
    _quant_case(X, g, flags, f"{M}x{K}/g{g}")


def test_quant_reorder_one_launch_reuses_workspace():
    # The one-launch path exchanges block maxima in the workspace under the
    # epoch protocol: consecutive calls on one (zero-initialised) workspace,
    # with different inputs and row counts, must each match the oracle.
    rrs = _rrs()
    K, g = 8192, 128
    ws = torch.zeros(rrs.reorder_workspace_bytes(16, K, g), dtype=torch.uint8, device="cuda")
    for i, M in enumerate((8, 16, 3, 8)):
        _, X, _ = _case(M, K, 16, g, 101 + i)
        act, order, _ = O.rotate_smooth_quant_reorder(X, g, BLOCK)
        print(f"[case] reorder one-launch reuse call {i} M={M}", flush=True)
        Xq, a, s, bo = rrs.rotate_smooth_quant_reorder(to_gpu(X), g, workspace=ws)
        np.testing.assert_array_equal(to_np(bo), order, err_msg=f"call {i}: block order")
        np.testing.assert_array_equal(to_np(s), act.s, err_msg=f"call {i}: s_group")
        np.testing.assert_array_equal(to_np(a), act.alpha, err_msg=f"call {i}: alpha")
        flips = check_codes(to_np(Xq), act, f"call {i}")
        assert flips == 0 or flips < 1e-6 * X.size


def test_quant_reorder_many_rows_reuses_workspace():
    # The many-token one-launch form: runs of workgroups and their leaders
    # change with the row count; consecutive calls on one workspace must each
    # match the oracle.
    rrs = _rrs()
    K, g = 4096, 128
    ws = torch.zeros(rrs.reorder_workspace_bytes(2048, K, g), dtype=torch.uint8, device="cuda")
    for i, M in enumerate((300, 2048, 17, 1000, 300)):
        _, X, _ = _case(M, K, 16, g, 211 + i)
        act, order, _ = O.rotate_smooth_quant_reorder(X, g, BLOCK)
        print(f"[case] reorder many-row reuse call {i} M={M}", flush=True)
        Xq, a, s, bo = rrs.rotate_smooth_quant_reorder(to_gpu(X), g, workspace=ws)
        np.testing.assert_array_equal(to_np(bo), order, err_msg=f"call {i}: block order")
        np.testing.assert_array_equal(to_np(s), act.s, err_msg=f"call {i}: s_group")
        np.testing.assert_array_equal(to_np(a), act.alpha, err_msg=f"call {i}: alpha")
        flips = check_codes(to_np(Xq), act, f"call {i}")
        assert flips == 0 or flips < 1e-6 * X.size


def test_quant_reorder_full_size():
    # The benchmark's prefill shape (the partial-row reduction at its largest:
    # 256 rows of K/32 block maxima).
    w = synth.WORKLOADS["qkv"]
    _quant_case(synth.activations(w), w.g, 0, "qkv")


@pytest.mark.parametrize("M,K", [(8, 1024), (8, 8192), (40, 8192)])
def test_quant_reorder_ties(M, K):
    # all-zero input: every key is 0, the order is the identity, all codes 0
    X = np.zeros((M, K), np.float16)
    act, order, (Xq, a, s, bo) = _quant_case(X, 128, 0, f"zeros {M}x{K}")
    np.testing.assert_array_equal(to_np(bo), np.arange(K // BLOCK))
    assert not to_np(Xq).any()


# Repeated blocks without rotation: every block is the same block scaled by 1,
# 2 or 4 (exact in fp16), so the K/32 keys take three values and equal keys
# fall in every list of 64 the ranking merges; equal keys keep increasing
# block index. One launch per row (M <= 16), the many-token one-launch kernel
# (K <= 4096) and the two-launch form (K = 8192 / 16384 with more rows).
@pytest.mark.parametrize("M,K", [(40, 4096), (3000, 4096), (1, 8192), (8, 8192), (16, 8192),
                                 (40, 8192), (20, 16384), (2, 512)])
def test_quant_reorder_repeated_blocks(M, K):
    rrs = _rrs()
    rng = np.random.default_rng(9 + M + K)
    base = rng.uniform(-1, 1, size=(M, BLOCK))
    scale = rng.choice([1.0, 2.0, 4.0], size=K // BLOCK)
    X = np.concatenate([base * c for c in scale], axis=1).astype(np.float16)
    act, order, _ = _quant_case(X, 128, rrs.SKIP_ROTATION, f"repeated blocks {M}x{K}")
    # the oracle's order itself: blocks of scale 4, then 2, then 1, each run in
    # increasing block index
    expect = np.concatenate([np.flatnonzero(scale == c) for c in (4.0, 2.0, 1.0)])
    np.testing.assert_array_equal(order, expect)


def _tol_terms(act_q, wq_q, s, g, M):
    """Partials and scales whose fp32 sum the kernel takes: the main kernel adds
    K/g group terms, the few-token (M <= 16) gather kernel K/32 block terms, each
    block scaled by its group's s (the tolerance bound is on that sum)."""
    if M > 16:
        return None, None
    return O.group_partials(act_q, wq_q, BLOCK), np.repeat(np.asarray(s), g // BLOCK)


def _gemm_ref(X, W, g, order, rotate=True):
    """Oracle layer for a given block order (sorted or not)."""
    perm = O.block_order_to_perm(order, BLOCK)
    act = O.rotate_smooth_quant(X, g, perm=perm, rotate=rotate)
    wq = O.prepare_weight(W, perm=perm, rotate=rotate)
    P = O.group_partials(act.q, wq.q, g)
    return act, wq, P


@pytest.mark.parametrize("M,K,N,g", [
    (300, 4096, 256, 128), (256, 1024, 400, 64), (77, 2048, 160, 256), (40, 512, 96, 512),
    (8, 8192, 128, 128), (1, 512, 32, 64), (16, 2048, 48, 512), (13, 4096, 80, 256),
])
@pytest.mark.parametrize("kind", ["runtime", "random"])
def test_gemm_reorder(M, K, N, g, kind):
    # The GEMM alone, on the oracle's codes: with the runtime order, and with a
    # random block order (the gather must not depend on the order being sorted).
    rrs = _rrs()
    w, X, W = _case(M, K, N, g, 17 + M + N)
    print(f"[case] reorder gemm {kind} M={M} K={K} N={N} g={g}", flush=True)
    if kind == "runtime":
        _, order, _ = O.rotate_smooth_quant_reorder(X, g, BLOCK)
    else:
        order = np.random.default_rng(M + K).permutation(K // BLOCK)
    act, wq, P = _gemm_ref(X, W, g, order)
    wnat = O.prepare_weight(W)                       # weights prepared once, natural order
    np.testing.assert_array_equal(wq.q, wnat.q[O.block_order_to_perm(order, BLOCK)])
    Y = rrs.w4a4_gemm_reorder(to_gpu(act.packed), to_gpu(act.alpha), to_gpu(act.s),
                              to_gpu(wnat.packed), to_gpu(wnat.beta),
                              to_gpu(order.astype(np.int32)), g)
    y_ref = O.output(P, act.s, act.alpha, wq.beta, norm=K)
    Pt, st = _tol_terms(act.q, wq.q, act.s, g, M)
    check_y(to_np(Y), y_ref, P if Pt is None else Pt, act.s if st is None else st, act.alpha,
            wq.beta, K, f"gemm {kind} {M}x{K}x{N}")


@pytest.mark.parametrize("M", [8, 300])
def test_gemm_reorder_table_entries_masked(M):
    # Entries are reduced modulo K/32 on the device: a table shifted by
    # multiples of K/32 (also negative ones) gives bit-identical outputs.
    rrs = _rrs()
    K, N, g = 2048, 128, 128
    w, X, W = _case(M, K, N, g, 5 + M)
    print(f"[case] reorder gemm masked table M={M}", flush=True)
    order = np.random.default_rng(3).permutation(K // BLOCK).astype(np.int32)
    act, wq, P = _gemm_ref(X, W, g, order)
    wnat = O.prepare_weight(W)
    args = (to_gpu(act.packed), to_gpu(act.alpha), to_gpu(act.s), to_gpu(wnat.packed),
            to_gpu(wnat.beta))
    Y0 = rrs.w4a4_gemm_reorder(*args, to_gpu(order), g)
    shifted = order + (K // BLOCK) * np.where(np.arange(order.size) % 2 == 0, 3, -1)
    Y1 = rrs.w4a4_gemm_reorder(*args, to_gpu(shifted.astype(np.int32)), g)
    assert torch.equal(Y0, Y1)


def _linear_case(w, X, W, flags=0, row_sample=None, col_sample=None, label=""):
    rrs = _rrs()
    rot = not (flags & rrs.SKIP_ROTATION)
    norm = w.K if rot else 1
    print(f"[case] reorder linear {label} M={w.M} K={w.K} N={w.N} g={w.g} flags={flags}",
          flush=True)
    Xg = to_gpu(X)
    Wq, beta = rrs.prepare_weight(to_gpu(W), flags=flags & rrs.SKIP_ROTATION)
    Xq, a, s, bo = rrs.rotate_smooth_quant_reorder(Xg, w.g, flags=flags)
    Y = rrs.w4a4_gemm_reorder(Xq, a, s, Wq, beta, bo, w.g, flags=flags)
    Y2 = rrs.linear_reorder(Xg, Wq, beta, w.g, flags=flags)
    assert torch.equal(Y, Y2), f"{label}: rrs_linear_reorder differs from quant + gemm"
    Y = to_np(Y).astype(np.float32)

    act, order, perm = O.rotate_smooth_quant_reorder(X, w.g, BLOCK, rotate=rot)
    np.testing.assert_array_equal(to_np(bo), order)
    np.testing.assert_array_equal(to_np(a), act.alpha)
    np.testing.assert_array_equal(to_np(s), act.s)
    check_codes(to_np(Xq), act, label)
    rows = np.arange(w.M) if row_sample is None else row_sample
    cols = np.arange(w.N) if col_sample is None else col_sample
    wq = O.prepare_weight(W[:, cols], perm=perm, rotate=rot)
    np.testing.assert_array_equal(to_np(beta)[cols], wq.beta)
    P = O.group_partials(act.q[rows], wq.q, w.g)
    y_ref = O.output(P, act.s, act.alpha[rows], wq.beta, norm=norm)
    Pt, st = _tol_terms(act.q[rows], wq.q, act.s, w.g, w.M)
    nw = check_y(Y[np.ix_(rows, cols)], y_ref, P if Pt is None else Pt,
                 act.s if st is None else st, act.alpha[rows], wq.beta, norm, label)
    print(f"{label}: normwise |dY|/|Y| = {nw:.3e}")


@pytest.mark.parametrize("M,K,N,g,flags", [
    (16, 512, 512, 128, 0), (130, 2048, 400, 512, 0), (77, 4096, 272, 128, 0),
    (5, 8192, 64, 64, 0), (300, 1024, 160, 256, 1), (9, 16384, 48, 128, 0),
])
def test_linear_reorder(M, K, N, g, flags):
    w, X, W = _case(M, K, N, g, 23 + M + K)
    _linear_case(w, X, W, flags, label=f"{M}x{K}x{N}/g{g}")


@pytest.mark.parametrize("name", ["qkv", "decode"])
def test_linear_reorder_full_size_sampled(name):
    # The benchmark's shapes and launch configuration; outputs on a sample of
    # rows x columns (plus the first/last row and column).
    w = synth.WORKLOADS[name]
    rng = np.random.default_rng(13)
    rows = np.unique(np.concatenate([[0, w.M - 1], rng.choice(w.M, min(w.M, 48),
                                                               replace=False)]))
    cols = np.unique(np.concatenate([[0, w.N - 1], rng.choice(w.N, 160, replace=False)]))
    _linear_case(w, synth.activations(w), synth.weights(w), row_sample=rows,
                 col_sample=cols, label=name)


def test_reorder_deterministic():
    rrs = _rrs()
    w, X, W = _case(512, 4096, 256, 128, 99)
    Xg = to_gpu(X)
    Wq, beta = rrs.prepare_weight(to_gpu(W))
    outs = [rrs.linear_reorder(Xg, Wq, beta, w.g) for _ in range(3)]
    for o in outs[1:]:
        assert torch.equal(o, outs[0])
