"""Bit-exact checks of the GEMM kernels exactly as rrs_w4a4_gemm runs them.

With alpha = beta = 1 and the group scales one-hot (s_b = 1 for one group b,
0 for the others) the output is Y = fp16(P_b / K): every other group enters
as an FMA by 0, and P_b / K is exact in binary32 (K is a power of two). The
oracle therefore predicts Y bit for bit (Eq. 3 for one block), which checks
each kernel's integer path and its accumulator encoding (the magic-number
seed of the production loop) through the timed entry point, for every kernel
the dispatch chooses: the weight-streaming kernel (up to 16 tokens with four
waves; 17 to 32 tokens at K = 8192 with eight waves and two token blocks; both
weight layouts), the few-token kernel (one, two or four blocks of 16 tokens;
two or four
column blocks per workgroup, with a partly filled last workgroup; both weight
layouts) and the main kernel (partial row and column tiles). With codes in
[-2, 2] every |P_b| <= 4 g <= 2048 is an integer that fp16 holds exactly, so
the whole partial is compared; with codes in [-7, 7] the comparison covers
P_b to fp16's 11 bits.

The partials hook (rrs_w4a4_gemm_partials) runs the same kernels with the same
seeding and returns P_b itself: it is compared bit for bit on row x column
slices of the full-size workloads (qkv, large, decode).
"""
import numpy as np
import pytest

import synth
from oracle import rrs_oracle as O
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


# (M, K, N, g, tiled): which kernel rrs_w4a4_gemm takes for each
CASES = [
    # weight-streaming kernel: row-major, M <= 16, K >= 4 g (R < 1 KB, = 1 KB, 2 KB per row)
    (1, 2048, 48, 64, False), (3, 512, 32, 128, False), (8, 4096, 80, 128, False),
    (16, 8192, 32, 256, False), (5, 16384, 16, 512, False), (11, 1024, 64, 256, False),
    # weight-streaming kernel, eight waves: 17..32 tokens at K = 8192 in two
    # token blocks (the second ragged or full), both layouts, g = 64 (8-byte
    # lane pieces) to g = 512 (no seed); N = 4112 gives the first workgroup a
    # second column block
    (17, 8192, 48, 128, False), (32, 8192, 48, 64, True), (24, 8192, 4112, 512, False),
    (20, 8192, 4112, 256, True),
    # few-token kernel, row-major: K < 4 g, and 17..64 tokens elsewhere (two or
    # four token blocks, four column blocks per workgroup, the last one partly
    # filled)
    (1, 1024, 48, 512, False), (17, 2048, 48, 128, False), (40, 4096, 80, 64, False),
    (64, 2048, 16, 256, False), (40, 8192, 48, 128, False), (64, 16384, 32, 256, False),
    # few-token kernel, tiled weights
    (8, 4096, 48, 128, True), (24, 2048, 80, 512, True), (64, 8192, 32, 64, True),
    (16, 1024, 32, 64, True),
    # main kernel, partial row and column tiles
    (65, 2048, 144, 128, False), (300, 4096, 272, 64, False), (257, 2048, 400, 512, True),
    (130, 1024, 128, 256, True),
    # main kernel, more tiles than one pass of workgroups (776 tiles: up to four
    # per workgroup, ragged last row and column tiles among them)
    (2000, 512, 12400, 128, False), (1800, 512, 12400, 64, True),
]


def _one_hot_case(qx, qw, g, tiled, label):
    rrs = _rrs()
    M, K = qx.shape
    N = qw.shape[1]
    G = K // g
    P = O.group_partials(qx, qw, g)
    xq = to_gpu(O.pack_int4(qx))
    rows = O.pack_int4(qw.T)
    wq = to_gpu(tile_wq(rows) if tiled else rows)
    ones_m = to_gpu(np.ones(M, np.float32))
    ones_n = to_gpu(np.ones(N, np.float32))
    flags = rrs.WEIGHT_TILED if tiled else 0
    for b in sorted({0, G // 2, G - 1}):
        s = np.zeros(G, np.float32)
        s[b] = 1.0
        print(f"[case] one-hot {label} M={M} K={K} N={N} g={g} tiled={tiled} b={b}", flush=True)
        Y = rrs.w4a4_gemm(xq, ones_m, to_gpu(s), wq, ones_n, g, flags=flags)
        got = to_np(Y).view(np.uint16)
        want = (P[b].astype(np.float64) / K).astype(np.float32).astype(np.float16).view(np.uint16)
        bad = got != want
        assert not bad.any(), (
            f"{label} b={b}: {int(bad.sum())} outputs differ; first at "
            f"{np.argwhere(bad)[:3].tolist()}")


@pytest.mark.parametrize("M,K,N,g,tiled", CASES)
def test_one_hot_scales_exact_small_codes(M, K, N, g, tiled):
    # codes in [-2, 2]: every partial is an integer of magnitude <= 4 g <= 2048,
    # which fp16 represents exactly, so Y carries P_b bit for bit.
    rng = np.random.default_rng(M * 131 + K + N + g)
    qx = rng.integers(-2, 3, size=(M, K)).astype(np.int8)
    qw = rng.integers(-2, 3, size=(K, N)).astype(np.int8)
    assert np.abs(O.group_partials(qx, qw, g)).max() <= 2048
    _one_hot_case(qx, qw, g, tiled, "small codes")


@pytest.mark.parametrize("M,K,N,g,tiled", CASES)
def test_one_hot_scales_exact_full_range(M, K, N, g, tiled):
    rng = np.random.default_rng(M * 137 + K + N + g + 1)
    qx = rng.integers(-7, 8, size=(M, K)).astype(np.int8)
    qw = rng.integers(-7, 8, size=(K, N)).astype(np.int8)
    qx[0, :] = 7           # one row and column at the extreme: |P_b| = 49 g there
    qw[:, 0] = -7
    _one_hot_case(qx, qw, g, tiled, "full range")


# ------------------------------------------------------------------ partials hook

def _partials_slice(act_q, qw_cols, g, label):
    rrs = _rrs()
    print(f"[case] partials slice {label} M={act_q.shape[0]} K={act_q.shape[1]} "
          f"N={qw_cols.shape[1]} g={g}", flush=True)
    Pg = rrs.w4a4_gemm_partials(to_gpu(O.pack_int4(act_q)), to_gpu(O.pack_int4(qw_cols.T)), g)
    want = O.group_partials(act_q, qw_cols, g)
    got = to_np(Pg)
    bad = got != want
    assert not bad.any(), (f"{label}: {int(bad.sum())} partials differ; first at "
                           f"{np.argwhere(bad)[:3].tolist()}")


def _sample(n, k, seed, mult=1):
    rng = np.random.default_rng(seed)
    idx = np.unique(np.concatenate([[0, n - 1], rng.choice(n, k, replace=False)]))
    extra = (-len(idx)) % mult
    if extra:
        rest = np.setdiff1d(np.arange(n), idx)
        idx = np.sort(np.concatenate([idx, rng.choice(rest, extra, replace=False)]))
    return idx


@pytest.mark.parametrize("name", ["qkv", "large"])
def test_partials_full_size_slices(name):
    # The workloads' own codes (oracle quantization of the synthetic X and W),
    # on sampled token rows x output columns at the full K: the main kernel at
    # its real K loop and group size, and the few-token kernel on 40 rows.
    w = synth.WORKLOADS[name]
    act = O.rotate_smooth_quant(synth.activations(w), w.g)
    cols = _sample(w.N, 300, 21, mult=16)
    wq = O.prepare_weight(synth.weights(w)[:, cols])
    rows = _sample(w.M, 290, 22)
    _partials_slice(act.q[rows], wq.q, w.g, f"{name} rows x cols")
    _partials_slice(act.q[rows[:40]], wq.q, w.g, f"{name} 40 rows")


def test_partials_decode_full_rows():
    # All 8 tokens of the decode workload (the weight-streaming kernel) against
    # sampled output channels at K = 8192.
    w = synth.WORKLOADS["decode"]
    act = O.rotate_smooth_quant(synth.activations(w), w.g)
    cols = _sample(w.N, 300, 23, mult=16)
    wq = O.prepare_weight(synth.weights(w)[:, cols])
    _partials_slice(act.q, wq.q, w.g, "decode")


@pytest.mark.parametrize("M,K,N,g", [
    (1, 512, 16, 64), (16, 16384, 32, 512), (9, 8192, 48, 256), (4, 1024, 64, 128),
    (2, 1024, 16, 512),   # K < 4 g: the few-token kernel
    # eight waves, two token blocks (K = 8192)
    (32, 8192, 48, 128), (18, 8192, 4112, 64), (25, 8192, 32, 512),
])
def test_partials_stream_kernel_edges(M, K, N, g):
    rng = np.random.default_rng(M + K + N + g)
    qx = rng.integers(-7, 8, size=(M, K)).astype(np.int8)
    qw = rng.integers(-7, 8, size=(K, N)).astype(np.int8)
    qx[-1] = -7
    qw[:, -1] = 7
    _partials_slice(qx, qw, g, "stream edges")
