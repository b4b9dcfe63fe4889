"""Host-only checks of the C ABI (no GPU needed): librrs.so loads, exports
every function include/rrs.h declares, and rejects invalid arguments with the
documented status code before touching any device.

The fake pointers used here are never dereferenced: every call below fails a
host-side check that comes before the device check. The one test that reaches
the device check only runs where no GPU is visible.
"""
import ctypes
import os
import re

import pytest

import paper_2409_20361_amd as rrs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rrs.h")

OK, NULL, SHAPE, GROUP, ALIGN, WS, NODEV, ARCH, HIP, FLAGS = 0, -1, -2, -3, -4, -5, -6, -7, -8, -9
PRECONDITION, TIMEOUT = -10, -11
P = 0x10000     # 16-byte aligned fake pointer (never dereferenced)
MIS = 0x10004   # misaligned fake pointer


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(rrs_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = rrs.lib()
    names = _declared()
    assert {"rrs_rotate_smooth_quant", "rrs_w4a4_gemm", "rrs_linear"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n
    # and they are real dynamic symbols of the shared object
    raw = ctypes.CDLL(rrs.lib_path())
    for n in names:
        getattr(raw, n)


def test_status_strings_and_version():
    for code in (OK, NULL, SHAPE, GROUP, ALIGN, WS, NODEV, ARCH, HIP, FLAGS, PRECONDITION,
                 TIMEOUT):
        s = rrs.status_string(code)
        assert s.startswith("RRS_") and s != "RRS_ERR_UNKNOWN"
    assert rrs.status_string(PRECONDITION).startswith("RRS_ERR_PRECONDITION")
    assert rrs.status_string(TIMEOUT).startswith("RRS_ERR_TIMEOUT")
    assert rrs.status_string(-99) == "RRS_ERR_UNKNOWN"
    assert rrs.version() >= 200   # 0.2.0: the _ex entry points


def test_workspace_queries():
    lib = rrs.lib()
    for M, K, g in ((16, 512, 128), (2048, 4096, 128), (8, 8192, 128), (8192, 8192, 64),
                    (3, 16384, 512)):
        q = lib.rrs_workspace_bytes(M, K, g)
        # a 256-byte header and 256 rows of K / 64 tagged 8-byte words (the
        # one-launch kernels), then 256 rows of K / 64 floats (the two-pass
        # kernels), each region 256-byte aligned
        a256 = lambda x: (x + 255) // 256 * 256  # noqa: E731
        assert q == 256 + a256(256 * (K // 64) * 8) + a256(256 * (K // 64) * 4)
        lw = lib.rrs_linear_workspace_bytes(M, K, g)
        a256 = lambda x: (x + 255) // 256 * 256  # noqa: E731
        assert lw == q + a256(M * K // 2) + a256(4 * M) + a256(4 * (K // g))
    for bad in ((0, 512, 128), (16, 500, 128), (16, 256, 64), (16, 32768, 128),
                (16, 512, 32), (16, 512, 1024), (16, 512, 96)):
        assert lib.rrs_workspace_bytes(*bad) == 0
        assert lib.rrs_linear_workspace_bytes(*bad) == 0


def _rsq(**kw):
    a = dict(X=P, M=16, K=512, g=128, perm=None, Xq=P, a=P, s=P, ws=P, wsb=1 << 30)
    a.update(kw)
    return rrs.lib().rrs_rotate_smooth_quant(a["X"], a["M"], a["K"], a["g"], a["perm"], a["Xq"],
                                             a["a"], a["s"], a["ws"], a["wsb"], None)


def _gemm(**kw):
    a = dict(Xq=P, a=P, s=P, Wq=P, w=P, M=16, N=512, K=512, g=128, Y=P)
    a.update(kw)
    return rrs.lib().rrs_w4a4_gemm(a["Xq"], a["a"], a["s"], a["Wq"], a["w"], a["M"], a["N"],
                                   a["K"], a["g"], a["Y"], None)


def _lin(**kw):
    a = dict(X=P, Wq=P, w=P, M=16, N=512, K=512, g=128, perm=None, Y=P, ws=P, wsb=1 << 30)
    a.update(kw)
    return rrs.lib().rrs_linear(a["X"], a["Wq"], a["w"], a["M"], a["N"], a["K"], a["g"],
                                a["perm"], a["Y"], a["ws"], a["wsb"], None)


def _prep(**kw):
    a = dict(W=P, K=512, N=512, perm=None, Wq=P, w=P)
    a.update(kw)
    return rrs.lib().rrs_prepare_weight(a["W"], a["K"], a["N"], a["perm"], a["Wq"], a["w"], None)


def _rsq_ex(**kw):
    a = dict(X=P, M=16, K=512, g=128, perm=None, flags=0, Xq=P, a=P, s=P, ws=P, wsb=1 << 30)
    a.update(kw)
    return rrs.lib().rrs_rotate_smooth_quant_ex(a["X"], a["M"], a["K"], a["g"], a["perm"],
                                                a["flags"], a["Xq"], a["a"], a["s"], a["ws"],
                                                a["wsb"], None)


def _gemm_ex(**kw):
    a = dict(Xq=P, a=P, s=P, Wq=P, w=P, M=16, N=512, K=512, g=128, flags=0, Y=P)
    a.update(kw)
    return rrs.lib().rrs_w4a4_gemm_ex(a["Xq"], a["a"], a["s"], a["Wq"], a["w"], a["M"], a["N"],
                                      a["K"], a["g"], a["flags"], a["Y"], None)


def _lin_ex(**kw):
    a = dict(X=P, Wq=P, w=P, M=16, N=512, K=512, g=128, perm=None, flags=0, Y=P, ws=P,
             wsb=1 << 30)
    a.update(kw)
    return rrs.lib().rrs_linear_ex(a["X"], a["Wq"], a["w"], a["M"], a["N"], a["K"], a["g"],
                                   a["perm"], a["flags"], a["Y"], a["ws"], a["wsb"], None)


def _prep_ex(**kw):
    a = dict(W=P, K=512, N=512, perm=None, flags=0, Wq=P, w=P)
    a.update(kw)
    return rrs.lib().rrs_prepare_weight_ex(a["W"], a["K"], a["N"], a["perm"], a["flags"],
                                           a["Wq"], a["w"], None)


def _parts(**kw):
    a = dict(Xq=P, Wq=P, M=16, N=512, K=512, g=128, P=P)
    a.update(kw)
    return rrs.lib().rrs_w4a4_gemm_partials(a["Xq"], a["Wq"], a["M"], a["N"], a["K"], a["g"],
                                            a["P"], None)


@pytest.mark.parametrize("fn,key", [
    (_rsq, "X"), (_rsq, "Xq"), (_rsq, "a"), (_rsq, "s"), (_rsq, "ws"),
    (_gemm, "Xq"), (_gemm, "a"), (_gemm, "s"), (_gemm, "Wq"), (_gemm, "w"), (_gemm, "Y"),
    (_lin, "X"), (_lin, "Wq"), (_lin, "w"), (_lin, "Y"), (_lin, "ws"),
    (_prep, "W"), (_prep, "Wq"), (_prep, "w"),
    (_parts, "Xq"), (_parts, "Wq"), (_parts, "P"),
])
def test_null_pointers(fn, key):
    assert fn(**{key: None}) == NULL


@pytest.mark.parametrize("fn,kw", [
    (_rsq_ex, dict(flags=8)), (_rsq_ex, dict(flags=-1)), (_rsq_ex, dict(flags=12)),
    (_gemm_ex, dict(flags=8)), (_gemm_ex, dict(flags=1 << 30)),
    (_lin_ex, dict(flags=8)), (_lin_ex, dict(flags=15)),
    (_prep_ex, dict(flags=2)), (_prep_ex, dict(flags=3)), (_prep_ex, dict(flags=6)),
    (_prep_ex, dict(flags=8)),
])
def test_bad_flags(fn, kw):
    assert fn(**kw) == FLAGS


@pytest.mark.parametrize("flags", [0, 1, 2, 3, 4, 5, 6, 7])
def test_good_flags_pass_the_flag_check(flags):
    # RRS_WEIGHT_TILED (4) is accepted everywhere, also where it has no effect
    # a valid flag word reaches the next check (alignment, workspace)
    assert _rsq_ex(flags=flags, Xq=MIS) == ALIGN
    assert _rsq_ex(flags=flags, wsb=0) == WS
    assert _gemm_ex(flags=flags, Y=MIS) == ALIGN
    assert _lin_ex(flags=flags, wsb=0) == WS
    if flags in (0, 1, 4, 5):
        assert _prep_ex(flags=flags, Wq=MIS) == ALIGN


def test_ex_check_order():
    # null beats shape beats group beats flags beats alignment beats workspace
    assert _rsq_ex(X=None, M=0, g=3, flags=8, Xq=MIS, wsb=0) == NULL
    assert _rsq_ex(M=0, g=3, flags=8, Xq=MIS, wsb=0) == SHAPE
    assert _rsq_ex(g=3, flags=8, Xq=MIS, wsb=0) == GROUP
    assert _rsq_ex(flags=8, Xq=MIS, wsb=0) == FLAGS
    assert _rsq_ex(Xq=MIS, wsb=0) == ALIGN
    assert _gemm_ex(Y=None, flags=8) == NULL
    assert _gemm_ex(N=8, flags=8) == SHAPE
    assert _prep_ex(K=1000, flags=2) == SHAPE
    assert _prep_ex(flags=2, W=MIS) == FLAGS


@pytest.mark.parametrize("fn,key", [
    (_rsq_ex, "X"), (_rsq_ex, "Xq"), (_rsq_ex, "ws"), (_gemm_ex, "s"), (_gemm_ex, "Y"),
    (_lin_ex, "X"), (_lin_ex, "ws"), (_prep_ex, "W"), (_prep_ex, "w"),
])
def test_ex_null_pointers(fn, key):
    assert fn(**{key: None}) == NULL


@pytest.mark.parametrize("kw", [dict(M=0), dict(M=-3), dict(K=500), dict(K=256),
                                dict(K=32768), dict(K=0)])
def test_bad_shapes_quant(kw):
    assert _rsq(**kw) == SHAPE


@pytest.mark.parametrize("fn", [_gemm, _lin, _parts])
@pytest.mark.parametrize("kw", [dict(N=0), dict(N=24), dict(N=-16), dict(M=0), dict(K=768),
                                dict(K=131072)])
def test_bad_shapes_gemm(fn, kw):
    assert fn(**kw) == SHAPE


@pytest.mark.parametrize("kw", [dict(K=1000), dict(N=8), dict(N=0)])
def test_bad_shapes_prep(kw):
    assert _prep(**kw) == SHAPE


@pytest.mark.parametrize("fn", [_rsq, _gemm, _lin, _parts])
@pytest.mark.parametrize("g", [0, 1, 32, 96, 1024, -128])
def test_bad_group(fn, g):
    assert fn(g=g) == GROUP


def test_group_must_divide_k():
    # g = K passes the group check and fails the later workspace check
    assert _rsq(K=512, g=512, wsb=0) == WS
    assert _rsq(K=512, g=1024) == GROUP
    assert _rsq(K=16384, g=512, wsb=0) == WS


@pytest.mark.parametrize("fn,key", [
    (_rsq, "X"), (_rsq, "Xq"), (_rsq, "a"), (_rsq, "s"), (_rsq, "ws"), (_rsq, "perm"),
    (_gemm, "Xq"), (_gemm, "Wq"), (_gemm, "Y"), (_gemm, "w"),
    (_lin, "X"), (_lin, "Y"), (_lin, "perm"), (_lin, "ws"),
    (_prep, "W"), (_prep, "Wq"), (_prep, "perm"),
    (_parts, "P"),
])
def test_misaligned(fn, key):
    assert fn(**{key: MIS}) == ALIGN


def test_workspace_too_small():
    need = rrs.workspace_bytes(16, 512, 128)
    assert _rsq(wsb=need - 1) == WS
    assert _rsq(wsb=0) == WS
    need_l = rrs.linear_workspace_bytes(16, 512, 128)
    assert _lin(wsb=need_l - 1) == WS


def test_check_order():
    # null beats shape beats group beats alignment beats workspace
    assert _rsq(X=None, M=0, g=3, Xq=MIS, wsb=0) == NULL
    assert _rsq(M=0, g=3, Xq=MIS, wsb=0) == SHAPE
    assert _rsq(g=3, Xq=MIS, wsb=0) == GROUP
    assert _rsq(Xq=MIS, wsb=0) == ALIGN


def _gpu_visible():
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:  # pragma: no cover
        return False


@pytest.mark.skipif(_gpu_visible(), reason="reaches the device check; only meaningful "
                    "(and only safe with fake pointers) where no GPU is visible")
def test_no_device():
    assert _rsq() == NODEV
    assert _gemm() == NODEV
    assert _lin() == NODEV
    assert _prep() == NODEV
    assert _parts() == NODEV
    for f in (0, 1, 2, 3):
        assert _rsq_ex(flags=f) == NODEV
        assert _gemm_ex(flags=f) == NODEV
        assert _lin_ex(flags=f) == NODEV
    assert _prep_ex(flags=1) == NODEV


# ------------------------------------------- kernel-comparison baselines (Section 4.5)

def _squant(**kw):
    a = dict(X=P, M=16, K=512, g=128, flags=0, Xq=P, a=P)
    a.update(kw)
    return rrs.lib().rrs_quantize_sub_channel(a["X"], a["M"], a["K"], a["g"], a["flags"],
                                              a["Xq"], a["a"], None)


def _sprep(**kw):
    a = dict(W=P, K=512, N=512, g=128, flags=0, Wq=P, w=P)
    a.update(kw)
    return rrs.lib().rrs_prepare_weight_sub_channel(a["W"], a["K"], a["N"], a["g"], a["flags"],
                                                    a["Wq"], a["w"], None)


def _scheme(**kw):
    a = dict(scheme=rrs.SCHEME_SUB_CHANNEL, Xq=P, x=P, s=None, Wq=P, w=P, M=16, N=512, K=512,
             g=128, flags=0, Y=P)
    a.update(kw)
    return rrs.lib().rrs_w4a4_gemm_scheme(a["scheme"], a["Xq"], a["x"], a["s"], a["Wq"], a["w"],
                                          a["M"], a["N"], a["K"], a["g"], a["flags"], a["Y"],
                                          None)


@pytest.mark.parametrize("fn,key", [
    (_squant, "X"), (_squant, "Xq"), (_squant, "a"),
    (_sprep, "W"), (_sprep, "Wq"), (_sprep, "w"),
    (_scheme, "Xq"), (_scheme, "x"), (_scheme, "Wq"), (_scheme, "w"), (_scheme, "Y"),
])
def test_baseline_null_pointers(fn, key):
    assert fn(**{key: None}) == NULL


def test_baseline_scheme_checks():
    # s_group is needed only by the Runtime Smooth scheme
    assert _scheme(scheme=rrs.SCHEME_RUNTIME_SMOOTH, s=None) == NULL
    assert _scheme(scheme=rrs.SCHEME_RUNTIME_SMOOTH, s=MIS) == ALIGN
    assert _scheme(scheme=7) == FLAGS
    assert _scheme(scheme=-1) == FLAGS
    assert _scheme(flags=8) == FLAGS
    assert _scheme(flags=4, Y=MIS) == ALIGN
    assert _scheme(N=20) == SHAPE
    assert _scheme(K=768) == SHAPE
    assert _scheme(g=96) == GROUP
    assert _scheme(x=MIS) == ALIGN
    assert _squant(flags=rrs.SKIP_SMOOTHING) == FLAGS   # only the rotation switch applies
    assert _squant(M=0) == SHAPE
    assert _squant(g=1024) == GROUP
    assert _squant(a=MIS) == ALIGN
    assert _sprep(flags=rrs.SKIP_SMOOTHING) == FLAGS
    assert _sprep(N=8) == SHAPE
    assert _sprep(g=32) == GROUP
    assert _sprep(Wq=MIS) == ALIGN


def _pc(**kw):
    a = dict(Xq=P, a=P, Wq=P, w=P, M=16, N=512, K=512, flags=0, Y=P)
    a.update(kw)
    return rrs.lib().rrs_w4a4_gemm_per_channel(a["Xq"], a["a"], a["Wq"], a["w"], a["M"], a["N"],
                                               a["K"], a["flags"], a["Y"], None)


@pytest.mark.parametrize("key", ["Xq", "a", "Wq", "w", "Y"])
def test_per_channel_null(key):
    assert _pc(**{key: None}) == NULL


def test_per_channel_checks():
    assert _pc(M=0) == SHAPE
    assert _pc(N=24) == SHAPE
    assert _pc(K=1000) == SHAPE
    assert _pc(flags=8) == FLAGS
    assert _pc(Y=MIS) == ALIGN


# ------------------------------------------- runtime channel reorder (Fig. 4 step (1))

def _rq(**kw):
    a = dict(X=P, M=16, K=512, g=128, flags=0, Xq=P, a=P, s=P, order=P, ws=P, wsb=1 << 30)
    a.update(kw)
    return rrs.lib().rrs_rotate_smooth_quant_reorder(a["X"], a["M"], a["K"], a["g"], a["flags"],
                                                     a["Xq"], a["a"], a["s"], a["order"],
                                                     a["ws"], a["wsb"], None)


def _rg(**kw):
    a = dict(Xq=P, a=P, s=P, Wq=P, w=P, order=P, M=16, N=512, K=512, g=128, flags=0, Y=P)
    a.update(kw)
    return rrs.lib().rrs_w4a4_gemm_reorder(a["Xq"], a["a"], a["s"], a["Wq"], a["w"], a["order"],
                                           a["M"], a["N"], a["K"], a["g"], a["flags"], a["Y"],
                                           None)


def _rl(**kw):
    a = dict(X=P, Wq=P, w=P, M=16, N=512, K=512, g=128, flags=0, Y=P, ws=P, wsb=1 << 30)
    a.update(kw)
    return rrs.lib().rrs_linear_reorder(a["X"], a["Wq"], a["w"], a["M"], a["N"], a["K"], a["g"],
                                        a["flags"], a["Y"], a["ws"], a["wsb"], None)


def test_reorder_workspace_queries():
    lib = rrs.lib()
    a256 = lambda x: (x + 255) // 256 * 256  # noqa: E731
    for M, K, g in ((16, 512, 128), (2048, 4096, 128), (8, 8192, 64), (3, 16384, 512)):
        q = lib.rrs_reorder_workspace_bytes(M, K, g)
        # the one-launch kernels' header and 16 rows of K/32 tagged words, then
        # 256 rows of K/32 block maxima (the two-launch path), then, at K <= 4096,
        # 256 rows of K/32 tagged words (the many-token one-launch kernel)
        words = a256(256 * (K // 32) * 8) if K <= 4096 else 0
        assert q == 256 + a256(16 * (K // 32) * 8) + a256(256 * (K // 32) * 4) + words
        lw = lib.rrs_linear_reorder_workspace_bytes(M, K, g)
        assert lw == q + a256(M * K // 2) + a256(4 * M) + a256(4 * (K // g)) + a256(4 * (K // 32))
    for bad in ((0, 512, 128), (16, 500, 128), (16, 512, 32), (16, 512, 1024)):
        assert lib.rrs_reorder_workspace_bytes(*bad) == 0
        assert lib.rrs_linear_reorder_workspace_bytes(*bad) == 0


@pytest.mark.parametrize("fn,key", [
    (_rq, "X"), (_rq, "Xq"), (_rq, "a"), (_rq, "s"), (_rq, "order"), (_rq, "ws"),
    (_rg, "Xq"), (_rg, "a"), (_rg, "s"), (_rg, "Wq"), (_rg, "w"), (_rg, "order"), (_rg, "Y"),
    (_rl, "X"), (_rl, "Wq"), (_rl, "w"), (_rl, "Y"), (_rl, "ws"),
])
def test_reorder_null_pointers(fn, key):
    assert fn(**{key: None}) == NULL


@pytest.mark.parametrize("fn", [_rq, _rg, _rl])
def test_reorder_checks(fn):
    assert fn(M=0) == SHAPE
    assert fn(K=768) == SHAPE
    assert fn(g=32) == GROUP
    assert fn(g=1024) == GROUP
    # only the rotation switch applies: without smoothing the order changes nothing
    assert fn(flags=rrs.SKIP_SMOOTHING) == FLAGS
    assert fn(flags=8) == FLAGS
    assert fn(flags=rrs.WEIGHT_TILED | rrs.SKIP_SMOOTHING) == FLAGS
    key = {_rq: "Xq", _rg: "order", _rl: "Y"}[fn]
    assert fn(**{key: MIS}) == ALIGN
    if fn is not _rq:
        assert fn(N=24) == SHAPE


def test_reorder_workspace_too_small():
    need = rrs.reorder_workspace_bytes(16, 512, 128)
    assert _rq(wsb=need - 1) == WS
    need_l = rrs.linear_reorder_workspace_bytes(16, 512, 128)
    assert _rl(wsb=need_l - 1) == WS


@pytest.mark.skipif(_gpu_visible(), reason="reaches the device check; only meaningful "
                    "(and only safe with fake pointers) where no GPU is visible")
def test_reorder_no_device():
    for f in (0, rrs.SKIP_ROTATION):
        assert _rq(flags=f) == NODEV
        assert _rg(flags=f) == NODEV
        assert _rl(flags=f) == NODEV


# ------------------------------------------------------------------ tiled Wq

@pytest.mark.parametrize("N,K", [(16, 512), (48, 1024), (32, 4096)])
def test_wq_tiling_helpers_follow_the_documented_layout(N, K):
    # include/rrs.h: packed byte j of row n sits at
    # (n/16) * 8K + (j/64) * 1024 + ((j%64)/16) * 256 + (n%16) * 16 + j%16.
    import numpy as np
    from tests._gpu_util import tile_wq, untile_wq
    rows = np.random.default_rng(N + K).integers(0, 256, (N, K // 2), dtype=np.uint8)
    flat = tile_wq(rows).reshape(-1)
    assert flat.size == N * K // 2
    for n in range(N):
        for j in range(K // 2):
            off = (n // 16) * 8 * K + (j // 64) * 1024 + ((j % 64) // 16) * 256 + (n % 16) * 16 \
                + j % 16
            assert flat[off] == rows[n, j]
    np.testing.assert_array_equal(untile_wq(tile_wq(rows)), rows)
    # a wave-sized slot (16 rows x 64 bytes of one K tile) is one contiguous 1 KB run
    slot = rows[16:32, 64:128] if N >= 32 and K >= 256 else rows[:16, :64]
    nb, c = (1, 1) if N >= 32 and K >= 256 else (0, 0)
    run = flat[nb * 8 * K + c * 1024: nb * 8 * K + c * 1024 + 1024]
    assert sorted(run.tolist()) == sorted(slot.reshape(-1).tolist())


def _qwait(**kw):
    a = dict(X=P, M=4, K=1024, g=128, extra=1, polls=8, Xq=P, a=P, s=P, ws=P, wsb=1 << 30,
             n=P)
    a.update(kw)
    return rrs.lib().rrs_test_quant_rows_wait(a["X"], a["M"], a["K"], a["g"], a["extra"],
                                              a["polls"], a["Xq"], a["a"], a["s"], a["ws"],
                                              a["wsb"], a["n"], None)


def test_quant_rows_wait_hook_checks():
    # the failure-path test hook validates like the quantizer, in the same order
    for key in ("X", "Xq", "a", "s", "ws", "n"):
        assert _qwait(**{key: None}) == NULL, key
    assert _qwait(M=1) == SHAPE       # one row: no exchange
    assert _qwait(M=65, K=8192) == SHAPE   # no one-launch kernel for this shape
    assert _qwait(M=33, K=8192, g=64) == SHAPE   # per-row up to 32 rows at g = K / 128
    assert _qwait(K=1000) == SHAPE
    assert _qwait(g=96) == GROUP
    assert _qwait(extra=-1) == FLAGS
    assert _qwait(polls=0) == FLAGS
    assert _qwait(M=4, extra=61) == FLAGS  # the per-row kernel waits for <= 64 rows
    assert _qwait(M=4, K=512, g=512, extra=13) == FLAGS  # <= 16 where one thread reads all
    assert _qwait(M=60, K=8192, extra=5) == FLAGS  # <= 64 rows at K = 8192, g = 128
    assert _qwait(M=30, K=8192, g=64, extra=3) == FLAGS  # <= 32 rows at g = 64
    assert _qwait(X=MIS) == ALIGN
    assert _qwait(wsb=16) == WS
    assert _qwait(M=65, K=8192, X=None) == NULL   # null pointers first


def _rwait(**kw):
    a = dict(X=P, M=4, K=1024, g=128, extra=1, polls=8, Xq=P, a=P, s=P, o=P, ws=P,
             wsb=1 << 30, n=P)
    a.update(kw)
    return rrs.lib().rrs_test_quant_reorder_wait(a["X"], a["M"], a["K"], a["g"], a["extra"],
                                                 a["polls"], a["Xq"], a["a"], a["s"], a["o"],
                                                 a["ws"], a["wsb"], a["n"], None)


def test_quant_reorder_wait_hook_checks():
    for key in ("X", "Xq", "a", "s", "o", "ws", "n"):
        assert _rwait(**{key: None}) == NULL, key
    assert _rwait(M=1) == SHAPE            # one row: no exchange
    assert _rwait(M=17, K=8192) == SHAPE   # more than 16 rows above K = 4096: two launches
    assert _rwait(M=5000, K=4096) == SHAPE  # more rows than one launch holds at K = 4096
    assert _rwait(K=16384) == SHAPE        # K > 8192: two launches
    assert _rwait(K=1000) == SHAPE
    assert _rwait(g=96) == GROUP
    assert _rwait(extra=-1) == FLAGS
    assert _rwait(polls=0) == FLAGS
    assert _rwait(M=4, extra=13) == FLAGS  # at most 16 rows in all
    assert _rwait(o=MIS) == ALIGN
    assert _rwait(wsb=16) == WS
    assert _rwait(M=17, X=None) == NULL    # null pointers first


def test_debug_checks_come_after_host_validation():
    # RRS_DEBUG only adds checks after the regular ones: invalid arguments still
    # get their usual codes, before any device access.
    old = os.environ.get("RRS_DEBUG")
    os.environ["RRS_DEBUG"] = "1"
    try:
        assert _rsq(X=None) == NULL
        assert _rsq(K=1000) == SHAPE
        assert _gemm(g=96) == GROUP
        assert _lin(ws=MIS) == ALIGN
        assert _prep(K=100) == SHAPE
    finally:
        if old is None:
            del os.environ["RRS_DEBUG"]
        else:
            os.environ["RRS_DEBUG"] = old
