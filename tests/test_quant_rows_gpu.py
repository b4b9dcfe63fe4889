"""rrs_rotate_smooth_quant through its one-launch kernels: one workgroup per
token row for up to 16 tokens (up to 32 or 64 where a group's threads share
the reads of the exchanged words), and the fused kernel (every row rotated
once, kept in registers) for more tokens at K <= 4096. Both exchange the workgroups'
group maxima within the launch as epoch-tagged words in the workspace. Codes
must equal the oracle's (boundary flips aside), alpha and s bit for bit, on a
zeroed workspace and when one workspace serves consecutive calls of any shape
and kernel (per-row, fused, two-pass): every exchange advances the epoch in
header word 0 by one and leaves word 1 (the last failed epoch) at 0."""
import numpy as np
import pytest

import synth
from oracle import rrs_oracle as O
from tests._gpu_util import check_codes, to_gpu, to_np

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


def _x(M, K, g, seed):
    w = synth.custom("qr", M, K, 16, g, seed, n_chan=max(1, K // 100), chan_factor=(20, 100),
                     n_spike=max(1, M * K // 2000), spike_mag=(100, 500))
    return synth.activations(w)


def _check(X, g, ws, label, flags=0):
    rrs = _rrs()
    Xq, a, s = rrs.rotate_smooth_quant(to_gpu(X), g, workspace=ws, flags=flags)
    act = O.rotate_smooth_quant(X, g, rotate=not (flags & rrs.SKIP_ROTATION))
    np.testing.assert_array_equal(to_np(a), act.alpha, err_msg=f"{label}: alpha")
    np.testing.assert_array_equal(to_np(s), act.s, err_msg=f"{label}: s")
    check_codes(to_np(Xq), act, label)


def _words(ws):
    return ws[:8].view(torch.int32).cpu().tolist()


def _zeros(M, K, g):
    return torch.zeros((_rrs().workspace_bytes(M, K, g),), dtype=torch.uint8, device="cuda")


@pytest.mark.parametrize("M", [1, 2, 3, 7, 8, 9, 16])
@pytest.mark.parametrize("K,g", [(8192, 128), (512, 64), (4096, 512), (16384, 256), (2048, 64),
                                 (512, 256), (1024, 512)])
def test_rows_match_oracle(M, K, g):
    print(f"[case] quant rows M={M} K={K} g={g}", flush=True)
    ws = _zeros(M, K, g)
    _check(_x(M, K, g, 5 * M + K + g), g, ws, f"rows {M}x{K}/g{g}")
    # one exchange (none for a single row): epoch 0 -> 1, no failure
    assert _words(ws)[:2] == ([1, 0] if M > 1 else [0, 0])


@pytest.mark.parametrize("M,K,g", [
    (17, 8192, 128), (33, 8192, 128), (64, 8192, 128), (32, 8192, 64), (50, 8192, 512),
    (64, 16384, 256), (32, 16384, 128), (20, 8192, 256),
    (40, 4096, 128), (64, 1024, 64), (33, 2048, 256), (64, 512, 64),
])
def test_rows_many_tokens_match_oracle(M, K, g):
    # 17..64 rows: one workgroup per row, the tps threads of a group reading
    # rows k, k + tps, ... of the exchanged words
    print(f"[case] quant rows (shared reads) M={M} K={K} g={g}", flush=True)
    ws = _zeros(M, K, g)
    _check(_x(M, K, g, 13 * M + K + g), g, ws, f"rows {M}x{K}/g{g}")
    assert _words(ws)[:2] == [1, 0]


@pytest.mark.parametrize("M", [4, 16])
def test_rows_without_rotation(M):
    rrs = _rrs()
    K, g = 4096, 128
    print(f"[case] quant rows without rotation M={M}", flush=True)
    ws = _zeros(M, K, g)
    _check(_x(M, K, g, 31 + M), g, ws, f"rows no-rot M={M}", flags=rrs.SKIP_ROTATION)
    assert _words(ws)[:2] == [1, 0]


@pytest.mark.parametrize("M,K,g", [(65, 4096, 128), (300, 4096, 64), (2048, 4096, 128),
                                   (4096, 4096, 128), (3000, 2048, 512), (777, 512, 128),
                                   (5000, 1024, 256), (1000, 2048, 256), (1024, 4096, 128)])
def test_fused_match_oracle(M, K, g):
    # more than 64 tokens at K <= 4096: the fused one-launch kernel (one or
    # two rows per wave; 4096 rows at K = 4096 is its largest single-slot
    # case, 5000 at K = 1024 takes two slots)
    print(f"[case] quant fused M={M} K={K} g={g}", flush=True)
    ws = _zeros(M, K, g)
    _check(_x(M, K, g, 9 * M + K + g), g, ws, f"fused {M}x{K}/g{g}")
    assert _words(ws)[:2] == [1, 0]


def test_one_workspace_for_every_kernel():
    # One zeroed workspace for consecutive calls with different shapes and
    # kernels: per-row (16, 5, 1, 12 tokens), fused (1000 tokens), two-pass
    # (static reorder: 300 tokens), per-row again. Each call is checked on its
    # own against the oracle; the epoch counts the exchanges.
    rrs = _rrs()
    K, g = 4096, 128
    ws = _zeros(4096, K, g)
    epoch = 0
    for i, M in enumerate([16, 5, 1, 12, 1000, 300, 8]):
        X = _x(M, K, g, 700 + i)
        if M == 300:
            perm = synth.permutation(K, 11)
            print(f"[case] shared workspace call {i}: two-pass M={M}", flush=True)
            Xq, a, s = rrs.rotate_smooth_quant(to_gpu(X), g, perm=to_gpu(perm), workspace=ws)
            act = O.rotate_smooth_quant(X, g, perm=perm)
            np.testing.assert_array_equal(to_np(a), act.alpha)
            np.testing.assert_array_equal(to_np(s), act.s)
            check_codes(to_np(Xq), act, f"shared call {i}")
        else:
            print(f"[case] shared workspace call {i}: M={M}", flush=True)
            _check(X, g, ws, f"shared call {i} M={M}")
            if M > 1:
                epoch += 1
        assert _words(ws)[:2] == [epoch, 0], f"call {i}"


def test_static_reorder_keeps_the_team_path():
    # With a static permutation the one-workgroup (team) kernel runs instead;
    # results still follow the oracle.
    rrs = _rrs()
    M, K, g = 6, 4096, 128
    print(f"[case] quant few tokens with perm M={M}", flush=True)
    X = _x(M, K, g, 77)
    perm = synth.permutation(K, 3)
    ws = _zeros(M, K, g)
    Xq, a, s = rrs.rotate_smooth_quant(to_gpu(X), g, perm=to_gpu(perm), workspace=ws)
    act = O.rotate_smooth_quant(X, g, perm=perm)
    np.testing.assert_array_equal(to_np(a), act.alpha)
    np.testing.assert_array_equal(to_np(s), act.s)
    check_codes(to_np(Xq), act, "perm")
