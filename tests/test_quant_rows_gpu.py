"""rrs_rotate_smooth_quant for up to 16 tokens without a static reorder: one
workgroup per token row, the rows' group maxima exchanged through the
workspace within the launch. Codes must equal the oracle's (boundary flips
aside), alpha and s bit for bit, whatever the workspace held before and when
one workspace serves consecutive calls with different row counts. After a call
with M > 1 the first two uint32 of the workspace read M rows arrived and no
wait that ran out."""
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


@pytest.mark.parametrize("M", [1, 2, 3, 7, 8, 9, 16])
@pytest.mark.parametrize("K,g", [(8192, 128), (512, 64), (4096, 512), (16384, 256), (2048, 64)])
def test_rows_match_oracle(M, K, g):
    rrs = _rrs()
    print(f"[case] quant rows M={M} K={K} g={g}", flush=True)
    ws = torch.empty((rrs.workspace_bytes(M, K, g),), dtype=torch.uint8, device="cuda")
    _check(_x(M, K, g, 5 * M + K + g), g, ws, f"rows {M}x{K}/g{g}")
    if M > 1:
        assert _words(ws) == [M, 0]


@pytest.mark.parametrize("M", [4, 16])
def test_rows_without_rotation(M):
    rrs = _rrs()
    K, g = 4096, 128
    print(f"[case] quant rows without rotation M={M}", flush=True)
    ws = torch.empty((rrs.workspace_bytes(M, K, g),), dtype=torch.uint8, device="cuda")
    _check(_x(M, K, g, 31 + M), g, ws, f"rows no-rot M={M}", flags=rrs.SKIP_ROTATION)
    assert _words(ws) == [M, 0]


def test_rows_garbage_workspace_and_reuse():
    # Workspace full of 0xFF (count included), then calls with 16, 5, 1 and 12
    # rows on it: each is checked against the oracle on its own.
    rrs = _rrs()
    K, g = 8192, 128
    ws = torch.full((rrs.workspace_bytes(16, K, g),), 255, dtype=torch.uint8, device="cuda")
    for i, M in enumerate([16, 5, 1, 12]):
        print(f"[case] quant rows reuse call {i} M={M}", flush=True)
        _check(_x(M, K, g, 700 + i), g, ws, f"reuse call {i} M={M}")
        if M > 1:
            assert _words(ws) == [M, 0]


def test_static_reorder_keeps_the_team_path():
    # With a static permutation the one-workgroup (team) kernel runs instead;
    # results still follow the oracle.
    rrs = _rrs()
    M, K, g = 6, 4096, 128
    print(f"[case] quant few tokens with perm M={M}", flush=True)
    X = _x(M, K, g, 77)
    perm = synth.permutation(K, 3)
    ws = torch.empty((rrs.workspace_bytes(M, K, g),), dtype=torch.uint8, device="cuda")
    Xq, a, s = rrs.rotate_smooth_quant(to_gpu(X), g, perm=to_gpu(perm), workspace=ws)
    act = O.rotate_smooth_quant(X, g, perm=perm)
    np.testing.assert_array_equal(to_np(a), act.alpha)
    np.testing.assert_array_equal(to_np(s), act.s)
    check_codes(to_np(Xq), act, "perm")
