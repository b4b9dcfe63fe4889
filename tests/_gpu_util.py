"""Shared helpers for the GPU parity tests (not collected by pytest)."""
import numpy as np

from oracle import rrs_oracle as O


def to_gpu(a, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def to_np(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def tile_wq(rows):
    """Row-major packed weights (N x K/2 bytes) -> the tiled layout that
    rrs_prepare_weight writes (include/rrs.h): 16-row blocks, each a run of K/128
    tiles of 1 KB; inside tile c of block nb, byte (q * 16 + r) * 16 + e holds
    packed byte 64 c + 16 q + e of row 16 nb + r. Returned as an N x K/2 array."""
    rows = np.ascontiguousarray(rows, dtype=np.uint8)
    N, Kh = rows.shape
    assert N % 16 == 0 and Kh % 64 == 0
    t = rows.reshape(N // 16, 16, Kh // 64, 4, 16).transpose(0, 2, 3, 1, 4)
    return np.ascontiguousarray(t).reshape(N, Kh)


def untile_wq(tiled):
    """Inverse of tile_wq: tiled weight bytes -> N x K/2 row-major packed rows."""
    tiled = np.ascontiguousarray(tiled, dtype=np.uint8)
    N, Kh = tiled.shape
    assert N % 16 == 0 and Kh % 64 == 0
    t = tiled.reshape(N // 16, Kh // 64, 4, 16, 16).transpose(0, 3, 1, 2, 4)
    return np.ascontiguousarray(t).reshape(N, Kh)


def near_half_integer(v, rel=1e-6):
    """Pre-rounding values within rel*|v| of a rounding boundary (k + 1/2)."""
    v = np.asarray(v, np.float64)
    return np.abs(np.abs(v - np.floor(v)) - 0.5) <= rel * np.maximum(np.abs(v), 1e-30)


def check_codes(gpu_packed, act, label):
    """GPU packed codes must equal the oracle's bit for bit; a code may differ
    only where the canonical pre-rounding value is within 1e-6 relative of a
    half-integer (counted and reported). Returns the number of such flips."""
    gq = O.unpack_int4(gpu_packed)
    diff = gq != act.q
    n = int(diff.sum())
    if n:
        flagged = near_half_integer(act.v)
        bad = diff & ~flagged
        assert not bad.any(), (
            f"{label}: {int(bad.sum())} code mismatches away from a rounding boundary; first at "
            f"{np.argwhere(bad)[:5].tolist()}")
        print(f"{label}: {n} boundary-flagged code flips")
    return n


def y_tolerance(P, s, alpha, beta, norm):
    """Elementwise bound for |Y_gpu - Y_ref|.

    1e-2 * max(|Y_ref|, 2^-14) is the contract; on top of it the rounding of
    the float32 sum over the G groups is bounded by (G + 3) * 2^-24 * T with
    T = |alpha beta| / norm * sum_b |s_b P_b| (any summation order), which only
    matters where the groups cancel to a tiny result.
    """
    G = P.shape[0]
    T = O.output_abs_terms(P, s, alpha, beta, norm)
    return T * (G + 3) * 2.0 ** -24


def check_y(y_gpu, y_ref, P, s, alpha, beta, norm, label):
    y_gpu = np.asarray(y_gpu, np.float64)
    y_ref = np.asarray(y_ref, np.float64)
    assert np.all(np.isfinite(y_gpu)), f"{label}: non-finite output"
    err = np.abs(y_gpu - y_ref)
    bound = 1e-2 * np.maximum(np.abs(y_ref), 2.0 ** -14) + y_tolerance(P, s, alpha, beta, norm)
    worst = np.argmax(err - bound)
    assert np.all(err <= bound), (
        f"{label}: {int((err > bound).sum())} outputs out of tolerance; worst at "
        f"{np.unravel_index(worst, err.shape)}: gpu={y_gpu.flat[worst]} ref={y_ref.flat[worst]}")
    # normwise: fp16 output rounding alone is 2^-11 relative
    nw = err.max() / max(np.abs(y_ref).max(), 1e-30)
    assert nw <= 2e-3, f"{label}: normwise error {nw}"
    return nw
