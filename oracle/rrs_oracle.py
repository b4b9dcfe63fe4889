"""CPU oracle for the Rotated Runtime Smooth (RRS) W4A4 linear layer.

TEST INFRASTRUCTURE ONLY. Only the test suite, the package's smoke check and
the benchmark's CPU-baseline leg may import this module. The product path (the
HIP library and its Python binding) never calls it, and it shares no code with
that path.

Paper: "Rotated Runtime Smooth: Training-Free Activation Smoother for accurate
INT4 inference" (arXiv 2409.20361).

Notation. The paper writes X in R^{N x K} (N tokens) and W in R^{M x K}
(Section 3.1). This module writes X: M x K (M tokens), W: K x N (N output
channels), the orientation of the library's interface. H_K is the +-1
Sylvester Hadamard matrix (H_K H_K^T = K I) and R = H_K / sqrt(K) (Eq. 4 and
Appendix A.1).

What is computed, step by step, in the paper's order:

  1. rotate each token: y_i = x_i H_K (Section 3.3 rotates the activations and
     then smooths them; Fig. 2(a) gives Y = (XR)(R^-1 W^T));
  2. optional static channel reorder pi (Fig. 4 step (1), Section 3.2);
  3. runtime channel maxima c_j = max_i |y_ij| (Eq. 1), grouped: the smoothing
     scale of group b is the largest c_j in it (Fig. 4 step (2), Section 3.2);
  4. per-token symmetric INT4 quantization of the smoothed activations,
     alpha = max|.| / 7 (Section 2.1, Eq. 2; per-token RTN per Section 4.1);
  5. weights rotated offline (H_K W) and quantized per output channel
     (Section 3.3 last paragraph; RTN stands in for GPTQ);
  6. per-group integer partial products P_b and the rescale
     Y = sum_b s_b P_b * alpha_i * beta_n / K (Eq. 3 with a block-constant
     scale, Section 3.2 and Fig. 4 step (3)).

Two arithmetic modes:

  * "fp32" (canonical): every floating-point step is one IEEE binary32
    operation with round-to-nearest-even, in a fixed order. The HIP path must
    reproduce codes, scales and partial sums of this mode bit for bit.
  * "fp64" (exact): the same steps in binary64. The FWHT of fp16 inputs is
    exact in binary64 for K <= 8192, so this mode gives the pre-rounding values
    that invariants and boundary reports use.

Readings of the paper (it is silent or loose on these points):

  * Hadamard matrix: Sylvester natural order, no random sign diagonal; the
    rotation is applied unnormalized (x H_K) and the 1/K of R R^T is folded
    into the output scale, which is exact (powers of two).
  * FWHT stage order: h = 1, 2, 4, ..., K/2; in each stage, for every index p
    with bit h clear, (y[p], y[p+h]) <- (y[p] + y[p+h], y[p] - y[p+h]).
  * Channel maxima run over all M tokens of the call (Eq. 1 takes the max over
    the token axis); one scale per channel group, shared by all tokens.
  * Smoothing divides by the scale: implemented as multiplication by the
    rounded reciprocal r_b = fl(1/s_b) (0 when s_b = 0).
  * Token scale: a_i = max_b fl(M_ib r_b) with M_ib = max_{j in b} |y_ij|;
    inv_i = fl(7 / a_i) (0 when a_i = 0), alpha_i = fl(a_i / 7).
  * Codes: q_ij = clamp(rint(fl(y_ij * fl(r_b * inv_i))), -7, 7), rint rounds
    half to even; -8 is never produced (symmetric range of Section 2.1).
  * Weights: u = H_K W (column FWHT), b_n = max_k |u_kn|, winv_n = fl(7/b_n),
    w_kn = clamp(rint(fl(u_kn winv_n)), -7, 7), beta_n = fl(b_n / 7).
  * Output: Y = fl32((alpha_i beta_n / K) * sum_b s_b P_b[i, n]), the sum and
    the products taken in binary64 (the group's smoothing scale multiplies
    each block's dequantized partial product, Fig. 4 step (3)).
  * Packing: two's-complement nibbles, two per byte, low nibble = even index.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np

QMAX = 7  # 2^(4-1) - 1, Section 2.1


def _dt(mode: str):
    if mode == "fp32":
        return np.float32
    if mode == "fp64":
        return np.float64
    raise ValueError(f"unknown mode {mode!r}")


# --------------------------------------------------------------------------
# Step 1: rotation (Section 3.3, Eq. 4, Appendix A.1)
# --------------------------------------------------------------------------

def fwht(x: np.ndarray, mode: str = "fp32", axis: int = -1) -> np.ndarray:
    """Unnormalized Walsh-Hadamard transform along `axis`: returns x H_K.

    Butterfly stages in the order h = 1, 2, 4, ..., K/2. In binary32 mode each
    butterfly output is one rounded add or subtract; this fixed order is the
    canonical rounding order the GPU reproduces.
    """
    dt = _dt(mode)
    y = np.moveaxis(np.array(x, dtype=dt, copy=True), axis, -1)
    y = np.ascontiguousarray(y)
    K = y.shape[-1]
    if K & (K - 1):
        raise ValueError("K must be a power of two")
    lead = y.shape[:-1]
    h = 1
    while h < K:
        v = y.reshape(*lead, K // (2 * h), 2, h)
        a = v[..., 0, :].copy()
        b = v[..., 1, :].copy()
        v[..., 0, :] = a + b
        v[..., 1, :] = a - b
        h *= 2
    return np.moveaxis(y, -1, axis)


def hadamard(K: int) -> np.ndarray:
    """Dense Sylvester H_K (float64), built by doubling: H_2K = [[H, H], [H, -H]]."""
    H = np.ones((1, 1), dtype=np.float64)
    while H.shape[0] < K:
        H = np.block([[H, H], [H, -H]])
    if H.shape[0] != K:
        raise ValueError("K must be a power of two")
    return H


# --------------------------------------------------------------------------
# Steps 2-4: reorder, runtime smoothing scales, per-token quantization
# (Eq. 1-2, Section 3.2, Fig. 4, Section 2.1)
# --------------------------------------------------------------------------

def channel_max(y: np.ndarray) -> np.ndarray:
    """c_j = max_i |y_ij| over all tokens (Eq. 1). Exact in any precision."""
    return np.abs(y).max(axis=0)


def group_scales(c: np.ndarray, g: int, mode: str = "fp32"):
    """s_b = max_{j in group b} c_j (Section 3.2); r_b = fl(1/s_b), 0 if s_b = 0."""
    dt = _dt(mode)
    K = c.shape[0]
    if K % g:
        raise ValueError("group size must divide K")
    s = c.reshape(K // g, g).max(axis=1).astype(dt)
    r = np.zeros_like(s)
    nz = s != 0
    r[nz] = dt(1) / s[nz]
    return s, r


def token_scales(y: np.ndarray, r: np.ndarray, g: int, mode: str = "fp32"):
    """a_i = max_b fl(M_ib r_b); inv_i = fl(7/a_i) (0 if a_i = 0); alpha_i = fl(a_i/7).

    M_ib is the largest |y_ij| of token i in group b; multiplying it by r_b is
    the smoothing X/s of Eq. 2 applied to the group maximum, and alpha is the
    symmetric INT4 scale of Section 2.1 taken per token.
    """
    dt = _dt(mode)
    M, K = y.shape
    Mib = np.abs(y).reshape(M, K // g, g).max(axis=2)
    a = (Mib * r[None, :]).astype(dt).max(axis=1)
    inv = np.zeros_like(a)
    nz = a != 0
    inv[nz] = dt(QMAX) / a[nz]
    alpha = a / dt(QMAX)
    return a, inv, alpha


def quantize_codes(y: np.ndarray, r: np.ndarray, inv: np.ndarray, g: int,
                   mode: str = "fp32", return_v: bool = False):
    """q_ij = clamp(rint(fl(y_ij * fl(r_b * inv_i))), -7, 7)  (Section 2.1)."""
    dt = _dt(mode)
    M, K = y.shape
    m = (r[None, :] * inv[:, None]).astype(dt)              # M x G
    v = (y.reshape(M, K // g, g) * m[:, :, None]).astype(dt).reshape(M, K)
    q = np.clip(np.rint(v), -QMAX, QMAX).astype(np.int8)
    return (q, v) if return_v else q


def pack_int4(q: np.ndarray) -> np.ndarray:
    """Two's-complement nibbles, low nibble = even index along the last axis."""
    q = np.asarray(q)
    if q.shape[-1] % 2:
        raise ValueError("last axis must be even")
    u = (q.astype(np.int16) & 0xF).astype(np.uint8)
    return (u[..., 0::2] | (u[..., 1::2] << 4)).astype(np.uint8)


def unpack_int4(p: np.ndarray) -> np.ndarray:
    """Inverse of pack_int4: bytes -> int8 codes in [-8, 7]."""
    p = np.asarray(p, dtype=np.uint8)
    lo = (p & 0xF).astype(np.int16)
    hi = (p >> 4).astype(np.int16)
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    out = np.empty(p.shape[:-1] + (2 * p.shape[-1],), dtype=np.int8)
    out[..., 0::2] = lo
    out[..., 1::2] = hi
    return out


@dataclass
class ActQuant:
    """Result of rotate + smooth + quantize for one call."""
    y: np.ndarray        # rotated (and reordered) activations, M x K
    c: np.ndarray        # channel maxima, K (in reordered positions)
    s: np.ndarray        # group smoothing scales, G
    r: np.ndarray        # their reciprocals, G
    a: np.ndarray        # token maxima after smoothing, M
    inv: np.ndarray      # 7 / a, M
    alpha: np.ndarray    # per-token scale, M
    q: np.ndarray        # codes, M x K int8
    v: np.ndarray        # pre-rounding values, M x K
    packed: np.ndarray   # M x K/2 uint8


def rotate_smooth_quant(X: np.ndarray, g: int, perm: Optional[np.ndarray] = None,
                        mode: str = "fp32", rotate: bool = True,
                        smooth: bool = True) -> ActQuant:
    """Online half of RRS for one linear layer (Section 3.3 then Section 3.2).

    `rotate=False` gives plain Runtime Smooth (Section 3.1); `smooth=False`
    sets every smoothing scale to 1, i.e. rotation followed by per-token
    quantization only (the QuaRot scheme of Section 2.3). Both are the paper's
    ablation baselines.
    """
    dt = _dt(mode)
    y = fwht(X, mode) if rotate else np.array(X, dtype=dt)
    if perm is not None:
        y = y[:, np.asarray(perm)]
    c = channel_max(y)
    if smooth:
        s, r = group_scales(c, g, mode)
    else:
        s = np.ones(y.shape[1] // g, dtype=dt)
        r = np.ones_like(s)
    a, inv, alpha = token_scales(y, r, g, mode)
    q, v = quantize_codes(y, r, inv, g, mode, return_v=True)
    return ActQuant(y, c, s, r, a, inv, alpha, q, v, pack_int4(q))


# --------------------------------------------------------------------------
# Step 5: offline weight preparation (Section 3.3 last paragraph)
# --------------------------------------------------------------------------

@dataclass
class WeightQuant:
    u: np.ndarray        # rotated (and reordered) weights, K x N
    b: np.ndarray        # per-output-channel maxima, N
    winv: np.ndarray     # 7 / b, N
    beta: np.ndarray     # per-output-channel scale, N
    q: np.ndarray        # codes, K x N int8
    packed: np.ndarray   # N x K/2 uint8 (K contiguous per output channel)


def prepare_weight(W: np.ndarray, perm: Optional[np.ndarray] = None, mode: str = "fp32",
                   rotate: bool = True) -> WeightQuant:
    """u = H_K W (each column rotated), rows reordered by pi, RTN per output channel."""
    dt = _dt(mode)
    u = fwht(W, mode, axis=0) if rotate else np.array(W, dtype=dt)
    if perm is not None:
        u = u[np.asarray(perm), :]
    b = np.abs(u).max(axis=0)
    winv = np.zeros_like(b)
    nz = b != 0
    winv[nz] = dt(QMAX) / b[nz]
    v = (u * winv[None, :]).astype(dt)
    q = np.clip(np.rint(v), -QMAX, QMAX).astype(np.int8)
    beta = b / dt(QMAX)
    return WeightQuant(u, b, winv, beta, q, pack_int4(q.T))


# --------------------------------------------------------------------------
# Step 6: grouped integer GEMM and rescale (Eq. 3, Section 3.2, Fig. 4 (3))
# --------------------------------------------------------------------------

def group_partials(qx: np.ndarray, qw: np.ndarray, g: int) -> np.ndarray:
    """P[b, i, n] = sum_{j in group b} qx[i, j] * qw[j, n], exact (int64).

    The products are taken with a float64 matrix product per group: every
    partial sum is an integer of magnitude <= 49 g < 2^53, so it is exact.
    """
    M, K = qx.shape
    K2, N = qw.shape
    if K != K2 or K % g:
        raise ValueError("shape mismatch")
    G = K // g
    P = np.empty((G, M, N), dtype=np.int64)
    for b in range(G):
        xs = qx[:, b * g:(b + 1) * g].astype(np.float64)
        ws = qw[b * g:(b + 1) * g, :].astype(np.float64)
        P[b] = np.rint(xs @ ws).astype(np.int64)
    return P


def output(P: np.ndarray, s: np.ndarray, alpha: np.ndarray, beta: np.ndarray, norm: int
           ) -> np.ndarray:
    """Y = fl32((alpha_i beta_n / norm) * sum_b s_b P_b[i, n]), in binary64 before the cast.

    norm = K when both operands were rotated (H_K H_K^T = K I undoes the
    unnormalized rotation), 1 when neither was.
    """
    acc = np.tensordot(np.asarray(s, dtype=np.float64), P.astype(np.float64), axes=(0, 0))
    scale = (np.asarray(alpha, np.float64)[:, None]
             * np.asarray(beta, np.float64)[None, :]) / norm
    return (acc * scale).astype(np.float32)


def output_abs_terms(P: np.ndarray, s: np.ndarray, alpha: np.ndarray, beta: np.ndarray,
                     norm: int) -> np.ndarray:
    """T = (|alpha_i| |beta_n| / norm) * sum_b |s_b P_b[i, n]|, the magnitude that
    bounds the rounding error of any order of the binary32 sum over groups."""
    acc = np.tensordot(np.abs(np.asarray(s, np.float64)), np.abs(P).astype(np.float64),
                       axes=(0, 0))
    scale = (np.abs(np.asarray(alpha, np.float64))[:, None]
             * np.abs(np.asarray(beta, np.float64))[None, :]) / norm
    return acc * scale


def linear(X: np.ndarray, W: np.ndarray, g: int, perm: Optional[np.ndarray] = None,
           mode: str = "fp32"):
    """The whole RRS linear layer: returns (Y fp32, ActQuant, WeightQuant, P)."""
    K = X.shape[1]
    act = rotate_smooth_quant(X, g, perm, mode)
    wq = prepare_weight(W, perm, mode)
    P = group_partials(act.q, wq.q, g)
    return output(P, act.s, act.alpha, wq.beta, norm=K), act, wq, P


# --------------------------------------------------------------------------
# Runtime channel reorder (Fig. 4 step (1), Section 3.2)
# --------------------------------------------------------------------------
#
# Fig. 4 step (1) reorders the channels by their channel-wise maxima before
# the grouping, so that channels of similar size share a smoothing scale.
# Taken at run time the order comes from this call's maxima c_j (Eq. 1, over
# the rotated activations of Section 3.3). Readings: channels move in blocks
# of `block` consecutive channels (block = 1 is a sort of single channels);
# a block's key is its largest c_j; keys are sorted largest first and equal
# keys keep increasing block index. The weight rows move with their channels,
# which leaves every product x_j w_j, and so the layer, unchanged up to the
# new grouping.

def runtime_block_order(c: np.ndarray, block: int) -> np.ndarray:
    """Block order of Fig. 4 step (1): position p takes block order[p]."""
    K = c.shape[0]
    if block < 1 or K % block:
        raise ValueError("block must divide K")
    nb = K // block
    key = c.reshape(nb, block).max(axis=1)
    return np.array(sorted(range(nb), key=lambda B: (-key[B], B)), dtype=np.int64)


def block_order_to_perm(order: np.ndarray, block: int) -> np.ndarray:
    """Channel permutation of a block order: position j takes channel perm[j]."""
    order = np.asarray(order, dtype=np.int64)
    return (order[:, None] * block + np.arange(block)[None, :]).reshape(-1)


def rotate_smooth_quant_reorder(X: np.ndarray, g: int, block: int = 32, mode: str = "fp32",
                                rotate: bool = True):
    """Rotate, reorder by this call's channel maxima, smooth and quantize.

    Returns (ActQuant, order, perm); the ActQuant holds the reordered
    activations, as rotate_smooth_quant with that perm.
    """
    dt = _dt(mode)
    y = fwht(X, mode) if rotate else np.array(X, dtype=dt)
    order = runtime_block_order(channel_max(y), block)
    perm = block_order_to_perm(order, block)
    return rotate_smooth_quant(X, g, perm, mode, rotate), order, perm


def linear_reorder(X: np.ndarray, W: np.ndarray, g: int, block: int = 32, mode: str = "fp32",
                   rotate: bool = True):
    """RRS linear layer with the runtime reorder: returns (Y, act, wq, P, order)."""
    K = X.shape[1]
    act, order, perm = rotate_smooth_quant_reorder(X, g, block, mode, rotate)
    wq = prepare_weight(W, perm, mode, rotate)
    P = group_partials(act.q, wq.q, g)
    Y = output(P, act.s, act.alpha, wq.beta, norm=K if rotate else 1)
    return Y, act, wq, P, order


# --------------------------------------------------------------------------
# Baselines of the kernel-efficiency comparison (Section 4.5, Fig. 6)
# --------------------------------------------------------------------------
#
# Per-channel A4W4 (the setting of Section 2.1 and of QuaRot/SpinQuant): one
# scale per token and one per output channel, no smoothing. Its quantizer is
# rotate_smooth_quant(..., smooth=False) with prepare_weight, and its output is
# output(P, ones, alpha, beta, norm): sum_b 1 * P_b is the plain integer dot
# product.
#
# Sub-channel A4W4 (Section 2.1 "sub-channel"): every row is split into groups
# of g channels, each (token, group) and each (output channel, group) has its
# own scale (shapes [M, L] and [N, L], L = K / g, Section 4.5), so the output
# multiplies every group partial by a matrix of scales instead of a scalar.

@dataclass
class SubChannelQuant:
    """Sub-channel quantization of the rows of a matrix (tokens, or weight
    columns seen as rows)."""
    y: np.ndarray        # rotated (or not) values, rows x K
    m: np.ndarray        # per (row, group) maxima, rows x G
    inv: np.ndarray      # fl(7 / m), 0 where m = 0
    scale: np.ndarray    # fl(m / 7), rows x G
    q: np.ndarray        # codes, rows x K int8
    v: np.ndarray        # pre-rounding values, rows x K
    packed: np.ndarray   # rows x K/2 uint8


def _sub_channel_rows(y: np.ndarray, g: int, mode: str) -> SubChannelQuant:
    """Symmetric RTN of every (row, group) block with its own absmax (Section 2.1)."""
    dt = _dt(mode)
    R, K = y.shape
    if K % g:
        raise ValueError("group size must divide K")
    G = K // g
    blocks = y.reshape(R, G, g)
    m = np.abs(blocks).max(axis=2).astype(dt)
    inv = np.zeros_like(m)
    nz = m != 0
    inv[nz] = dt(QMAX) / m[nz]
    v = (blocks * inv[:, :, None]).astype(dt).reshape(R, K)
    q = np.clip(np.rint(v), -QMAX, QMAX).astype(np.int8)
    scale = (m / dt(QMAX)).astype(dt)
    return SubChannelQuant(y, m, inv, scale, q, v, pack_int4(q))


def sub_channel_quant(X: np.ndarray, g: int, mode: str = "fp32",
                      rotate: bool = True) -> SubChannelQuant:
    """Activations: y = x H_K (or x), then one scale per (token, group)."""
    dt = _dt(mode)
    y = fwht(X, mode) if rotate else np.array(X, dtype=dt)
    return _sub_channel_rows(y, g, mode)


def sub_channel_weight(W: np.ndarray, g: int, mode: str = "fp32",
                       rotate: bool = True) -> SubChannelQuant:
    """Weights: u = H_K W (or W); output channel n is row n of u^T, one scale per
    (output channel, group). The packed result is N x K/2 like prepare_weight's."""
    dt = _dt(mode)
    u = fwht(W, mode, axis=0) if rotate else np.array(W, dtype=dt)
    return _sub_channel_rows(np.ascontiguousarray(u.T), g, mode)


def output_sub_channel(P: np.ndarray, a_sub: np.ndarray, b_sub: np.ndarray, norm: int
                       ) -> np.ndarray:
    """Y = fl32((1/norm) * sum_b a_ib b_nb P_b[i, n]), in binary64 before the cast.

    a_sub: M x G token-group scales, b_sub: N x G channel-group scales.
    """
    a = np.asarray(a_sub, np.float64)
    b = np.asarray(b_sub, np.float64)
    acc = np.einsum("ib,nb,bin->in", a, b, P.astype(np.float64))
    return (acc / norm).astype(np.float32)


def output_sub_channel_abs_terms(P: np.ndarray, a_sub: np.ndarray, b_sub: np.ndarray,
                                 norm: int) -> np.ndarray:
    """T = (1/norm) sum_b |a_ib b_nb P_b[i, n]|, the magnitude bounding the
    rounding of any binary32 order of the sub-channel sum."""
    a = np.abs(np.asarray(a_sub, np.float64))
    b = np.abs(np.asarray(b_sub, np.float64))
    return np.einsum("ib,nb,bin->in", a, b, np.abs(P).astype(np.float64)) / norm


# --------------------------------------------------------------------------
# Diagnostics (Section 2.3, Appendix A.1, A.2): smoothness and victim measures
# --------------------------------------------------------------------------

def smoothness_rms(t: np.ndarray) -> np.ndarray:
    """mu = absmax(t) / RMS(t) per token (Section 2.3)."""
    t = np.asarray(t, np.float64)
    return np.abs(t).max(axis=-1) / np.sqrt((t * t).mean(axis=-1))


def smoothness_l2(t: np.ndarray) -> np.ndarray:
    """mu = absmax(t) / ||t||_2 per token (Appendix A.2)."""
    t = np.asarray(t, np.float64)
    return np.abs(t).max(axis=-1) / np.sqrt((t * t).sum(axis=-1))


def victim_measure(scale: np.ndarray) -> float:
    """u = max|x_smooth| / RMS|x_smooth| with x_smooth = 1 / scale (Appendix A.1)."""
    xs = 1.0 / np.asarray(scale, np.float64)
    return float(np.abs(xs).max() / np.sqrt((xs * xs).mean()))


def fp64_reference(X: np.ndarray, W: np.ndarray) -> np.ndarray:
    """The unquantized product X W in binary64 (for quantization-error reports only)."""
    return np.asarray(X, np.float64) @ np.asarray(W, np.float64)
