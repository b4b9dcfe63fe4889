"""Seeded synthetic inputs for the RRS linear layer.

This module only draws random numbers. It holds none of the method's
arithmetic (no rotation, scale, quantization or product), so both the CPU
oracle and the HIP path can be fed from it without sharing code.

The paper's workloads are LLaMA/Qwen/Mistral linear-layer activations on
WikiText-2 (Section 4.1). Neither the models nor the dataset are available, so
these generators stand in for them: token activations are standard normal with
two kinds of outliers laid on top, the channel-wise outliers (whole columns
scaled up) and the spike outliers (isolated large entries) that Section 2.2 and
Appendix A.1 describe. Weights are N(0, 0.02^2), the scale of a randomly
initialised LLaMA-7B linear layer.

Recipe, per workload and seed:
  * streams = default_rng(SeedSequence(seed).spawn(2)): one for X, one for W;
  * X0 = standard normal, M x K, float32;
  * n_chan = round(chan_frac * K) outlier channels chosen without replacement;
    each whole column is multiplied by its factor (a fixed factor, or one drawn
    log-uniformly from [lo, hi]);
  * n_spike spike positions chosen uniformly without replacement over the M*K
    entries are overwritten with sign * magnitude (a fixed magnitude, or one
    drawn uniformly from [lo, hi]; signs uniform);
  * X = float16(X0);
  * W = float16(0.02 * standard normal), K x N, drawn row-block by row-block
    (the stream is consumed in row-major order, so the result does not depend
    on the block size).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    M: int            # tokens
    K: int            # input channels (power of two)
    N: int            # output channels
    g: int            # smoothing group size
    seed: int
    n_chan: int       # number of channel-wise outlier columns
    chan_factor: Tuple[float, float]   # (lo, hi); lo == hi means a fixed factor
    n_spike: int      # number of spike entries
    spike_mag: Tuple[float, float]     # (lo, hi); lo == hi means a fixed magnitude
    extra_seeds: Tuple[int, ...] = field(default_factory=tuple)

    @property
    def G(self) -> int:
        return self.K // self.g


def _round_half_up(x: float) -> int:
    return int(np.floor(x + 0.5))


# The five workloads: a tiny case, the LLaMA-7B fused QKV and gate/up
# projections, a decode-shaped memory-bound case and a large prefill case.
WORKLOADS = {
    "tiny": Workload("tiny", 16, 512, 512, 128, 1, 4, (50.0, 50.0), 3, (200.0, 200.0),
                     extra_seeds=(2, 3, 4)),
    "qkv": Workload("qkv", 2048, 4096, 12288, 128, 2,
                    _round_half_up(0.01 * 4096), (20.0, 100.0),
                    _round_half_up(1e-4 * 2048 * 4096), (100.0, 500.0)),
    "gateup": Workload("gateup", 4096, 4096, 22016, 128, 3,
                       _round_half_up(0.01 * 4096), (20.0, 100.0),
                       _round_half_up(1e-4 * 4096 * 4096), (100.0, 500.0)),
    "decode": Workload("decode", 8, 8192, 28672, 128, 4,
                       _round_half_up(0.01 * 8192), (50.0, 50.0), 2, (100.0, 500.0)),
    "large": Workload("large", 8192, 8192, 28672, 64, 5,
                      _round_half_up(0.02 * 8192), (20.0, 100.0),
                      _round_half_up(5e-4 * 8192 * 8192), (100.0, 500.0)),
}


def custom(name: str, M: int, K: int, N: int, g: int, seed: int, *, n_chan: int = 0,
           chan_factor=(50.0, 50.0), n_spike: int = 0, spike_mag=(200.0, 200.0)) -> Workload:
    """A workload of any shape with the same recipe (used for ragged test cases)."""
    return Workload(name, M, K, N, g, seed, n_chan, tuple(chan_factor), n_spike,
                    tuple(spike_mag))


def _streams(seed: int):
    ss = np.random.SeedSequence(seed).spawn(2)
    return np.random.default_rng(ss[0]), np.random.default_rng(ss[1])


def _draw(rng, lohi, size):
    lo, hi = lohi
    if lo == hi:
        return np.full(size, lo, dtype=np.float64)
    return rng.uniform(lo, hi, size)


def _draw_log(rng, lohi, size):
    lo, hi = lohi
    if lo == hi:
        return np.full(size, lo, dtype=np.float64)
    return np.exp(rng.uniform(np.log(lo), np.log(hi), size))


def activations(w: Workload, seed: Optional[int] = None) -> np.ndarray:
    """X: M x K float16, standard normal with channel and spike outliers."""
    rx, _ = _streams(w.seed if seed is None else seed)
    M, K = w.M, w.K
    x = rx.standard_normal((M, K), dtype=np.float32)
    if w.n_chan:
        cols = rx.choice(K, size=w.n_chan, replace=False)
        fac = _draw_log(rx, w.chan_factor, w.n_chan).astype(np.float32)
        x[:, cols] *= fac[None, :]
    if w.n_spike:
        pos = rx.choice(M * K, size=w.n_spike, replace=False)
        mag = _draw(rx, w.spike_mag, w.n_spike)
        sgn = rx.choice(np.array([-1.0, 1.0]), size=w.n_spike)
        x.reshape(-1)[pos] = (sgn * mag).astype(np.float32)
    return x.astype(np.float16)


_W_BLOCK_ROWS = 256


def weights(w: Workload, seed: Optional[int] = None, cols: Optional[np.ndarray] = None
            ) -> np.ndarray:
    """W: K x N float16 ~ N(0, 0.02^2), or only the columns `cols` of it."""
    _, rw = _streams(w.seed if seed is None else seed)
    K, N = w.K, w.N
    ncols = N if cols is None else len(cols)
    out = np.empty((K, ncols), dtype=np.float16)
    for r0 in range(0, K, _W_BLOCK_ROWS):
        r1 = min(K, r0 + _W_BLOCK_ROWS)
        blk = rw.standard_normal((r1 - r0, N), dtype=np.float32)
        if cols is not None:
            blk = blk[:, cols]
        out[r0:r1] = (np.float32(0.02) * blk).astype(np.float16)
    return out


def permutation(K: int, seed: int) -> np.ndarray:
    """A seeded channel permutation (int32), for the optional static reorder."""
    rng = np.random.default_rng(np.random.SeedSequence(seed).spawn(3)[2])
    return rng.permutation(K).astype(np.int32)
