"""Quantization error of the runtime channel reorder (Fig. 4 step (1)) by block
size, on the synthetic stand-ins of the five workloads: TEST INFRASTRUCTURE
(an oracle-only report; it calls nothing but oracle/ and the seeded input
generators).

For each workload the layer is computed by the oracle three ways: RRS without
a reorder, RRS with the runtime reorder moving blocks of 32 channels (what the
GPU path does), and RRS with the literal per-channel reorder (block = 1). Each
is compared with the unquantized product X W in binary64 on a sample of output
columns (all tokens). Printed per workload: the relative Frobenius error
||Y - XW|| / ||XW|| and the mean over tokens of the per-token relative error.

    python -m oracle.reorder_report [--cols 256]
"""
from __future__ import annotations

import argparse
import sys
import os

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import synth  # noqa: E402
from oracle import rrs_oracle as O  # noqa: E402


def errors(Y: np.ndarray, ref: np.ndarray):
    d = np.asarray(Y, np.float64) - ref
    fro = np.linalg.norm(d) / np.linalg.norm(ref)
    per_tok = np.linalg.norm(d, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-300)
    return fro, float(per_tok.mean())


def report(name: str, ncols: int, seed: int = 17):
    w = synth.WORKLOADS[name]
    rng = np.random.default_rng(seed)
    cols = np.sort(rng.choice(w.N, min(ncols, w.N), replace=False))
    X = synth.activations(w)
    W = synth.weights(w, cols=cols)
    ref = O.fp64_reference(X, W)
    out = {}
    act = O.rotate_smooth_quant(X, w.g)
    wq = O.prepare_weight(W)
    P = O.group_partials(act.q, wq.q, w.g)
    out["none"] = errors(O.output(P, act.s, act.alpha, wq.beta, norm=w.K), ref)
    for block in (32, 1):
        Y, *_ = O.linear_reorder(X, W, w.g, block=block)
        out[f"block {block}"] = errors(Y, ref)
    return w, len(cols), out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--cols", type=int, default=256)
    ap.add_argument("--workloads", default="tiny,qkv,gateup,decode,large")
    args = ap.parse_args()
    print("| workload | M x K x N (cols sampled), g | reorder | rel. Frobenius error | "
          "mean per-token rel. error |")
    print("|---|---|---|---|---|")
    for name in args.workloads.split(","):
        w, nc, out = report(name, args.cols)
        for k, (fro, tok) in out.items():
            print(f"| {name} | {w.M} x {w.K} x {w.N} ({nc}), {w.g} | {k} | {fro:.5f} | {tok:.5f} |",
                  flush=True)


if __name__ == "__main__":
    main()
