"""Writes workload/thresholds.json: the fp32 gate thresholds of the threshold-mode
workloads, chosen from the oracle's fp64 gate probabilities so that the
causal-block sparsity hits each workload's target.

Calls only the oracle (and the seeded input generators).  Run from the repo
root:  python -m workload.make_thresholds

Recipe, per workload (global threshold) or per head (per-head targets): with
F the forced blocks (first and diagonal) and C the other causal blocks, the
number of blocks to keep is round((1 - s) * causal); the threshold is the
geometric mean of the n-th and (n+1)-th largest probability in C, with
n = keep - |F|, so that Eq. 4's strict comparison keeps exactly n of C.
"""
from __future__ import annotations

import json
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workload as W  # noqa: E402


def _threshold_for(ell_heads: np.ndarray, target: float) -> float:
    """ell_heads [H, nb, nb] log-scores sharing one threshold."""
    H, nb, _ = ell_heads.shape
    tri = np.tril(np.ones((nb, nb), bool))
    forced = np.zeros((nb, nb), bool)
    forced[:, 0] = True
    forced[np.arange(nb), np.arange(nb)] = True
    cand = tri & ~forced
    causal = H * int(tri.sum())
    n_forced = H * int(forced.sum())
    keep = int(round((1.0 - target) * causal))
    n = max(0, min(keep - n_forced, H * int(cand.sum())))
    vals = np.sort(ell_heads[:, cand].reshape(-1))[::-1]
    if n == 0:
        return 1.0
    if n >= vals.size:
        return 0.0
    return float(math.exp(0.5 * (vals[n - 1] + vals[n])))


def thresholds_for(w: W.Workload) -> dict:
    q = W.make_tensor(w, "q")
    k = W.make_tensor(w, "k")
    wq, wk = W.make_weights(w)
    _, ell = oracle.gate(q, k, wq, wk)
    ell = ell[0] if w.batch == 1 else ell.reshape(-1, *ell.shape[-2:])
    if w.per_head_sparsity is not None:
        thr = [_threshold_for(ell[h:h + 1], s) for h, s in enumerate(w.per_head_sparsity)]
    else:
        thr = [_threshold_for(ell, w.target_sparsity)]
    thr32 = np.asarray(thr, np.float32)
    sel = oracle.select(ell[None] if w.batch == 1 else ell, oracle.THRESHOLD, thresholds=thr32)
    nb = w.n_blocks
    causal = nb * (nb + 1) // 2
    per_head = 1.0 - sel["count"].reshape(-1, nb).sum(-1) / causal
    return dict(thresholds=[float(t) for t in thr32],
                achieved_sparsity=float(1.0 - sel["count"].sum() / (causal * w.heads_q * w.batch)),
                achieved_per_head=[round(float(x), 6) for x in per_head],
                target=w.per_head_sparsity if w.per_head_sparsity is not None else w.target_sparsity)


def main() -> None:
    out = {}
    for name, w in W.WORKLOADS.items():
        if w.select != W.SEL_THRESHOLD:
            continue
        out[name] = thresholds_for(w)
        print(name, "sparsity", round(out[name]["achieved_sparsity"], 4), flush=True)
    with open(W.THRESHOLDS_FILE, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")


if __name__ == "__main__":
    main()
