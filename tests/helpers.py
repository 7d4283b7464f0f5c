"""Shared helpers for the parity tests: seeded inputs, oracle runs, comparisons.

Inputs flow one way: numpy (seeded) -> oracle and -> GPU.  Nothing computed by
the HIP path is ever fed to the oracle or used as an expected value.
"""
from __future__ import annotations

import math
import zlib

import numpy as np

import oracle
import workload as W

MASK_BAND = 1e-4      # log-score distance to the selection cut within which masks may differ
ATOL_F32 = 1e-4       # attention max-abs tolerance, fp32 path
ATOL_BF16 = 2e-2      # attention max-abs tolerance, bf16 path


def to_device(x: np.ndarray, device="cuda"):
    """Stored elements (fp32 or uint16 bf16 bits) -> torch tensor of the same bytes."""
    import torch
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(x).to(device)


def from_device(t) -> np.ndarray:
    import torch
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def as_f64(x: np.ndarray) -> np.ndarray:
    return W.bf16_bits_to_f32(x).astype(np.float64) if x.dtype == np.uint16 else x.astype(np.float64)


def stable_seed(*parts) -> int:
    """Process-independent seed from any printable parts."""
    return zlib.crc32(repr(parts).encode()) % 100000


def lists_from_dense(m: np.ndarray):
    """count [.., nb] and ascending idx [.., nb, nb] (uint16) of a 0/1 mask."""
    nb = m.shape[-1]
    count = (m != 0).sum(-1).astype(np.int32)
    idx = np.zeros(m.shape, np.uint16)
    flat_m = m.reshape(-1, nb)
    flat_i = idx.reshape(-1, nb)
    for r in range(flat_m.shape[0]):
        js = np.nonzero(flat_m[r])[0]
        flat_i[r, :js.size] = js
    return count, idx


def small_inputs(B, Hq, Hkv, S, D, dtype, seed, Dg=None, spikes=False, w_sigma2=None):
    """Seeded Q, K, V, Wq, Wk of a small case (stored as the GPU receives them)."""
    Dg = Dg or D
    w = W.Workload(f"case{seed}", seed, B, Hq, Hkv, D, S, dtype, Dg,
                   w_sigma2 if w_sigma2 is not None else 1.0 / Dg,
                   "spikes" if spikes else "plain", W.SEL_TOPK_RATIO, topk_ratio=0.5)
    q = W.make_tensor(w, "q")
    k = W.make_tensor(w, "k")
    v = W.make_tensor(w, "v")
    wq, wk = W.make_weights(w)
    return w, q, k, v, wq, wk


def oracle_gate(q, k, wq, wk, mode, rho=0.0, kfix=0, thresholds=None, keep_first=1, keep_diag=1,
                w_per_head=True, rope_theta=0.0):
    L, ell = oracle.gate(q, k, wq, wk, 64, w_per_head, rope_theta=rope_theta)
    sel = oracle.select(ell, mode, rho=rho, k=kfix, thresholds=thresholds,
                        keep_first=keep_first, keep_diag=keep_diag)
    sel["L"] = L
    sel["ell"] = ell
    return sel


def dense_from_lists(count: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """0/1 [.., nb, nb] mask from count [.., nb] and ascending idx [.., nb, nb]."""
    nb = count.shape[-1]
    out = np.zeros(count.shape + (nb,), np.uint8)
    flat_c = count.reshape(-1)
    flat_i = idx.reshape(-1, nb)
    flat_o = out.reshape(-1, nb)
    for r in range(flat_c.size):
        c = int(flat_c[r])
        assert 0 <= c <= nb
        js = flat_i[r, :c].astype(np.int64)
        assert np.all(np.diff(js) > 0), "index list must be strictly ascending"
        flat_o[r, js] = 1
    return out


def gpu_mask_numpy(mask):
    count = mask.count.cpu().numpy()
    idx = mask.idx.cpu().numpy().view(np.uint16)
    return count, idx, dense_from_lists(count, idx)


def check_mask(gpu_dense: np.ndarray, gpu_count: np.ndarray, orc: dict, topk: bool,
               band: float = MASK_BAND):
    """Mask rule: entries may differ only where the oracle log-score lies within
    `band` of the row's selection cut; TopK rows hold exactly the oracle's count.
    Returns a dict of statistics; raises AssertionError on a violation."""
    om = orc["mask"]
    diff = gpu_dense != om
    n_diff = int(diff.sum())
    stats = dict(entries=int(om.size), active=int(om.sum()), differ=n_diff, outside_band=0)
    if n_diff:
        ell = orc["ell"]
        cut = orc["cut"][..., None]
        dist = np.abs(ell - cut)
        bad = diff & ~(dist <= band)
        stats["outside_band"] = int(bad.sum())
        if bad.any():
            loc = np.argwhere(bad)[:5]
            raise AssertionError(f"mask mismatch outside the cut band at {loc.tolist()} "
                                 f"(ell={ell[tuple(loc[0])]}, cut={orc['cut'][tuple(loc[0][:-1])]})")
        # literal reading of the rule: |P - cut probability| <= band
        pc = np.exp(np.clip(cut, -700, 0))
        stats["outside_literal"] = int((diff & ~(np.abs(np.exp(ell) - pc) <= band)).sum())
    if topk:
        np.testing.assert_array_equal(gpu_count, orc["count"])
    return stats


def upload_mask(count: np.ndarray, idx: np.ndarray, device="cuda", block: int = 64):
    import torch
    import paper_2410_13276_amd as seer
    return seer.BlockMask(count=torch.from_numpy(np.ascontiguousarray(count, np.int32)).to(device),
                          idx=torch.from_numpy(np.ascontiguousarray(idx).view(np.int16)).to(device),
                          block=block)


def sample_rows(B, Hq, nb, n, seed):
    """Seeded, row-stratified sample of (b, h, i) q-block rows, always including
    the first and last rows."""
    rng = np.random.default_rng(seed)
    rows = {(0, 0, 0), (B - 1, Hq - 1, nb - 1)}
    strata = np.linspace(0, nb, num=min(n, nb) + 1).astype(int)
    for s in range(len(strata) - 1):
        i = int(rng.integers(strata[s], max(strata[s] + 1, strata[s + 1])))
        rows.add((int(rng.integers(B)), int(rng.integers(Hq)), min(i, nb - 1)))
    return np.array(sorted(rows), dtype=np.int32)


def gather_rows(o: np.ndarray, rows: np.ndarray, block: int = 64) -> np.ndarray:
    """[n, block, D] slices of a [B, H, S, D] array at q-block rows."""
    return np.stack([o[b, h, i * block:(i + 1) * block] for b, h, i in rows])


def attn_flops(count_total: int, D: int) -> float:
    return 4.0 * 64 * 64 * D * count_total


def causal_blocks(nb: int) -> int:
    return nb * (nb + 1) // 2


def sparsity(count: np.ndarray) -> float:
    nb = count.shape[-1]
    return 1.0 - float(count.sum()) / (causal_blocks(nb) * (count.size // nb))


def log_cut(thr: float) -> float:
    return math.log(thr)
