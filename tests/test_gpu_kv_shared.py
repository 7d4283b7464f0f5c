"""GPU parity for the shared-mask variant: one block mask per KV group (not the
paper's per-head gate).  The gate scores block j of query-block row i by the
mean over the group's query heads of their gate probabilities and selects on
that score; attention applies row (b, g, i) to every query head of group g and
loads each K/V tile once for several of them (up to 4 heads per workgroup).

Bars as for per-head masks: masks outside the 1e-4 cut band of the oracle's
group log-score (TopK rows keep exactly the oracle's count), attention 1e-4
(fp32) / 2e-2 (bf16) max-abs against the fp64 oracle run on the group mask
repeated for each query head.  Attention on a shared mask must also equal,
bit for bit, the per-head kernel run on that repeated mask."""
import os

import numpy as np
import pytest

import oracle
import workload as W
from helpers import (ATOL_BF16, ATOL_F32, as_f64, check_mask, from_device, gather_rows,
                     gpu_mask_numpy, sample_rows, small_inputs, stable_seed, to_device, upload_mask)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")

CASES = [
    # B, Hq, Hkv, S, D, dtype, Dg
    (1, 8, 2, 1024, 128, "bf16", 128),   # GQA 4:1 (4 heads per workgroup)
    (2, 4, 2, 640, 128, "bf16", 128),    # GQA 2:1 (2 heads per workgroup)
    (1, 7, 1, 1280, 128, "bf16", 128),   # GQA 7:1 (one head per workgroup)
    (1, 8, 1, 4160, 64, "bf16", 64),     # GQA 8:1, D 64, nb = 65
    (1, 4, 1, 1000, 64, "bf16", 32),     # partial last block
    (1, 4, 2, 576, 128, "f32", 128),     # fp32 kernel
    (1, 4, 4, 448, 128, "bf16", 64),     # GQA 1:1: shared = per head
]


def _tol(dtype):
    return ATOL_F32 if dtype == "f32" else ATOL_BF16


def _nb(S):
    return -(-S // 64)


def _group_select(q, k, wq, wk, Hkv, mode, rho=0.0, kfix=0, thresholds=None, keep_first=1, keep_diag=1):
    _, ell = oracle.gate(q, k, wq, wk, 64, True)
    ellg = oracle.group_logscore(ell, Hkv)
    sel = oracle.select(ellg, mode, rho=rho, k=kfix, thresholds=thresholds,
                        keep_first=keep_first, keep_diag=keep_diag)
    sel["ell"] = ellg
    return sel


def _upload_kv(count, idx):
    m = upload_mask(count, idx)
    m.kv_shared = True
    return m


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("sel", ["ratio", "fixed", "thr", "thr_kv", "noforce"])
def test_kv_gate_mask_parity(case, sel):
    B, Hq, Hkv, S, D, dt, Dg = case
    print(f"[kv gate] {case} {sel}", flush=True)
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed("kv", case, sel), Dg=Dg,
                                      spikes=True)
    qd, kd = to_device(q), to_device(k)
    wqd, wkd = torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda()
    kw = dict(keep_first=1, keep_diag=1)
    if sel == "ratio":
        mode, args, gargs = oracle.TOPK_RATIO, dict(rho=0.3), dict(mode=seer.TOPK_RATIO, topk_ratio=0.3)
    elif sel == "fixed":
        mode, args, gargs = oracle.TOPK_FIXED, dict(kfix=3), dict(mode=seer.TOPK_FIXED, topk_k=3)
    elif sel == "thr":
        mode, args = oracle.THRESHOLD, dict(thresholds=np.float32(0.02))
        gargs = dict(mode=seer.THRESHOLD, threshold=0.02)
    elif sel == "thr_kv":  # one threshold per KV group
        thr = np.linspace(0.005, 0.1, Hkv).astype(np.float32)
        mode, args = oracle.THRESHOLD, dict(thresholds=thr)
        gargs = dict(mode=seer.THRESHOLD, head_thresholds=torch.from_numpy(thr).cuda())
    else:
        mode, args, gargs = oracle.TOPK_RATIO, dict(rho=0.25), dict(mode=seer.TOPK_RATIO, topk_ratio=0.25)
        kw = dict(keep_first=0, keep_diag=0)
    orc = _group_select(q, k, wq, wk, Hkv, mode, **args, **kw)
    mask = seer.gate(qd, kd, wqd, wkd, **gargs, **kw, kv_shared=True, dense_out=True)
    torch.cuda.synchronize()
    assert tuple(mask.count.shape) == (B, Hkv, _nb(S))
    count, idx, dense = gpu_mask_numpy(mask)
    np.testing.assert_array_equal(dense, mask.dense.cpu().numpy())
    check_mask(dense, count, orc, topk=mode != oracle.THRESHOLD)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("cap", [4, 2, 1])
def test_kv_attention_parity(case, cap):
    """Attention on the oracle's group mask, with at most `cap` query heads per
    workgroup, against the oracle on the mask repeated per head."""
    B, Hq, Hkv, S, D, dt, Dg = case
    G = Hq // Hkv
    print(f"[kv attn] {case} cap {cap}", flush=True)
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed("kva", case), Dg=Dg)
    orc = _group_select(q, k, wq, wk, Hkv, oracle.TOPK_RATIO, rho=0.35)
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    o, lse = seer.bsattn(qd, kd, vd, _upload_kv(orc["count"], orc["idx"]), want_lse=True,
                         opts={"heads_per_wg": cap})
    torch.cuda.synchronize()
    per_head = np.repeat(orc["mask"], G, axis=1)
    O_ref, lse_ref = oracle.attn(q, k, v, mask=per_head)
    nb = _nb(S)
    og = as_f64(from_device(o)).reshape(B, Hq, nb, 64, D) if S % 64 == 0 else None
    if og is None:  # partial last block: compare the rows that exist
        ref = O_ref.reshape(B, Hq, nb * 64, D)[:, :, :S]
        err = float(np.abs(as_f64(from_device(o)) - ref).max())
        lerr = float(np.abs(lse.cpu().numpy() - lse_ref.reshape(B, Hq, nb * 64)[:, :, :S]).max())
    else:
        err = float(np.abs(og - O_ref.reshape(B, Hq, nb, 64, D)).max())
        lerr = float(np.abs(lse.cpu().numpy().reshape(B, Hq, nb, 64) - lse_ref.reshape(B, Hq, nb, 64)).max())
    assert err <= _tol(dt), err
    assert lerr <= 1e-3, lerr


@pytest.mark.parametrize("case", [c for c in CASES if c[5] == "bf16"], ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("pattern", ["gate", "random", "empty_rows"])
def test_kv_attention_equals_per_head_kernel(case, pattern):
    """The shared-row workgroup computes, per head, exactly what the per-head
    kernel computes on the repeated mask (same tiles, same order)."""
    B, Hq, Hkv, S, D, dt, Dg = case
    G = Hq // Hkv
    nb = _nb(S)
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed("kvb", case, pattern), Dg=Dg)
    if pattern == "gate":
        om = _group_select(q, k, wq, wk, Hkv, oracle.TOPK_RATIO, rho=0.3)["mask"]
    else:
        kind = "random" if pattern == "random" else "empty_rows"
        om = np.stack([np.stack([W.pattern_mask(kind, nb, 100 * b + g, 0.3) for g in range(Hkv)])
                       for b in range(B)])
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    dev_om = torch.from_numpy(om).cuda()
    kv_mask = seer.mask_from_dense(dev_om, kv_shared=True)
    ph_mask = seer.mask_from_dense(torch.from_numpy(np.repeat(om, G, axis=1)).cuda(), heads_kv=Hkv)
    o1, l1 = seer.bsattn(qd, kd, vd, kv_mask, want_lse=True)
    o2, l2 = seer.bsattn(qd, kd, vd, ph_mask, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1, l2)


def test_kv_full_size_llama_128k():
    """Headline shape (32 query / 8 KV heads, D 128, 131072 tokens) with a shared
    TopK-0.1 mask: masks against the oracle in full, attention on sampled rows."""
    w = W.WORKLOADS["llama_s128k"]
    print("[kv 128k] generating inputs", flush=True)
    q, k, v = (W.make_tensor(w, t) for t in "qkv")
    wq, wk = W.make_weights(w)
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    mask = seer.gate(qd, kd, torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda(), mode=seer.TOPK_RATIO,
                     topk_ratio=w.topk_ratio, kv_shared=True)
    o, _ = seer.bsattn(qd, kd, vd, mask)
    torch.cuda.synchronize()
    count, idx, dense = gpu_mask_numpy(mask)
    print("[kv 128k] device path done", flush=True)
    orc = _group_select(q, k, wq, wk, w.heads_kv, oracle.TOPK_RATIO, rho=w.topk_ratio)
    stats = check_mask(dense, count, orc, topk=True)
    print(f"[kv 128k] masks {stats}", flush=True)
    G = w.heads_q // w.heads_kv
    rows = sample_rows(w.batch, w.heads_q, w.n_blocks, 48, seed=7)
    same = np.array([(dense[b, h // G, i] == orc["mask"][b, h // G, i]).all() for b, h, i in rows])
    rows = rows[same]
    assert len(rows) >= 40
    O_ref, _ = oracle.attn(q, k, v, mask=np.repeat(orc["mask"], G, axis=1), rows=rows)
    err = float(np.abs(as_f64(gather_rows(from_device(o), rows)) - O_ref).max())
    print(f"[kv 128k] attention max-abs {err:.3e} over {len(rows)} rows", flush=True)
    assert err <= ATOL_BF16
