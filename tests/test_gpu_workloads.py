"""GPU parity at the full sizes of the five workloads, in the launch
configuration bench.py times (whole tensors, one gate call, one attention call
with the key-range split workspace wherever the shape splits).

Masks are compared in full against the oracle's fp64 gate (mismatches allowed
only within 1e-4 of the selection cut in log-score, TopK rows exactly k).
Attention is compared on a seeded, row-stratified sample of query-block rows
that the oracle computes one by one: the block-sparse kernel on the oracle's
own mask (uploaded), the end-to-end path (device gate -> device attention) on
sampled rows whose device mask equals the oracle's, and, at 128k tokens, the
dense kernel."""
import numpy as np
import pytest

import oracle
import workload as W
from helpers import (ATOL_BF16, ATOL_F32, as_f64, check_mask, from_device, gather_rows,
                     gpu_mask_numpy, sample_rows, to_device, upload_mask)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")

ROWS = 256  # sampled query-block rows per workload (row-stratified)


def _gate_kwargs(w):
    kw = dict(keep_first=w.keep_first, keep_diag=w.keep_diag)
    if w.select == W.SEL_THRESHOLD:
        thr = W.load_thresholds(w)
        if thr.size == 1:
            kw.update(mode=seer.THRESHOLD, threshold=float(thr[0]))
        else:
            kw.update(mode=seer.THRESHOLD, head_thresholds=torch.from_numpy(thr).cuda())
        return kw, dict(mode=oracle.THRESHOLD, thresholds=thr)
    if w.select == W.SEL_TOPK_RATIO:
        kw.update(mode=seer.TOPK_RATIO, topk_ratio=w.topk_ratio)
        return kw, dict(mode=oracle.TOPK_RATIO, rho=w.topk_ratio)
    kw.update(mode=seer.TOPK_FIXED, topk_k=w.topk_k)
    return kw, dict(mode=oracle.TOPK_FIXED, k=w.topk_k)


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_workload_full_size(name):
    w = W.WORKLOADS[name]
    print(f"[workload] {name}: generating inputs", flush=True)
    q, k, v = (W.make_tensor(w, t) for t in "qkv")
    wq, wk = W.make_weights(w)
    gkw, okw = _gate_kwargs(w)

    # device path, exactly as bench.py runs it (with the key-range split workspace)
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    nws = seer.attn_workspace_bytes(qd, kd, vd)
    aws = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda") if nws else None
    print(f"[workload] {name}: split workspace {nws} bytes", flush=True)
    mask = seer.gate(qd, kd, torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda(), **gkw)
    o_e2e, _ = seer.bsattn(qd, kd, vd, mask, workspace=aws)
    torch.cuda.synchronize()
    count, idx, dense = gpu_mask_numpy(mask)
    o_e2e = from_device(o_e2e)
    print(f"[workload] {name}: device path done", flush=True)

    # oracle gate in full
    _, ell = oracle.gate(q, k, wq, wk)
    sel = oracle.select(ell, okw["mode"], rho=okw.get("rho", 0.0), k=okw.get("k", 0),
                        thresholds=okw.get("thresholds"), keep_first=w.keep_first,
                        keep_diag=w.keep_diag)
    sel["ell"] = ell
    stats = check_mask(dense, count, sel, topk=w.select != W.SEL_THRESHOLD)
    del ell
    print(f"[workload] {name}: masks {stats}", flush=True)

    nb = w.n_blocks
    rows = sample_rows(w.batch, w.heads_q, nb, ROWS, seed=nb)
    tol = ATOL_F32 if w.dtype == "f32" else ATOL_BF16

    # block-sparse kernel on the oracle's mask
    o_sp, lse = seer.bsattn(qd, kd, vd, upload_mask(sel["count"], sel["idx"]), want_lse=True, workspace=aws)
    torch.cuda.synchronize()
    O_ref, lse_ref = oracle.attn(q, k, v, mask=sel["mask"], rows=rows)
    err = float(np.abs(as_f64(gather_rows(from_device(o_sp), rows)) - O_ref).max())
    lse_g = np.stack([lse.cpu().numpy()[b, h, i * 64:(i + 1) * 64] for b, h, i in rows])
    lse_err = float(np.abs(lse_g - lse_ref).max())
    print(f"[workload] {name}: sparse attention max-abs {err:.3e}, lse {lse_err:.3e}", flush=True)
    assert err <= tol
    assert lse_err <= 1e-3

    # end to end on rows whose device mask equals the oracle's
    same = np.array([(dense[b, h, i] == sel["mask"][b, h, i]).all() for b, h, i in rows])
    e2e_rows = rows[same]
    assert same.mean() >= 0.9, f"only {same.mean():.2f} of sampled rows have identical masks"
    if len(e2e_rows):
        O_ref2, _ = oracle.attn(q, k, v, mask=sel["mask"], rows=e2e_rows)
        err2 = float(np.abs(as_f64(gather_rows(o_e2e, e2e_rows)) - O_ref2).max())
        print(f"[workload] {name}: end-to-end max-abs {err2:.3e} over {len(e2e_rows)} rows", flush=True)
        assert err2 <= tol

    # the dense comparison kernel at the headline size
    if name == W.HEADLINE:
        od, _ = seer.dense_attn(qd, kd, vd, workspace=aws)
        torch.cuda.synchronize()
        drows = rows[:: max(1, len(rows) // 12)]
        O_ref3, _ = oracle.attn(q, k, v, rows=drows)
        err3 = float(np.abs(as_f64(gather_rows(from_device(od), drows)) - O_ref3).max())
        print(f"[workload] {name}: dense max-abs {err3:.3e} over {len(drows)} rows", flush=True)
        assert err3 <= tol
