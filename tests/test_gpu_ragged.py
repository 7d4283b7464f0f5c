"""GPU parity for sequences that are not a multiple of the block: the last
block is partial (it pools over the tokens it holds; its rows past the end are
neither queries nor keys).

Outputs are written into buffers with guard rows behind the sequence, filled
with a sentinel; every test also checks that no kernel wrote past the end.
Bars as for whole blocks (masks outside the 1e-4 cut band, logits 1e-5 relative,
attention 1e-4 fp32 / 2e-2 bf16 max-abs, LSE 1e-3, pooled map 2e-4 relative)."""
import numpy as np
import pytest

import oracle
import workload as W
from helpers import (ATOL_BF16, ATOL_F32, as_f64, check_mask, from_device, gpu_mask_numpy,
                     lists_from_dense, small_inputs, stable_seed, to_device, upload_mask)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")

GUARD = 64
SENTINEL = -12288.0  # exact in bf16 and fp32

CASES = [
    # B, Hq, Hkv, S, D, dtype, Dg
    (1, 2, 1, 1000, 64, "f32", 64),      # 16 tiles, 40 rows in the last
    (2, 4, 2, 650, 128, "bf16", 128),    # 11 tiles, 10 rows in the last
    (1, 7, 1, 2069, 128, "bf16", 128),   # GQA 7:1, 33 tiles, 21 rows in the last
    (1, 2, 2, 4097, 128, "bf16", 64),    # 65 tiles, 1 row in the last
    (1, 3, 1, 63, 64, "bf16", 32),       # one partial tile
    (1, 2, 1, 5, 128, "bf16", 64),       # five tokens
]


def _ceil(a, b):
    return -(-a // b)


def _guarded_out(like, S):
    """A [B, H, S, D] view into a buffer with GUARD sentinel rows per head."""
    B, H, _, D = like.shape
    buf = torch.full((B, H, S + GUARD, D), SENTINEL, dtype=like.dtype, device=like.device)
    return buf, buf[:, :, :S]


def _guards_intact(buf, S):
    return bool((buf[:, :, S:].float() == SENTINEL).all())


def _rows_valid(O_blocks, B, H, S, block, D):
    return O_blocks.reshape(B, H, -1, D)[:, :, :S]


def _inputs(case, tag, spikes=True):
    B, Hq, Hkv, S, D, dt, Dg = case
    return small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed(case, tag), Dg=Dg, spikes=spikes and S >= 3)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("block", [64, 128])
def test_ragged_gate_parity(case, block):
    B, Hq, Hkv, S, D, dt, Dg = case
    w, q, k, v, wq, wk = _inputs(case, ("gate", block))
    nb = _ceil(S, block)
    L, ell = oracle.gate(q, k, wq, wk, block)
    orc = oracle.select(ell, oracle.TOPK_RATIO, rho=0.3)
    orc["L"], orc["ell"] = L, ell
    qd, kd = to_device(q), to_device(k)
    logits = torch.empty((B, Hq, nb, nb), dtype=torch.float32, device="cuda")
    mask = seer.gate(qd, kd, torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda(),
                     mode=seer.TOPK_RATIO, topk_ratio=0.3, block=block, dense_out=True, logits_out=logits)
    torch.cuda.synchronize()
    assert mask.n_blocks == nb
    count, idx, dense = gpu_mask_numpy(mask)
    tri = np.tril(np.ones((nb, nb), bool))
    err = np.abs(logits.cpu().numpy().astype(np.float64) - L)[..., tri].max()
    assert err <= 1e-5 * max(1.0, np.abs(L[..., tri]).max()), err
    check_mask(dense, count, orc, topk=True)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("pattern,causal", [("gate", True), ("random", True), ("vertical", False),
                                            ("empty_rows", True), ("random", False)])
@pytest.mark.parametrize("block", [64, 128])
def test_ragged_bsattn_parity(case, pattern, causal, block):
    B, Hq, Hkv, S, D, dt, Dg = case
    nb = _ceil(S, block)
    w, q, k, v, wq, wk = _inputs(case, ("attn", pattern, causal, block), spikes=False)
    if pattern == "gate":
        _, ell = oracle.gate(q, k, wq, wk, block)
        om = oracle.select(ell, oracle.TOPK_RATIO, rho=0.4)["mask"]
    else:
        om = np.stack([np.stack([W.pattern_mask(pattern, nb, 30 * b + h, 0.4) for h in range(Hq)])
                       for b in range(B)])
        if not causal:
            om = np.maximum(om, np.triu(np.stack([np.stack([W.pattern_mask("random", nb, 7 + h, 0.3).T
                                                            for h in range(Hq)]) for _ in range(B)]), 1))
    count, idx = lists_from_dense(om)
    O_ref, lse_ref = oracle.attn(q, k, v, block=block, mask=om, causal=causal)
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    buf, o = _guarded_out(qd, S)
    lse_buf = torch.full((B * Hq * S + GUARD,), SENTINEL, dtype=torch.float32, device="cuda")
    lse = lse_buf[:B * Hq * S].view(B, Hq, S)
    seer.bsattn(qd, kd, vd, upload_mask(count, idx, block=block), causal=causal, out=o, lse=lse)
    torch.cuda.synchronize()
    assert _guards_intact(buf, S) and bool((lse_buf[B * Hq * S:] == SENTINEL).all())
    O = as_f64(from_device(o.contiguous()))
    ref = _rows_valid(O_ref, B, Hq, S, block, D)
    err = float(np.abs(O - ref).max())
    assert err <= (ATOL_F32 if dt == "f32" else ATOL_BF16), err
    lref = lse_ref.reshape(B, Hq, -1)[:, :, :S]
    lg = lse.cpu().numpy().astype(np.float64)
    fin = np.isfinite(lref)
    np.testing.assert_array_equal(np.isfinite(lg), fin)
    if fin.any():
        assert float(np.abs(lg[fin] - lref[fin]).max()) <= 1e-3
    assert np.all(O[~fin] == 0.0)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("causal", [True, False])
def test_ragged_dense_and_split_parity(case, causal):
    split = {"split": 1, "split_width": 3}
    B, Hq, Hkv, S, D, dt, Dg = case
    w, q, k, v, _, _ = _inputs(case, ("dense", causal))
    O_ref, lse_ref = oracle.attn(q, k, v, causal=causal)
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    n = seer.attn_workspace_bytes(qd, kd, vd, causal=causal, opts=split)
    ws = torch.empty(max(n, 1), dtype=torch.uint8, device="cuda")
    ref = _rows_valid(O_ref, B, Hq, S, 64, D)
    for workspace in (None, ws):
        buf, o = _guarded_out(qd, S)
        _, lse = seer.dense_attn(qd, kd, vd, causal=causal, out=o, want_lse=True, workspace=workspace,
                                 opts=split)
        torch.cuda.synchronize()
        assert _guards_intact(buf, S)
        O = as_f64(from_device(o.contiguous()))
        assert float(np.abs(O - ref).max()) <= (ATOL_F32 if dt == "f32" else ATOL_BF16)
        lref = lse_ref.reshape(B, Hq, -1)[:, :, :S]
        assert float(np.abs(lse.cpu().numpy() - lref).max()) <= 1e-3


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("causal", [True, False])
def test_ragged_ground_truth_parity(case, causal):
    B, Hq, Hkv, S, D, dt, Dg = case
    w, q, k, v, _, _ = _inputs(case, ("gt", causal))
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    buf, o = _guarded_out(qd, S)
    _, _, gt = seer.attn_gt(qd, kd, vd, causal=causal, out=o)
    torch.cuda.synchronize()
    assert _guards_intact(buf, S)
    ref = oracle.maxpool_gt(q, k, causal=causal)
    g = gt.cpu().numpy().astype(np.float64)
    bad = np.abs(g - ref) > 2e-4 * ref + 1e-6
    assert not bad.any(), float(np.abs(g - ref).max())


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_ragged_distill_parity(case):
    B, Hq, Hkv, S, D, dt, Dg = case
    w, q, k, v, _, _ = _inputs(case, "distill")
    rng = np.random.default_rng(stable_seed(case, "dw"))
    wq = (rng.standard_normal((Hq, D, Dg)) / np.sqrt(D)).astype(np.float32)
    wk = (rng.standard_normal((Hkv, 3 * D, Dg)) / np.sqrt(3 * D)).astype(np.float32)
    nb = _ceil(S, 64)
    gt = np.tril(np.exp(-2.0 * np.abs(rng.standard_normal((B, Hq, nb, nb))))).astype(np.float32)
    loss, dwq, dwk = seer.gate_distill(to_device(q), to_device(k), torch.from_numpy(wq).cuda(),
                                       torch.from_numpy(wk).cuda(), torch.from_numpy(gt).cuda())
    torch.cuda.synchronize()
    l_ref, dwq_ref, dwk_ref = oracle.distill(q, k, wq, wk, gt)
    assert abs(float(loss.item()) - l_ref) <= 1e-4 * abs(l_ref) + 1e-9
    for got, ref in ((dwq, dwq_ref), (dwk, dwk_ref)):
        err = float(np.abs(got.cpu().numpy().astype(np.float64) - ref).max())
        assert err <= 2e-4 * float(np.abs(ref).max()) + 1e-12, err
