"""GPU parity with 128-token gate blocks and masks (the paper's sparse kernel
takes blocks of 64 or 128 tokens, section 3.3): the gate pools, scores and
selects 128-token blocks; attention runs a 128-token mask as its 64-key tiles.

Bars as for 64-token blocks: masks identical outside the 1e-4 cut band (TopK
rows exactly k), logits within 1e-5 relative, attention max-abs 1e-4 (fp32) /
2e-2 (bf16) against the fp64 oracle at block 128."""
import numpy as np
import pytest

import oracle
import workload as W
from helpers import (ATOL_BF16, ATOL_F32, as_f64, check_mask, from_device, gpu_mask_numpy,
                     lists_from_dense, oracle_gate, small_inputs, stable_seed, to_device, upload_mask)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")

BLK = 128

CASES = [
    # B, Hq, Hkv, S, D, dtype, Dg
    (1, 2, 1, 1024, 64, "f32", 64),
    (2, 4, 2, 1280, 128, "bf16", 128),
    (1, 4, 1, 8320, 128, "bf16", 128),    # nb = 65: two select words
    (1, 3, 3, 512, 64, "bf16", 32),
    (1, 2, 1, 128, 128, "bf16", 64),      # a single block
]


def _gate_args(sel, Hq):
    if sel == "ratio":
        return oracle.TOPK_RATIO, dict(rho=0.3), dict(mode=seer.TOPK_RATIO, topk_ratio=0.3)
    if sel == "fixed":
        return oracle.TOPK_FIXED, dict(kfix=3), dict(mode=seer.TOPK_FIXED, topk_k=3)
    return oracle.THRESHOLD, dict(thresholds=np.float32(0.03)), dict(mode=seer.THRESHOLD, threshold=0.03)


def _oracle_gate128(q, k, wq, wk, mode, **args):
    L, ell = oracle.gate(q, k, wq, wk, BLK)
    sel = oracle.select(ell, mode, rho=args.get("rho", 0.0), k=args.get("kfix", 0),
                        thresholds=args.get("thresholds"))
    sel["L"], sel["ell"] = L, ell
    return sel


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("sel", ["ratio", "fixed", "thr"])
def test_gate_block128_mask_parity(case, sel):
    B, Hq, Hkv, S, D, dt, Dg = case
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed(case, sel, BLK), Dg=Dg,
                                      spikes=True)
    mode, args, gargs = _gate_args(sel, Hq)
    orc = _oracle_gate128(q, k, wq, wk, mode, **args)
    nb = S // BLK
    qd, kd = to_device(q), to_device(k)
    logits = torch.empty((B, Hq, nb, nb), dtype=torch.float32, device="cuda")
    mask = seer.gate(qd, kd, torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda(), **gargs,
                     block=BLK, dense_out=True, logits_out=logits)
    torch.cuda.synchronize()
    assert mask.n_blocks == nb
    count, idx, dense = gpu_mask_numpy(mask)
    tri = np.tril(np.ones((nb, nb), bool))
    err = np.abs(logits.cpu().numpy().astype(np.float64) - orc["L"])[..., tri].max()
    assert err <= 1e-5 * max(1.0, np.abs(orc["L"][..., tri]).max()), err
    check_mask(dense, count, orc, topk=mode != oracle.THRESHOLD)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("pattern", ["gate", "random", "vertical", "slash", "empty_rows"])
def test_bsattn_block128_parity(case, pattern):
    B, Hq, Hkv, S, D, dt, Dg = case
    nb = S // BLK
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed(case, pattern, "b128"), Dg=Dg)
    if pattern == "gate":
        om = _oracle_gate128(q, k, wq, wk, oracle.TOPK_RATIO, rho=0.4)["mask"]
    else:
        om = np.stack([np.stack([W.pattern_mask(pattern, nb, 50 * b + h, 0.3) for h in range(Hq)])
                       for b in range(B)])
    count, idx = lists_from_dense(om)
    O_ref, lse_ref = oracle.attn(q, k, v, block=BLK, mask=om)
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    m = upload_mask(count, idx, block=BLK)
    ws = torch.empty(max(1, seer.attn_workspace_bytes(qd, kd, vd)), dtype=torch.uint8, device="cuda")
    o, lse = seer.bsattn(qd, kd, vd, m, want_lse=True)
    o_ws, _ = seer.bsattn(qd, kd, vd, m, workspace=ws)  # a 128-token mask never splits
    torch.cuda.synchronize()
    O = as_f64(from_device(o)).reshape(-1, BLK, D)
    err = float(np.abs(O - O_ref).max()) if O_ref.size else 0.0
    assert err <= (ATOL_F32 if dt == "f32" else ATOL_BF16), err
    lse_g = lse.cpu().numpy().reshape(-1, BLK).astype(np.float64)
    fin = np.isfinite(lse_ref)
    np.testing.assert_array_equal(np.isfinite(lse_g), fin)
    if fin.any():
        assert float(np.abs(lse_g[fin] - lse_ref[fin]).max()) <= 1e-3
    assert np.all(O[~fin.any(axis=1)] == 0.0)
    assert torch.equal(o.view(torch.int16) if o.dtype == torch.bfloat16 else o,
                       o_ws.view(torch.int16) if o_ws.dtype == torch.bfloat16 else o_ws)


def test_block128_equals_expanded_64_mask():
    """A 128-token mask and its expansion to 64-token blocks give the same tiles,
    hence bit-identical outputs when both rows walk their tiles in ascending
    order (128-token rows always do; 64-token rows are asked to)."""
    B, Hq, Hkv, S, D = 1, 4, 2, 2048, 128
    nb = S // BLK
    w, q, k, v, _, _ = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("b128exp"))
    om = np.stack([W.pattern_mask("random", nb, h, 0.3) for h in range(Hq)])[None]
    om[..., np.arange(nb), np.arange(nb)] = 1
    om64 = np.kron(om, np.ones((2, 2), np.uint8)) & np.tril(np.ones((2 * nb, 2 * nb), np.uint8))
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    o128, l128 = seer.bsattn(qd, kd, vd, upload_mask(*lists_from_dense(om), block=BLK), want_lse=True)
    o64, l64 = seer.bsattn(qd, kd, vd, upload_mask(*lists_from_dense(om64)), want_lse=True,
                           opts={"walk_classes": 1})
    torch.cuda.synchronize()
    assert torch.equal(o128.view(torch.int16), o64.view(torch.int16))
    assert torch.equal(l128, l64)


def test_block128_long_rows_refill_the_list_window():
    """Long rows of a 128-token mask: 33024 tokens (258 blocks of 128, 516
    tiles per row), every causal block active, against the dense kernel in full
    (bit for bit: both walk ascending) and the oracle on sampled rows."""
    B, Hq, Hkv, S, D = 1, 1, 1, 33024, 64
    nb = S // BLK
    w, q, k, v, _, _ = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("b128long"))
    om = np.tril(np.ones((nb, nb), np.uint8))[None, None]
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    m = seer.mask_from_dense(torch.from_numpy(om).cuda(), heads_kv=Hkv, block=BLK)
    o, _ = seer.bsattn(qd, kd, vd, m)
    od, _ = seer.dense_attn(qd, kd, vd)
    torch.cuda.synchronize()
    assert int(m.count.max().item()) == nb
    diff = float((o.float() - od.float()).abs().max())
    assert diff == 0.0, diff
    rows = np.array([[0, 0, nb - 1], [0, 0, 257], [0, 0, 130]], np.int32)
    O_ref, _ = oracle.attn(q, k, v, block=BLK, mask=om, rows=rows)
    O = as_f64(from_device(o))
    got = np.stack([O[b, h, i * BLK:(i + 1) * BLK] for b, h, i in rows])
    assert float(np.abs(got - O_ref).max()) <= ATOL_BF16
