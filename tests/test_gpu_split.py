"""GPU parity of the key-range split (seer_bsattn_ws / seer_dense_attn_ws): rows
cut into ranges of w key blocks computed as separate tasks by persistent
workgroups; each row's last task merges the bf16 partials.

The split runs only on request (the split option), with ranges sized to the L2
(128 blocks at head_dim 128); these tests request it with a small range width
(the split_width option) so that small shapes reach many ranges (a partial last
range, rows with empty ranges, rows with a single non-empty range written
directly, ragged GQA layouts).  Bars as for the unsplit kernel (max-abs 2e-2
against the fp64 oracle, LSE 1e-3, empty rows O = 0 and LSE = -inf); the split
result also stays within 1e-2 of the unsplit one (the partials' bf16 rounding)
and is bitwise reproducible (the merge order is fixed, whichever task arrives
last)."""
import numpy as np
import pytest

import oracle
import workload as W
from helpers import (ATOL_BF16, as_f64, from_device, lists_from_dense, oracle_gate, small_inputs,
                     stable_seed, to_device, upload_mask)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")

CASES = [
    # B, Hq, Hkv, S, D, w   (w: key blocks per range)
    (1, 2, 1, 1024, 128, 1),   # 1 KV group: 16 ranges of 1 block
    (2, 4, 2, 2048, 128, 3),   # 4 groups: 11 ranges, the last of 2 blocks
    (1, 4, 1, 4096, 64, 4),    # D 64: 16 ranges of 4
    (1, 8, 2, 1536, 128, 5),   # nb 24: 5 ranges, the last of 4 blocks
    (1, 7, 1, 2048, 128, 2),   # GQA 7:1, 16 ranges
]


def _opts(wr):
    return {"split": 1, "split_width": wr}


def _ws(qd, kd, vd, wr):
    n = seer.attn_workspace_bytes(qd, kd, vd, opts=_opts(wr))
    return n, torch.empty(max(n, 1), dtype=torch.uint8, device="cuda")


def _check(o, lse, O_ref, lse_ref, D):
    O = as_f64(from_device(o)).reshape(-1, 64, D)
    err = float(np.abs(O - O_ref).max())
    assert err <= ATOL_BF16, err
    lse_g = lse.cpu().numpy().reshape(-1, 64).astype(np.float64)
    fin = np.isfinite(lse_ref)
    np.testing.assert_array_equal(np.isfinite(lse_g), fin)
    if fin.any():
        assert float(np.abs(lse_g[fin] - lse_ref[fin]).max()) <= 1e-3
    empty = ~fin.any(axis=1)
    assert np.all(O[empty] == 0.0)
    return err


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("pattern", ["gate", "random", "vertical", "slash", "a_shape", "empty_rows"])
def test_split_bsattn_parity(case, pattern):
    B, Hq, Hkv, S, D, wr = case
    nb = S // 64
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed(case, pattern, "split"))
    if pattern == "gate":
        orc = oracle_gate(q, k, wq, wk, oracle.TOPK_RATIO, rho=0.3)
        count, idx, om = orc["count"], orc["idx"], orc["mask"]
    else:
        om = np.stack([np.stack([W.pattern_mask(pattern, nb, 100 * b + h, 0.3) for h in range(Hq)])
                       for b in range(B)])
        count, idx = lists_from_dense(om)
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    n, ws = _ws(qd, kd, vd, wr)
    assert n > 0, "the split must be enabled for this shape"
    m = upload_mask(count, idx)
    print(f"[split] case {case} pattern {pattern} workspace {n}", flush=True)
    assert seer.attn_launches(qd, kd, vd, m, opts=_opts(wr), workspace_bytes=n) == 1  # one persistent launch
    o, lse = seer.bsattn(qd, kd, vd, m, want_lse=True, workspace=ws, opts=_opts(wr))
    o2, lse2 = seer.bsattn(qd, kd, vd, m, want_lse=True, workspace=ws, opts=_opts(wr))
    o0, _ = seer.bsattn(qd, kd, vd, m)
    torch.cuda.synchronize()
    O_ref, lse_ref = oracle.attn(q, k, v, mask=om)
    _check(o, lse, O_ref, lse_ref, D)
    assert torch.equal(o.view(torch.int16), o2.view(torch.int16)) and torch.equal(lse, lse2)
    diff = float((o.float() - o0.float()).abs().max())
    assert diff <= 1e-2, diff


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_split_dense_parity(case):
    B, Hq, Hkv, S, D, wr = case
    w, q, k, v, _, _ = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed(case, "splitdense"))
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    n, ws = _ws(qd, kd, vd, wr)
    o, lse = seer.dense_attn(qd, kd, vd, want_lse=True, workspace=ws, opts=_opts(wr))
    torch.cuda.synchronize()
    O_ref, lse_ref = oracle.attn(q, k, v)
    _check(o, lse, O_ref, lse_ref, D)


def test_split_small_workspace_and_noncausal_fall_back_to_unsplit():
    B, Hq, Hkv, S, D = 1, 4, 2, 2048, 128
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("splitfb"))
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    orc = oracle_gate(q, k, wq, wk, oracle.TOPK_RATIO, rho=0.3)
    m = upload_mask(orc["count"], orc["idx"])
    n, _ = _ws(qd, kd, vd, 4)
    small = torch.empty(n // 2, dtype=torch.uint8, device="cuda")
    o_small, _ = seer.bsattn(qd, kd, vd, m, workspace=small, opts=_opts(4))
    o_plain, _ = seer.bsattn(qd, kd, vd, m)
    o_nc, _ = seer.dense_attn(qd, kd, vd, causal=False, workspace=small, opts=_opts(4))
    o_nc0, _ = seer.dense_attn(qd, kd, vd, causal=False)
    torch.cuda.synchronize()
    assert torch.equal(o_small.view(torch.int16), o_plain.view(torch.int16))
    assert torch.equal(o_nc.view(torch.int16), o_nc0.view(torch.int16))


def test_split_is_opt_in():
    """Without the split option a call with a workspace is the unsplit one."""
    B, Hq, Hkv, S, D = 1, 4, 2, 2048, 128
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("splitoptin"))
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    orc = oracle_gate(q, k, wq, wk, oracle.TOPK_RATIO, rho=0.3)
    m = upload_mask(orc["count"], orc["idx"])
    n, ws = _ws(qd, kd, vd, 4)
    assert n > 0 and seer.attn_workspace_bytes(qd, kd, vd) == 0
    o_ws, _ = seer.bsattn(qd, kd, vd, m, workspace=ws)
    o_ws0, _ = seer.bsattn(qd, kd, vd, m, workspace=ws, opts={"split_width": 4})
    o_plain, _ = seer.bsattn(qd, kd, vd, m)
    torch.cuda.synchronize()
    assert torch.equal(o_ws.view(torch.int16), o_plain.view(torch.int16))
    assert torch.equal(o_ws0.view(torch.int16), o_plain.view(torch.int16))
