"""The residue-class walk of sparse rows (seer_attn_opts.walk_classes): a row
visits its blocks j = S q + c in the order (c, q).  Only the order in which a
row's tiles are summed changes, so every class count must match the fp64
oracle within the usual bars, be reproducible bit for bit, and treat list
entries above the diagonal (a caller's mask) exactly as the ascending walk
does: they are not part of the row."""
import numpy as np
import pytest

import oracle
import workload as W
from helpers import (ATOL_BF16, ATOL_F32, as_f64, from_device, lists_from_dense, small_inputs, stable_seed,
                     to_device, upload_mask)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")

CASES = [
    # B, Hq, Hkv, S, D, dtype
    (1, 4, 1, 4160, 128, "bf16"),   # nb = 65: lists longer than one ballot word, uneven class sizes
    (2, 4, 2, 2048, 64, "bf16"),
    (1, 2, 1, 1024, 128, "bf16"),
    (1, 2, 2, 768, 64, "f32"),      # the fp32 kernel ignores the option
]
PATTERNS = ["random", "vertical", "slash", "a_shape"]


def _mask(pattern, B, H, nb, seed):
    return np.stack([np.stack([W.pattern_mask(pattern, nb, seed + 1000 * b + h, 0.35) for h in range(H)])
                     for b in range(B)])


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("pattern", PATTERNS)
def test_walk_classes_parity_and_determinism(case, pattern):
    B, Hq, Hkv, S, D, dt = case
    nb = S // 64
    print(f"[walk] {case} {pattern}", flush=True)
    _, q, k, v, _, _ = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed("walk", case, pattern))
    om = _mask(pattern, B, Hq, nb, stable_seed("walkmask", case, pattern) % 100000)
    count, idx = lists_from_dense(om)
    O_ref, _ = oracle.attn(q, k, v, mask=om)
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    mask = upload_mask(count, idx)
    tol = ATOL_F32 if dt == "f32" else ATOL_BF16
    outs = {}
    for s in (1, 2, 4, 8, 16):
        o, lse = seer.bsattn(qd, kd, vd, mask, want_lse=True, opts={"walk_classes": s})
        o2, lse2 = seer.bsattn(qd, kd, vd, mask, want_lse=True, opts={"walk_classes": s})
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16) if o.dtype == torch.bfloat16 else o,
                           o2.view(torch.int16) if o2.dtype == torch.bfloat16 else o2), s
        assert torch.equal(lse, lse2), s
        got = from_device(o).reshape(B, Hq, S, D)
        ref = O_ref.reshape(B, Hq, S, D)
        err = float(np.abs(as_f64(got) - ref).max())
        assert err <= tol, (s, err)
        outs[s] = got
    # the default is one of the walks above
    o, _ = seer.bsattn(qd, kd, vd, mask)
    torch.cuda.synchronize()
    assert any(np.array_equal(from_device(o).reshape(B, Hq, S, D), outs[s]) for s in outs)


@pytest.mark.parametrize("s", [1, 4, 16])
def test_walk_drops_entries_above_the_diagonal(s):
    """A caller's causal mask may list blocks above the diagonal; they are the
    ascending list's tail and take no part, whatever the walk."""
    B, Hq, Hkv, S, D = 1, 2, 1, 2048, 128
    nb = S // 64
    _, q, k, v, _, _ = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("walkdiag", s))
    base = _mask("random", B, Hq, nb, 77)
    rng = np.random.default_rng(5)
    extra = base | (rng.random(base.shape) < 0.3)  # adds blocks anywhere, above the diagonal too
    causal_part = extra & np.tril(np.ones((nb, nb), bool))
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    o1, l1 = seer.bsattn(qd, kd, vd, upload_mask(*lists_from_dense(extra)), want_lse=True,
                         opts={"walk_classes": s})
    o2, l2 = seer.bsattn(qd, kd, vd, upload_mask(*lists_from_dense(causal_part)), want_lse=True,
                         opts={"walk_classes": s})
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1, l2)


def test_rows_longer_than_the_list_window():
    """Rows of more than 2048 entries cross the kernel's LDS list window (it is
    refilled as the row advances) and walk ascending; shorter rows of the same
    call take the residue-class walk.  133120 tokens (2080 blocks), one head,
    every causal block active: the ascending walk equals the dense kernel bit
    for bit; the default walk matches the oracle on rows on both sides of 2048."""
    B, Hq, Hkv, S, D = 1, 1, 1, 2080 * 64, 64
    nb = S // 64
    _, q, k, v, _, _ = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("walkwin"))
    om = np.tril(np.ones((nb, nb), np.uint8))[None, None]
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    m = seer.mask_from_dense(torch.from_numpy(om).cuda(), heads_kv=Hkv)
    o_asc, _ = seer.bsattn(qd, kd, vd, m, opts={"walk_classes": 1})
    o_def, _ = seer.bsattn(qd, kd, vd, m)
    od, _ = seer.dense_attn(qd, kd, vd)
    torch.cuda.synchronize()
    assert int(m.count.max().item()) == nb
    assert torch.equal(o_asc.view(torch.int16), od.view(torch.int16))
    rows = np.array([[0, 0, nb - 1], [0, 0, 2048], [0, 0, 2047], [0, 0, 700]], np.int32)
    O_ref, _ = oracle.attn(q, k, v, mask=om, rows=rows)
    O = as_f64(from_device(o_def))
    got = np.stack([O[b, h, i * 64:(i + 1) * 64] for b, h, i in rows])
    assert float(np.abs(got - O_ref).max()) <= ATOL_BF16
