"""Dense attention and the ground-truth kernel with several query heads per
workgroup.  Dense rows are the same for every query head of a KV group, so a
workgroup takes 2 (or 4) heads of one group for the same query block and loads
each K/V tile once for all of them (the heads_per_wg option caps the count; 1
is one head per workgroup).

Bars: O and LSE against the fp64 oracle (2e-2 bf16 max-abs, LSE 1e-3), the
pooled map within the ground-truth test's relative band, and O, LSE and the
pooled map bitwise equal for 1, 2 and 4 heads per workgroup: each head's
arithmetic is the same, in the same tile order."""
import numpy as np
import pytest

import oracle
from helpers import ATOL_BF16, as_f64, from_device, small_inputs, stable_seed, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")

GT_RTOL, GT_ATOL = 2e-4, 1e-6

CASES = [
    # B, Hq, Hkv, S, D
    (1, 8, 2, 1024, 128),    # GQA 4:1: 4 heads per workgroup possible
    (2, 4, 2, 640, 128),     # GQA 2:1, batch 2
    (1, 6, 2, 1000, 64),     # GQA 3:1 (one head per workgroup), partial last block
    (1, 8, 1, 4160, 64),     # GQA 8:1, nb = 65
    (1, 4, 1, 130, 128),     # 3 blocks, the last of 2 rows
]


def _run(qd, kd, vd, causal, cap):
    opts = {"heads_per_wg": cap}
    o, lse = seer.dense_attn(qd, kd, vd, causal=causal, want_lse=True, opts=opts)
    og, lseg, gt = seer.attn_gt(qd, kd, vd, causal=causal, want_lse=True, opts=opts)
    torch.cuda.synchronize()
    return o, lse, og, lseg, gt


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("causal", [True, False])
def test_dense_and_ground_truth_with_shared_row_workgroups(case, causal):
    B, Hq, Hkv, S, D = case
    print(f"[shared rows] {case} causal={causal}", flush=True)
    w, q, k, v, _, _ = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("shared-rows", case, causal),
                                    spikes=True)
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    runs = {cap: _run(qd, kd, vd, causal, cap) for cap in (1, 2, 4)}
    for cap in (2, 4):
        for name, a, b in zip(("O", "LSE", "O (gt)", "LSE (gt)", "pooled map"), runs[1], runs[cap]):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"{cap} heads per workgroup: {name}"
    o, lse, og, lseg, gt = runs[2]
    assert torch.equal(o.view(torch.int16), og.view(torch.int16)) and torch.equal(lse, lseg)
    nb = -(-S // 64)
    O_ref, lse_ref = oracle.attn(q, k, v, causal=causal)
    ref = O_ref.reshape(B, Hq, nb * 64, D)[:, :, :S]
    assert float(np.abs(as_f64(from_device(o)) - ref).max()) <= ATOL_BF16
    lref = lse_ref.reshape(B, Hq, nb * 64)[:, :, :S]
    assert float(np.abs(lse.cpu().numpy() - lref).max()) <= 1e-3
    gt_ref = oracle.maxpool_gt(q, k, causal=causal)
    g = gt.cpu().numpy().astype(np.float64)
    assert not (np.abs(g - gt_ref) > GT_RTOL * gt_ref + GT_ATOL).any(), float(np.abs(g - gt_ref).max())
