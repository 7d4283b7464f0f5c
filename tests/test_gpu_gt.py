"""GPU parity of dense attention with the 2D max-pooled attention map
(seer_attn_gt; Eq. 2, computed as in appendix A.1) against the fp64 oracle.

Bars: O and LSE as for dense attention (the ground-truth kernel is the dense
kernel plus the row-max stores and the pooling epilogue); the pooled map within
GT_RTOL relative + GT_ATOL absolute of the oracle's (fp32 score arithmetic:
an exponent error of ~1e-6 makes a relative error of the same order), exact
zeros where the tile holds no visible key."""
import numpy as np
import pytest

import oracle
import workload as W
from helpers import (ATOL_BF16, ATOL_F32, as_f64, from_device, gather_rows, sample_rows,
                     small_inputs, stable_seed, to_device)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")

GT_RTOL = 2e-4
GT_ATOL = 1e-6

CASES = [
    # B, Hq, Hkv, S, D, dtype
    (1, 2, 1, 1024, 64, "f32"),
    (2, 4, 2, 640, 128, "bf16"),
    (1, 7, 1, 1280, 128, "bf16"),
    (1, 3, 3, 448, 64, "bf16"),
    (1, 2, 1, 64, 128, "bf16"),   # a single block
    (1, 2, 2, 576, 128, "f32"),
]


def _check_gt(gt_gpu, gt_ref, causal):
    g = gt_gpu.astype(np.float64)
    bad = np.abs(g - gt_ref) > GT_RTOL * gt_ref + GT_ATOL
    assert not bad.any(), (np.argwhere(bad)[:5].tolist(), float(np.abs(g - gt_ref).max()))
    if causal:
        nb = g.shape[-1]
        upper = np.triu(np.ones((nb, nb), bool), 1)
        assert np.all(g[..., upper] == 0.0)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("causal", [True, False])
def test_attn_gt_parity(case, causal):
    B, Hq, Hkv, S, D, dt = case
    w, q, k, v, _, _ = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed(case, causal, "gt"),
                                    spikes=True)
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    print(f"[gt] case {case} causal={causal}", flush=True)
    o, lse, gt = seer.attn_gt(qd, kd, vd, causal=causal, want_lse=True)
    o_dense, lse_dense = seer.dense_attn(qd, kd, vd, causal=causal, want_lse=True)
    torch.cuda.synchronize()
    O_ref, lse_ref = oracle.attn(q, k, v, causal=causal)
    gt_ref = oracle.maxpool_gt(q, k, causal=causal)
    O = from_device(o).reshape(-1, 64, D)
    tol = ATOL_F32 if dt == "f32" else ATOL_BF16
    assert float(np.abs(as_f64(O) - O_ref).max()) <= tol
    assert float(np.abs(lse.cpu().numpy().reshape(-1, 64) - lse_ref).max()) <= 1e-3
    _check_gt(gt.cpu().numpy(), gt_ref, causal)
    # the extra stores leave the attention arithmetic untouched
    assert torch.equal(o.view(torch.int16) if o.dtype == torch.bfloat16 else o,
                       o_dense.view(torch.int16) if o_dense.dtype == torch.bfloat16 else o_dense)
    assert torch.equal(lse, lse_dense)


@pytest.mark.parametrize("kv_groups", [1, 3])
def test_attn_gt_chunked_workspace_matches_one_launch(kv_groups):
    B, Hq, Hkv, S, D = 2, 8, 2, 640, 128  # 4 KV groups of 4 query heads
    w, q, k, v, _, _ = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("gtchunk", kv_groups))
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    o1, l1, g1 = seer.attn_gt(qd, kd, vd, want_lse=True)
    need = seer.attn_gt_workspace_bytes(qd, kd, vd, kv_groups)
    assert need * 4 // kv_groups == seer.attn_gt_workspace_bytes(qd, kd, vd, 0)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    o2, l2, g2 = seer.attn_gt(qd, kd, vd, want_lse=True, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1, l2)
    assert torch.equal(g1, g2)


def test_attn_gt_strided_views_and_scale():
    # Q/K/V as head-interleaved views of one [B, S, H, D] buffer, custom scale
    B, Hq, Hkv, S, D = 1, 4, 2, 384, 64
    w, q, k, v, _, _ = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("gtstride"))
    qd, kd, vd = (to_device(np.ascontiguousarray(x.transpose(0, 2, 1, 3))).transpose(1, 2)
                  for x in (q, k, v))
    o, _, gt = seer.attn_gt(qd, kd, vd, sm_scale=0.07)
    torch.cuda.synchronize()
    _check_gt(gt.cpu().numpy(), oracle.maxpool_gt(q, k, scale=0.07), True)


@pytest.mark.slow
def test_attn_gt_full_size_32k_sampled_rows():
    """32768 tokens, 32 query / 8 KV heads: two KV groups per launch, sampled
    rows of the pooled map and of O against the oracle."""
    w = W.WORKLOADS["llama_s32k"]
    print("[gt] llama_s32k: generating inputs", flush=True)
    q, k, v = (W.make_tensor(w, t) for t in "qkv")
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    ws = torch.empty(seer.attn_gt_workspace_bytes(qd, kd, vd, 2), dtype=torch.uint8, device="cuda")
    o, lse, gt = seer.attn_gt(qd, kd, vd, want_lse=True, workspace=ws)
    torch.cuda.synchronize()
    print("[gt] llama_s32k: device done", flush=True)
    nb = w.n_blocks
    rows = sample_rows(w.batch, w.heads_q, nb, 16, seed=nb + 7)
    gt_ref = oracle.maxpool_gt(q, k, rows=rows)
    g = gt.cpu().numpy()
    _check_gt(np.stack([g[b, h, i] for b, h, i in rows]), gt_ref, False)
    upper = np.triu(np.ones((nb, nb), bool), 1)
    assert np.all(g[..., upper] == 0.0)
    O_ref, _ = oracle.attn(q, k, v, rows=rows)
    err = float(np.abs(as_f64(gather_rows(from_device(o), rows)) - O_ref).max())
    assert err <= ATOL_BF16, err
    # every query's probabilities sum to 1, so a row's pooled maxima cover at
    # least 1/64 of each query's mass: sum_j gt[i][j] >= 1/64 for every row
    assert float(g.sum(-1).min()) >= 1.0 / 64 - 1e-6
