"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle.

Bars: block masks identical except where the oracle log-score lies within 1e-4
of the row's selection cut (TopK rows keep exactly the oracle's count);
attention max-abs error <= 1e-4 (fp32) and <= 2e-2 (bf16).  Attention is
compared on the oracle's own mask, uploaded to the device, so that a near-cut
mask difference cannot mask an attention error; the end-to-end test then runs
gate -> attention entirely on the device."""
import numpy as np
import pytest

import oracle
import workload as W
from helpers import (ATOL_BF16, ATOL_F32, as_f64, check_mask, from_device, gather_rows,
                     gpu_mask_numpy, lists_from_dense, oracle_gate, sample_rows, small_inputs,
                     stable_seed, to_device, upload_mask)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")


def _tol(dtype):
    return ATOL_F32 if dtype == "f32" else ATOL_BF16


def _gpu(q, k, v, wq, wk):
    return tuple(to_device(x) for x in (q, k, v)) + (torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda())


def _max_abs(gpu_o, ref):
    return float(np.max(np.abs(as_f64(gpu_o) - ref))) if ref.size else 0.0


# --------------------------------------------------------------------------
# small shapes: several tiles, ragged block grids, GQA ratios, both dtypes
# --------------------------------------------------------------------------

CASES = [
    # B, Hq, Hkv, S, D, dtype, Dg
    (1, 2, 1, 1024, 64, "f32", 64),
    (2, 4, 2, 640, 128, "bf16", 128),
    (1, 7, 1, 1280, 128, "bf16", 128),
    (1, 3, 3, 448, 64, "bf16", 32),
    (1, 2, 1, 64, 128, "bf16", 64),       # a single block
    (1, 4, 1, 4160, 128, "bf16", 128),    # nb = 65: two select words, ragged logit tiles
    (1, 2, 2, 576, 128, "f32", 128),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("sel", ["ratio", "fixed", "thr", "thr_head", "noforce"])
@pytest.mark.parametrize("path", ["workspace", "logits"])
def test_gate_mask_parity(case, sel, path):
    """path 'workspace': the logits live in the gate's workspace; 'logits': they
    are written to the caller's buffer and also checked against the oracle's."""
    B, Hq, Hkv, S, D, dt, Dg = case
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed(case, sel), Dg=Dg,
                                      spikes=True)
    qd, kd, _, wqd, wkd = _gpu(q, k, v, wq, wk)
    kw = dict(keep_first=1, keep_diag=1)
    if sel == "ratio":
        mode, args = oracle.TOPK_RATIO, dict(rho=0.3)
        gargs = dict(mode=seer.TOPK_RATIO, topk_ratio=0.3)
    elif sel == "fixed":
        mode, args = oracle.TOPK_FIXED, dict(kfix=3)
        gargs = dict(mode=seer.TOPK_FIXED, topk_k=3)
    elif sel == "thr":
        mode, args = oracle.THRESHOLD, dict(thresholds=np.float32(0.02))
        gargs = dict(mode=seer.THRESHOLD, threshold=0.02)
    elif sel == "thr_head":
        thr = np.linspace(0.005, 0.1, Hq).astype(np.float32)
        mode, args = oracle.THRESHOLD, dict(thresholds=thr)
        gargs = dict(mode=seer.THRESHOLD, head_thresholds=torch.from_numpy(thr).cuda())
    else:
        mode, args = oracle.TOPK_RATIO, dict(rho=0.25)
        gargs = dict(mode=seer.TOPK_RATIO, topk_ratio=0.25)
        kw = dict(keep_first=0, keep_diag=0)
    orc = oracle_gate(q, k, wq, wk, mode, **args, **kw)
    logits = None
    if path == "logits":
        logits = torch.empty((B, Hq, S // 64, S // 64), dtype=torch.float32, device="cuda")
    mask = seer.gate(qd, kd, wqd, wkd, **gargs, **kw, dense_out=True, logits_out=logits)
    torch.cuda.synchronize()
    count, idx, dense = gpu_mask_numpy(mask)
    np.testing.assert_array_equal(dense, mask.dense.cpu().numpy())
    if logits is not None:
        # the raw gate logits agree with the oracle's on the causal triangle
        nb = S // 64
        tri = np.tril(np.ones((nb, nb), bool))
        gl = logits.cpu().numpy().astype(np.float64)
        err = np.abs(gl - orc["L"])[..., tri].max()
        assert err <= 1e-5 * max(1.0, np.abs(orc["L"][..., tri]).max()), err
    check_mask(dense, count, orc, topk=mode != oracle.THRESHOLD)


ROPE_CASES = [CASES[0], CASES[1], CASES[3], CASES[5]]


@pytest.mark.parametrize("case", ROPE_CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("theta,sel", [(10000.0, "ratio"), (500000.0, "thr"), (1e6, "fixed")])
def test_gate_block_rope_parity(case, theta, sel):
    """Block-level RoPE in the gate (section 3.1): logits and masks against the
    oracle with the same rope base."""
    B, Hq, Hkv, S, D, dt, Dg = case
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed(case, theta), Dg=Dg,
                                      spikes=True)
    qd, kd, _, wqd, wkd = _gpu(q, k, v, wq, wk)
    if sel == "ratio":
        mode, args, gargs = oracle.TOPK_RATIO, dict(rho=0.3), dict(mode=seer.TOPK_RATIO, topk_ratio=0.3)
    elif sel == "thr":
        mode, args = oracle.THRESHOLD, dict(thresholds=np.float32(0.02))
        gargs = dict(mode=seer.THRESHOLD, threshold=0.02)
    else:
        mode, args, gargs = oracle.TOPK_FIXED, dict(kfix=4), dict(mode=seer.TOPK_FIXED, topk_k=4)
    orc = oracle_gate(q, k, wq, wk, mode, **args, rope_theta=theta)
    nb = S // 64
    logits = torch.empty((B, Hq, nb, nb), dtype=torch.float32, device="cuda")
    mask = seer.gate(qd, kd, wqd, wkd, **gargs, rope_theta=theta, dense_out=True, logits_out=logits)
    torch.cuda.synchronize()
    count, idx, dense = gpu_mask_numpy(mask)
    tri = np.tril(np.ones((nb, nb), bool))
    gl = logits.cpu().numpy().astype(np.float64)
    err = np.abs(gl - orc["L"])[..., tri].max()
    assert err <= 1e-5 * max(1.0, np.abs(orc["L"][..., tri]).max()), err
    check_mask(dense, count, orc, topk=mode != oracle.THRESHOLD)
    if nb > 1:
        # the rotation changes the scores: the rope-free logits differ
        L0, _ = oracle.gate(q, k, wq, wk, 64, True)
        assert np.abs(L0[..., tri] - orc["L"][..., tri]).max() > 10 * err


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("pattern", ["gate", "a_shape", "vertical", "slash", "random", "empty_rows"])
def test_bsattn_parity(case, pattern):
    B, Hq, Hkv, S, D, dt, Dg = case
    nb = S // 64
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed(case, pattern), Dg=Dg)
    if pattern == "gate":
        orc = oracle_gate(q, k, wq, wk, oracle.TOPK_RATIO, rho=0.4)
        count, idx = orc["count"], orc["idx"]
        om = orc["mask"]
    else:
        om = np.stack([np.stack([W.pattern_mask(pattern, nb, 1000 * b + h, 0.3) for h in range(Hq)])
                       for b in range(B)])
        count, idx = lists_from_dense(om)
    O_ref, lse_ref = oracle.attn(q, k, v, mask=om)
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    o, lse = seer.bsattn(qd, kd, vd, upload_mask(count, idx), want_lse=True)
    torch.cuda.synchronize()
    O = from_device(o).reshape(B * Hq * nb, 64, D)
    err = _max_abs(O, O_ref)
    assert err <= _tol(dt), err
    lse_g = lse.cpu().numpy().reshape(-1, 64).astype(np.float64)
    fin = np.isfinite(lse_ref)
    np.testing.assert_array_equal(np.isfinite(lse_g), fin)
    if fin.any():
        assert np.max(np.abs(lse_g[fin] - lse_ref[fin])) <= 1e-3
    empty = ~fin.any(axis=1)
    assert np.all(as_f64(O)[empty] == 0.0)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("causal", [True, False])
def test_dense_parity(case, causal):
    B, Hq, Hkv, S, D, dt, Dg = case
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed(case, causal), Dg=Dg)
    O_ref, lse_ref = oracle.attn(q, k, v, causal=causal)
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    o, lse = seer.dense_attn(qd, kd, vd, causal=causal, want_lse=True)
    torch.cuda.synchronize()
    O = from_device(o).reshape(-1, 64, D)
    assert _max_abs(O, O_ref) <= _tol(dt)
    assert np.max(np.abs(lse.cpu().numpy().reshape(-1, 64) - lse_ref)) <= 1e-3


@pytest.mark.parametrize("pattern", ["vertical", "random", "empty_rows"])
def test_mask_from_dense_is_exact(pattern):
    B, Hq, nb = 2, 3, 70
    om = np.stack([np.stack([W.pattern_mask(pattern, nb, 10 * b + h, 0.3) for h in range(Hq)])
                   for b in range(B)])
    om[0, 0, 5, 6:] = 1  # entries above the diagonal are kept verbatim
    m = seer.mask_from_dense(torch.from_numpy(om).cuda())
    torch.cuda.synchronize()
    count, idx, dense = gpu_mask_numpy(m)
    np.testing.assert_array_equal(dense, om)
    np.testing.assert_array_equal(count, om.sum(-1))


def test_end_to_end_gate_then_bsattn():
    B, Hq, Hkv, S, D = 1, 8, 2, 2048, 128
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=77, spikes=True)
    qd, kd, vd, wqd, wkd = _gpu(q, k, v, wq, wk)
    mask = seer.gate(qd, kd, wqd, wkd, mode=seer.TOPK_RATIO, topk_ratio=0.2)
    o, _ = seer.bsattn(qd, kd, vd, mask)
    torch.cuda.synchronize()
    orc = oracle_gate(q, k, wq, wk, oracle.TOPK_RATIO, rho=0.2)
    count, idx, dense = gpu_mask_numpy(mask)
    check_mask(dense, count, orc, topk=True)
    nb = S // 64
    same = (dense == orc["mask"]).all(-1)  # rows whose mask equals the oracle's
    rows = np.argwhere(same).astype(np.int32)
    O_ref, _ = oracle.attn(q, k, v, mask=orc["mask"], rows=rows)
    assert _max_abs(gather_rows(from_device(o), rows), O_ref) <= ATOL_BF16
    assert same.mean() > 0.9


def test_deterministic_bitwise():
    B, Hq, Hkv, S, D = 1, 4, 1, 2048, 128
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=5)
    qd, kd, vd, wqd, wkd = _gpu(q, k, v, wq, wk)
    outs = []
    for _ in range(2):
        m = seer.gate(qd, kd, wqd, wkd, mode=seer.THRESHOLD, threshold=0.01)
        o, lse = seer.bsattn(qd, kd, vd, m, want_lse=True)
        od, _ = seer.dense_attn(qd, kd, vd)
        torch.cuda.synchronize()
        outs.append((m.count.cpu(), gpu_mask_numpy(m)[2], o.cpu(), lse.cpu(), od.cpu()))
    for a, b in zip(*outs):
        assert torch.equal(torch.as_tensor(a), torch.as_tensor(b))


def test_strided_views():
    # Q/K/V as views into a packed [B, S, H, D] buffer (sequence-major layout)
    B, Hq, Hkv, S, D = 1, 4, 2, 512, 128
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=11)
    qd = to_device(np.ascontiguousarray(q.transpose(0, 2, 1, 3))).transpose(1, 2)
    kd = to_device(np.ascontiguousarray(k.transpose(0, 2, 1, 3))).transpose(1, 2)
    vd = to_device(np.ascontiguousarray(v.transpose(0, 2, 1, 3))).transpose(1, 2)
    O_ref, _ = oracle.attn(q, k, v)
    o, _ = seer.dense_attn(qd, kd, vd)
    torch.cuda.synchronize()
    assert _max_abs(from_device(o.contiguous()).reshape(-1, 64, D), O_ref) <= ATOL_BF16


@pytest.mark.parametrize("case", [(1, 8, 2, 4096, 128, 64), (2, 4, 1, 3000, 64, 64), (1, 4, 4, 2048, 128, 64),
                                  (1, 4, 2, 4096, 128, 128)],
                         ids=lambda c: "x".join(map(str, c)))
def test_batched_launches_equal_single_launch(case):
    """Long sparse rows launch in batches of the resident workgroups (task ids
    continue across batches); forced here on small shapes with small batches,
    the outputs must equal the single launch's bit for bit."""
    B, Hq, Hkv, S, D, blk = case
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("batches", case), spikes=True)
    qd, kd, vd = (to_device(x) for x in (q, k, v))
    mask = seer.gate(qd, kd, torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda(), mode=seer.TOPK_RATIO,
                     topk_ratio=0.3, block=blk)
    o1, l1 = seer.bsattn(qd, kd, vd, mask, want_lse=True, opts={"batch_min_blocks": -1})
    outs = []
    for wgs in (64, 24, 8):
        opts = {"batch_min_blocks": 1, "batch_wgs": wgs}
        assert seer.attn_launches(qd, kd, vd, mask, opts=opts) > 1
        outs.append(seer.bsattn(qd, kd, vd, mask, want_lse=True, opts=opts))
    torch.cuda.synchronize()
    for o2, l2 in outs:
        assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
        assert torch.equal(l1, l2)
