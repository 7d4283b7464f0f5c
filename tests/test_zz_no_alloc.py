"""The gate for callers that cannot allocate (seer_gate_noalloc): no workspace,
its scratch a static device array, the logits formed and selected in one kernel.

Through the C ABI (the binding only marshals arguments), against seer_gate on
the same inputs: masks equal except where the oracle log-score lies within 1e-4
of the row's selection cut (the two form the logits in a different summation
order), TopK rows with exactly the oracle's count.  Two calls in a row, the
second on a smaller input (the shared scratch keeps the first call's contents);
oracle parity of the masks on small shapes (several tiles, ragged block grids,
GQA, both dtypes, every selection mode); exact ties bit for bit."""
import numpy as np
import pytest

import oracle
import workload as W
from helpers import check_mask, gpu_mask_numpy, oracle_gate, small_inputs, stable_seed, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")


def _gpu(q, k, wq, wk):
    return to_device(q), to_device(k), torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda()


def _masks(qd, kd, wqd, wkd, B, H, S, **gargs):
    """(seer_gate's mask, seer_gate_noalloc's mask) as numpy (count, dense)."""
    ref = seer.gate(qd, kd, wqd, wkd, **gargs, dense_out=True)
    out = seer.alloc_mask(B, H, S, "cuda", dense=True)
    seer.gate_noalloc(qd, kd, wqd, wkd, out, **gargs)
    torch.cuda.synchronize()
    rc, _, rd = gpu_mask_numpy(ref)
    nc, _, nd = gpu_mask_numpy(out)
    return (rc, rd), (nc, nd)


def test_noalloc_matches_gate_on_two_calls_in_a_row():
    """A larger call, then a smaller one on new inputs: the scratch left by the
    first must not leak into the second."""
    for B, Hq, Hkv, S, D, dt, Dg, tag in ((1, 8, 2, 8192, 128, "bf16", 128, "first"),
                                          (2, 4, 1, 1280, 64, "bf16", 64, "second")):
        print(f"[no-alloc] {tag} call: B{B} Hq{Hq} Hkv{Hkv} S{S} D{D} Dg{Dg}", flush=True)
        w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed("noalloc", tag), Dg=Dg,
                                          spikes=True)
        qd, kd, wqd, wkd = _gpu(q, k, wq, wk)
        orc = oracle_gate(q, k, wq, wk, oracle.TOPK_RATIO, rho=0.2)
        (rc, rd), (nc, nd) = _masks(qd, kd, wqd, wkd, B, Hq, S, mode=seer.TOPK_RATIO, topk_ratio=0.2)
        check_mask(rd, rc, orc, topk=True)
        check_mask(nd, nc, orc, topk=True)
        diff = nd != rd
        if diff.any():  # seer_gate vs seer_gate_noalloc: only inside the cut band
            dist = np.abs(orc["ell"] - orc["cut"][..., None])
            assert not np.any(diff & ~(dist <= 1e-4))
        np.testing.assert_array_equal(nc, rc)


CASES = [
    # B, Hq, Hkv, S, D, dtype, Dg
    (1, 2, 1, 1024, 64, "f32", 64),
    (2, 4, 2, 640, 128, "bf16", 128),
    (1, 7, 1, 1280, 128, "bf16", 128),
    (1, 3, 3, 448, 64, "bf16", 32),
    (1, 2, 1, 64, 128, "bf16", 64),       # a single block
    (1, 4, 1, 4160, 128, "bf16", 128),    # nb = 65: two select words, a partial column tile
    (1, 2, 1, 3000, 128, "bf16", 128),    # a partial last block
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("sel", ["ratio", "fixed", "thr", "thr_head", "noforce", "rope"])
def test_noalloc_mask_parity(case, sel):
    B, Hq, Hkv, S, D, dt, Dg = case
    w, q, k, v, wq, wk = small_inputs(B, Hq, Hkv, S, D, dt, seed=stable_seed("noalloc", case, sel), Dg=Dg,
                                      spikes=True)
    qd, kd, wqd, wkd = _gpu(q, k, wq, wk)
    kw = dict(keep_first=1, keep_diag=1)
    extra = {}
    if sel in ("ratio", "rope"):
        mode, args, gargs = oracle.TOPK_RATIO, dict(rho=0.3), dict(mode=seer.TOPK_RATIO, topk_ratio=0.3)
        if sel == "rope":
            extra = dict(rope_theta=500000.0)
    elif sel == "fixed":
        mode, args, gargs = oracle.TOPK_FIXED, dict(kfix=3), dict(mode=seer.TOPK_FIXED, topk_k=3)
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
    orc = oracle_gate(q, k, wq, wk, mode, **args, **kw, **extra)
    out = seer.alloc_mask(B, Hq, S, "cuda", dense=True)
    seer.gate_noalloc(qd, kd, wqd, wkd, out, **gargs, **kw, **extra)
    torch.cuda.synchronize()
    count, idx, dense = gpu_mask_numpy(out)
    np.testing.assert_array_equal(dense, out.dense.cpu().numpy())
    check_mask(dense, count, orc, topk=mode != oracle.THRESHOLD)


def _blockwise_integers(rng, B, H, nb, D, lo, hi):
    a = rng.integers(lo, hi + 1, size=(B, H, nb, D)).astype(np.float32)
    return W.f32_to_bf16_bits(np.ascontiguousarray(np.repeat(a, 64, axis=2)))


@pytest.mark.parametrize("case", [(1, 4, 2, 130, 64, 64, (-2, 2)), (1, 2, 2, 1100, 64, 32, (0, 1))],
                         ids=lambda c: "x".join(map(str, c[:6])))
def test_noalloc_exact_ties_match_oracle(case):
    """Block-constant integer Q and K with weights passing the pooled mean: every
    logit is exact, so the mask must equal the oracle's bit for bit, including
    which tied blocks it keeps (the smaller index)."""
    B, Hq, Hkv, nb, D, Dg, (lo, hi) = case
    rng = np.random.default_rng(stable_seed("noalloc ties", case))
    q = _blockwise_integers(rng, B, Hq, nb, D, lo, hi)
    k = _blockwise_integers(rng, B, Hkv, nb, D, lo, hi)
    wq = np.zeros((Hq, D, Dg), np.float32)
    wk = np.zeros((Hkv, 3 * D, Dg), np.float32)
    for d in range(Dg):
        wq[:, d, d] = 1.0
        wk[:, 2 * D + d, d] = 1.0
    _, ell = oracle.gate(q, k, wq, wk, 64, True)
    orc = oracle.select(ell, oracle.TOPK_RATIO, rho=0.3)
    out = seer.alloc_mask(B, Hq, 64 * nb, "cuda", dense=True)
    seer.gate_noalloc(to_device(q), to_device(k), torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda(), out,
                      mode=seer.TOPK_RATIO, topk_ratio=0.3)
    torch.cuda.synchronize()
    count, _, dense = gpu_mask_numpy(out)
    np.testing.assert_array_equal(count, orc["count"])
    assert not np.any(dense != orc["mask"])


def test_noalloc_refuses_what_it_cannot_hold():
    """Beyond the static scratch, or unsupported, the call returns an error and
    writes nothing."""
    B, Hq, Hkv, S, D = 1, 2, 1, 64 * 2049, 64
    q = torch.zeros((B, Hq, S, D), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((B, Hkv, S, D), dtype=torch.bfloat16, device="cuda")
    wq = torch.zeros((Hq, D, 64), dtype=torch.float32, device="cuda")
    wk = torch.zeros((Hkv, 3 * D, 64), dtype=torch.float32, device="cuda")
    out = seer.alloc_mask(B, Hq, S, "cuda")
    out.count.fill_(-7)
    with pytest.raises(seer.SeerError) as e:
        seer.gate_noalloc(q, k, wq, wk, out, mode=seer.TOPK_RATIO, topk_ratio=0.1)
    assert e.value.status == seer.ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert bool((out.count == -7).all())
