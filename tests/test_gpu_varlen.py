"""GPU parity for packed variable-length batches (seer_gate_varlen,
seer_bsattn_varlen): Q/K/V/O packed [tokens, heads, head_dim], sequence b at
tokens [cu[b], cu[b+1]).  Each sequence is its own problem; the lengths mix
whole and partial blocks, a single token and an empty sequence.

Bars: masks and attention against the fp64 oracle per sequence (mask cut band
1e-4, bf16 attention 2e-2 max-abs, LSE 1e-3), and bit-for-bit equality with
separate batch-1 calls on views of the same packed tensors."""
import numpy as np
import pytest

import oracle
from helpers import ATOL_BF16, as_f64, check_mask, from_device, small_inputs, stable_seed, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")

LENGTHS = [1000, 64, 0, 1, 2500, 130]
HQ, HKV, D, DG = 4, 2, 128, 64


def _nb(n):
    return -(-n // 64)


def _packed_inputs(lengths, seed):
    """Per-sequence seeded [1, H, len, D] tensors, packed token-major, and one gate."""
    seqs = []
    for b, n in enumerate(lengths):
        if n == 0:
            seqs.append(None)
            continue
        _, q, k, v, _, _ = small_inputs(1, HQ, HKV, n, D, "bf16", seed=seed + 17 * b, Dg=DG, spikes=n >= 64)
        seqs.append((q, k, v))
    _, _, _, _, wq, wk = small_inputs(1, HQ, HKV, 64, D, "bf16", seed=seed, Dg=DG)

    def pack(j, H):
        parts = [s[j][0].transpose(1, 0, 2) for s in seqs if s is not None]
        return np.ascontiguousarray(np.concatenate(parts, axis=0)) if parts else np.zeros((0, H, D), np.uint16)

    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    return seqs, pack(0, HQ), pack(1, HKV), pack(2, HKV), wq, wk, cu


def _view(t, cu, b):
    """[1, H, len_b, D] view of sequence b of a packed [T, H, D] tensor."""
    return t[int(cu[b]):int(cu[b + 1])].permute(1, 0, 2).unsqueeze(0)


@pytest.mark.parametrize("sel", ["ratio", "thr"])
def test_varlen_gate_and_attention(sel):
    print(f"[varlen] {sel}", flush=True)
    seqs, q, k, v, wq, wk, cu = _packed_inputs(LENGTHS, stable_seed("varlen", sel))
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    wqd, wkd = torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda()
    if sel == "ratio":
        gargs, mode, oargs = dict(mode=seer.TOPK_RATIO, topk_ratio=0.3), oracle.TOPK_RATIO, dict(rho=0.3)
    else:
        gargs, mode, oargs = dict(mode=seer.THRESHOLD, threshold=0.02), oracle.THRESHOLD, dict(
            thresholds=np.float32(0.02))
    mask = seer.gate_varlen(qd, kd, wqd, wkd, cu, **gargs)
    o, lse = seer.bsattn_varlen(qd, kd, vd, cu, mask, want_lse=True)
    torch.cuda.synchronize()
    o_np = from_device(o)
    lse_np = lse.cpu().numpy()
    for b, n in enumerate(LENGTHS):
        if n == 0:
            continue
        qb, kb, vb = seqs[b]
        _, ell = oracle.gate(qb, kb, wq, wk, 64, True)
        orc = oracle.select(ell, mode, **oargs)
        orc["ell"] = ell
        cnt, idx = mask.sequence(b)
        cnt = cnt.cpu().numpy()[None]
        idx = idx.cpu().numpy().view(np.uint16)[None]
        nb = _nb(n)
        dense = np.zeros((1, HQ, nb, nb), np.uint8)
        for h in range(HQ):
            for i in range(nb):
                dense[0, h, i, idx[0, h, i, :cnt[0, h, i]].astype(np.int64)] = 1
        check_mask(dense, cnt, orc, topk=mode != oracle.THRESHOLD)
        # attention against the oracle on the device's own mask (identical outside the cut band)
        O_ref, lse_ref = oracle.attn(qb, kb, vb, mask=dense)
        ref = O_ref.reshape(HQ, nb * 64, D)[:, :n]
        got = as_f64(o_np[int(cu[b]):int(cu[b + 1])]).transpose(1, 0, 2)
        err = float(np.abs(got - ref).max())
        lerr = float(np.abs(lse_np[HQ * int(cu[b]):HQ * int(cu[b + 1])].reshape(HQ, n)
                            - lse_ref.reshape(HQ, nb * 64)[:, :n]).max())
        print(f"[varlen] seq {b} len {n}: attention {err:.2e}, lse {lerr:.2e}", flush=True)
        assert err <= ATOL_BF16 and lerr <= 1e-3


@pytest.mark.parametrize("kv_shared", [False, True])
def test_varlen_equals_separate_calls(kv_shared):
    seqs, q, k, v, wq, wk, cu = _packed_inputs(LENGTHS, stable_seed("varlen-eq", kv_shared))
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    wqd, wkd = torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda()
    kw = dict(mode=seer.TOPK_RATIO, topk_ratio=0.25, kv_shared=kv_shared)
    mask = seer.gate_varlen(qd, kd, wqd, wkd, cu, **kw)
    o, _ = seer.bsattn_varlen(qd, kd, vd, cu, mask)
    o_sep = torch.zeros_like(qd)
    torch.cuda.synchronize()
    for b, n in enumerate(LENGTHS):
        if n == 0:
            continue
        qb, kb, vb = _view(qd, cu, b), _view(kd, cu, b), _view(vd, cu, b)
        m = seer.gate(qb, kb, wqd, wkd, **kw)
        seer.bsattn(qb, kb, vb, m, out=_view(o_sep, cu, b))
        torch.cuda.synchronize()
        cnt, idx = mask.sequence(b)
        assert torch.equal(cnt, m.count[0])
        c = m.count[0].cpu().numpy()
        a, bb = idx.cpu().numpy(), m.idx[0].cpu().numpy()
        for h in range(c.shape[0]):
            for i in range(c.shape[1]):
                assert np.array_equal(a[h, i, :c[h, i]], bb[h, i, :c[h, i]])
    assert torch.equal(o.view(torch.int16), o_sep.view(torch.int16))


def test_varlen_attention_on_uploaded_masks_matches_oracle():
    """Caller-made per-sequence masks (random patterns incl. empty rows with forcing off)."""
    lengths = [700, 0, 190, 4096]
    seqs, q, k, v, wq, wk, cu = _packed_inputs(lengths, stable_seed("varlen-up"))
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    rng = np.random.default_rng(5)
    dense_all, counts, idxs = [], [], []
    for n in lengths:
        nb = _nb(n)
        m = (rng.random((HQ, nb, nb)) < 0.3).astype(np.uint8) * np.tril(np.ones((nb, nb), np.uint8))
        dense_all.append(m)
        c = m.sum(-1).astype(np.int32)
        ix = np.zeros((HQ, nb, nb), np.uint16)
        for h in range(HQ):
            for i in range(nb):
                js = np.nonzero(m[h, i])[0]
                ix[h, i, :js.size] = js
        counts.append(c.reshape(-1))
        idxs.append(ix.reshape(-1))
    vm = seer.VarlenMask(count=torch.from_numpy(np.concatenate(counts)).cuda(),
                         idx=torch.from_numpy(np.concatenate(idxs).view(np.int16)).cuda(),
                         cu_seqlens=[int(x) for x in cu], heads=HQ)
    o, _ = seer.bsattn_varlen(qd, kd, vd, cu, vm)
    torch.cuda.synchronize()
    o_np = from_device(o)
    for b, n in enumerate(lengths):
        if n == 0:
            continue
        nb = _nb(n)
        O_ref, _ = oracle.attn(*seqs[b], mask=dense_all[b][None])
        ref = np.nan_to_num(O_ref.reshape(HQ, nb * 64, D)[:, :n])
        got = as_f64(o_np[int(cu[b]):int(cu[b + 1])]).transpose(1, 0, 2)
        assert float(np.abs(got - ref).max()) <= ATOL_BF16
