"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Nothing here re-types the oracle's own formulas: each check compares the oracle
with a closed form, an invariant stated in the paper, a hand-derived fixture
(tests/golden/), a brute force over tiny inputs, or an independent library
routine (torch.nn.functional pooling / scaled_dot_product_attention, in fp64).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from workload import bf16_bits_to_f32, f32_to_bf16_bits, pattern_mask

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def _rand(shape, seed, dtype=np.float32):
    return np.random.default_rng(seed).standard_normal(shape).astype(dtype)


def _as_f64(x):
    return bf16_bits_to_f32(x).astype(np.float64) if x.dtype == np.uint16 else x.astype(np.float64)


# --------------------------------------------------------------------------
# pooling (section 3.1)
# --------------------------------------------------------------------------

def test_pool_constant_block_closed_form():
    x = np.repeat(np.arange(4, dtype=np.float32)[None, None, :, None], 64, axis=2)  # [1,1,256,1]
    x = np.ascontiguousarray(np.repeat(x, 3, axis=3))
    q = oracle.pool(x, 64, oracle.POOL_AVG)
    k = oracle.pool(x, 64, oracle.POOL_MAX_MIN_AVG)
    for i in range(4):
        assert np.all(q[0, 0, i] == i)
        assert np.all(k[0, 0, i] == i)


def test_pool_ramp_closed_form():
    # x[t, d] = a_d + c_d * t inside each block: mean is the midpoint, max and
    # min sit at the block ends (which end depends on the sign of c_d).
    block, nb, D = 64, 3, 4
    a = np.array([0.5, -1.0, 2.0, 0.0])
    c = np.array([0.25, -0.5, 0.0, 1.0])
    t = np.arange(nb * block)
    x = (a[None, :] + c[None, :] * t[:, None]).astype(np.float32)[None, None]
    k = oracle.pool(np.ascontiguousarray(x), block, oracle.POOL_MAX_MIN_AVG)
    for i in range(nb):
        first = a + c * (i * block)
        last = a + c * (i * block + block - 1)
        np.testing.assert_allclose(k[0, 0, i, :D], np.maximum(first, last), rtol=0, atol=0)
        np.testing.assert_allclose(k[0, 0, i, D:2 * D], np.minimum(first, last), rtol=0, atol=0)
        np.testing.assert_allclose(k[0, 0, i, 2 * D:], (first + last) / 2, rtol=1e-15, atol=1e-15)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_pool_matches_torch_pooling(dtype):
    B, H, S, D, blk = 2, 3, 256, 8, 64
    xf = _rand((B, H, S, D), 1)
    x = xf if dtype == "f32" else f32_to_bf16_bits(xf)
    ref = torch.from_numpy(_as_f64(x))  # [B,H,S,D]
    t = ref.permute(0, 1, 3, 2).reshape(B * H, D, S)
    avg = F.avg_pool1d(t, blk, blk).reshape(B, H, D, -1).permute(0, 1, 3, 2)
    mx = F.max_pool1d(t, blk, blk).reshape(B, H, D, -1).permute(0, 1, 3, 2)
    mn = -F.max_pool1d(-t, blk, blk).reshape(B, H, D, -1).permute(0, 1, 3, 2)
    q = oracle.pool(x, blk, oracle.POOL_AVG)
    k = oracle.pool(x, blk, oracle.POOL_MAX_MIN_AVG)
    np.testing.assert_allclose(q, avg.numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_array_equal(k[..., :D], mx.numpy())          # max first
    np.testing.assert_array_equal(k[..., D:2 * D], mn.numpy())     # then min
    np.testing.assert_allclose(k[..., 2 * D:], avg.numpy(), rtol=1e-14, atol=1e-15)  # then avg


def test_pool_128_combines_two_64_halves():
    # a 128-token block pools to max of maxes, min of mins, mean of means of its halves
    x = _rand((2, 3, 512, 8), 4)
    k64 = oracle.pool(x, 64, oracle.POOL_MAX_MIN_AVG)
    k128 = oracle.pool(x, 128, oracle.POOL_MAX_MIN_AVG)
    q64, q128 = oracle.pool(x, 64, oracle.POOL_AVG), oracle.pool(x, 128, oracle.POOL_AVG)
    D = 8
    a, b = k64[:, :, 0::2], k64[:, :, 1::2]
    np.testing.assert_array_equal(k128[..., :D], np.maximum(a[..., :D], b[..., :D]))
    np.testing.assert_array_equal(k128[..., D:2 * D], np.minimum(a[..., D:2 * D], b[..., D:2 * D]))
    np.testing.assert_allclose(k128[..., 2 * D:], (a[..., 2 * D:] + b[..., 2 * D:]) / 2, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(q128, (q64[:, :, 0::2] + q64[:, :, 1::2]) / 2, rtol=1e-14, atol=1e-15)


def test_pool_strided_input_matches_contiguous():
    x = _rand((1, 4, 128, 16), 2)
    view = x[:, ::2]  # non-contiguous head stride
    a = oracle.pool(np.ascontiguousarray(view), 64, oracle.POOL_MAX_MIN_AVG)
    b = oracle.pool(view, 64, oracle.POOL_MAX_MIN_AVG)
    np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("blk", [64, 128])
def test_pool_partial_last_block(blk):
    # a sequence that is not a multiple of the block: the last block pools over
    # the tokens it holds (blocks do not overlap, section 3.1)
    S = 3 * blk + 37
    x = _rand((1, 2, S, 4), 3)
    q = oracle.pool(x, blk, oracle.POOL_AVG)
    k = oracle.pool(x, blk, oracle.POOL_MAX_MIN_AVG)
    assert q.shape[2] == 4 and k.shape[2] == 4
    tail = x[:, :, 3 * blk:].astype(np.float64)
    np.testing.assert_allclose(q[:, :, 3], tail.mean(axis=2), rtol=1e-14, atol=1e-15)
    np.testing.assert_array_equal(k[:, :, 3, :4], tail.max(axis=2))
    np.testing.assert_array_equal(k[:, :, 3, 4:8], tail.min(axis=2))
    np.testing.assert_allclose(k[:, :, 2, 8:], x[:, :, 2 * blk:3 * blk].astype(np.float64).mean(axis=2),
                               rtol=1e-14, atol=1e-15)


@pytest.mark.parametrize("causal", [True, False])
def test_partial_last_block_attention_matches_sdpa(causal):
    B, Hq, Hkv, S, D = 1, 2, 1, 64 * 5 + 23, 16
    q, k, v = _rand((B, Hq, S, D), 51), _rand((B, Hkv, S, D), 52), _rand((B, Hkv, S, D), 53)
    nb = 6
    bm = np.stack([pattern_mask("random", nb, 7 + h, 0.5) for h in range(Hq)])[None]
    bm[..., np.arange(nb), np.arange(nb)] = 1
    O, lse = oracle.attn(q, k, v, mask=bm, causal=causal)
    tok = np.kron(bm, np.ones((64, 64), np.uint8))[..., :S, :S].astype(bool)
    if causal:
        tok &= np.tril(np.ones((S, S), bool))
    ref = _sdpa(q, k, v, attn_mask=torch.from_numpy(tok))
    Of = O.reshape(B, Hq, nb * 64, D)
    np.testing.assert_allclose(Of[:, :, :S], ref, rtol=1e-10, atol=1e-12)
    assert np.isnan(Of[:, :, S:]).all() and np.isnan(lse.reshape(B, Hq, nb * 64)[:, :, S:]).all()


def test_partial_last_block_maxpool_matches_torch_ceil_mode():
    B, Hq, S, D = 1, 2, 64 * 3 + 50, 8
    q, k = _rand((B, Hq, S, D), 54), _rand((B, 1, S, D), 55)
    gt = oracle.maxpool_gt(q, k)
    tq = torch.from_numpy(q.astype(np.float64))
    tk = torch.from_numpy(k.astype(np.float64)).repeat_interleave(Hq, dim=1)
    sc = (tq @ tk.transpose(-1, -2)) / math.sqrt(D)
    sc = sc.masked_fill(~torch.ones(S, S, dtype=torch.bool).tril(), float("-inf"))
    ref = F.max_pool2d(torch.softmax(sc, -1), 64, 64, ceil_mode=True).numpy()
    np.testing.assert_allclose(gt, ref, rtol=1e-12, atol=0)


def test_partial_last_block_distill_gradients():
    rng = np.random.default_rng(56)
    S, D, Dg = 64 * 3 + 29, 16, 8
    q = rng.standard_normal((1, 2, S, D)).astype(np.float32)
    k = rng.standard_normal((1, 1, S, D)).astype(np.float32)
    wq, wk = rng.standard_normal((2, D, Dg)) * 0.4, rng.standard_normal((1, 3 * D, Dg)) * 0.4
    gt = oracle.maxpool_gt(q, k)
    loss, dwq, dwk = oracle.distill(q, k, wq, wk, gt)
    h = 1e-6
    for idx in [(0, 3, 2), (1, 15, 7)]:
        Wp, Wm = wq.copy(), wq.copy()
        Wp[idx] += h
        Wm[idx] -= h
        fd = (oracle.distill(q, k, Wp, wk, gt)[0] - oracle.distill(q, k, Wm, wk, gt)[0]) / (2 * h)
        assert abs(fd - dwq[idx]) <= 1e-6 * max(1e-3, abs(fd)) + 1e-9


# --------------------------------------------------------------------------
# gate (Eq. 1)
# --------------------------------------------------------------------------

def test_gate_hand_fixture():
    g = json.load(open(os.path.join(GOLDEN, "tiny_gate.json")))
    blk = g["block"]
    q = np.asarray(g["q"], dtype=np.float32)[None, None]
    k = np.asarray(g["k"], dtype=np.float32)[None, None]
    wq = np.asarray(g["wq"], dtype=np.float32)[None]
    wk = np.asarray(g["wk"], dtype=np.float32)[None]
    qp = oracle.pool(q, blk, oracle.POOL_AVG)
    kp = oracle.pool(k, blk, oracle.POOL_MAX_MIN_AVG)
    np.testing.assert_array_equal(qp[0, 0], np.asarray(g["pooled_q"], dtype=np.float64))
    np.testing.assert_array_equal(kp[0, 0], np.asarray(g["pooled_k"], dtype=np.float64))
    qg = oracle.linear(qp, wq)
    kg = oracle.linear(kp, wk)
    np.testing.assert_array_equal(qg[0, 0], np.asarray(g["qg"], dtype=np.float64))
    np.testing.assert_array_equal(kg[0, 0], np.asarray(g["kg"], dtype=np.float64))
    L = oracle.gate_logits(qg, kg)
    env = {"sqrt": math.sqrt, "exp": math.exp, "inf": math.inf}
    want_L = np.array([[eval(s, env) for s in row] for row in g["logits"]])
    np.testing.assert_allclose(L[0, 0], want_L, rtol=1e-15)
    ell = oracle.gate_logscore(L)
    want_P = np.array([[eval(s, env) for s in row] for row in g["probs"]])
    np.testing.assert_allclose(np.exp(ell[0, 0]), want_P, rtol=1e-14, atol=0)
    sel = oracle.select(ell, oracle.TOPK_FIXED, k=1, keep_first=0, keep_diag=0)
    np.testing.assert_array_equal(sel["mask"][0, 0], g["topk_fixed_k1_no_forcing"])
    for key, thr, kd in [("threshold_0p5_no_forcing", 0.5, 0), ("threshold_0p1_no_forcing", 0.1, 0),
                         ("threshold_0p5_keep_diag", 0.5, 1)]:
        sel = oracle.select(ell, oracle.THRESHOLD, thresholds=np.float32(thr), keep_first=0, keep_diag=kd)
        np.testing.assert_array_equal(sel["mask"][0, 0], g[key], err_msg=key)


def _torch_gate_special(q, k, part):
    """Gate with Wq = I and Wk selecting one pooled part of K, built from torch ops."""
    B, H, S, D = q.shape
    blk = 64
    tq = torch.from_numpy(_as_f64(q)).permute(0, 1, 3, 2).reshape(B * H, D, S)
    tk = torch.from_numpy(_as_f64(k)).permute(0, 1, 3, 2).reshape(B * H, D, S)
    qp = F.avg_pool1d(tq, blk, blk).reshape(B, H, D, -1).transpose(-1, -2)
    if part == 0:
        kp = F.max_pool1d(tk, blk, blk)
    elif part == 1:
        kp = -F.max_pool1d(-tk, blk, blk)
    else:
        kp = F.avg_pool1d(tk, blk, blk)
    kp = kp.reshape(B, H, D, -1).transpose(-1, -2)
    logits = qp @ kp.transpose(-1, -2) / math.sqrt(D)
    nb = S // blk
    causal = torch.ones(nb, nb, dtype=torch.bool).tril()
    logits = logits.masked_fill(~causal, float("-inf"))
    return torch.softmax(logits, dim=-1).numpy()


@pytest.mark.parametrize("part", [0, 1, 2])  # which slot of max | min | avg Wk reads
def test_gate_reduces_to_pooled_attention(part):
    B, H, S, D = 1, 2, 512, 16
    q = _rand((B, H, S, D), 10 + part)
    k = _rand((B, H, S, D), 20 + part)
    wq = np.broadcast_to(np.eye(D, dtype=np.float32), (H, D, D)).copy()
    wk = np.zeros((H, 3 * D, D), dtype=np.float32)
    wk[:, part * D:(part + 1) * D, :] = np.eye(D, dtype=np.float32)
    L, ell = oracle.gate(q, k, wq, wk)
    ref = _torch_gate_special(q, k, part)
    np.testing.assert_allclose(np.exp(ell), ref, rtol=1e-12, atol=1e-300)


def test_gate_rows_sum_to_one_and_size():
    # the gate output of a head is [seq/B, seq/B], 1/4096 of the attention map at
    # B = 64 (section 3.1); every softmax row sums to 1 (section 3.2)
    B, Hq, Hkv, S, D, Dg = 1, 4, 2, 1024, 32, 24
    q, k = _rand((B, Hq, S, D), 5), _rand((B, Hkv, S, D), 6)
    wq, wk = _rand((Hq, D, Dg), 7) * 0.3, _rand((Hkv, 3 * D, Dg), 8) * 0.3
    L, ell = oracle.gate(q, k, wq, wk)
    assert L.shape[-2] * L.shape[-1] * 4096 == S * S
    np.testing.assert_allclose(np.exp(ell).sum(-1), 1.0, rtol=1e-13)
    assert np.all(np.isneginf(np.triu(L[0, 0], 1)[np.triu_indices(16, 1)]))


def test_gate_gqa_equals_replicated_kv():
    B, Hq, Hkv, S, D, Dg = 1, 6, 2, 256, 16, 8
    q, k = _rand((B, Hq, S, D), 30), _rand((B, Hkv, S, D), 31)
    wq, wk = _rand((Hq, D, Dg), 32), _rand((Hkv, 3 * D, Dg), 33)
    L, _ = oracle.gate(q, k, wq, wk)
    k_rep = np.ascontiguousarray(np.repeat(k, Hq // Hkv, axis=1))
    wk_rep = np.ascontiguousarray(np.repeat(wk, Hq // Hkv, axis=0))
    L_rep, _ = oracle.gate(q, k_rep, wq, wk_rep)
    np.testing.assert_array_equal(L, L_rep)


def test_gate_shared_weights_equal_tiled_weights():
    B, H, S, D, Dg = 1, 3, 256, 8, 8
    x = _rand((B, H, S, D), 40)
    w = _rand((1, D, Dg), 41)
    a = oracle.linear(oracle.pool(x, 64, oracle.POOL_AVG), w, w_per_head=False)
    b = oracle.linear(oracle.pool(x, 64, oracle.POOL_AVG), np.repeat(w, H, axis=0), w_per_head=True)
    np.testing.assert_array_equal(a, b)
    ref = np.einsum("bhnc,cd->bhnd", oracle.pool(x, 64, oracle.POOL_AVG), w[0].astype(np.float64))
    np.testing.assert_allclose(a, ref, rtol=1e-13, atol=1e-15)


# --------------------------------------------------------------------------
# selection (Eq. 3 / Eq. 4)
# --------------------------------------------------------------------------

def _rand_ell(B, H, nb, seed, ties=False):
    rng = np.random.default_rng(seed)
    L = rng.standard_normal((B, H, nb, nb))
    if ties:
        L = np.round(L * 2) / 2  # many exact ties
    L = np.where(np.tril(np.ones((nb, nb), bool)), L, -np.inf)
    return oracle.gate_logscore(L)


def test_topk_schedule_fixture():
    g = json.load(open(os.path.join(GOLDEN, "topk_schedule.json")))
    nb = g["n_blocks"]
    ell = _rand_ell(1, 2, nb, 50)
    sel = oracle.select(ell, oracle.TOPK_RATIO, rho=g["ratio"])
    for h in range(2):
        np.testing.assert_array_equal(sel["count"][0, h], g["k"])
        assert int(sel["mask"][0, h].sum()) == g["total"]
    assert nb * (nb + 1) // 2 == g["causal_total"]


@pytest.mark.parametrize("kf,kd", [(1, 1), (0, 0), (1, 0), (0, 1)])
@pytest.mark.parametrize("ties", [False, True])
def test_topk_brute_force(kf, kd, ties):
    nb = 8
    ell = _rand_ell(1, 3, nb, 60 + kf + 2 * kd, ties=ties)
    for k in range(1, nb + 1):
        sel = oracle.select(ell, oracle.TOPK_FIXED, k=k, keep_first=kf, keep_diag=kd)
        for h in range(3):
            for i in range(nb):
                forced = set()
                if kf:
                    forced.add(0)
                if kd:
                    forced.add(i)
                kk = min(i + 1, max(len(forced), k))
                cands = [j for j in range(i + 1) if j not in forced]
                best = None
                for subset in itertools.combinations(cands, kk - len(forced)):
                    # rank: values descending, then indices ascending on ties
                    key = sorted(((-ell[0, h, i, j], j) for j in subset))
                    if best is None or key < best[0]:
                        best = (key, subset)
                want = np.zeros(nb, np.uint8)
                want[list(forced | set(best[1]))] = 1
                np.testing.assert_array_equal(sel["mask"][0, h, i], want, err_msg=f"k={k} h={h} i={i}")
                assert sel["count"][0, h, i] == kk


def test_topk_ratio_one_keeps_all_causal_blocks():
    nb = 12
    sel = oracle.select(_rand_ell(1, 2, nb, 70), oracle.TOPK_RATIO, rho=1.0)
    np.testing.assert_array_equal(sel["mask"][0, 0], np.tril(np.ones((nb, nb), np.uint8)))


def test_topk_nested_in_k():
    nb = 16
    ell = _rand_ell(1, 2, nb, 71)
    prev = None
    for k in range(1, nb + 1):
        m = oracle.select(ell, oracle.TOPK_FIXED, k=k)["mask"]
        if prev is not None:
            assert np.all(prev <= m)
        prev = m


def test_select_idx_is_ascending_compaction_of_mask():
    nb = 20
    ell = _rand_ell(2, 3, nb, 72)
    for sel in (oracle.select(ell, oracle.TOPK_RATIO, rho=0.3),
                oracle.select(ell, oracle.THRESHOLD, thresholds=np.float32(0.05))):
        for b, h, i in itertools.product(range(2), range(3), range(nb)):
            c = sel["count"][b, h, i]
            np.testing.assert_array_equal(sel["idx"][b, h, i, :c], np.nonzero(sel["mask"][b, h, i])[0])


def test_threshold_monotone_and_limits():
    nb = 24
    ell = _rand_ell(1, 4, nb, 80)
    causal = np.tril(np.ones((nb, nb), np.uint8))
    prev = None
    for thr in [1e-30, 1e-4, 1e-3, 1e-2, 0.05, 0.2, 0.5, 1.0]:
        m = oracle.select(ell, oracle.THRESHOLD, thresholds=np.float32(thr))["mask"]
        if prev is not None:
            assert np.all(m <= prev)
        prev = m
    tiny = oracle.select(ell, oracle.THRESHOLD, thresholds=np.float32(1e-30))["mask"]
    np.testing.assert_array_equal(tiny[0, 0], causal)
    one = oracle.select(ell, oracle.THRESHOLD, thresholds=np.float32(1.0))["mask"]
    forced = np.zeros((nb, nb), np.uint8)
    forced[:, 0] = 1
    forced[np.arange(nb), np.arange(nb)] = 1
    np.testing.assert_array_equal(one[0, 2], forced)
    # Eq. 4 is a strict comparison: row 0 has a single causal block whose
    # probability is exactly 1, so a threshold of 1 keeps nothing unforced
    none = oracle.select(ell, oracle.THRESHOLD, thresholds=np.float32(1.0), keep_first=0, keep_diag=0)
    assert none["mask"].sum() == 0 and np.all(none["count"] == 0)


def test_threshold_per_head_equals_global_per_head():
    nb = 16
    ell = _rand_ell(1, 4, nb, 81)
    thr = np.array([1e-3, 0.02, 0.1, 0.3], np.float32)
    per = oracle.select(ell, oracle.THRESHOLD, thresholds=thr)["mask"]
    for h in range(4):
        one = oracle.select(ell, oracle.THRESHOLD, thresholds=thr[h])["mask"]
        np.testing.assert_array_equal(per[0, h], one[0, h])


# --------------------------------------------------------------------------
# masked causal attention (section 3.3) and the dense path
# --------------------------------------------------------------------------

def _sdpa(q, k, v, attn_mask=None, causal=False):
    Hq, Hkv = q.shape[1], k.shape[1]
    tq = torch.from_numpy(_as_f64(q))
    tk = torch.from_numpy(_as_f64(k)).repeat_interleave(Hq // Hkv, dim=1)
    tv = torch.from_numpy(_as_f64(v)).repeat_interleave(Hq // Hkv, dim=1)
    return F.scaled_dot_product_attention(tq, tk, tv, attn_mask=attn_mask, is_causal=causal).numpy()


def _o_full(O, B, H, S, D):
    return O.reshape(B, H, S, D)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("Hq,Hkv", [(2, 2), (4, 1), (6, 2)])
def test_dense_causal_matches_sdpa(dtype, Hq, Hkv):
    B, S, D = 1, 256, 32
    mk = (lambda x: x) if dtype == "f32" else f32_to_bf16_bits
    q, k, v = (mk(_rand((B, h, S, D), s)) for h, s in [(Hq, 1), (Hkv, 2), (Hkv, 3)])
    O, lse = oracle.attn(q, k, v)
    ref = _sdpa(q, k, v, causal=True)
    np.testing.assert_allclose(_o_full(O, B, Hq, S, D), ref, rtol=1e-10, atol=1e-12)
    # an all-ones block mask is the same thing
    ones = np.ones((B, Hq, S // 64, S // 64), np.uint8)
    O1, lse1 = oracle.attn(q, k, v, mask=ones)
    np.testing.assert_array_equal(O1, O)
    np.testing.assert_array_equal(lse1, lse)


def test_dense_noncausal_matches_sdpa():
    B, H, S, D = 1, 2, 192, 16
    q, k, v = (_rand((B, H, S, D), s) for s in (4, 5, 6))
    O, _ = oracle.attn(q, k, v, causal=False)
    np.testing.assert_allclose(_o_full(O, B, H, S, D), _sdpa(q, k, v), rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("blk", [64, 128])
@pytest.mark.parametrize("kind", ["a_shape", "vertical", "slash", "random"])
def test_block_masked_matches_sdpa_with_token_mask(kind, blk):
    B, Hq, Hkv, S, D = 1, 4, 2, 512, 16
    nb = S // blk
    q, k, v = _rand((B, Hq, S, D), 7), _rand((B, Hkv, S, D), 8), _rand((B, Hkv, S, D), 9)
    bm = np.stack([pattern_mask(kind, nb, 100 + h, 0.3) for h in range(Hq)])[None]
    bm[..., np.arange(nb), np.arange(nb)] = 1  # keep the diagonal so no row is empty
    O, lse = oracle.attn(q, k, v, mask=bm, block=blk)
    tok = np.kron(bm, np.ones((blk, blk), np.uint8)).astype(bool) & np.tril(np.ones((S, S), bool))
    ref = _sdpa(q, k, v, attn_mask=torch.from_numpy(tok))
    np.testing.assert_allclose(_o_full(O, B, Hq, S, D), ref, rtol=1e-10, atol=1e-12)
    # LSE against torch.logsumexp of the masked score matrix
    tq = torch.from_numpy(q.astype(np.float64))
    tk = torch.from_numpy(k.astype(np.float64)).repeat_interleave(Hq // Hkv, dim=1)
    sc = (tq @ tk.transpose(-1, -2)) / math.sqrt(D)
    sc = sc.masked_fill(~torch.from_numpy(tok), float("-inf"))
    np.testing.assert_allclose(lse.reshape(B, Hq, S), torch.logsumexp(sc, -1).numpy(), rtol=1e-12)


def test_constant_v_gives_constant_output():
    B, Hq, Hkv, S, D = 1, 2, 1, 256, 8
    q, k = _rand((B, Hq, S, D), 11), _rand((B, Hkv, S, D), 12)
    v = np.broadcast_to(np.linspace(-2, 3, D, dtype=np.float32), (B, Hkv, S, D)).copy()
    bm = np.stack([pattern_mask("random", 4, h, 0.5) for h in range(Hq)])[None]
    bm[..., np.arange(4), np.arange(4)] = 1
    O, _ = oracle.attn(q, k, v, mask=bm)
    np.testing.assert_allclose(O, np.broadcast_to(v[0, 0, 0], O.shape), rtol=1e-14, atol=1e-14)


def test_diagonal_only_mask_is_local_attention():
    # only the diagonal 64-block: each query sees keys of its own block up to itself
    B, H, S, D, blk = 1, 1, 256, 8, 64
    q, k, v = (_rand((B, H, S, D), s) for s in (13, 14, 15))
    bm = np.eye(S // blk, dtype=np.uint8)[None, None]
    O, _ = oracle.attn(q, k, v, mask=bm)
    for i in range(S // blk):
        sl = slice(i * blk, (i + 1) * blk)
        ref = _sdpa(q[:, :, sl], k[:, :, sl], v[:, :, sl], causal=True)
        np.testing.assert_allclose(O[i], ref[0, 0], rtol=1e-10, atol=1e-12)


def test_empty_row_gives_zero_and_neg_inf():
    B, H, S, D = 1, 1, 256, 8
    q, k, v = (_rand((B, H, S, D), s) for s in (16, 17, 18))
    bm = np.tril(np.ones((4, 4), np.uint8))[None, None].copy()
    bm[0, 0, 2, :] = 0
    O, lse = oracle.attn(q, k, v, mask=bm)
    assert np.all(O[2] == 0.0) and np.all(np.isneginf(lse[2]))
    assert np.all(np.isfinite(lse[[0, 1, 3]]))


def test_gqa_attention_equals_replicated_kv():
    B, Hq, Hkv, S, D = 1, 4, 2, 256, 16
    q, k, v = _rand((B, Hq, S, D), 19), _rand((B, Hkv, S, D), 20), _rand((B, Hkv, S, D), 21)
    bm = np.stack([pattern_mask("vertical", 4, h, 0.5) for h in range(Hq)])[None]
    a, la = oracle.attn(q, k, v, mask=bm)
    rep = lambda x: np.ascontiguousarray(np.repeat(x, Hq // Hkv, axis=1))
    b, lb = oracle.attn(q, rep(k), rep(v), mask=bm)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(la, lb)


def test_row_subset_equals_full():
    B, Hq, Hkv, S, D = 2, 2, 1, 256, 8
    q, k, v = _rand((B, Hq, S, D), 22), _rand((B, Hkv, S, D), 23), _rand((B, Hkv, S, D), 24)
    Ofull, lfull = oracle.attn(q, k, v)
    rows = np.array([[1, 1, 3], [0, 0, 0], [1, 0, 2]], np.int32)
    O, l = oracle.attn(q, k, v, rows=rows)
    for r, (b, h, i) in enumerate(rows):
        flat = (b * Hq + h) * (S // 64) + i
        np.testing.assert_array_equal(O[r], Ofull[flat])
        np.testing.assert_array_equal(l[r], lfull[flat])


# --------------------------------------------------------------------------
# distillation target (Eq. 2)
# --------------------------------------------------------------------------

def test_maxpool_gt_matches_torch():
    B, Hq, Hkv, S, D, blk = 1, 2, 1, 256, 16, 64
    q, k = _rand((B, Hq, S, D), 25), _rand((B, Hkv, S, D), 26)
    gt = oracle.maxpool_gt(q, k)
    tq = torch.from_numpy(q.astype(np.float64))
    tk = torch.from_numpy(k.astype(np.float64)).repeat_interleave(2, dim=1)
    sc = (tq @ tk.transpose(-1, -2)) / math.sqrt(D)
    sc = sc.masked_fill(~torch.ones(S, S, dtype=torch.bool).tril(), float("-inf"))
    p = torch.softmax(sc, -1)
    ref = F.max_pool2d(p, blk, blk).numpy()
    np.testing.assert_allclose(gt, ref, rtol=1e-12, atol=0)


def test_maxpool_gt_noncausal_matches_torch_and_rows_subset():
    B, Hq, Hkv, S, D, blk = 2, 3, 1, 192, 8, 64
    q, k = _rand((B, Hq, S, D), 27), _rand((B, Hkv, S, D), 28)
    gt = oracle.maxpool_gt(q, k, causal=False)
    tq = torch.from_numpy(q.astype(np.float64))
    tk = torch.from_numpy(k.astype(np.float64)).repeat_interleave(Hq, dim=1)
    p = torch.softmax((tq @ tk.transpose(-1, -2)) / math.sqrt(D), -1)
    ref = F.max_pool2d(p, blk, blk).numpy()
    np.testing.assert_allclose(gt, ref, rtol=1e-12, atol=0)
    # a row subset in any order returns those rows of the full map
    rows = np.array([[1, 2, 0], [0, 0, 2], [1, 0, 1]], np.int32)
    sub = oracle.maxpool_gt(q, k, causal=False, rows=rows)
    np.testing.assert_array_equal(sub, gt[rows[:, 0], rows[:, 1], rows[:, 2]])


def test_maxpool_gt_uniform_attention_closed_form():
    # K = 0 makes every visible score equal: query t spreads 1/(t+1) uniformly,
    # so tile (i, j <= i) pools to its first query's 1/(64 i + 1); j > i is 0
    B, Hq, S, D, blk = 1, 1, 320, 16, 64
    q = _rand((B, Hq, S, D), 29)
    k = np.zeros((B, Hq, S, D), np.float32)
    gt = oracle.maxpool_gt(q, k)[0, 0]
    nb = S // blk
    want = np.tril(np.ones((nb, nb))) / (blk * np.arange(nb) + 1.0)[:, None]
    np.testing.assert_allclose(gt, want, rtol=1e-14, atol=0)


# --------------------------------------------------------------------------
# block-level RoPE in the gate (section 3.1)
# --------------------------------------------------------------------------

def test_block_rope_matches_complex_rotation():
    # independent formulation: plane (d, d + Dg/2) as the complex number
    # x_d + i x_{d+Dg/2}, multiplied by exp(i * pos * (theta/B)^(-2d/Dg))
    B, H, nb, Dg, theta, blk = 1, 2, 37, 16, 500000.0, 64
    x = np.random.default_rng(90).standard_normal((B, H, nb, Dg))
    y = oracle.block_rope(x, theta, blk)
    half = Dg // 2
    z = x[..., :half] + 1j * x[..., half:]
    w = (theta / blk) ** (-2.0 * np.arange(half) / Dg)
    rot = np.exp(1j * np.arange(nb)[:, None] * w[None, :])
    zr = z * rot
    np.testing.assert_allclose(y[..., :half], zr.real, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y[..., half:], zr.imag, rtol=1e-12, atol=1e-12)


def test_block_rope_invariants():
    B, H, nb, Dg = 1, 3, 50, 32
    x = np.random.default_rng(91).standard_normal((B, H, nb, Dg))
    y = oracle.block_rope(x, 10000.0, 64)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    np.testing.assert_array_equal(y[..., 0, :], x[..., 0, :])  # position 0 is not rotated


def test_block_rope_logits_depend_on_relative_position_only():
    # identical rows for every block: the rotated logits depend on i - j only
    B, Hq, Hkv, nb, Dg = 1, 2, 1, 40, 16
    rng = np.random.default_rng(92)
    qg = np.broadcast_to(rng.standard_normal(Dg), (B, Hq, nb, Dg)).copy()
    kg = np.broadcast_to(rng.standard_normal(Dg), (B, Hkv, nb, Dg)).copy()
    L = oracle.gate_logits(oracle.block_rope(qg, 500000.0), oracle.block_rope(kg, 500000.0))
    for d in range(nb):
        diag = np.diagonal(L[0, 0], offset=-d)
        np.testing.assert_allclose(diag, diag[0], rtol=1e-11, atol=1e-12)
    assert np.ptp(L[0, 0][np.tril_indices(nb)]) > 1e-3  # and does vary with i - j


def test_gate_with_rope_equals_manual_composition():
    B, Hq, Hkv, S, D, Dg = 1, 2, 1, 512, 16, 8
    q, k = _rand((B, Hq, S, D), 93), _rand((B, Hkv, S, D), 94)
    wq, wk = _rand((Hq, D, Dg), 95), _rand((Hkv, 3 * D, Dg), 96)
    L, _ = oracle.gate(q, k, wq, wk, rope_theta=500000.0)
    qg = oracle.block_rope(oracle.linear(oracle.pool(q, 64, oracle.POOL_AVG), wq), 500000.0)
    kg = oracle.block_rope(oracle.linear(oracle.pool(k, 64, oracle.POOL_MAX_MIN_AVG), wk), 500000.0)
    np.testing.assert_array_equal(L, oracle.gate_logits(qg, kg))


# --------------------------------------------------------------------------
# gate distillation step (Eq. 2): KL(gt || score) and weight gradients
# --------------------------------------------------------------------------

def _distill_case(seed, Hq=2, Hkv=1, S=256, D=16, Dg=8, per_head=True):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((1, Hq, S, D)).astype(np.float32)
    k = rng.standard_normal((1, Hkv, S, D)).astype(np.float32)
    nw_q, nw_k = (Hq, Hkv) if per_head else (1, 1)
    wq = rng.standard_normal((nw_q, D, Dg)) * 0.4
    wk = rng.standard_normal((nw_k, 3 * D, Dg)) * 0.4
    gt = oracle.maxpool_gt(q, k)
    return q, k, wq, wk, gt


@pytest.mark.parametrize("per_head,theta", [(True, 0.0), (True, 10000.0), (False, 0.0), (False, 500000.0)])
def test_distill_gradients_match_finite_differences(per_head, theta):
    q, k, wq, wk, gt = _distill_case(31 + int(per_head), per_head=per_head)
    loss, dwq, dwk = oracle.distill(q, k, wq, wk, gt, w_per_head=per_head, rope_theta=theta)
    assert loss > 0
    rng = np.random.default_rng(5)
    h = 1e-6
    for W, dW, which in ((wq, dwq, "q"), (wk, dwk, "k")):
        for _ in range(12):
            idx = tuple(int(rng.integers(n)) for n in W.shape)
            Wp, Wm = W.copy(), W.copy()
            Wp[idx] += h
            Wm[idx] -= h
            args = lambda X: (X, wk) if which == "q" else (wq, X)
            lp = oracle.distill(q, k, *args(Wp), gt, w_per_head=per_head, rope_theta=theta)[0]
            lm = oracle.distill(q, k, *args(Wm), gt, w_per_head=per_head, rope_theta=theta)[0]
            fd = (lp - lm) / (2 * h)
            assert abs(fd - dW[idx]) <= 1e-6 * max(1e-3, abs(fd)) + 1e-9, (which, idx, fd, dW[idx])


def test_distill_loss_matches_torch_kl_div_on_the_gate_softmax():
    # P from the C gate oracle (an independent path), KL from torch's kl_div
    q, k, wq, wk, gt = _distill_case(41)
    loss = oracle.distill(q, k, wq, wk, gt)[0]
    _, ell = oracle.gate(q, k, wq.astype(np.float32), wk.astype(np.float32))
    nb = ell.shape[-1]
    tri = np.tril(np.ones((nb, nb), bool))
    T = np.where(tri, gt, 0.0)
    T = T / T.sum(-1, keepdims=True)
    logp = torch.from_numpy(np.where(tri, ell, -1e300))
    kl = F.kl_div(logp, torch.from_numpy(T), reduction="sum").item() / (ell.size // nb)
    # weights rounded to fp32 for the C path: compare with the same rounding
    loss32 = oracle.distill(q, k, wq.astype(np.float32), wk.astype(np.float32), gt)[0]
    assert abs(kl - loss32) <= 1e-12 * max(1.0, kl)
    assert abs(loss - loss32) < 1e-3 * loss


def test_distill_zero_at_the_optimum_and_descent():
    q, k, wq, wk, _ = _distill_case(43)
    _, ell = oracle.gate(q, k, wq.astype(np.float32), wk.astype(np.float32))
    nb = ell.shape[-1]
    tri = np.tril(np.ones((nb, nb), bool))
    target = np.where(tri, np.exp(ell), 0.0) * 0.37  # any positive row scale: rows renormalise
    w32q, w32k = wq.astype(np.float32).astype(np.float64), wk.astype(np.float32).astype(np.float64)
    loss, dwq, dwk = oracle.distill(q, k, w32q, w32k, target)
    assert abs(loss) < 1e-13
    assert np.abs(dwq).max() < 1e-12 and np.abs(dwk).max() < 1e-12
    # away from the optimum a small step against the gradient lowers the loss
    q2, k2, wq2, wk2, gt2 = _distill_case(44)
    l0, gq, gk = oracle.distill(q2, k2, wq2, wk2, gt2)
    l1 = oracle.distill(q2, k2, wq2 - 1e-2 * gq / np.abs(gq).max(), wk2 - 1e-2 * gk / np.abs(gk).max(), gt2)[0]
    assert l1 < l0


# --------------------------------------------------------------------------
# shared-mask variant: one mask per KV group, scored by the mean of the
# group's head probabilities (the paper's gate is per head, section 3.1)
# --------------------------------------------------------------------------

def test_group_select_hand_fixture():
    g = json.load(open(os.path.join(GOLDEN, "group_select.json")))
    nb, i = g["n_blocks"], g["row"]
    ell = np.full((1, g["heads_q"], nb, nb), -np.inf)
    for h in range(g["heads_q"]):
        for r in range(nb):  # rows other than the asserted one: uniform over their causal blocks
            ell[0, h, r, :r + 1] = -math.log(r + 1)
    ell[0, 0, i, :] = np.log(g["p_head0"])
    ell[0, 1, i, :] = np.log(g["p_head1"])
    ellg = oracle.group_logscore(ell, g["heads_kv"])
    modes = {"topk_fixed": oracle.TOPK_FIXED, "topk_ratio": oracle.TOPK_RATIO, "threshold": oracle.THRESHOLD}
    for c in g["cases"]:
        sel = oracle.select(ellg, modes[c["mode"]], rho=c.get("rho", 0.0), k=c.get("k", 0),
                            thresholds=np.array([c.get("threshold", 0.0)], np.float32),
                            keep_first=c["keep_first"], keep_diag=c["keep_diag"])
        want = np.zeros(nb, np.uint8)
        want[c["selected"]] = 1
        np.testing.assert_array_equal(sel["mask"][0, 0, i], want, err_msg=str(c))


def test_group_score_of_one_head_is_the_head_score():
    ell = oracle.gate_logscore(_rand((2, 3, 9, 9), 80).astype(np.float64) + np.triu(np.full((9, 9), -np.inf), 1))
    np.testing.assert_array_equal(oracle.group_logscore(ell, 3), ell)
    for mode, kw in ((oracle.TOPK_RATIO, dict(rho=0.4)), (oracle.THRESHOLD, dict(thresholds=np.float32(0.1)))):
        a = oracle.select(oracle.group_logscore(ell, 3), mode, **kw)
        b = oracle.select(ell, mode, **kw)
        np.testing.assert_array_equal(a["mask"], b["mask"])


def test_group_score_of_identical_heads_and_row_sums():
    nb = 11
    tri = np.triu(np.full((nb, nb), -np.inf), 1)
    one = oracle.gate_logscore(_rand((1, 2, nb, nb), 81).astype(np.float64) + tri)
    ell = np.repeat(one, 4, axis=1)  # 2 KV groups of 4 identical heads
    ellg = oracle.group_logscore(ell, 2)
    np.testing.assert_allclose(ellg, one, rtol=0, atol=1e-13)
    # the group's scores are a distribution over the causal blocks of each row
    mixed = oracle.gate_logscore(_rand((1, 8, nb, nb), 82).astype(np.float64) + tri)
    p = np.exp(oracle.group_logscore(mixed, 2))
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=0, atol=1e-12)
    assert np.all(p[..., np.triu_indices(nb, 1)[0], np.triu_indices(nb, 1)[1]] == 0)
