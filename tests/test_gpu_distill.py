"""GPU parity of the gate distillation step (seer_gate_distill; section 3.2,
Eq. 2) against the fp64 oracle: the mean KL(renormalised gt || gate softmax)
and the gradients of the gate weights.

Bars: the loss within DIST_RTOL relative; each gradient within GRAD_RTOL of the
largest oracle gradient entry (fp32-accurate forward logits and products against an
fp64 reference), and every entry of at least ELEM_FLOOR of the largest within
ELEM_RTOL of its own value.  The ground truth fed to both sides is seeded synthetic data in
[0, 1] with exact zeros and one all-zero row, stored as fp32."""
import numpy as np
import pytest

import oracle
from helpers import small_inputs, stable_seed, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")

DIST_RTOL = 1e-4
GRAD_RTOL = 2e-4

# Element-wise bar beside the max-scaled one: every gradient entry of at least
# 1% of the largest is within 0.1% of the oracle's value, so small entries are
# checked on their own scale too (measured: 0.5-10e-6 of the largest entry, and
# 2e-5 to 7.2e-4 relative at the floor, the largest at nb = 65; the same with
# fp32-MFMA products, so the fp32 forward sets them).
ELEM_FLOOR = 1e-2
ELEM_RTOL = 1e-3


def _check_grad_elementwise(g, ref, rtol=ELEM_RTOL):
    top = float(np.abs(ref).max())
    if top == 0.0:  # (a single block: every gradient is exactly zero, checked above)
        return
    big = np.abs(ref) >= ELEM_FLOOR * top
    rel = np.abs(g[big] - ref[big]) / np.abs(ref[big])
    print(f"[distill] element-wise relative error {float(rel.max()):.3e} over {int(big.sum())} entries",
          flush=True)
    assert float(rel.max()) <= rtol, float(rel.max())


CASES = [
    # B, Hq, Hkv, S, D, dtype, Dg, per_head, rope_theta
    (1, 2, 1, 1024, 64, "f32", 64, True, 0.0),
    (2, 4, 2, 640, 128, "bf16", 128, True, 0.0),
    (1, 4, 1, 1280, 128, "bf16", 64, False, 10000.0),
    (1, 3, 3, 448, 64, "bf16", 32, True, 500000.0),
    (1, 2, 1, 64, 128, "bf16", 64, True, 0.0),       # a single block
    (1, 4, 1, 4160, 128, "bf16", 128, True, 0.0),    # nb = 65: ragged GEMM tiles
    (2, 2, 1, 576, 128, "f32", 128, False, 0.0),
]


def synthetic_gt(B, Hq, nb, seed):
    """Seeded 2D-max-pool-like target: causal rows of values in (0, 1] with a
    strong diagonal, ~10% exact zeros, and row (0, 0, nb - 1) all zero."""
    rng = np.random.default_rng(seed)
    g = np.exp(-3.0 * np.abs(rng.standard_normal((B, Hq, nb, nb))))
    g[rng.random(g.shape) < 0.1] = 0.0
    idx = np.arange(nb)
    g[..., idx, idx] = 1.0
    g *= np.tril(np.ones((nb, nb)))
    g[0, 0, nb - 1, :] = 0.0
    return g.astype(np.float32)


def _weights(B, Hq, Hkv, D, Dg, per_head, seed):
    rng = np.random.default_rng(seed)
    nq, nk = (Hq, Hkv) if per_head else (1, 1)
    wq = (rng.standard_normal((nq, D, Dg)) / np.sqrt(D)).astype(np.float32)
    wk = (rng.standard_normal((nk, 3 * D, Dg)) / np.sqrt(3 * D)).astype(np.float32)
    return wq, wk


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("opts", [None, {"gemm_min_chunks": 1}, {"gemm_tile_n": 128},
                                  {"gemm_tile_n": 128, "gemm_min_chunks": 1}],
                         ids=["default", "split", "wide", "wide_split"])
def test_gate_distill_parity(case, opts):
    """`split`: every backward product cut into as many K parts as it has
    K chunks (empty parts included), summed by the reduction kernel.  `wide`:
    128-column output tiles for every product (ragged where gate_dim < 128),
    which the default takes only for long rows at gate_dim 128."""
    B, Hq, Hkv, S, D, dt, Dg, per_head, theta = case
    seed = stable_seed(case, "distill")
    _, q, k, _, _, _ = small_inputs(B, Hq, Hkv, S, D, dt, seed=seed, spikes=True)
    wq, wk = _weights(B, Hq, Hkv, D, Dg, per_head, seed + 1)
    nb = S // 64
    gt = synthetic_gt(B, Hq, nb, seed + 2)
    print(f"[distill] case {case}", flush=True)
    qd, kd = to_device(q), to_device(k)
    loss, dwq, dwk = seer.gate_distill(qd, kd, torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda(),
                                       torch.from_numpy(gt).cuda(), w_per_head=per_head, rope_theta=theta,
                                       opts=opts)
    torch.cuda.synchronize()
    l_ref, dwq_ref, dwk_ref = oracle.distill(q, k, wq, wk, gt, w_per_head=per_head, rope_theta=theta)
    l_gpu = float(loss.item())
    assert abs(l_gpu - l_ref) <= DIST_RTOL * abs(l_ref) + 1e-9, (l_gpu, l_ref)
    for got, ref in ((dwq, dwq_ref), (dwk, dwk_ref)):
        g = got.cpu().numpy().astype(np.float64)
        assert g.shape == ref.shape
        err = float(np.abs(g - ref).max())
        print(f"[distill] grad err {err:.3e} of max {float(np.abs(ref).max()):.3e}", flush=True)
        assert err <= GRAD_RTOL * float(np.abs(ref).max()) + 1e-12, (err, float(np.abs(ref).max()))
        _check_grad_elementwise(g, ref)


# Long rows (one query head): nb = 1100 and 2048 hold the whole row in registers
# (eight 16-byte chunks per lane), nb = 2052 streams it in two passes.  The
# element-wise bar is looser here: the fp32 row softmax of a long row carries a
# larger absolute error (its log-sum-exp and logits round at a larger scale), and
# the small gradient entries are sums with heavy cancellation of P - T.
# Measured: 1.6e-3 at nb = 1024, 2.3e-3 at nb = 1100 (both KL row kernels give
# the same within 10%), while the max-scaled error stays at 1-4e-5 of the
# largest entry.
LONG_ROWS = [1100, 2048, 2052]
ELEM_RTOL_LONG = 5e-3


@pytest.mark.parametrize("nb", LONG_ROWS)
def test_gate_distill_long_rows(nb):
    B, Hq, Hkv, S, D, Dg = 1, 1, 1, 64 * nb, 64, 32
    seed = stable_seed("distlong", nb)
    _, q, k, _, _, _ = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=seed, spikes=True)
    wq, wk = _weights(B, Hq, Hkv, D, Dg, True, seed + 1)
    gt = synthetic_gt(B, Hq, nb, seed + 2)
    print(f"[distill] long rows nb = {nb}", flush=True)
    loss, dwq, dwk = seer.gate_distill(to_device(q), to_device(k), torch.from_numpy(wq).cuda(),
                                       torch.from_numpy(wk).cuda(), torch.from_numpy(gt).cuda())
    torch.cuda.synchronize()
    l_ref, dwq_ref, dwk_ref = oracle.distill(q, k, wq, wk, gt)
    assert abs(float(loss.item()) - l_ref) <= DIST_RTOL * abs(l_ref), (float(loss.item()), l_ref)
    for got, ref in ((dwq, dwq_ref), (dwk, dwk_ref)):
        g = got.cpu().numpy().astype(np.float64)
        err = float(np.abs(g - ref).max())
        print(f"[distill] grad err {err:.3e} of max {float(np.abs(ref).max()):.3e}", flush=True)
        assert err <= GRAD_RTOL * float(np.abs(ref).max()), err
        _check_grad_elementwise(g, ref, ELEM_RTOL_LONG)


def test_gate_distill_deterministic_and_workspace_reuse():
    B, Hq, Hkv, S, D, Dg = 1, 4, 2, 1024, 128, 128
    _, q, k, _, _, _ = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("distdet"))
    wq, wk = _weights(B, Hq, Hkv, D, Dg, True, 7)
    gt = torch.from_numpy(synthetic_gt(B, Hq, S // 64, 8)).cuda()
    qd, kd = to_device(q), to_device(k)
    wqd, wkd = torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda()
    l1, a1, b1 = seer.gate_distill(qd, kd, wqd, wkd, gt, rope_theta=500000.0)
    r1 = (l1.clone(), a1.clone(), b1.clone())
    l2, a2, b2 = seer.gate_distill(qd, kd, wqd, wkd, gt, rope_theta=500000.0)
    torch.cuda.synchronize()
    for x, y in zip(r1, (l2, a2, b2)):
        assert torch.equal(x, y)


def test_distill_on_device_ground_truth_decreases_loss():
    """End to end on the device: ground truth from seer_attn_gt, one plain
    gradient step on the gate weights lowers the distillation loss."""
    B, Hq, Hkv, S, D, Dg = 1, 4, 1, 2048, 128, 128
    _, q, k, v, _, _ = small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("diste2e"), spikes=True)
    wq, wk = _weights(B, Hq, Hkv, D, Dg, True, 11)
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    _, _, gt = seer.attn_gt(qd, kd, vd)
    wqd, wkd = torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda()
    l0, gq, gk = seer.gate_distill(qd, kd, wqd, wkd, gt)
    l0 = float(l0.item())
    step = 0.5 / max(float(gq.abs().max()), float(gk.abs().max()))
    l1, _, _ = seer.gate_distill(qd, kd, wqd - step * 1e-2 * gq, wkd - step * 1e-2 * gk, gt)
    assert float(l1.item()) < l0


@pytest.mark.slow
@pytest.mark.parametrize("name", ["llama_s32k", "qwen_s64k"])
def test_gate_distill_full_size(name):
    """Full workload shapes (32 query / 8 KV heads at 32768 tokens; 28 / 4 at
    65536): loss and gradients against the oracle in full."""
    import workload as W
    w = W.WORKLOADS[name]
    print(f"[distill] {name}: generating inputs", flush=True)
    q, k = W.make_tensor(w, "q"), W.make_tensor(w, "k")
    wq, wk = _weights(w.batch, w.heads_q, w.heads_kv, w.head_dim, w.gate_dim, True, w.seed + 5)
    gt = synthetic_gt(w.batch, w.heads_q, w.n_blocks, w.seed + 6)
    loss, dwq, dwk = seer.gate_distill(to_device(q), to_device(k), torch.from_numpy(wq).cuda(),
                                       torch.from_numpy(wk).cuda(), torch.from_numpy(gt).cuda(),
                                       rope_theta=500000.0)
    torch.cuda.synchronize()
    print(f"[distill] {name}: device done", flush=True)
    l_ref, dwq_ref, dwk_ref = oracle.distill(q, k, wq, wk, gt, rope_theta=500000.0)
    assert abs(float(loss.item()) - l_ref) <= DIST_RTOL * abs(l_ref), (float(loss.item()), l_ref)
    for got, ref in ((dwq, dwq_ref), (dwk, dwk_ref)):
        g = got.cpu().numpy().astype(np.float64)
        err = float(np.abs(g - ref).max())
        print(f"[distill] {name}: grad err {err:.3e} of max {float(np.abs(ref).max()):.3e}", flush=True)
        assert err <= GRAD_RTOL * float(np.abs(ref).max()), err
        _check_grad_elementwise(g, ref)
