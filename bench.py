"""Benchmark of the SeerAttention prefill hot path on one MI355X.

One step = the whole path on one batch of seeded synthetic input already
resident in HBM: the AttnGate (pool + linear, gate logits, TopK/threshold
selection; seer_gate) followed by block-sparse causal attention over the
active tiles (seer_bsattn).  The dense causal kernel (seer_dense_attn) is timed
at the same shape for the speedup.  Default workload: Llama-3-8B head layout
(32 query / 8 KV heads, head_dim 128), 131072 tokens, bf16, TopK keeping 10%
of each query-block row's causal blocks.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--workload llama_s128k]

Prints one JSON line on stdout (diagnostics go to stderr).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workload as W  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA (published)
PEAK_F32_TFLOPS = 157.3     # MI355X dense fp32 MFMA (published)
PEAK_HBM_GBS = 8000.0
ROPE_BASE = 500000.0         # Llama 3.1's RoPE base, for the gate's block-level RoPE
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_traffic.json")
ATTN_SRC = os.path.join(ROOT, "paper_2410_13276_amd", "csrc", "attn_kernels.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _dev(x: np.ndarray):
    import torch
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(x).cuda()


def _src_hash() -> str:
    with open(ATTN_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def _traffic(workload: str):
    """HBM bytes per attention launch from committed rocprofv3 counters, if they
    were taken on the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        rec = t.get(workload)
        if rec and rec.get("kernel_src_sha256_16") == _src_hash():
            return rec["bytes_per_launch"]
    except (OSError, ValueError, KeyError):
        pass
    return None


def cpu_baseline(w: W.Workload, q, k, v, wq, wk, n_rows: int):
    """The fp64 oracle, as it stands, on a bounded sample of the same workload."""
    import oracle
    threads = oracle.set_threads(0)
    t0 = time.perf_counter()
    _, ell = oracle.gate(q, k, wq, wk)
    if w.select == W.SEL_THRESHOLD:
        sel = oracle.select(ell, oracle.THRESHOLD, thresholds=W.load_thresholds(w))
    else:
        sel = oracle.select(ell, oracle.TOPK_RATIO if w.select == W.SEL_TOPK_RATIO else oracle.TOPK_FIXED,
                            rho=w.topk_ratio, k=w.topk_k)
    t_gate = time.perf_counter() - t0
    del ell
    nb = w.n_blocks
    rng = np.random.default_rng(7)
    strata = np.linspace(0, nb, n_rows + 1).astype(int)
    rows = np.array([(int(rng.integers(w.batch)), int(rng.integers(w.heads_q)),
                      int(rng.integers(strata[s], max(strata[s] + 1, strata[s + 1]))))
                     for s in range(n_rows)], dtype=np.int32)
    rows[:, 2] = np.minimum(rows[:, 2], nb - 1)
    t0 = time.perf_counter()
    oracle.attn(q, k, v, mask=sel["mask"], rows=rows)
    t_attn = time.perf_counter() - t0
    tiles = int(sum(sel["count"][b, h, i] for b, h, i in rows))
    flops = 4.0 * 64 * 64 * w.head_dim * tiles
    return dict(value=flops / t_attn / 1e12, unit="TFLOP/s", cores=threads, kind="oracle",
                sample=(f"{n_rows} row-stratified (head, query-block) rows of {w.name} "
                        f"({tiles} active 64x64 tiles, {flops / 1e9:.1f} GFLOP) through the fp64 "
                        f"attention oracle on the oracle's own mask; value = active-tile flops / "
                        f"{t_attn:.2f} s. The full fp64 gate oracle took {t_gate:.2f} s."),
                gate_seconds=round(t_gate, 3), attn_seconds=round(t_attn, 3),
                host_cpus=len(os.sched_getaffinity(0)), cpu_model=platform.processor() or platform.machine())


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=W.HEADLINE, choices=sorted(W.WORKLOADS))
    ap.add_argument("--dense-runs", type=int, default=3)
    ap.add_argument("--gt-runs", type=int, default=2, help="timed runs of the ground-truth kernel (0: skip)")
    ap.add_argument("--extra-runs", type=int, default=3,
                    help="timed runs of the gate with block RoPE and of the distillation step (0: skip)")
    ap.add_argument("--cpu-rows", type=int, default=4096, help="oracle sample size (q-block rows)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy three times (the known-size "
                         "reference for scaling HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the SeerAttention prefill path here is the "
              "single-GPU kernel pair (gate + block-sparse attention); multi-GPU runs are not "
              "supported (the path would shard by KV-head group, one group set per GPU).",
              file=sys.stderr)
        return 2

    import torch
    import paper_2410_13276_amd as seer

    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": src.numel() * 4, "copies": 3}))
        return 0

    w = W.WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    q, k, v = (W.make_tensor(w, t) for t in "qkv")
    wq, wk = W.make_weights(w)
    log(f"[bench] inputs for {w.name} generated in {time.perf_counter() - t0:.1f}s")
    qd, kd, vd = _dev(q), _dev(k), _dev(v)
    wqd, wkd = torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda()
    thr = W.load_thresholds(w)
    gate_kw = dict(keep_first=w.keep_first, keep_diag=w.keep_diag)
    if w.select == W.SEL_THRESHOLD:
        if thr.size == 1:
            gate_kw.update(mode=seer.THRESHOLD, threshold=float(thr[0]))
        else:
            gate_kw.update(mode=seer.THRESHOLD, head_thresholds=torch.from_numpy(thr).cuda())
    elif w.select == W.SEL_TOPK_RATIO:
        gate_kw.update(mode=seer.TOPK_RATIO, topk_ratio=w.topk_ratio)
    else:
        gate_kw.update(mode=seer.TOPK_FIXED, topk_k=w.topk_k)

    # everything the timed region touches is allocated up front
    mask = seer.alloc_mask(w.batch, w.heads_q, w.seq_len)
    ws = torch.empty(max(1, seer.gate_workspace_bytes(qd, kd, w.gate_dim)), dtype=torch.uint8, device="cuda")
    o = torch.empty_like(qd)
    od = torch.empty_like(qd)
    # key-range split workspace (sparse and dense get the same treatment)
    n_aws = seer.attn_workspace_bytes(qd, kd, vd)  # 0: the split is opt-in
    aws = torch.empty(n_aws, dtype=torch.uint8, device="cuda") if n_aws else None
    stream = torch.cuda.current_stream()

    def step():
        seer.gate(qd, kd, wqd, wkd, **gate_kw, mask=mask, workspace=ws)
        seer.bsattn(qd, kd, vd, mask, out=o, workspace=aws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    active = int(mask.count.sum().item())
    # active diagonal tiles (half of each is above the causal diagonal): a row's
    # list is ascending, so the diagonal is active iff its last entry is i
    cnt = mask.count.long()
    last = mask.idx.gather(-1, (cnt - 1).clamp(min=0).unsqueeze(-1)).squeeze(-1).long() & 0xFFFF
    rows_i = torch.arange(cnt.shape[-1], device=cnt.device)
    active_diag = int(((cnt > 0) & (last == rows_i)).sum().item())
    nb = w.n_blocks
    causal_tiles = w.batch * w.heads_q * nb * (nb + 1) // 2
    sparsity = 1.0 - active / causal_tiles
    flops_tile = 4.0 * 64 * 64 * w.head_dim
    log(f"[bench] active tiles {active} / {causal_tiles} causal (sparsity {sparsity:.4f})")

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for s in range(args.steps):
        ev[s][0].record(stream)
        seer.gate(qd, kd, wqd, wkd, **gate_kw, mask=mask, workspace=ws)
        ev[s][1].record(stream)
        seer.bsattn(qd, kd, vd, mask, out=o, workspace=aws)
        ev[s][2].record(stream)
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_step = total_ms / args.steps
    gate_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    attn_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    attn_min = float(np.min([e[1].elapsed_time(e[2]) for e in ev]))

    # dense comparison at the same shape, same cache treatment
    seer.dense_attn(qd, kd, vd, out=od, workspace=aws)
    torch.cuda.synchronize()
    dts = []
    for _ in range(args.dense_runs):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        seer.dense_attn(qd, kd, vd, out=od, workspace=aws)
        b.record(stream)
        torch.cuda.synchronize()
        dts.append(a.elapsed_time(b))
    dense_ms = float(np.median(dts))
    dense_flops = flops_tile * causal_tiles

    # distillation ground truth (2D max-pooled attention map) at the same shape,
    # with a workspace of one KV group per launch
    gt_ms, gt_ws_bytes = None, 0
    if args.gt_runs > 0:
        gt_ws_bytes = seer.attn_gt_workspace_bytes(qd, kd, vd, 1)
        gt_ws = torch.empty(gt_ws_bytes, dtype=torch.uint8, device="cuda")
        gt_map = torch.empty((w.batch, w.heads_q, nb, nb), dtype=torch.float32, device="cuda")
        seer.attn_gt(qd, kd, vd, out=od, gt=gt_map, workspace=gt_ws)
        torch.cuda.synchronize()
        gts = []
        for _ in range(args.gt_runs):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            seer.attn_gt(qd, kd, vd, out=od, gt=gt_map, workspace=gt_ws)
            b.record(stream)
            torch.cuda.synchronize()
            gts.append(a.elapsed_time(b))
        gt_ms = float(np.median(gts))
        del gt_ws

    def timed(fn, runs):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(runs):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts))

    # the gate with block-level RoPE (section 3.1: pre-RoPE q/k, rotation at block
    # positions after the linear layers), Llama 3.1's RoPE base
    rope_ms, distill_ms = None, None
    if args.extra_runs > 0:
        rope_ms = timed(lambda: seer.gate(qd, kd, wqd, wkd, **gate_kw, rope_theta=ROPE_BASE, mask=mask,
                                          workspace=ws), args.extra_runs)
    # one gate distillation step (Eq. 2: KL against the pooled ground truth,
    # gradients of both gate weights) at the same shape
    if args.extra_runs > 0 and args.gt_runs > 0 and w.dtype == "bf16":
        dwq, dwk = torch.empty_like(wqd), torch.empty_like(wkd)
        loss = torch.empty(1, dtype=torch.float32, device="cuda")
        dws = torch.empty(max(1, seer.gate_distill_workspace_bytes(qd, kd, wqd, wkd)), dtype=torch.uint8,
                          device="cuda")
        distill_ms = timed(lambda: seer.gate_distill(qd, kd, wqd, wkd, gt_map, dwq=dwq, dwk=dwk, loss=loss,
                                                     workspace=dws), args.extra_runs)
        del dwq, dwk, dws
    if args.gt_runs > 0:
        del gt_map

    # variant: one mask per KV group (the mean of the group's head probabilities
    # selects; attention loads each K/V tile once for two query heads), same
    # TopK setting, at the same shape
    kv = None
    if args.extra_runs > 0 and w.dtype == "bf16" and w.heads_q > w.heads_kv and w.select != W.SEL_THRESHOLD:
        mkv = seer.alloc_mask(w.batch, w.heads_kv, w.seq_len, kv_shared=True)
        kv_gate_ms = timed(lambda: seer.gate(qd, kd, wqd, wkd, **gate_kw, kv_shared=True, mask=mkv, workspace=ws),
                           args.extra_runs)
        kv_attn_ms = timed(lambda: seer.bsattn(qd, kd, vd, mkv, out=od, workspace=aws), args.extra_runs)
        kv_active = int(mkv.count.sum().item()) * (w.heads_q // w.heads_kv)
        kv_sp = 1.0 - kv_active / causal_tiles
        kv = {"what": "shared-mask variant (not the paper's per-head gate): one mask per KV group selected "
                      "from the mean of its query heads' gate probabilities; attention loads each K/V tile "
                      "once for two query heads of the group",
              "gate_ms": round(kv_gate_ms, 4), "attn_ms": round(kv_attn_ms, 4),
              "attn_tflops": round(flops_tile * kv_active / (kv_attn_ms * 1e-3) / 1e12, 2),
              "sparsity": round(kv_sp, 5), "active_tiles": kv_active,
              "speedup_vs_dense": round(dense_ms / kv_attn_ms, 3),
              "speedup_tracking": round(dense_ms / kv_attn_ms * (1.0 - kv_sp), 3)}
        del mkv

    active_flops = flops_tile * active
    D = w.head_dim
    attn_kernels = f"attn_fwd_bf16_kernel<{D}, true, false, {'true' if w.seq_len % 64 else 'false'}, 1>"
    attn_tflops = active_flops / (attn_ms * 1e-3) / 1e12
    # launches of the attention kernel one seer_bsattn call makes (the library's own count)
    launches = seer.attn_launches(qd, kd, vd, mask, workspace_bytes=0 if aws is None else aws.numel())
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    traffic = _traffic(w.name)
    es = 2 if w.dtype == "bf16" else 4
    alg_bytes = es * w.batch * w.seq_len * w.head_dim * (2 * w.heads_q + 2 * w.heads_kv)  # Q, O, K, V
    speedup = dense_ms / attn_ms
    result = {
        "metric": "block-sparse prefill attn TFLOPS (active tiles) + speedup vs dense @128k",
        "value": round(active_flops / (ms_step * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded Llama-shaped Q/K/V with key spikes and local smoothing; random gate weights)",
        "config": {"workload": w.name, "batch": w.batch, "heads_q": w.heads_q, "heads_kv": w.heads_kv,
                   "head_dim": w.head_dim, "seq_len": w.seq_len, "block": 64, "gate_dim": w.gate_dim,
                   "selection": {W.SEL_TOPK_RATIO: f"topk_ratio={w.topk_ratio}",
                                 W.SEL_TOPK_FIXED: f"topk_k={w.topk_k}",
                                 W.SEL_THRESHOLD: "threshold"}[w.select],
                   "parallelism": "single GPU"},
        "value_definition": "active-tile attention flops / (gate + block-sparse attention) step time",
        "attn_tflops": round(attn_tflops, 2),
        "useful_attn_tflops": round(flops_tile * (active - 0.5 * active_diag) / (attn_ms * 1e-3) / 1e12, 2),
        "attn_ms": round(attn_ms, 4),
        "attn_ms_min": round(attn_min, 4),
        "gate_ms": round(gate_ms, 4),
        "dense_ms": round(dense_ms, 3),
        "dense_tflops": round(dense_flops / (dense_ms * 1e-3) / 1e12, 2),
        "useful_dense_tflops": round(flops_tile * (causal_tiles - 0.5 * w.batch * w.heads_q * nb)
                                     / (dense_ms * 1e-3) / 1e12, 2),
        "useful_flops_note": "useful_* count each diagonal tile as half (its upper triangle is masked)",
        "sparsity": round(sparsity, 5),
        "active_tiles": active,
        "speedup_vs_dense": round(speedup, 3),
        "speedup_vs_dense_incl_gate": round(dense_ms / ms_step, 3),
        "ideal_speedup": round(1.0 / (1.0 - sparsity), 3),
        "speedup_tracking": round(speedup * (1.0 - sparsity), 3),
        "ground_truth": None if gt_ms is None else {
            "what": "dense attention + 2D max-pooled attention map (seer_attn_gt), one KV group per launch",
            "ms": round(gt_ms, 3), "dense_ms": round(dense_ms, 3),
            "overhead_vs_dense": round(gt_ms / dense_ms - 1.0, 4),
            "workspace_bytes": gt_ws_bytes, "map_bytes": 4 * w.batch * w.heads_q * nb * nb},
        "gate_block_rope": None if rope_ms is None else {
            "what": f"seer_gate with block-level RoPE (base {ROPE_BASE:g}) at the same shape",
            "ms": round(rope_ms, 4), "overhead_vs_gate": round(rope_ms / gate_ms - 1.0, 4)},
        "kv_shared": kv,
        "distill": None if distill_ms is None else {
            "what": "seer_gate_distill: gate forward, KL(renormalised ground truth || gate), dWq and dWk",
            "ms": round(distill_ms, 3)},
        "roofline": {"bound": "mfma", "kernel": attn_kernels,
                     "achieved": round(attn_tflops, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(attn_tflops / peak, 4), "traffic": traffic,
                     "launches_per_call": launches,
                     "flops_per_launch": active_flops / launches,
                     "launch_avg_ms": round(attn_ms / launches, 4),
                     "algorithmic_bytes_per_launch": alg_bytes / launches,
                     "traffic_tb_per_s": None if traffic is None else
                     round(traffic / (attn_ms / launches * 1e-3) / 1e12, 3),
                     "note": "achieved = active-tile flops of one call / the call's mean HIP-event "
                             "duration = flops_per_launch / launch_avg_ms (the call's launches run "
                             "back to back on the stream). traffic = bytes past L2 per launch "
                             "(scaled rocprofv3 FETCH_SIZE + WRITE_SIZE); traffic_tb_per_s = traffic "
                             "/ launch_avg_ms, against algorithmic_bytes_per_launch (Q, K, V read "
                             "once, O written once): tiles of near-random masks are reused little "
                             "in a 4 MB L2, so the launch streams K/V from the Infinity Cache"},
    }
    log(f"[bench] step {ms_step:.3f} ms (gate {gate_ms:.3f} + attn {attn_ms:.3f}); "
        f"attn {attn_tflops:.1f} TF/s; dense {dense_ms:.2f} ms; speedup {speedup:.2f}x "
        f"(ideal {1 / (1 - sparsity):.2f}x)")
    if not args.no_cpu_baseline:
        del qd, kd, vd, o, od, ws, aws
        result["cpu_baseline"] = cpu_baseline(w, q, k, v, wq, wk, args.cpu_rows)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
