"""Benchmark of the SeerAttention prefill hot path on one MI355X.

One step = the whole path on one batch of seeded synthetic input already
resident in HBM: the AttnGate (pool + linear, gate logits, TopK/threshold
selection; seer_gate) followed by block-sparse causal attention over the
active tiles (seer_bsattn).  The dense causal kernel (seer_dense_attn) is timed
at the same shape for the speedup.  Default workload: Llama-3-8B head layout
(32 query / 8 KV heads, head_dim 128), 131072 tokens, bf16, TopK keeping 10%
of each query-block row's causal blocks.  The other workloads of the
measurement plan (1k fp32, 8k, 32k, 64k GQA 7:1) are timed and checked under
`configs`.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--workload llama_s128k]

Prints one JSON line on stdout (diagnostics go to stderr).  Timings of single
calls are medians over runs, with the minimum beside them; `value` is the
active-tile flops of a step over the mean step time of the timed K steps.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import subprocess
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
CUS, BF16_FLOP_PER_CLK_CU, F32_FLOP_PER_CLK_CU = 256, 4096, 256  # peak = CUs x flop/clk x clock
ROPE_BASE = 500000.0         # Llama 3.1's RoPE base, for the gate's block-level RoPE
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_traffic.json")
ATTN_SRC = os.path.join(ROOT, "paper_2410_13276_amd", "csrc", "attn_kernels.hip")
MASK_BAND = 1e-4             # log-score distance to the selection cut within which masks may differ
CONFIG_WORKLOADS = ("tiny_f32_s1k", "llama_s8k", "llama_s32k", "qwen_s64k")


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
    """Bytes past L2 per attention launch from committed rocprofv3 counters, if
    they were taken on the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        rec = t.get(workload)
        if rec and rec.get("kernel_src_sha256_16") == _src_hash():
            return rec["bytes_per_launch"]
    except (OSError, ValueError, KeyError):
        pass
    return None


def _stats(ts):
    ts = np.asarray(ts, dtype=np.float64)
    return {"median": round(float(np.median(ts)), 4), "min": round(float(ts.min()), 4),
            "mean": round(float(ts.mean()), 4), "runs": int(ts.size)}


# ---------------------------------------------------------------------------
# clocks: a helper process samples amd-smi during the run
# ---------------------------------------------------------------------------
#
# The helper is started before this process touches the GPU (it never touches
# it either), and it alone starts amd-smi.  Under rocprofv3, whose preloaded
# library initialises the GPU in every process it starts, no helper runs.

_SAMPLER = r"""
import json, subprocess, sys, time
end = time.time() + float(sys.argv[1])
while time.time() < end:
    try:
        r = subprocess.run(["amd-smi", "metric", "-g", "0", "--clock", "--json"], capture_output=True,
                           text=True, timeout=10)
        d = json.loads(r.stdout)
        gpu = d["gpu_data"][0] if isinstance(d, dict) else d[0]
        vals = [float(v["clk"]["value"]) for k, v in gpu["clock"].items()
                if k.startswith("gfx") and isinstance(v, dict)]
        if vals:
            print(f"{time.time():.4f} {sum(vals) / len(vals):.1f}", flush=True)
    except Exception:
        pass
    time.sleep(0.05)
"""


def _under_profiler() -> bool:
    return any(k.startswith("ROCPROF") for k in os.environ) or "rocprof" in os.environ.get("LD_PRELOAD", "")


class ClockSampler:
    """The XCDs' mean gfx clock (MHz), read by a helper process (amd-smi reads 50 ms apart)."""

    def __init__(self, max_seconds: float = 900.0):
        self.proc = None
        if _under_profiler():
            return
        try:
            self.proc = subprocess.Popen([sys.executable, "-c", _SAMPLER, str(max_seconds)],
                                         stdout=subprocess.PIPE, stderr=subprocess.DEVNULL, text=True)
        except OSError:
            self.proc = None

    def samples(self):
        """(time, MHz) pairs; stops the helper."""
        if self.proc is None:
            return []
        self.proc.terminate()
        try:
            out, _ = self.proc.communicate(timeout=20)
        except subprocess.TimeoutExpired:
            self.proc.kill()
            out, _ = self.proc.communicate()
        pairs = []
        for line in out.splitlines():
            try:
                t, c = line.split()
                pairs.append((float(t), float(c)))
            except ValueError:
                continue
        return pairs


CLOCK_WINDOW_S = 1.5      # back-to-back sparse calls while the clock is sampled
CLOCK_MIN_SAMPLES = 3


def _clock_summary(pairs, t_win0, t_win1, t_first, t_last):
    """Clock before the run, under load (samples at or above 1000 MHz inside the
    clock window, after its first 0.25 s; idle XCDs drop to ~100 MHz) and after
    it.  The median under load is given only from CLOCK_MIN_SAMPLES samples."""
    if not pairs:
        return None
    before = [c for t, c in pairs if t <= t_first]
    busy = [] if t_win0 is None else [c for t, c in pairs if t_win0 + 0.25 <= t <= t_win1 and c >= 1000.0]
    after = [c for t, c in pairs if t >= t_last]
    ok = len(busy) >= CLOCK_MIN_SAMPLES
    return {"before": round(before[-1], 1) if before else None,
            "under_load_median": round(float(np.median(busy)), 1) if ok else None,
            "under_load_min": round(min(busy), 1) if ok else None,
            "under_load_max": round(max(busy), 1) if ok else None,
            "under_load_samples": len(busy),
            "after": round(after[0], 1) if after else None,
            "what": "gfx clock (mean over the 8 XCDs) from amd-smi, read back to back (one read takes a few "
                    "hundred ms): the last sample before the run; the median, min and max of the samples at "
                    f"or above 1000 MHz while the sparse attention call runs back to back for {CLOCK_WINDOW_S} s "
                    "after the timed steps (untimed; the first 0.25 s skipped), given from "
                    f"{CLOCK_MIN_SAMPLES} samples on; the first sample after the run"}


# ---------------------------------------------------------------------------
# timing helpers (HIP events on the launch stream)
# ---------------------------------------------------------------------------

def _timed(fn, runs, stream):
    import torch
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
    return ts


def _gate_kernel_split(fn, runs):
    """Per-call device time of the gate's kernels by stage (torch.profiler): pool
    + linear (pool_proj_kernel) and score + select (the logits and selection
    kernels, also given apart; the fused kernel counts as both).  None under
    rocprofv3 (one tracer at a time)."""
    if _under_profiler():
        return None
    import torch
    from torch.profiler import ProfilerActivity, profile
    fn()
    torch.cuda.synchronize()
    with profile(activities=[ProfilerActivity.CUDA]) as prof:
        for _ in range(runs):
            fn()
        torch.cuda.synchronize()
    pool = logits = select = fused = 0.0
    for e in prof.key_averages():
        t = getattr(e, "device_time_total", None)
        if t is None:
            t = getattr(e, "cuda_time_total", 0.0)
        if "pool_proj_kernel" in e.key:
            pool += t
        elif "gate_logits_kernel" in e.key:
            logits += t
        elif "select_kernel" in e.key:
            select += t
        elif "gate_fused_kernel" in e.key:
            fused += t
    score = logits + select + fused
    if pool <= 0 and score <= 0:
        return None
    ms = lambda t: round(t / runs / 1e3, 4)
    out = {"pool_linear_ms": ms(pool), "score_select_ms": ms(score)}
    if fused > 0:
        out["fused_score_select_ms"] = ms(fused)
    else:
        out["logits_ms"] = ms(logits)
        out["select_ms"] = ms(select)
    out["source"] = "torch.profiler kernel device times, per call"
    return out


def _gate_kwargs(w, seer):
    import torch
    kw = dict(keep_first=w.keep_first, keep_diag=w.keep_diag)
    if w.select == W.SEL_THRESHOLD:
        thr = W.load_thresholds(w)
        if thr.size == 1:
            kw.update(mode=seer.THRESHOLD, threshold=float(thr[0]))
        else:
            kw.update(mode=seer.THRESHOLD, head_thresholds=torch.from_numpy(thr).cuda())
    elif w.select == W.SEL_TOPK_RATIO:
        kw.update(mode=seer.TOPK_RATIO, topk_ratio=w.topk_ratio)
    else:
        kw.update(mode=seer.TOPK_FIXED, topk_k=w.topk_k)
    return kw


def _selection_str(w):
    return {W.SEL_TOPK_RATIO: f"topk_ratio={w.topk_ratio}", W.SEL_TOPK_FIXED: f"topk_k={w.topk_k}",
            W.SEL_THRESHOLD: "threshold (per head)" if w.per_head_sparsity else "threshold (global)"}[w.select]


# ---------------------------------------------------------------------------
# the oracle: selection on the full gate, attention on sampled rows
# ---------------------------------------------------------------------------

def _oracle_select(w, ell, oracle):
    if w.select == W.SEL_THRESHOLD:
        return oracle.select(ell, oracle.THRESHOLD, thresholds=W.load_thresholds(w),
                             keep_first=w.keep_first, keep_diag=w.keep_diag)
    mode = oracle.TOPK_RATIO if w.select == W.SEL_TOPK_RATIO else oracle.TOPK_FIXED
    return oracle.select(ell, mode, rho=w.topk_ratio, k=w.topk_k, keep_first=w.keep_first, keep_diag=w.keep_diag)


def _sample_rows(w, n_rows, seed=7):
    """Row-stratified (b, h, i) query-block rows: one per equal slice of i."""
    nb = w.n_blocks
    n_rows = min(n_rows, w.batch * w.heads_q * nb)
    rng = np.random.default_rng(seed)
    strata = np.linspace(0, nb, n_rows + 1).astype(int)
    rows = np.array([(int(rng.integers(w.batch)), int(rng.integers(w.heads_q)),
                      int(rng.integers(strata[s], max(strata[s] + 1, strata[s + 1]))))
                     for s in range(n_rows)], dtype=np.int32)
    rows[:, 2] = np.minimum(rows[:, 2], nb - 1)
    return rows


def _gpu_dense_mask(mask, nb):
    """0/1 [B, H, nb, nb] host copy of a device mask (count + ascending idx)."""
    count = mask.count.cpu().numpy().astype(np.int64)
    idx = mask.idx.cpu().numpy().view(np.uint16)
    rows = count.reshape(-1)
    flat = idx.reshape(-1, nb)
    out = np.zeros((rows.size, nb), np.uint8)
    r = np.repeat(np.arange(rows.size), rows)
    c = flat[np.arange(nb)[None, :] < rows[:, None]]
    out[r, c] = 1
    return count, out.reshape(count.shape + (nb,))


def _mask_parity(gpu_count, gpu_dense, sel, ell, topk):
    """Mask mismatches against the oracle: entries may differ only where the
    oracle log-score lies within MASK_BAND of the row's cut; TopK rows must
    hold exactly the oracle's count."""
    diff = gpu_dense != sel["mask"]
    n = int(diff.sum())
    out_band = 0
    if n:
        dist = np.abs(ell[diff] - np.broadcast_to(sel["cut"][..., None], ell.shape)[diff])
        out_band = int((dist > MASK_BAND).sum())
    return {"entries": int(diff.size), "differ": n, "differ_in_cut_band": n - out_band,
            "differ_outside_cut_band": out_band,
            "topk_rows_count_mismatch": int((gpu_count != sel["count"]).sum()) if topk else None}


def _attn_parity(o_gpu, w, q, k, v, sel, rows, gpu_dense, oracle):
    """Max-abs error of the device output on the sampled rows against the fp64
    oracle on its own mask, over the rows whose device mask equals it."""
    same = np.array([bool(np.array_equal(gpu_dense[b, h, i], sel["mask"][b, h, i])) for b, h, i in rows])
    use = rows[same]
    t0 = time.perf_counter()
    O_ref, _ = oracle.attn(q, k, v, mask=sel["mask"], rows=use)
    t = time.perf_counter() - t0
    if len(use) == 0:
        return None, t, 0
    got = np.stack([o_gpu[b, h, 64 * i:64 * (i + 1)].float().cpu().numpy() for b, h, i in use]).astype(np.float64)
    n = min(64, w.seq_len)
    return float(np.abs(got[:, :n] - O_ref[:, :n]).max()), t, int(len(use))


# ---------------------------------------------------------------------------
# one workload on the device: gate, sparse attention, dense attention
# ---------------------------------------------------------------------------

def _run_config(name, seer, runs, dense_runs, with_oracle, rows_per_config):
    import oracle
    import torch
    w = W.WORKLOADS[name]
    stream = torch.cuda.current_stream()
    q, k, v = (W.make_tensor(w, t) for t in "qkv")
    wq, wk = W.make_weights(w)
    qd, kd, vd = _dev(q), _dev(k), _dev(v)
    wqd, wkd = torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda()
    gkw = _gate_kwargs(w, seer)
    mask = seer.alloc_mask(w.batch, w.heads_q, w.seq_len)
    ws = torch.empty(max(1, seer.gate_workspace_bytes(qd, kd, w.gate_dim)), dtype=torch.uint8, device="cuda")
    o, od = torch.empty_like(qd), torch.empty_like(qd)
    gate = lambda: seer.gate(qd, kd, wqd, wkd, **gkw, mask=mask, workspace=ws)
    attn = lambda: seer.bsattn(qd, kd, vd, mask, out=o)
    gate_ts = _timed(gate, runs, stream)
    attn_ts = _timed(attn, runs, stream)
    dense_ts = _timed(lambda: seer.dense_attn(qd, kd, vd, out=od), dense_runs, stream)
    nb = w.n_blocks
    active = int(mask.count.sum().item())
    causal_tiles = w.batch * w.heads_q * nb * (nb + 1) // 2
    sp = 1.0 - active / causal_tiles
    flops = 4.0 * 64 * 64 * w.head_dim * active
    a_ms, d_ms = float(np.median(attn_ts)), float(np.median(dense_ts))
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    rec = {"shape": f"B{w.batch} Hq{w.heads_q}/Hkv{w.heads_kv} D{w.head_dim} S{w.seq_len} {w.dtype}",
           "selection": _selection_str(w), "sparsity": round(sp, 5), "active_tiles": active,
           "gate_ms": _stats(gate_ts), "gate_stages": _gate_kernel_split(gate, max(3, runs // 2)),
           "attn_ms": _stats(attn_ts), "attn_tflops": round(flops / (a_ms * 1e-3) / 1e12, 2),
           "attn_frac_of_peak": round(flops / (a_ms * 1e-3) / 1e12 / peak, 4), "peak_tflops": peak,
           "attn_launches": seer.attn_launches(qd, kd, vd, mask),
           "dense_ms": _stats(dense_ts), "speedup_vs_dense": round(d_ms / a_ms, 3),
           "ideal_speedup": round(1.0 / (1.0 - sp), 3), "speedup_tracking": round(d_ms / a_ms * (1.0 - sp), 3)}
    if with_oracle:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        _, ell = oracle.gate(q, k, wq, wk)
        sel = _oracle_select(w, ell, oracle)
        t_gate = time.perf_counter() - t0
        gc, gd = _gpu_dense_mask(mask, nb)
        par = _mask_parity(gc, gd, sel, ell, w.select != W.SEL_THRESHOLD)
        del ell
        rows = _sample_rows(w, rows_per_config if w.name != "tiny_f32_s1k" else w.batch * w.heads_q * nb)
        err, t_attn, n_used = _attn_parity(o, w, q, k, v, sel, rows, gd, oracle)
        par.update({"attn_max_abs": err, "attn_rows_checked": n_used, "attn_rows_sampled": int(len(rows)),
                    "attn_tolerance": 1e-4 if w.dtype == "f32" else 2e-2,
                    "oracle_gate_s": round(t_gate, 2), "oracle_attn_s": round(t_attn, 2)})
        rec["parity"] = par
    del qd, kd, vd, o, od, ws, mask
    torch.cuda.empty_cache()
    return rec


# ---------------------------------------------------------------------------
# CPU baseline: the oracle as it stands on the host's cores
# ---------------------------------------------------------------------------

def cpu_baseline(w, q, k, v, wq, wk, n_rows, seer_mask, o_gpu):
    """The fp64 oracle on a bounded sample of the workload (the full gate, the
    attention of n_rows query-block rows), its rate in the metric's unit, and
    the parity of the device's mask and output against it."""
    import oracle
    threads = oracle.set_threads(0)
    t0 = time.perf_counter()
    _, ell = oracle.gate(q, k, wq, wk)
    sel = _oracle_select(w, ell, oracle)
    t_gate = time.perf_counter() - t0
    nb = w.n_blocks
    gc, gd = _gpu_dense_mask(seer_mask, nb)
    mask_par = _mask_parity(gc, gd, sel, ell, w.select != W.SEL_THRESHOLD)
    del ell
    rows = _sample_rows(w, n_rows)
    t0 = time.perf_counter()
    O_ref, _ = oracle.attn(q, k, v, mask=sel["mask"], rows=rows)
    t_attn = time.perf_counter() - t0
    tiles = int(sum(sel["count"][b, h, i] for b, h, i in rows))
    flops = 4.0 * 64 * 64 * w.head_dim * tiles
    total_tiles = int(sel["count"].sum())
    # parity of the device output on the sampled rows whose device mask equals the oracle's
    same = np.array([bool(np.array_equal(gd[b, h, i], sel["mask"][b, h, i])) for b, h, i in rows])
    got = np.stack([o_gpu[b, h, 64 * i:64 * (i + 1)].float().cpu().numpy()
                    for b, h, i in rows[same]]).astype(np.float64)
    err = float(np.abs(got - O_ref[same]).max()) if same.any() else None
    base = dict(value=flops / t_attn / 1e12, unit="TFLOP/s", cores=threads, kind="oracle",
                sample=(f"{len(rows)} row-stratified (head, query-block) rows of {w.name} ({tiles} active 64x64 "
                        f"tiles, {flops / 1e9:.1f} GFLOP) through the fp64 attention oracle on the oracle's own "
                        f"mask; value = active-tile flops / {t_attn:.2f} s. The full fp64 gate oracle took "
                        f"{t_gate:.2f} s."),
                gate_seconds=round(t_gate, 3), attn_seconds=round(t_attn, 3),
                attn_full_seconds_extrapolated=round(t_attn * total_tiles / max(tiles, 1), 1),
                extrapolation="extrapolated: the sample's time scaled by all active tiles / the sample's tiles",
                host_cpus=len(os.sched_getaffinity(0)), cpu_model=platform.processor() or platform.machine())
    parity = dict(mask=mask_par, attn_max_abs=err, attn_rows_checked=int(same.sum()),
                  attn_rows_sampled=int(len(rows)), attn_tolerance=2e-2 if w.dtype == "bf16" else 1e-4)
    return base, parity


def cpu_baseline_tiny_threads():
    """The oracle on the 1k fp32 workload (gate + full attention), on one thread
    and on all of the host's cores."""
    import oracle
    w = W.WORKLOADS["tiny_f32_s1k"]
    q, k, v = (W.make_tensor(w, t) for t in "qkv")
    wq, wk = W.make_weights(w)
    out = {}
    for label, n in (("1_thread", 1), ("all_threads", len(os.sched_getaffinity(0)))):
        used = oracle.set_threads(n)
        t0 = time.perf_counter()
        _, ell = oracle.gate(q, k, wq, wk)
        sel = _oracle_select(w, ell, oracle)
        oracle.attn(q, k, v, mask=sel["mask"])
        t = time.perf_counter() - t0
        flops = 4.0 * 64 * 64 * w.head_dim * int(sel["count"].sum())
        out[label] = {"threads": used, "seconds": round(t, 4), "attn_tflops": round(flops / t / 1e12, 6)}
    oracle.set_threads(0)
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=W.HEADLINE, choices=sorted(W.WORKLOADS))
    ap.add_argument("--dense-runs", type=int, default=3)
    ap.add_argument("--gt-runs", type=int, default=2, help="timed runs of the ground-truth kernel (0: skip)")
    ap.add_argument("--extra-runs", type=int, default=3,
                    help="timed runs of the gate with block RoPE, the distillation step and the shared-mask "
                         "variant (0: skip)")
    ap.add_argument("--cpu-rows", type=int, default=4096, help="oracle sample size (q-block rows)")
    ap.add_argument("--config-runs", type=int, default=10, help="timed runs per call of the other workloads")
    ap.add_argument("--config-rows", type=int, default=256, help="oracle attention rows per other workload")
    ap.add_argument("--no-configs", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle (baseline and parity)")
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

    sampler = None if args.calibrate_copy else ClockSampler()
    time.sleep(1.0 if sampler and sampler.proc else 0.0)  # samples of the clock before the run
    t_first = time.time()

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
    gate_kw = _gate_kwargs(w, seer)

    # everything the timed region touches is allocated up front
    mask = seer.alloc_mask(w.batch, w.heads_q, w.seq_len)
    ws = torch.empty(max(1, seer.gate_workspace_bytes(qd, kd, w.gate_dim)), dtype=torch.uint8, device="cuda")
    o = torch.empty_like(qd)
    od = torch.empty_like(qd)
    stream = torch.cuda.current_stream()

    def step():
        seer.gate(qd, kd, wqd, wkd, **gate_kw, mask=mask, workspace=ws)
        seer.bsattn(qd, kd, vd, mask, out=o)

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
    t_start = time.time()
    start.record(stream)
    for s in range(args.steps):
        ev[s][0].record(stream)
        seer.gate(qd, kd, wqd, wkd, **gate_kw, mask=mask, workspace=ws)
        ev[s][1].record(stream)
        seer.bsattn(qd, kd, vd, mask, out=o)
        ev[s][2].record(stream)
    end.record(stream)
    torch.cuda.synchronize()
    # dense comparison at the same shape, same cache treatment
    dense_ts = _timed(lambda: seer.dense_attn(qd, kd, vd, out=od), args.dense_runs, stream)
    t_end = time.time()
    # clock window (untimed): the sparse call back to back, so that the clock
    # sampler sees this kernel's steady load
    t_win0 = t_win1 = None
    if sampler and sampler.proc:
        t_win0 = time.time()
        while time.time() - t_win0 < CLOCK_WINDOW_S:
            for _ in range(4):
                seer.bsattn(qd, kd, vd, mask, out=o)
            torch.cuda.synchronize()
        t_win1 = time.time()
    total_ms = start.elapsed_time(end)
    ms_step = total_ms / args.steps
    gate_ts = [e[0].elapsed_time(e[1]) for e in ev]
    attn_ts = [e[1].elapsed_time(e[2]) for e in ev]
    gate_ms, attn_ms = float(np.median(gate_ts)), float(np.median(attn_ts))
    dense_ms = float(np.median(dense_ts))
    dense_flops = flops_tile * causal_tiles
    gate_stages = _gate_kernel_split(lambda: seer.gate(qd, kd, wqd, wkd, **gate_kw, mask=mask, workspace=ws), 5)

    # distillation ground truth (2D max-pooled attention map) at the same shape,
    # with a workspace of one KV group per launch
    gt_ms, gt_ws_bytes = None, 0
    if args.gt_runs > 0:
        gt_ws_bytes = seer.attn_gt_workspace_bytes(qd, kd, vd, 1)
        gt_ws = torch.empty(gt_ws_bytes, dtype=torch.uint8, device="cuda")
        gt_map = torch.empty((w.batch, w.heads_q, nb, nb), dtype=torch.float32, device="cuda")
        gt_ms = float(np.median(_timed(lambda: seer.attn_gt(qd, kd, vd, out=od, gt=gt_map, workspace=gt_ws),
                                       args.gt_runs, stream)))
        del gt_ws

    # the gate with block-level RoPE (section 3.1: pre-RoPE q/k, rotation at block
    # positions after the linear layers), Llama 3.1's RoPE base
    rope_ms, distill_ms = None, None
    if args.extra_runs > 0:
        mask_rope = seer.alloc_mask(w.batch, w.heads_q, w.seq_len)  # (the step's mask is checked later)
        rope_ms = float(np.median(_timed(lambda: seer.gate(qd, kd, wqd, wkd, **gate_kw, rope_theta=ROPE_BASE,
                                                           mask=mask_rope, workspace=ws), args.extra_runs, stream)))
        del mask_rope
    # one gate distillation step (Eq. 2: KL against the pooled ground truth,
    # gradients of both gate weights) at the same shape
    if args.extra_runs > 0 and args.gt_runs > 0 and w.dtype == "bf16":
        dwq, dwk = torch.empty_like(wqd), torch.empty_like(wkd)
        loss = torch.empty(1, dtype=torch.float32, device="cuda")
        dws = torch.empty(max(1, seer.gate_distill_workspace_bytes(qd, kd, wqd, wkd)), dtype=torch.uint8,
                          device="cuda")
        distill_ms = float(np.median(_timed(lambda: seer.gate_distill(qd, kd, wqd, wkd, gt_map, dwq=dwq, dwk=dwk,
                                                                      loss=loss, workspace=dws),
                                            args.extra_runs, stream)))
        del dwq, dwk, dws
    if args.gt_runs > 0:
        del gt_map

    # variant: one mask per KV group (the mean of the group's head probabilities
    # selects; attention loads each K/V tile once for two query heads), same
    # TopK setting, at the same shape
    kv = None
    if args.extra_runs > 0 and w.dtype == "bf16" and w.heads_q > w.heads_kv and w.select != W.SEL_THRESHOLD:
        mkv = seer.alloc_mask(w.batch, w.heads_kv, w.seq_len, kv_shared=True)
        kv_ws = torch.empty(max(1, seer.gate_workspace_bytes(qd, kd, w.gate_dim)), dtype=torch.uint8,
                            device="cuda")
        kv_gate_ms = float(np.median(_timed(lambda: seer.gate(qd, kd, wqd, wkd, **gate_kw, kv_shared=True, mask=mkv,
                                                              workspace=kv_ws), args.extra_runs, stream)))
        kv_attn_ms = float(np.median(_timed(lambda: seer.bsattn(qd, kd, vd, mkv, out=od), args.extra_runs, stream)))
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
        del mkv, kv_ws
    t_last = time.time()
    time.sleep(0.2 if sampler and sampler.proc else 0.0)  # a sample after the run
    clocks = _clock_summary(sampler.samples() if sampler else [], t_win0, t_win1, t_first, t_last)

    active_flops = flops_tile * active
    D = w.head_dim
    attn_kernel = f"attn_fwd_bf16_kernel<{D}, true, false, {'true' if w.seq_len % 64 else 'false'}, 1>"
    attn_tflops = active_flops / (attn_ms * 1e-3) / 1e12
    # launches of the attention kernel one seer_bsattn call makes (the library's own count)
    launches = seer.attn_launches(qd, kd, vd, mask)
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    clk_load = clocks["under_load_median"] if clocks else None
    peak_at_clk = None if clk_load is None else \
        CUS * (BF16_FLOP_PER_CLK_CU if w.dtype == "bf16" else F32_FLOP_PER_CLK_CU) * clk_load * 1e6 / 1e12
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
                   "selection": _selection_str(w), "parallelism": "single GPU"},
        "value_definition": "active-tile attention flops / mean (gate + block-sparse attention) step time of "
                            "the timed steps",
        "timing": "gate, attention and dense: HIP events on the launch stream; median over runs, min and "
                  "mean beside it",
        "attn_tflops": round(attn_tflops, 2),
        "useful_attn_tflops": round(flops_tile * (active - 0.5 * active_diag) / (attn_ms * 1e-3) / 1e12, 2),
        "attn_ms": round(attn_ms, 4),
        "attn_ms_stats": _stats(attn_ts),
        "gate_ms": round(gate_ms, 4),
        "gate_ms_stats": _stats(gate_ts),
        "gate_stages": gate_stages,
        "dense_ms": round(dense_ms, 3),
        "dense_ms_stats": _stats(dense_ts),
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
        "clocks_mhz": clocks,
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
        "roofline": {"bound": "mfma", "kernel": attn_kernel,
                     "achieved": round(attn_tflops, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(attn_tflops / peak, 4), "traffic": traffic,
                     "peak_at_measured_clock": None if peak_at_clk is None else round(peak_at_clk, 1),
                     "frac_at_measured_clock": None if peak_at_clk is None else round(attn_tflops / peak_at_clk, 4),
                     "launches_per_call": launches,
                     "flops_per_launch": active_flops / launches,
                     "launch_avg_ms": round(attn_ms / launches, 4),
                     "algorithmic_bytes_per_launch": alg_bytes / launches,
                     "traffic_tb_per_s": None if traffic is None else
                     round(traffic / (attn_ms / launches * 1e-3) / 1e12, 3),
                     "note": "achieved = active-tile flops of one call / the call's median HIP-event duration "
                             "= flops_per_launch / launch_avg_ms (the call's launches run back to back on "
                             "the stream; launches_per_call is the library's own count, seer_attn_launches). "
                             "peak_at_measured_clock = 256 CUs x 4096 bf16 flop/clk x the median gfx clock "
                             "under load. traffic = bytes past L2 per launch (scaled rocprofv3 FETCH_SIZE + "
                             "WRITE_SIZE); traffic_tb_per_s = traffic / launch_avg_ms, against "
                             "algorithmic_bytes_per_launch (Q, K, V read once, O written once): the "
                             "active tiles request far more K/V than that (32 KiB each), and what the XCD "
                             "L2s do not reuse comes from the Infinity Cache or HBM"},
    }
    log(f"[bench] step {ms_step:.3f} ms (gate {gate_ms:.3f} + attn {attn_ms:.3f}); "
        f"attn {attn_tflops:.1f} TF/s; dense {dense_ms:.2f} ms; speedup {speedup:.2f}x "
        f"(ideal {1 / (1 - sparsity):.2f}x); clock under load {clk_load}")

    del qd, kd, vd, od, ws
    torch.cuda.empty_cache()
    if not args.no_configs:
        result["configs"] = {}
        for name in CONFIG_WORKLOADS:
            if name == w.name:
                continue
            t0 = time.perf_counter()
            result["configs"][name] = _run_config(name, seer, args.config_runs, args.dense_runs,
                                                  not args.no_cpu_baseline, args.config_rows)
            c = result["configs"][name]
            log(f"[bench] {name}: attn {c['attn_ms']['median']:.3f} ms ({c['attn_tflops']} TF/s), "
                f"dense {c['dense_ms']['median']:.3f} ms, gate {c['gate_ms']['median']:.3f} ms "
                f"({time.perf_counter() - t0:.1f}s)")
    if not args.no_cpu_baseline:
        base, parity = cpu_baseline(w, q, k, v, wq, wk, args.cpu_rows, mask, o)
        base["tiny_f32_s1k_full"] = cpu_baseline_tiny_threads()
        result["cpu_baseline"] = base
        result["parity"] = parity
        log(f"[bench] parity: {json.dumps(parity)}")
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
