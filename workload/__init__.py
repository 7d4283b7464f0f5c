"""Seeded synthetic inputs for the SeerAttention prefill path.

This module is shared by the HIP path's tests/bench and by the oracle's callers.
It holds none of the method's arithmetic: only random draws, the fp32 -> bf16
rounding of the stored inputs (round to nearest even), and the shape and
selection parameters of each workload.

The paper measures on Llama-3.1-8B-Instruct activations over PG19/RULER text;
neither the model nor the data is available, so these seeded tensors with the
same head layout stand in for them:

* Q, K, V ~ N(0, 1) drawn per (tensor, batch, head) from
  ``numpy.random.Generator(PCG64(SeedSequence(seed, spawn_key=(tensor, b, h))))``
  so that any single head can be regenerated on its own.
* "spikes": each KV head gets a rank-1 spike ``2*sqrt(D)*u_g`` added to its keys at
  3 seeded positions (attention-sink / vertical-stripe structure).
* "smooth": keys are first replaced by a trailing 256-token box average of their
  noise, rescaled to unit variance (local-window correlation), spikes after.
* Gate weights ~ N(0, sigma^2) in fp32, one matrix per head (Wq [Hq, D, Dg],
  Wk [Hkv, 3D, Dg]).
"""
from __future__ import annotations

import dataclasses
import json
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np

BLOCK = 64

# tensor ids for the seed spawn keys
_T_Q, _T_K, _T_V, _T_WQ, _T_WK, _T_STRUCT, _T_PERM = 0, 1, 2, 3, 4, 5, 6

SEL_TOPK_RATIO = 0
SEL_TOPK_FIXED = 1
SEL_THRESHOLD = 2

_HERE = os.path.dirname(os.path.abspath(__file__))
THRESHOLDS_FILE = os.path.join(_HERE, "thresholds.json")


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    batch: int
    heads_q: int
    heads_kv: int
    head_dim: int
    seq_len: int
    dtype: str  # "f32" or "bf16"
    gate_dim: int
    w_sigma2: float
    structure: str  # "plain", "spikes", "smooth"
    select: int  # SEL_*
    topk_ratio: float = 0.0
    topk_k: int = 0
    # threshold workloads: target causal-block sparsity (global) or per-head spread
    target_sparsity: float = 0.0
    per_head_sparsity: Optional[tuple] = None
    keep_first: int = 1
    keep_diag: int = 1

    @property
    def n_blocks(self) -> int:
        return self.seq_len // BLOCK

    @property
    def group(self) -> int:
        return self.heads_q // self.heads_kv

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _qwen_sparsity(n_heads: int, seed: int) -> tuple:
    """Per-head target sparsity 0.60 + 0.35*pi(h)/(n-1), pi a seeded permutation."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(_T_PERM,))))
    perm = rng.permutation(n_heads)
    return tuple(float(0.60 + 0.35 * p / (n_heads - 1)) for p in perm)


WORKLOADS = {
    # 2 query heads sharing 1 KV head, D 64, 1024 tokens, fp32; TopK keeps 50% of
    # the causal blocks of each query-block row, first and diagonal always kept.
    "tiny_f32_s1k": Workload("tiny_f32_s1k", 1001, 1, 2, 1, 64, 1024, "f32", 64, 1.0 / 64,
                             "plain", SEL_TOPK_RATIO, topk_ratio=0.5),
    # Llama-3-8B head layout (32 q / 8 kv, D 128), 8k tokens, bf16; one global
    # threshold giving about 50% block sparsity.
    "llama_s8k": Workload("llama_s8k", 1002, 1, 32, 8, 128, 8192, "bf16", 128, 1.0 / 128,
                          "spikes", SEL_THRESHOLD, target_sparsity=0.5),
    # same layout, 32k tokens, local-window keys, TopK for 80% sparsity
    "llama_s32k": Workload("llama_s32k", 1003, 1, 32, 8, 128, 32768, "bf16", 128, 1.0 / 128,
                           "smooth", SEL_TOPK_RATIO, topk_ratio=0.2),
    # same layout, 128k tokens, TopK for 90% sparsity (the headline workload)
    "llama_s128k": Workload("llama_s128k", 1004, 1, 32, 8, 128, 131072, "bf16", 128, 1.0 / 128,
                            "smooth", SEL_TOPK_RATIO, topk_ratio=0.1),
    # Qwen-style GQA 7:1 (28 q / 4 kv), 64k tokens, per-head thresholds for
    # sparsity spread over 60..95% across heads
    "qwen_s64k": Workload("qwen_s64k", 1005, 1, 28, 4, 128, 65536, "bf16", 128, 1.0 / 128,
                          "spikes", SEL_THRESHOLD,
                          per_head_sparsity=_qwen_sparsity(28, 1005)),
}

HEADLINE = "llama_s128k"


# ----------------------------------------------------------------------------
# storage rounding
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _rng(seed: int, *key) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=tuple(key))))


# ----------------------------------------------------------------------------
# per-head draws
# ----------------------------------------------------------------------------

def _spike(w: Workload, b: int, g: int):
    rng = _rng(w.seed, _T_STRUCT, b, g)
    pos = rng.choice(w.seq_len, size=3, replace=False)
    u = rng.standard_normal(w.head_dim)
    u /= np.linalg.norm(u)
    return np.sort(pos), (2.0 * math.sqrt(w.head_dim)) * u


def _head(w: Workload, tensor: int, b: int, h: int) -> np.ndarray:
    """fp32 [S, D] values of one head before storage rounding."""
    S, D = w.seq_len, w.head_dim
    rng = _rng(w.seed, tensor, b, h)
    if tensor == _T_K and w.structure == "smooth":
        win = 256
        z = rng.standard_normal((S + win - 1, D))
        c = np.cumsum(z, axis=0)
        c = np.concatenate([np.zeros((1, D)), c], axis=0)
        x = (c[win:] - c[:-win]) / win * math.sqrt(win)  # unit variance
    else:
        x = rng.standard_normal((S, D), dtype=np.float32)
    x = np.asarray(x, dtype=np.float32)
    if tensor == _T_K and w.structure in ("spikes", "smooth"):
        pos, vec = _spike(w, b, h)
        x = x.copy()
        x[pos, :] += vec.astype(np.float32)
    return x


def _store(w: Workload, x: np.ndarray) -> np.ndarray:
    return x if w.dtype == "f32" else f32_to_bf16_bits(x)


def head_tensor(w: Workload, which: str, b: int, h: int) -> np.ndarray:
    """Stored elements ([S, D] fp32 or bf16 bits) of head h of 'q', 'k' or 'v'."""
    t = {"q": _T_Q, "k": _T_K, "v": _T_V}[which]
    return _store(w, _head(w, t, b, h))


def make_tensor(w: Workload, which: str, threads: int = 8) -> np.ndarray:
    """Full stored tensor [B, H, S, D] of 'q', 'k' or 'v' (fp32 or uint16 bf16 bits)."""
    H = w.heads_q if which == "q" else w.heads_kv
    dt = np.float32 if w.dtype == "f32" else np.uint16
    out = np.empty((w.batch, H, w.seq_len, w.head_dim), dtype=dt)

    def fill(bh):
        b, h = bh
        out[b, h] = head_tensor(w, which, b, h)

    jobs = [(b, h) for b in range(w.batch) for h in range(H)]
    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        list(ex.map(fill, jobs))
    return out


def make_weights(w: Workload):
    """Gate weights Wq [Hq, D, Dg] and Wk [Hkv, 3D, Dg], fp32 ~ N(0, sigma^2)."""
    s = math.sqrt(w.w_sigma2)
    wq = _rng(w.seed, _T_WQ).standard_normal((w.heads_q, w.head_dim, w.gate_dim)) * s
    wk = _rng(w.seed, _T_WK).standard_normal((w.heads_kv, 3 * w.head_dim, w.gate_dim)) * s
    return wq.astype(np.float32), wk.astype(np.float32)


# ----------------------------------------------------------------------------
# selection parameters
# ----------------------------------------------------------------------------

def load_thresholds(w: Workload) -> Optional[np.ndarray]:
    """fp32 thresholds for a threshold workload: shape [1] (global) or [Hq]."""
    if w.select != SEL_THRESHOLD:
        return None
    with open(THRESHOLDS_FILE) as f:
        table = json.load(f)
    if w.name not in table:
        raise KeyError(f"no stored thresholds for workload {w.name}; run workload/make_thresholds.py")
    return np.asarray(table[w.name]["thresholds"], dtype=np.float32)


# ----------------------------------------------------------------------------
# synthetic block-mask pattern classes (the five families the paper's mask
# visualisation shows: A-shape, vertical, slash, diagonal-block, random)
# ----------------------------------------------------------------------------

def pattern_mask(kind: str, nb: int, seed: int, density: float = 0.2) -> np.ndarray:
    """uint8 [nb, nb] block mask, block-causal (j <= i), of one pattern class.

    The diagonal is NOT forced here, so rows may be empty (user masks)."""
    kinds = ("a_shape", "vertical", "slash", "diagonal", "random", "empty_rows")
    if kind not in kinds:
        raise ValueError(kind)
    rng = _rng(seed, 99, kinds.index(kind))
    i = np.arange(nb)[:, None]
    j = np.arange(nb)[None, :]
    causal = j <= i
    if kind == "a_shape":
        m = (j < max(1, nb // 16)) | (i - j < max(1, nb // 8))
    elif kind == "vertical":
        cols = rng.choice(nb, size=max(1, int(density * nb)), replace=False)
        m = np.isin(j, cols) | (i == j)
    elif kind == "slash":
        offs = rng.choice(nb, size=max(1, int(density * nb)), replace=False)
        m = np.isin(i - j, offs)
    elif kind == "diagonal":
        m = i == j
    elif kind == "random":
        m = rng.random((nb, nb)) < density
    else:  # empty_rows
        m = rng.random((nb, nb)) < density
        m[rng.choice(nb, size=max(1, nb // 4), replace=False), :] = False
    return (m & causal).astype(np.uint8)
