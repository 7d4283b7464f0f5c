"""Python access to the fp64 CPU oracle (seer_oracle.c).

TEST INFRASTRUCTURE ONLY: the independent checker of the HIP library.  It shares
no code with paper_2410_13276_amd/ and imports nothing from it.  Only tests/,
__graft_entry__.smoke() and the cpu_baseline leg of bench.py use it.

Every function follows one step of the SeerAttention prefill path
(arXiv 2410.13276): pooling and gate (section 3.1, Eq. 1), block selection
(Eq. 3 TopK, Eq. 4 threshold), masked causal attention (section 3.3), and the
MaxPool2D distillation target (Eq. 2).  Pooling, gate, selection, attention and
the pooled target are computed in the C file, this module only marshals numpy
arrays for them; distill() (the KL loss of Eq. 2 and its weight gradients) is
written here in numpy fp64 on top of the C gate.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "seer_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

F32, BF16 = 0, 1
POOL_AVG, POOL_MAX_MIN_AVG = 0, 1
TOPK_RATIO, TOPK_FIXED, THRESHOLD = 0, 1, 2

_lib = None


def build(force: bool = False) -> str:
    """Compile liboracle.so with gcc (-O2, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        build()
        L = C.CDLL(_LIB_PATH)
        p = C.c_void_p
        i = C.c_int
        L.orc_version.restype = i
        L.orc_set_threads.argtypes = [i]
        L.orc_set_threads.restype = i
        L.orc_pool.argtypes = [p, i, i, i, i, i, p, i, i, p]
        L.orc_pool.restype = i
        L.orc_linear.argtypes = [p, i, i, i, i, p, i, i, p]
        L.orc_linear.restype = None
        L.orc_block_rope.argtypes = [p, C.c_int64, i, i, C.c_double, i]
        L.orc_block_rope.restype = None
        L.orc_gate_logits.argtypes = [p, p, i, i, i, i, i, p]
        L.orc_gate_logits.restype = None
        L.orc_gate_logscore.argtypes = [p, C.c_int64, i, p]
        L.orc_gate_logscore.restype = None
        L.orc_group_logscore.argtypes = [p, i, i, i, i, p]
        L.orc_group_logscore.restype = None
        L.orc_topk_k.argtypes = [i, i, C.c_double, i, i]
        L.orc_topk_k.restype = i
        L.orc_select.argtypes = [p, i, i, i, i, C.c_double, i, p, i, i, i, p, p, p, p]
        L.orc_select.restype = i
        L.orc_attn.argtypes = [p, p, p, i, i, i, i, i, i, p, p, p, i, i, C.c_double,
                               p, p, i, p, p]
        L.orc_attn.restype = i
        L.orc_maxpool_gt.argtypes = [p, p, i, i, i, i, i, i, p, p, i, i, C.c_double, p,
                                     C.c_int64, p]
        L.orc_maxpool_gt.restype = i
        _lib = L
    return _lib


def set_threads(n: int) -> int:
    """Set the OpenMP thread count (n <= 0 keeps it); returns the count in use."""
    return lib().orc_set_threads(int(n))


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _dtype_code(x: np.ndarray) -> int:
    if x.dtype == np.float32:
        return F32
    if x.dtype == np.uint16:
        return BF16
    raise TypeError("oracle inputs are fp32 arrays or uint16 bf16 bit patterns")


def _strides(x: np.ndarray) -> np.ndarray:
    """(batch, head, seq) strides in elements of a [B, H, S, D] array with unit D stride."""
    assert x.ndim == 4 and x.strides[3] == x.itemsize
    return np.asarray([s // x.itemsize for s in x.strides[:3]], dtype=np.int64)


def pool(x: np.ndarray, block: int, kind: int) -> np.ndarray:
    """Sequence pooling of [B, H, S, D]: avg -> [B,H,nb,D]; max|min|avg -> [B,H,nb,3D]."""
    B, H, S, D = x.shape
    nb = -(-S // block)  # the last block may be partial
    out = np.empty((B, H, nb, D if kind == POOL_AVG else 3 * D), dtype=np.float64)
    st = _strides(x)
    rc = lib().orc_pool(_ptr(x), _dtype_code(x), B, H, S, D, _ptr(st), block, kind, _ptr(out))
    if rc != 0:
        raise ValueError("bad pooling arguments")
    return out


def linear(pooled: np.ndarray, W: np.ndarray, w_per_head: bool = True) -> np.ndarray:
    """Gate linear layer: [B,H,nb,din] x W[H or 1, din, dout] -> [B,H,nb,dout]."""
    pooled = np.ascontiguousarray(pooled, dtype=np.float64)
    W = np.ascontiguousarray(W, dtype=np.float32)
    B, H, nb, din = pooled.shape
    assert W.shape[1] == din
    dout = W.shape[2]
    out = np.empty((B, H, nb, dout), dtype=np.float64)
    lib().orc_linear(_ptr(pooled), B, H, nb, din, _ptr(W), int(bool(w_per_head)), dout, _ptr(out))
    return out


def block_rope(x: np.ndarray, theta: float, block: int = 64) -> np.ndarray:
    """Block-level RoPE of gate rows [B, H, nb, Dg] (a rotated copy)."""
    x = np.array(x, dtype=np.float64, order="C", copy=True)
    B, H, nb, Dg = x.shape
    lib().orc_block_rope(_ptr(x), B * H, nb, Dg, float(theta), int(block))
    return x


def gate_logits(Qg: np.ndarray, Kg: np.ndarray) -> np.ndarray:
    Qg = np.ascontiguousarray(Qg, dtype=np.float64)
    Kg = np.ascontiguousarray(Kg, dtype=np.float64)
    B, Hq, nb, Dg = Qg.shape
    Hkv = Kg.shape[1]
    L = np.empty((B, Hq, nb, nb), dtype=np.float64)
    lib().orc_gate_logits(_ptr(Qg), _ptr(Kg), B, Hq, Hkv, nb, Dg, _ptr(L))
    return L


def gate_logscore(L: np.ndarray) -> np.ndarray:
    L = np.ascontiguousarray(L, dtype=np.float64)
    nb = L.shape[-1]
    ell = np.empty_like(L)
    lib().orc_gate_logscore(_ptr(L), L.size // nb, nb, _ptr(ell))
    return ell


def group_logscore(ell: np.ndarray, heads_kv: int) -> np.ndarray:
    """Log of the mean gate probability over each KV group's query heads
    [B, Hkv, nb, nb] (the shared-mask variant's score)."""
    ell = np.ascontiguousarray(ell, dtype=np.float64)
    B, Hq, nb, _ = ell.shape
    if Hq % heads_kv != 0:
        raise ValueError("heads_q must be a multiple of heads_kv")
    out = np.empty((B, heads_kv, nb, nb), dtype=np.float64)
    lib().orc_group_logscore(_ptr(ell), B, Hq, heads_kv, nb, _ptr(out))
    return out


def topk_k(mode: int, i: int, rho: float, k_fixed: int, n_forced: int) -> int:
    return lib().orc_topk_k(mode, i, rho, k_fixed, n_forced)


def select(ell: np.ndarray, mode: int, rho: float = 0.0, k: int = 0,
           thresholds: Optional[np.ndarray] = None, keep_first: int = 1, keep_diag: int = 1):
    """Block selection on log-scores [B, Hq, nb, nb].

    Returns dict(mask uint8 [B,Hq,nb,nb], count int32 [B,Hq,nb],
    idx uint16 [B,Hq,nb,nb], cut float64 [B,Hq,nb])."""
    ell = np.ascontiguousarray(ell, dtype=np.float64)
    B, Hq, nb, _ = ell.shape
    thr = None
    n_thr = 0
    if mode == THRESHOLD:
        thr = np.ascontiguousarray(np.atleast_1d(thresholds), dtype=np.float32)
        n_thr = thr.size
    mask = np.zeros((B, Hq, nb, nb), dtype=np.uint8)
    count = np.zeros((B, Hq, nb), dtype=np.int32)
    idx = np.zeros((B, Hq, nb, nb), dtype=np.uint16)
    cut = np.zeros((B, Hq, nb), dtype=np.float64)
    rc = lib().orc_select(_ptr(ell), B, Hq, nb, mode, float(rho), int(k), _ptr(thr), n_thr,
                          int(keep_first), int(keep_diag), _ptr(mask), _ptr(count), _ptr(idx),
                          _ptr(cut))
    if rc != 0:
        raise ValueError(f"orc_select failed ({rc})")
    return dict(mask=mask, count=count, idx=idx, cut=cut)


def gate(q: np.ndarray, k: np.ndarray, wq: np.ndarray, wk: np.ndarray, block: int = 64,
         w_per_head: bool = True, rope_theta: float = 0.0):
    """Pool, linear, optional block-level RoPE (rope_theta > 0) and logits of the
    gate.  Returns (L, ell) [B, Hq, nb, nb]."""
    qp = pool(q, block, POOL_AVG)
    kp = pool(k, block, POOL_MAX_MIN_AVG)
    qg = linear(qp, wq, w_per_head)
    kg = linear(kp, wk, w_per_head)
    if rope_theta > 0:
        qg = block_rope(qg, rope_theta, block)
        kg = block_rope(kg, rope_theta, block)
    L = gate_logits(qg, kg)
    return L, gate_logscore(L)


def attn(q: np.ndarray, k: np.ndarray, v: np.ndarray, block: int = 64, causal: bool = True,
         scale: Optional[float] = None, mask: Optional[np.ndarray] = None,
         rows: Optional[np.ndarray] = None):
    """Masked (block-sparse) causal attention in fp64.

    q [B,Hq,S,D], k/v [B,Hkv,S,D] (fp32 or bf16 bits, same type); mask uint8
    [B,Hq,nb,nb] or None (dense); rows int32 [n,3] of (b,h,i) or None (all).
    Returns (O [n, block, D], LSE [n, block]) with n = len(rows) or B*Hq*nb; rows
    past the end of a partial last block are NaN."""
    assert q.dtype == k.dtype == v.dtype
    B, Hq, S, D = q.shape
    Hkv = k.shape[1]
    nb = -(-S // block)  # the last block may be partial
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    if mask is not None:
        mask = np.ascontiguousarray(mask, dtype=np.uint8)
        assert mask.shape == (B, Hq, nb, nb)
    n = B * Hq * nb
    if rows is not None:
        rows = np.ascontiguousarray(rows, dtype=np.int32).reshape(-1, 3)
        n = rows.shape[0]
    O = np.empty((n, block, D), dtype=np.float64)
    lse = np.empty((n, block), dtype=np.float64)
    rc = lib().orc_attn(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), B, Hq, Hkv, S, D,
                        _ptr(_strides(q)), _ptr(_strides(k)), _ptr(_strides(v)), block,
                        int(bool(causal)), float(scale), _ptr(mask), _ptr(rows),
                        n if rows is not None else 0, _ptr(O), _ptr(lse))
    if rc != 0:
        raise ValueError(f"orc_attn failed ({rc})")
    return O, lse


def maxpool_gt(q: np.ndarray, k: np.ndarray, block: int = 64, scale: Optional[float] = None,
               causal: bool = True, rows: Optional[np.ndarray] = None):
    """Eq. 2 target: block-wise max of the attention probabilities.
    Returns [B,Hq,nb,nb], or [n, nb] for rows int32 [n,3] of (b,h,i)."""
    B, Hq, S, D = q.shape
    Hkv = k.shape[1]
    nb = -(-S // block)  # the last block may be partial
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    n = B * Hq * nb
    if rows is not None:
        rows = np.ascontiguousarray(rows, dtype=np.int32).reshape(-1, 3)
        n = rows.shape[0]
    gt = np.empty((n, nb), dtype=np.float64)
    rc = lib().orc_maxpool_gt(_ptr(q), _ptr(k), _dtype_code(q), B, Hq, Hkv, S, D,
                              _ptr(_strides(q)), _ptr(_strides(k)), block, int(bool(causal)),
                              float(scale), _ptr(rows), n if rows is not None else 0, _ptr(gt))
    if rc != 0:
        raise ValueError(f"orc_maxpool_gt failed ({rc})")
    return gt if rows is not None else gt.reshape(B, Hq, nb, nb)


# ---------------------------------------------------------------------------
# gate distillation step (Eq. 2): KL(ground truth || gate score) and its
# gradients with respect to the gate weights, in fp64 numpy
# ---------------------------------------------------------------------------

def _rope_angles(nb: int, Dg: int, theta: float, block: int) -> np.ndarray:
    """[nb, Dg/2] rotation angles of the block-level RoPE: position i, plane d
    rotates by i * (theta / block)^(-2d/Dg)."""
    half = Dg // 2
    w = (theta / block) ** (-2.0 * np.arange(half) / Dg)
    return np.arange(nb, dtype=np.float64)[:, None] * w[None, :]


def _rotate(x: np.ndarray, ang: np.ndarray, inverse: bool) -> np.ndarray:
    """Rotates plane (d, d + Dg/2) of rows [.., nb, Dg] by +ang (or -ang)."""
    half = x.shape[-1] // 2
    c, s = np.cos(ang), np.sin(ang)
    if inverse:
        s = -s
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def distill(q: np.ndarray, k: np.ndarray, wq: np.ndarray, wk: np.ndarray, gt: np.ndarray,
            block: int = 64, w_per_head: bool = True, rope_theta: float = 0.0,
            parts: bool = False):
    """One gate distillation step (section 3.2, Eq. 2) in fp64.

    The gate's block-causal softmax P (Eq. 1, the forward of `gate`) is fitted
    to the ground truth: each row of gt [B,Hq,nb,nb] (the 2D max-pooled
    attention map, j <= i) is renormalised to a distribution T, and
        loss = mean over the B*Hq*nb rows of KL(T || P) = sum_j T log(T / P)
    with 0 log 0 = 0.  Gradients follow the chain rule backwards through the
    softmax (dloss/dL = (P sum(T) - T) / rows), the logits, the optional
    block-level RoPE (its inverse rotation) and the linear layers.
    Returns (loss, dwq, dwk), dwq/dwk shaped like wq/wk; with parts=True also
    a dict of the intermediate P, T and logits."""
    B, Hq, S, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    nb = -(-S // block)  # the last block may be partial
    Wq = np.asarray(wq, dtype=np.float64).reshape(-1, D, wq.shape[-1])
    Wk = np.asarray(wk, dtype=np.float64).reshape(-1, 3 * D, wk.shape[-1])
    Dg = Wq.shape[-1]
    qp = pool(q, block, POOL_AVG)                  # [B,Hq,nb,D]
    kp = pool(k, block, POOL_MAX_MIN_AVG)          # [B,Hkv,nb,3D]
    wq_h = Wq if w_per_head else np.broadcast_to(Wq[:1], (Hq, D, Dg))
    wk_g = Wk if w_per_head else np.broadcast_to(Wk[:1], (Hkv, 3 * D, Dg))
    qg = qp @ wq_h
    kg = kp @ wk_g
    if rope_theta > 0:
        ang = _rope_angles(nb, Dg, rope_theta, block)
        qg = _rotate(qg, ang, False)
        kg = _rotate(kg, ang, False)
    kg_h = np.repeat(kg, G, axis=1)                # KV head of each query head
    causal = np.tril(np.ones((nb, nb), dtype=bool))
    L = (qg @ np.swapaxes(kg_h, -1, -2)) / np.sqrt(Dg)
    L = np.where(causal, L, -np.inf)
    m = L.max(axis=-1, keepdims=True)
    e = np.where(causal, np.exp(L - m), 0.0)
    P = e / e.sum(axis=-1, keepdims=True)
    logP = np.where(causal, L - m - np.log(e.sum(axis=-1, keepdims=True)), 0.0)

    g = np.where(causal, np.asarray(gt, dtype=np.float64), 0.0)
    gs = g.sum(axis=-1, keepdims=True)
    T = np.divide(g, gs, out=np.zeros_like(g), where=gs > 0)
    logT = np.log(np.where(T > 0, T, 1.0))
    rows = B * Hq * nb
    loss = float(np.sum(T * (logT - logP)) / rows)

    Tsum = T.sum(axis=-1, keepdims=True)
    dL = np.where(causal, P * Tsum - T, 0.0) / rows
    dqg = (dL @ kg_h) / np.sqrt(Dg)
    dkg_h = (np.swapaxes(dL, -1, -2) @ qg) / np.sqrt(Dg)
    dkg = dkg_h.reshape(B, Hkv, G, nb, Dg).sum(axis=2)
    if rope_theta > 0:
        dqg = _rotate(dqg, ang, True)
        dkg = _rotate(dkg, ang, True)
    dwq = (np.swapaxes(qp, -1, -2) @ dqg).sum(axis=0)
    dwk = (np.swapaxes(kp, -1, -2) @ dkg).sum(axis=0)
    if not w_per_head:
        dwq = dwq.sum(axis=0, keepdims=True)
        dwk = dwk.sum(axis=0, keepdims=True)
    dwq = dwq.reshape(np.shape(wq))
    dwk = dwk.reshape(np.shape(wk))
    if parts:
        return loss, dwq, dwk, dict(P=P, T=T, L=L)
    return loss, dwq, dwk
