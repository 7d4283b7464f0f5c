"""Python binding of libseer.so, the MI355X (gfx950) SeerAttention prefill library.

Argument marshalling only: every step of the path runs in the library's HIP
kernels (include/seer.h documents the C ABI).  PyTorch supplies device memory
and the current stream.  Importing this package does not load the library;
the first call does, and raises if libseer.so has not been built -- there is
no CPU fallback.

    mask = seer.gate(q, k, wq, wk, mode=seer.TOPK_RATIO, topk_ratio=0.1)
    o, lse = seer.bsattn(q, k, v, mask)
    o_dense, _ = seer.dense_attn(q, k, v)
    o_dense, lse, gt = seer.attn_gt(q, k, v, want_lse=True)   # distillation target
    loss, dwq, dwk = seer.gate_distill(q, k, wq, wk, gt)      # KL(gt || gate) and gradients
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libseer.so")

BLOCK = 64
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = 0, 1, 2, 3, 4
BF16, F32 = 0, 1
TOPK_RATIO, TOPK_FIXED, THRESHOLD = 0, 1, 2


class AttnDesc(C.Structure):
    _fields_ = [("batch", C.c_int32), ("heads_q", C.c_int32), ("heads_kv", C.c_int32),
                ("seq_len", C.c_int32), ("head_dim", C.c_int32), ("dtype", C.c_int32),
                ("q_stride", C.c_int64 * 3), ("k_stride", C.c_int64 * 3),
                ("v_stride", C.c_int64 * 3), ("o_stride", C.c_int64 * 3)]


class GateDesc(C.Structure):
    _fields_ = [("block", C.c_int32), ("gate_dim", C.c_int32), ("w_per_head", C.c_int32),
                ("mode", C.c_int32), ("topk_ratio", C.c_double), ("topk_k", C.c_int32),
                ("threshold", C.c_float), ("head_thresholds", C.c_void_p),
                ("keep_first", C.c_int32), ("keep_diag", C.c_int32), ("rope_theta", C.c_double),
                ("kv_shared", C.c_int32)]


class AttnOpts(C.Structure):
    """seer_attn_opts: launch options of the attention calls (zero fields: defaults)."""
    _fields_ = [("split", C.c_int32), ("split_width", C.c_int32), ("heads_per_wg", C.c_int32),
                ("batch_min_blocks", C.c_int32), ("batch_wgs", C.c_int32), ("walk_classes", C.c_int32)]


class DistillOpts(C.Structure):
    """seer_distill_opts (zero fields: defaults)."""
    _fields_ = [("gemm_min_chunks", C.c_int32), ("gemm_tile_n", C.c_int32)]


def _opts_ref(opts, cls):
    """None, a dict of fields, or a ctypes options struct -> pointer argument."""
    if opts is None:
        return None
    if isinstance(opts, dict):
        opts = cls(**opts)
    if not isinstance(opts, cls):
        raise TypeError(f"options must be a dict or {cls.__name__}")
    return C.byref(opts)


class BlockMaskStruct(C.Structure):
    _fields_ = [("n_blocks", C.c_int32), ("count", C.c_void_p), ("idx", C.c_void_p),
                ("dense", C.c_void_p), ("kv_shared", C.c_int32)]


# every symbol include/seer.h declares, with its ctypes signature
_P = C.c_void_p
_SIGS = {
    "seer_abi_version": ([], C.c_int),
    "seer_status_str": ([C.c_int], C.c_char_p),
    "seer_gate_workspace_bytes": ([_P, _P, C.c_int32], C.c_size_t),
    "seer_mask_idx_elems": ([_P, C.c_int32], C.c_size_t),
    "seer_gate": ([_P, _P, _P, _P, _P, _P, _P, _P, _P, C.c_size_t, _P], C.c_int),
    "seer_gate_noalloc": ([_P, _P, _P, _P, _P, _P, _P, _P], C.c_int),
    "seer_gate_noalloc_max_bytes": ([], C.c_size_t),
    "seer_bsattn": ([_P, C.c_int32, _P, C.c_int32, C.c_float, _P, _P, _P, _P, _P, _P], C.c_int),
    "seer_dense_attn": ([_P, C.c_int32, C.c_float, _P, _P, _P, _P, _P, _P], C.c_int),
    "seer_mask_from_dense": ([_P, C.c_int32, _P, _P, _P], C.c_int),
    "seer_attn_gt_workspace_bytes": ([_P, C.c_int32, C.c_int32], C.c_size_t),
    "seer_gate_distill_workspace_bytes": ([_P, _P, _P], C.c_size_t),
    "seer_attn_workspace_bytes": ([_P, C.c_int32, C.c_int32, _P], C.c_size_t),
    "seer_bsattn_ws": ([_P, C.c_int32, _P, C.c_int32, C.c_float, _P, _P, _P, _P, _P, _P, C.c_size_t, _P, _P],
                       C.c_int),
    "seer_dense_attn_ws": ([_P, C.c_int32, C.c_float, _P, _P, _P, _P, _P, _P, C.c_size_t, _P, _P], C.c_int),
    "seer_attn_launches": ([_P, C.c_int32, C.c_int32, C.c_int32, _P, C.c_size_t], C.c_int32),
    "seer_gate_distill": ([_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, C.c_size_t, _P, _P], C.c_int),
    "seer_attn_gt": ([_P, C.c_int32, C.c_int32, C.c_float, _P, _P, _P, _P, _P, _P, _P, C.c_size_t, _P, _P],
                     C.c_int),
    "seer_varlen_mask_elems": ([_P, _P, C.c_int32, C.c_int32, _P], C.c_size_t),
    "seer_gate_varlen_workspace_bytes": ([_P, _P, _P], C.c_size_t),
    "seer_gate_varlen": ([_P, _P, _P, _P, _P, _P, _P, _P, _P, C.c_size_t, _P], C.c_int),
    "seer_bsattn_varlen": ([_P, _P, C.c_int32, _P, C.c_int32, C.c_float, _P, _P, _P, _P, _P, _P], C.c_int),
}

_lib = None


class SeerError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_str(status)} ({status})")


def lib():
    """The loaded libseer.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2410_13276_amd.build` (no CPU fallback exists)")
        L = C.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def status_str(status: int) -> str:
    return lib().seer_status_str(int(status)).decode()


def abi_version() -> int:
    return lib().seer_abi_version()


# ---------------------------------------------------------------------------
# marshalling helpers
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}: Q/K/V are bfloat16 or float32")


def make_desc(q, k, v=None, o=None) -> AttnDesc:
    """Descriptor of [B, H, S, D] tensors (element strides, D contiguous)."""
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o)):
        if t is not None and (t.dim() != 4 or t.stride(3) != 1):
            raise ValueError(f"{name} must be [batch, heads, seq, head_dim] with unit last stride")
    d = AttnDesc()
    d.batch, d.heads_q, d.seq_len, d.head_dim = q.shape[0], q.shape[1], q.shape[2], q.shape[3]
    d.heads_kv = k.shape[1]
    d.dtype = _dtype_code(q)
    for field, t in (("q_stride", q), ("k_stride", k), ("v_stride", v if v is not None else k),
                     ("o_stride", o if o is not None else q)):
        arr = getattr(d, field)
        for e in range(3):
            arr[e] = t.stride(e)
    return d


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _check(status: int, where: str):
    if status != OK:
        raise SeerError(status, where)


@dataclass
class BlockMask:
    """Compacted block mask: idx[b, h, i, :count[b, h, i]] ascending (device tensors)
    of `block`-token blocks (64 or 128; the last block may be partial).  With
    kv_shared the rows are per KV head (h = KV head) and apply to every query
    head of the group."""
    count: object  # int32 [B, H, nb]  (H = Hq, or Hkv when kv_shared)
    idx: object    # int16 storage of uint16 [B, H, nb, nb]
    dense: Optional[object] = None  # uint8 [B, H, nb, nb]
    block: int = BLOCK
    kv_shared: bool = False

    @property
    def n_blocks(self) -> int:
        return self.count.shape[-1]

    def struct(self) -> BlockMaskStruct:
        m = BlockMaskStruct()
        m.n_blocks = self.n_blocks
        m.count = _ptr(self.count)
        m.idx = _ptr(self.idx)
        m.dense = _ptr(self.dense)
        m.kv_shared = int(bool(self.kv_shared))
        return m

    def indices(self):
        """idx as non-negative int32 (block indices are < 65536)."""
        return self.idx.to(_torch().int32) & 0xFFFF


def alloc_mask(batch: int, heads: int, seq_len: int, device="cuda", dense: bool = False,
               block: int = BLOCK, kv_shared: bool = False) -> BlockMask:
    """Mask buffers for `heads` row sets: the query heads, or the KV heads of a
    kv_shared mask."""
    torch = _torch()
    nb = -(-seq_len // block)  # the last block may be partial
    return BlockMask(
        count=torch.empty((batch, heads, nb), dtype=torch.int32, device=device),
        idx=torch.empty((batch, heads, nb, nb), dtype=torch.int16, device=device),
        dense=torch.empty((batch, heads, nb, nb), dtype=torch.uint8, device=device) if dense else None,
        block=block, kv_shared=kv_shared)


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------

def gate_desc(gate_dim: int, mode: int, topk_ratio: float = 0.0, topk_k: int = 0,
              threshold: float = 0.0, head_thresholds=None, keep_first: bool = True,
              keep_diag: bool = True, w_per_head: bool = True, rope_theta: float = 0.0,
              block: int = BLOCK, kv_shared: bool = False) -> GateDesc:
    g = GateDesc()
    g.block = block
    g.gate_dim = gate_dim
    g.w_per_head = int(bool(w_per_head))
    g.mode = mode
    g.topk_ratio = float(topk_ratio)
    g.topk_k = int(topk_k)
    g.threshold = float(threshold)
    g.head_thresholds = _ptr(head_thresholds)
    g.keep_first = int(bool(keep_first))
    g.keep_diag = int(bool(keep_diag))
    g.rope_theta = float(rope_theta)
    g.kv_shared = int(bool(kv_shared))
    return g


def gate_workspace_bytes(q, k, gate_dim: int, mode: int = TOPK_RATIO, topk_ratio: float = 1.0,
                         logits_in_workspace: bool = True) -> int:
    d = make_desc(q, k)
    g = gate_desc(gate_dim, mode, topk_ratio=topk_ratio, topk_k=1, threshold=0.0)
    return lib().seer_gate_workspace_bytes(C.byref(d), C.byref(g), int(logits_in_workspace))


def gate(q, k, wq, wk, *, mode: int, topk_ratio: float = 0.0, topk_k: int = 0,
         threshold: float = 0.0, head_thresholds=None, keep_first: bool = True,
         keep_diag: bool = True, w_per_head: bool = True, rope_theta: float = 0.0,
         block: int = BLOCK, kv_shared: bool = False, mask: Optional[BlockMask] = None,
         dense_out: bool = False, logits_out=None, workspace=None, stream=None) -> BlockMask:
    """AttnGate + block selection (seer_gate).  Returns the block mask (of
    `block`-token blocks, 64 or 128).  With rope_theta > 0 (the model's RoPE
    base) q and k are pre-RoPE and the gate applies its block-level RoPE.  With
    kv_shared one mask per KV group is selected from the mean of the group's
    head probabilities."""
    torch = _torch()
    d = make_desc(q, k)
    gd = gate_desc(wq.shape[-1], mode, topk_ratio, topk_k, threshold, head_thresholds,
                   keep_first, keep_diag, w_per_head, rope_theta, block, kv_shared)
    if mask is None:
        heads = k.shape[1] if kv_shared else q.shape[1]
        mask = alloc_mask(q.shape[0], heads, q.shape[2], q.device, dense=dense_out, block=block,
                          kv_shared=kv_shared)
    mask.block = block
    need = lib().seer_gate_workspace_bytes(C.byref(d), C.byref(gd), int(logits_out is None))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    ms = mask.struct()
    st = lib().seer_gate(C.byref(d), C.byref(gd), _ptr(q), _ptr(k), _ptr(wq), _ptr(wk),
                         C.byref(ms), _ptr(logits_out), _ptr(workspace), workspace.numel(),
                         _stream(stream))
    _check(st, "seer_gate")
    return mask


def gate_noalloc(q, k, wq, wk, mask: "BlockMask", *, mode: int, topk_ratio: float = 0.0, topk_k: int = 0,
                 threshold: float = 0.0, head_thresholds=None, keep_first: bool = True,
                 keep_diag: bool = True, w_per_head: bool = True, rope_theta: float = 0.0,
                 block: int = BLOCK, stream=None) -> "BlockMask":
    """seer_gate_noalloc: the gate without a workspace and without any
    allocation (its scratch is a static device array of
    gate_noalloc_max_bytes()); the caller passes the output mask.  Calls that
    overlap on one device share the scratch and race."""
    if mask is None:
        raise ValueError("gate_noalloc allocates nothing: pass the output mask")
    d = make_desc(q, k)
    gd = gate_desc(wq.shape[-1], mode, topk_ratio, topk_k, threshold, head_thresholds,
                   keep_first, keep_diag, w_per_head, rope_theta, block, False)
    mask.block = block
    ms = mask.struct()
    st = lib().seer_gate_noalloc(C.byref(d), C.byref(gd), _ptr(q), _ptr(k), _ptr(wq), _ptr(wk), C.byref(ms),
                                 _stream(stream))
    _check(st, "seer_gate_noalloc")
    return mask


def gate_noalloc_max_bytes() -> int:
    """Size of seer_gate_noalloc's static device scratch."""
    return lib().seer_gate_noalloc_max_bytes()


def attn_workspace_bytes(q, k, v=None, causal: bool = True, opts=None) -> int:
    """Workspace that enables the key-range split of bsattn / dense_attn for
    this shape and options (0: the call does not split)."""
    d = make_desc(q, k, v)
    return lib().seer_attn_workspace_bytes(C.byref(d), BLOCK, int(bool(causal)), _opts_ref(opts, AttnOpts))


def attn_launches(q, k, v=None, mask: Optional["BlockMask"] = None, *, causal: bool = True, opts=None,
                  workspace_bytes: int = 0) -> int:
    """Attention-kernel launches one bsattn (mask given) or dense_attn call with
    these arguments makes on the current device (seer_attn_launches)."""
    d = make_desc(q, k, v)
    kind = 0 if mask is None else (2 if mask.kv_shared else 1)
    block = BLOCK if mask is None else mask.block
    n = lib().seer_attn_launches(C.byref(d), block, kind, int(bool(causal)), _opts_ref(opts, AttnOpts),
                                 int(workspace_bytes))
    if n < 0:
        raise ValueError("seer_attn_launches: invalid arguments")
    return n


def _ws_args(workspace):
    if workspace is None:
        return None, 0
    return _ptr(workspace), workspace.numel() * workspace.element_size()


def bsattn(q, k, v, mask: BlockMask, *, causal: bool = True, sm_scale: float = 0.0, out=None,
           lse: Optional[object] = None, want_lse: bool = False, workspace=None, opts=None, stream=None):
    """Block-sparse attention (seer_bsattn; seer_bsattn_ws with a workspace or
    launch options -- a dict of seer_attn_opts fields or an AttnOpts).
    Returns (O, LSE or None)."""
    torch = _torch()
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
    d = make_desc(q, k, v, out)
    ms = mask.struct()
    block = mask.block  # 64- or 128-token mask blocks
    if workspace is None and opts is None:
        st = lib().seer_bsattn(C.byref(d), block, C.byref(ms), int(bool(causal)), float(sm_scale),
                               _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), _stream(stream))
        _check(st, "seer_bsattn")
    else:
        wp, wn = _ws_args(workspace)
        st = lib().seer_bsattn_ws(C.byref(d), block, C.byref(ms), int(bool(causal)), float(sm_scale),
                                  _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), wp, wn,
                                  _opts_ref(opts, AttnOpts), _stream(stream))
        _check(st, "seer_bsattn_ws")
    return out, lse


def dense_attn(q, k, v, *, causal: bool = True, sm_scale: float = 0.0, out=None,
               lse: Optional[object] = None, want_lse: bool = False, workspace=None, opts=None, stream=None):
    """Dense attention over every (causal) block (seer_dense_attn; seer_dense_attn_ws
    with a workspace or launch options).  Returns (O, LSE or None)."""
    torch = _torch()
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
    d = make_desc(q, k, v, out)
    if workspace is None and opts is None:
        st = lib().seer_dense_attn(C.byref(d), int(bool(causal)), float(sm_scale), _ptr(q), _ptr(k),
                                   _ptr(v), _ptr(out), _ptr(lse), _stream(stream))
        _check(st, "seer_dense_attn")
    else:
        wp, wn = _ws_args(workspace)
        st = lib().seer_dense_attn_ws(C.byref(d), int(bool(causal)), float(sm_scale), _ptr(q), _ptr(k),
                                      _ptr(v), _ptr(out), _ptr(lse), wp, wn, _opts_ref(opts, AttnOpts),
                                      _stream(stream))
        _check(st, "seer_dense_attn_ws")
    return out, lse


def attn_gt_workspace_bytes(q, k, v=None, kv_groups: int = 0) -> int:
    """Workspace of attn_gt running `kv_groups` KV groups per launch (0: all)."""
    d = make_desc(q, k, v)
    return lib().seer_attn_gt_workspace_bytes(C.byref(d), BLOCK, int(kv_groups))


def attn_gt(q, k, v, *, causal: bool = True, sm_scale: float = 0.0, out=None,
            lse: Optional[object] = None, want_lse: bool = False, gt=None, workspace=None,
            kv_groups: int = 0, opts=None, stream=None):
    """Dense attention plus the 2D max-pooled attention map (seer_attn_gt).
    Returns (O, LSE or None, gt [B, Hq, nb, nb] fp32).  Without a workspace,
    one sized for `kv_groups` KV groups per launch (0: all) is allocated."""
    torch = _torch()
    B, Hq, S, _ = q.shape
    nb = -(-S // BLOCK)  # the last block may be partial
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
    if gt is None:
        gt = torch.empty((B, Hq, nb, nb), dtype=torch.float32, device=q.device)
    d = make_desc(q, k, v, out)
    if workspace is None:
        n = lib().seer_attn_gt_workspace_bytes(C.byref(d), BLOCK, int(kv_groups))
        workspace = torch.empty(max(n, 1), dtype=torch.uint8, device=q.device)
    st = lib().seer_attn_gt(C.byref(d), BLOCK, int(bool(causal)), float(sm_scale), _ptr(q), _ptr(k),
                            _ptr(v), _ptr(out), _ptr(lse), _ptr(gt), _ptr(workspace),
                            workspace.numel() * workspace.element_size(), _opts_ref(opts, AttnOpts),
                            _stream(stream))
    _check(st, "seer_attn_gt")
    return out, lse, gt


def gate_distill_workspace_bytes(q, k, wq, wk, *, w_per_head: bool = True, rope_theta: float = 0.0,
                                 opts=None) -> int:
    """Workspace of gate_distill for these shapes and options."""
    d = make_desc(q, k)
    gd = gate_desc(wq.shape[-1], TOPK_RATIO, topk_ratio=1.0, w_per_head=w_per_head, rope_theta=rope_theta)
    return lib().seer_gate_distill_workspace_bytes(C.byref(d), C.byref(gd), _opts_ref(opts, DistillOpts))


def gate_distill(q, k, wq, wk, gt, *, w_per_head: bool = True, rope_theta: float = 0.0,
                 dwq=None, dwk=None, loss=None, workspace=None, opts=None, stream=None):
    """One gate distillation step (seer_gate_distill): returns (loss [1], dwq, dwk)
    as device fp32 tensors; loss is the mean KL(renormalised gt || gate softmax)."""
    torch = _torch()
    d = make_desc(q, k)
    gd = gate_desc(wq.shape[-1], TOPK_RATIO, topk_ratio=1.0, w_per_head=w_per_head,
                   rope_theta=rope_theta)
    if dwq is None:
        dwq = torch.empty_like(wq)
    if dwk is None:
        dwk = torch.empty_like(wk)
    if loss is None:
        loss = torch.empty(1, dtype=torch.float32, device=q.device)
    if workspace is None:
        n = lib().seer_gate_distill_workspace_bytes(C.byref(d), C.byref(gd), _opts_ref(opts, DistillOpts))
        workspace = torch.empty(max(n, 1), dtype=torch.uint8, device=q.device)
    st = lib().seer_gate_distill(C.byref(d), C.byref(gd), _ptr(q), _ptr(k), _ptr(wq), _ptr(wk),
                                 _ptr(gt), _ptr(loss), _ptr(dwq), _ptr(dwk), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), _opts_ref(opts, DistillOpts),
                                 _stream(stream))
    _check(st, "seer_gate_distill")
    return loss, dwq, dwk


def mask_from_dense(dense, heads_kv: int = 1, mask: Optional[BlockMask] = None,
                    block: int = BLOCK, kv_shared: bool = False, stream=None) -> BlockMask:
    """Compacts a uint8 [B, H, nb, nb] device mask of `block`-token blocks
    (seer_mask_from_dense); H = Hq, or Hkv for a kv_shared mask."""
    torch = _torch()
    B, H, nb, _ = dense.shape
    if mask is None:
        mask = alloc_mask(B, H, nb * block, dense.device, block=block, kv_shared=kv_shared)
    mask.block = block
    mask.kv_shared = kv_shared
    d = AttnDesc()
    d.batch, d.heads_q, d.heads_kv, d.seq_len, d.head_dim, d.dtype = B, H, (H if kv_shared else heads_kv), \
        nb * block, 128, BF16
    ms = mask.struct()
    st = lib().seer_mask_from_dense(C.byref(d), block, _ptr(dense.contiguous()), C.byref(ms),
                                    _stream(stream))
    _check(st, "seer_mask_from_dense")
    return mask


# ---------------------------------------------------------------------------
# packed variable-length batches
# ---------------------------------------------------------------------------

def make_varlen_desc(q, k, cu_seqlens, v=None, o=None) -> AttnDesc:
    """Descriptor of packed [T, H, D] tensors holding len(cu_seqlens) - 1 sequences."""
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o)):
        if t is not None and (t.dim() != 3 or t.stride(2) != 1):
            raise ValueError(f"{name} must be packed [tokens, heads, head_dim] with unit last stride")
    d = AttnDesc()
    d.batch = len(cu_seqlens) - 1
    d.heads_q, d.seq_len, d.head_dim = q.shape[1], q.shape[0], q.shape[2]
    d.heads_kv = k.shape[1]
    d.dtype = _dtype_code(q)
    for field, t in (("q_stride", q), ("k_stride", k), ("v_stride", v if v is not None else k),
                     ("o_stride", o if o is not None else q)):
        arr = getattr(d, field)
        arr[0], arr[1], arr[2] = 0, t.stride(1), t.stride(0)
    return d


def _cu_host(cu_seqlens):
    cu = [int(x) for x in (cu_seqlens.tolist() if hasattr(cu_seqlens, "tolist") else cu_seqlens)]
    return (C.c_int32 * len(cu))(*cu), cu


@dataclass
class VarlenMask:
    """Block masks of a packed batch: sequence b's count rows [H, nb_b] and idx rows
    [H, nb_b, nb_b] stored back to back in flat device arrays."""
    count: object  # int32 [sum_b H nb_b]
    idx: object    # int16 storage of uint16 [sum_b H nb_b^2]
    cu_seqlens: list
    heads: int
    block: int = BLOCK
    kv_shared: bool = False
    dense: Optional[object] = None  # uint8, same layout as idx

    def struct(self) -> BlockMaskStruct:
        m = BlockMaskStruct()
        m.n_blocks = 0
        m.count = _ptr(self.count)
        m.idx = _ptr(self.idx)
        m.dense = _ptr(self.dense)
        m.kv_shared = int(bool(self.kv_shared))
        return m

    def sequence(self, b: int):
        """(count [H, nb_b], idx [H, nb_b, nb_b]) views of sequence b."""
        nbs = [-(-(self.cu_seqlens[s + 1] - self.cu_seqlens[s]) // self.block) for s in range(len(self.cu_seqlens) - 1)]
        c0 = sum(self.heads * n for n in nbs[:b])
        i0 = sum(self.heads * n * n for n in nbs[:b])
        nb = nbs[b]
        return (self.count[c0:c0 + self.heads * nb].view(self.heads, nb),
                self.idx[i0:i0 + self.heads * nb * nb].view(self.heads, nb, nb))


def alloc_varlen_mask(q, k, cu_seqlens, block: int = BLOCK, kv_shared: bool = False,
                      dense: bool = False) -> VarlenMask:
    torch = _torch()
    cu_arr, cu = _cu_host(cu_seqlens)
    d = make_varlen_desc(q, k, cu)
    n_count = C.c_size_t(0)
    n_idx = lib().seer_varlen_mask_elems(C.byref(d), cu_arr, block, int(bool(kv_shared)), C.byref(n_count))
    if n_idx == 0 and cu[-1] > 0:
        raise ValueError("invalid packed batch description")
    heads = k.shape[1] if kv_shared else q.shape[1]
    return VarlenMask(count=torch.empty(max(n_count.value, 1), dtype=torch.int32, device=q.device),
                      idx=torch.empty(max(n_idx, 1), dtype=torch.int16, device=q.device), cu_seqlens=cu,
                      heads=heads, block=block, kv_shared=kv_shared,
                      dense=torch.empty(max(n_idx, 1), dtype=torch.uint8, device=q.device) if dense else None)


def gate_varlen(q, k, wq, wk, cu_seqlens, *, mode: int, topk_ratio: float = 0.0, topk_k: int = 0,
                threshold: float = 0.0, head_thresholds=None, keep_first: bool = True, keep_diag: bool = True,
                w_per_head: bool = True, rope_theta: float = 0.0, block: int = BLOCK, kv_shared: bool = False,
                mask: Optional[VarlenMask] = None, dense_out: bool = False, workspace=None,
                stream=None) -> VarlenMask:
    """seer_gate_varlen: the gate of every sequence of a packed [T, H, D] batch."""
    torch = _torch()
    cu_arr, cu = _cu_host(cu_seqlens)
    d = make_varlen_desc(q, k, cu)
    gd = gate_desc(wq.shape[-1], mode, topk_ratio, topk_k, threshold, head_thresholds,
                   keep_first, keep_diag, w_per_head, rope_theta, block, kv_shared)
    if mask is None:
        mask = alloc_varlen_mask(q, k, cu, block, kv_shared, dense_out)
    need = lib().seer_gate_varlen_workspace_bytes(C.byref(d), cu_arr, C.byref(gd))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    ms = mask.struct()
    st = lib().seer_gate_varlen(C.byref(d), cu_arr, C.byref(gd), _ptr(q), _ptr(k), _ptr(wq), _ptr(wk),
                                C.byref(ms), _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "seer_gate_varlen")
    return mask


def bsattn_varlen(q, k, v, cu_seqlens, mask: VarlenMask, *, causal: bool = True, sm_scale: float = 0.0,
                  out=None, lse=None, want_lse: bool = False, stream=None):
    """seer_bsattn_varlen: block-sparse attention of every sequence of a packed batch.
    Returns (O [T, Hq, D], LSE or None); LSE is flat, sequence b's [Hq, len_b] block
    starting at element Hq * cu[b]."""
    torch = _torch()
    cu_arr, cu = _cu_host(cu_seqlens)
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(max(q.shape[0] * q.shape[1], 1), dtype=torch.float32, device=q.device)
    d = make_varlen_desc(q, k, cu, v, out)
    ms = mask.struct()
    st = lib().seer_bsattn_varlen(C.byref(d), cu_arr, mask.block, C.byref(ms), int(bool(causal)),
                                  float(sm_scale), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse),
                                  _stream(stream))
    _check(st, "seer_bsattn_varlen")
    return out, lse
