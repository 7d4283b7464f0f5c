"""Host-side checks of the C ABI (no GPU needed): the library loads, exports every
symbol include/seer.h declares, and rejects invalid arguments before any launch.

Every call below returns from argument validation, which touches no device."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "seer.h")

seer = pytest.importorskip("paper_2410_13276_amd")
if not os.path.exists(seer.LIB_PATH):
    pytest.skip("libseer.so not built", allow_module_level=True)


def declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(seer_[a-z_]+)\s*\(", txt)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) == 22, names
    L = C.CDLL(seer.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(seer._SIGS)


def test_version_and_status_strings():
    assert seer.abi_version() == 5
    assert seer.status_str(0) == "SEER_OK"
    assert seer.status_str(3) == "SEER_ERR_WORKSPACE"
    assert seer.status_str(99) == "SEER_ERR_UNKNOWN"


def _desc(B=1, Hq=4, Hkv=2, S=1024, D=128, dtype=0):
    d = seer.AttnDesc()
    d.batch, d.heads_q, d.heads_kv, d.seq_len, d.head_dim, d.dtype = B, Hq, Hkv, S, D, dtype
    for f, H in (("q_stride", Hq), ("k_stride", Hkv), ("v_stride", Hkv), ("o_stride", Hq)):
        arr = getattr(d, f)
        arr[0], arr[1], arr[2] = H * S * D, S * D, D
    return d


def _gate(**kw):
    g = seer.gate_desc(128, seer.TOPK_RATIO, topk_ratio=0.5)
    for k, v in kw.items():
        setattr(g, k, v)
    return g


FAKE = 0x1000  # a 16-byte aligned non-NULL address; never dereferenced on these paths


def _call_gate(d, g, ws_bytes=1 << 40, mask_nb=None, q=FAKE, ws=FAKE * 16):
    L = seer.lib()
    m = seer.BlockMaskStruct()
    m.n_blocks = (d.seq_len // 64) if mask_nb is None else mask_nb
    m.count, m.idx, m.dense = FAKE, FAKE, None
    return L.seer_gate(C.byref(d), C.byref(g), q, FAKE, FAKE, FAKE, C.byref(m), None, ws, ws_bytes, None)


def _sr(nb):
    """Rows of one head's split gate rows (whole 32-row groups)."""
    return -(-nb // 32) * 32


def test_workspace_size_formula():
    d, g = _desc(B=2, Hq=4, Hkv=2, S=1024), _gate()
    L = seer.lib()
    nb = 16
    up = lambda x: (x + 255) // 256 * 256
    # Qg, Kg as three bf16 parts per element (the logits kernel; the fp32 rows
    # of the fused kernel share that region)
    want = up(2 * 4 * _sr(nb) * 3 * 128 * 2) + up(2 * 2 * _sr(nb) * 3 * 128 * 2)
    assert L.seer_gate_workspace_bytes(C.byref(d), C.byref(g), 0) == want
    assert L.seer_gate_workspace_bytes(C.byref(d), C.byref(g), 1) == want + up(2 * 4 * nb * nb * 4)
    assert L.seer_gate_noalloc_max_bytes() == 64 << 20
    assert L.seer_mask_idx_elems(C.byref(d), 64) == 2 * 4 * nb * nb
    assert L.seer_mask_idx_elems(C.byref(d), 128) == 2 * 4 * (nb // 2) ** 2   # 128-token blocks
    assert L.seer_mask_idx_elems(C.byref(d), 96) == 0


@pytest.mark.parametrize("field,value,status", [
    ("heads_kv", 3, seer.ERR_INVALID_ARG),     # heads_q % heads_kv != 0
    ("seq_len", 0, seer.ERR_INVALID_ARG),
    ("head_dim", 96, seer.ERR_UNSUPPORTED),
    ("dtype", 7, seer.ERR_INVALID_ARG),
    ("batch", 0, seer.ERR_INVALID_ARG),
])
def test_gate_rejects_bad_desc(field, value, status):
    d = _desc()
    setattr(d, field, value)
    assert _call_gate(d, _gate()) == status


@pytest.mark.parametrize("field,value,status", [
    ("block", 96, seer.ERR_UNSUPPORTED),
    ("gate_dim", 48, seer.ERR_UNSUPPORTED),
    ("mode", 9, seer.ERR_INVALID_ARG),
    ("topk_ratio", 0.0, seer.ERR_INVALID_ARG),
    ("topk_ratio", 1.5, seer.ERR_INVALID_ARG),
    ("rope_theta", -1.0, seer.ERR_INVALID_ARG),
    ("rope_theta", float("nan"), seer.ERR_INVALID_ARG),
    ("rope_theta", float("inf"), seer.ERR_INVALID_ARG),
])
def test_gate_rejects_bad_gate(field, value, status):
    assert _call_gate(_desc(), _gate(**{field: value})) == status


def test_gate_rejects_fixed_k_zero_and_nan_threshold():
    assert _call_gate(_desc(), _gate(mode=seer.TOPK_FIXED, topk_k=0)) == seer.ERR_INVALID_ARG
    assert _call_gate(_desc(), _gate(mode=seer.THRESHOLD, threshold=float("nan"))) == seer.ERR_INVALID_ARG


def test_gate_rejects_short_workspace_null_and_mask_shape():
    d, g = _desc(), _gate()
    need = seer.lib().seer_gate_workspace_bytes(C.byref(d), C.byref(g), 1)
    assert _call_gate(d, g, ws_bytes=need - 1) == seer.ERR_WORKSPACE
    assert _call_gate(d, g, ws=None) == seer.ERR_WORKSPACE
    assert _call_gate(d, g, q=None) == seer.ERR_INVALID_ARG
    assert _call_gate(d, g, q=FAKE + 2) == seer.ERR_INVALID_ARG  # misaligned
    assert _call_gate(d, g, mask_nb=15) == seer.ERR_INVALID_ARG


def test_attention_rejects_bad_args():
    L = seer.lib()
    d = _desc()
    m = seer.BlockMaskStruct()
    m.n_blocks, m.count, m.idx, m.dense = 16, FAKE, FAKE, None
    args = (FAKE, FAKE, FAKE, FAKE, None, None)
    assert L.seer_bsattn(C.byref(d), 96, C.byref(m), 1, 0.0, *args) == seer.ERR_UNSUPPORTED
    assert L.seer_bsattn(C.byref(d), 128, C.byref(m), 1, 0.0, *args) == seer.ERR_INVALID_ARG  # nb 16 != 8
    assert L.seer_bsattn(C.byref(d), 64, None, 1, 0.0, *args) == seer.ERR_INVALID_ARG
    m.n_blocks = 8
    assert L.seer_bsattn(C.byref(d), 64, C.byref(m), 1, 0.0, *args) == seer.ERR_INVALID_ARG
    assert L.seer_dense_attn(C.byref(d), 1, float("nan"), *args) == seer.ERR_INVALID_ARG
    assert L.seer_dense_attn(C.byref(d), 1, 0.0, None, FAKE, FAKE, FAKE, None, None) == seer.ERR_INVALID_ARG
    d.q_stride[2] = 100  # not a multiple of 8 bf16 elements (16 bytes)
    assert L.seer_dense_attn(C.byref(d), 1, 0.0, *args) == seer.ERR_UNSUPPORTED
    d = _desc()
    d.o_stride[2] = 64  # rows would overlap (stride < head_dim)
    assert L.seer_dense_attn(C.byref(d), 1, 0.0, *args) == seer.ERR_INVALID_ARG


def test_mask_from_dense_rejects_bad_args():
    L = seer.lib()
    d = _desc()
    m = seer.BlockMaskStruct()
    m.n_blocks, m.count, m.idx, m.dense = 16, FAKE, FAKE, None
    assert L.seer_mask_from_dense(C.byref(d), 64, None, C.byref(m), None) == seer.ERR_INVALID_ARG
    assert L.seer_mask_from_dense(C.byref(d), 32, FAKE, C.byref(m), None) == seer.ERR_UNSUPPORTED
    m.n_blocks = 3
    assert L.seer_mask_from_dense(C.byref(d), 64, FAKE, C.byref(m), None) == seer.ERR_INVALID_ARG


def test_attn_gt_workspace_and_rejects_bad_args():
    L = seer.lib()
    d = _desc(B=2, Hq=4, Hkv=2, S=1024, D=128)
    per_head = 16 * 16 * 64 * 4
    assert L.seer_attn_gt_workspace_bytes(C.byref(d), 64, 0) == 2 * 4 * per_head
    assert L.seer_attn_gt_workspace_bytes(C.byref(d), 64, 1) == 2 * per_head   # G = 2
    assert L.seer_attn_gt_workspace_bytes(C.byref(d), 64, 9) == 2 * 4 * per_head
    assert L.seer_attn_gt_workspace_bytes(C.byref(d), 128, 0) == 0
    args = (FAKE, FAKE, FAKE, FAKE, None)
    assert L.seer_attn_gt(C.byref(d), 64, 1, 0.0, *args, None, FAKE * 16, 1 << 40, None, None) == \
        seer.ERR_INVALID_ARG                                                  # no gt
    assert L.seer_attn_gt(C.byref(d), 64, 1, 0.0, *args, FAKE, FAKE * 16, 2 * per_head - 1, None, None) == \
        seer.ERR_WORKSPACE
    assert L.seer_attn_gt(C.byref(d), 64, 1, 0.0, *args, FAKE, None, 1 << 40, None, None) == seer.ERR_WORKSPACE
    assert L.seer_attn_gt(C.byref(d), 64, 1, 0.0, *args, FAKE, FAKE * 16 + 16, 1 << 40, None, None) == \
        seer.ERR_INVALID_ARG                                                  # misaligned workspace
    assert L.seer_attn_gt(C.byref(d), 128, 1, 0.0, *args, FAKE, FAKE * 16, 1 << 40, None, None) == \
        seer.ERR_UNSUPPORTED


def test_gate_distill_workspace_and_rejects_bad_args():
    L = seer.lib()
    d, g = _desc(B=1, Hq=4, Hkv=2, S=1024, D=128), _gate()
    nb, up = 16, (lambda x: (x + 255) // 256 * 256)
    # Qg, Kg, their bf16 parts, Qp, Kp, logits, dQg, dKg, row losses + 64 partial sums; no
    # product splits at this size
    want = (up(4 * nb * 128 * 4) + up(2 * nb * 128 * 4) + up(4 * _sr(nb) * 3 * 128 * 2) + up(2 * _sr(nb) * 3 * 128 * 2)
            + up(4 * nb * 128 * 4) + up(2 * nb * 384 * 4)
            + up(4 * nb * nb * 4) + up(4 * nb * 128 * 4) + up(2 * nb * 128 * 4) + up((4 * nb + 64) * 8))
    need = L.seer_gate_distill_workspace_bytes(C.byref(d), C.byref(g), None)
    assert need == want
    g.mode = 9  # the selection mode is not used by the distillation step
    assert L.seer_gate_distill_workspace_bytes(C.byref(d), C.byref(g), None) == want
    call = lambda gt=FAKE, ws=FAKE * 16, n=need, gd=g: L.seer_gate_distill(
        C.byref(d), C.byref(gd), FAKE, FAKE, FAKE, FAKE, gt, FAKE, FAKE, FAKE, ws, n, None, None)
    assert call(gt=None) == seer.ERR_INVALID_ARG
    assert call(n=need - 1) == seer.ERR_WORKSPACE
    assert call(ws=None) == seer.ERR_WORKSPACE
    assert call(ws=FAKE * 16 + 16) == seer.ERR_INVALID_ARG
    assert call(gd=_gate(gate_dim=48)) == seer.ERR_UNSUPPORTED
    assert call(gd=_gate(rope_theta=-2.0)) == seer.ERR_INVALID_ARG


def _gemm_tile_n(N, K2, tile_n=0):
    """Output tile width of a distillation product: the option when set, else
    128 columns for N >= 128 with a contraction of at least 1024, else 64."""
    if tile_n in (64, 128):
        return tile_n
    return 128 if N >= 128 and K2 >= 1024 else 64


def _gemm_splits(M, N, K1, K2, Z, min_chunks=8, tile_n=0):
    """The split rule of the distillation products: about 2048 workgroups of
    64x64 output tiles, or 1024 of 64x128 ones, when the tiles are fewer, at
    least `min_chunks` 32-wide K chunks per part, at most 64 parts."""
    tn = _gemm_tile_n(N, K2, tile_n)
    tiles = -(-N // tn) * -(-M // 64) * Z
    chunks = K1 * -(-K2 // 32)
    return max(1, min(-(-(2048 * 64 // tn) // tiles), chunks // min_chunks, 64))


@pytest.mark.parametrize("nb,min_chunks,tile_n", [(512, None, 0), (512, 1, 0), (512, None, 128),
                                                  (1024, None, 0), (1024, 2, 64), (2048, None, 0)])
def test_gate_distill_workspace_split_products(nb, min_chunks, tile_n):
    """32 q / 8 kv heads: the backward products split their K range; the
    workspace holds the largest product's parts (gemm_min_chunks: at least that
    many K chunks per part; gemm_tile_n: the output tile width)."""
    fields = {}
    if min_chunks is not None:
        fields["gemm_min_chunks"] = min_chunks
    if tile_n:
        fields["gemm_tile_n"] = tile_n
    opts = C.byref(seer.DistillOpts(**fields)) if fields else None
    mc = min_chunks or 8
    L = seer.lib()
    B, Hq, Hkv, D, Dg = 1, 32, 8, 128, 128
    d, g = _desc(B=B, Hq=Hq, Hkv=Hkv, S=64 * nb, D=D), _gate()
    up = lambda x: (x + 255) // 256 * 256
    base = (up(Hq * nb * Dg * 4) + up(Hkv * nb * Dg * 4) + up(Hq * _sr(nb) * 3 * Dg * 2) + up(Hkv * _sr(nb) * 3 * Dg * 2)
            + up(Hq * nb * D * 4) + up(Hkv * nb * 3 * D * 4)
            + up(Hq * nb * nb * 4) + up(Hq * nb * Dg * 4) + up(Hkv * nb * Dg * 4) + up((Hq * nb + 64) * 8))
    products = [(nb, Dg, 1, nb, Hq), (nb, Dg, Hq // Hkv, nb, Hkv), (D, Dg, 1, nb, Hq), (3 * D, Dg, 1, nb, Hkv)]
    part = 0
    for M, N, K1, K2, Z in products:
        sp = _gemm_splits(M, N, K1, K2, Z, mc, tile_n)
        if sp > 1:
            part = max(part, Z * sp * M * N)
    assert part > 0
    assert L.seer_gate_distill_workspace_bytes(C.byref(d), C.byref(g), opts) == base + up(4 * part)


def test_gate_distill_rejects_bad_tile_width():
    L = seer.lib()
    d, g = _desc(B=1, Hq=2, Hkv=1, S=1024, D=64), _gate()
    for t in (32, 96, 256, -64):
        assert L.seer_gate_distill_workspace_bytes(C.byref(d), C.byref(g),
                                                   C.byref(seer.DistillOpts(gemm_tile_n=t))) == 0
    assert L.seer_gate_distill_workspace_bytes(C.byref(d), C.byref(g),
                                               C.byref(seer.DistillOpts(gemm_tile_n=64))) > 0


def test_attn_workspace_bytes_formula():
    L = seer.lib()
    up = lambda x: (x + 255) // 256 * 256
    opt = lambda **kw: C.byref(seer.AttnOpts(**kw))

    def want(Hq, nb, w, D):
        P = -(-nb // w)
        slots = sum(i // w + 1 for i in range(nb))
        return up(Hq * nb * (P + 3) * 4) + up(8 * 4) + up(Hq * slots * 64 * 4) + up(Hq * slots * 64 * D * 2)

    d = _desc(B=1, Hq=32, Hkv=8, S=131072, D=128)
    assert L.seer_attn_workspace_bytes(C.byref(d), 64, 1, None) == 0            # the split is opt-in
    assert L.seer_attn_workspace_bytes(C.byref(d), 64, 1, opt()) == 0
    # ranges sized to the L2: 128 blocks (4 MiB of K and V) at head_dim 128
    assert L.seer_attn_workspace_bytes(C.byref(d), 64, 1, opt(split=1)) == want(32, 2048, 128, 128)
    assert L.seer_attn_workspace_bytes(C.byref(d), 64, 0, opt(split=1)) == 0    # non-causal: no split
    assert L.seer_attn_workspace_bytes(C.byref(d), 64, 1, opt(split=1, split_width=300)) == \
        want(32, 2048, 300, 128)                                                # a partial last range
    assert L.seer_attn_workspace_bytes(C.byref(d), 64, 1, opt(split=2)) == 0     # invalid option
    d.dtype = 1
    assert L.seer_attn_workspace_bytes(C.byref(d), 64, 1, opt(split=1)) == 0    # fp32: no split
    d = _desc(B=1, Hq=4, Hkv=2, S=8192, D=64)                                  # nb 128 <= 256 at D 64
    assert L.seer_attn_workspace_bytes(C.byref(d), 64, 1, opt(split=1)) == 0
    assert L.seer_attn_workspace_bytes(C.byref(d), 64, 1, opt(split=1, split_width=5)) == want(4, 128, 5, 64)


def test_gate_noalloc_rejects_unsupported_and_oversized():
    """The no-allocation gate validates before touching its scratch: the shared
    mask and rows of more than 2048 blocks are unsupported, and shapes whose
    projected rows exceed the 64 MiB scratch are refused (SEER_ERR_WORKSPACE)."""
    L = seer.lib()
    m = seer.BlockMaskStruct()
    call = lambda d, g, nb: (setattr(m, "n_blocks", nb), setattr(m, "count", FAKE), setattr(m, "idx", FAKE),
                             setattr(m, "kv_shared", g.kv_shared),
                             L.seer_gate_noalloc(C.byref(d), C.byref(g), FAKE, FAKE, FAKE, FAKE, C.byref(m),
                                                 None))[-1]
    assert call(_desc(S=64 * 2049), _gate(), 2049) == seer.ERR_UNSUPPORTED          # > 2048 blocks
    assert call(_desc(), _gate(kv_shared=1), 16) == seer.ERR_UNSUPPORTED            # shared mask
    # (64 + 8) heads x 2048 blocks x 128 x 4 B = 72 MiB of projected rows > 64 MiB
    assert call(_desc(Hq=64, Hkv=8, S=131072), _gate(), 2048) == seer.ERR_WORKSPACE
    assert call(_desc(), _gate(), 15) == seer.ERR_INVALID_ARG                        # mask shape
    assert L.seer_gate_noalloc(C.byref(_desc()), C.byref(_gate()), None, FAKE, FAKE, FAKE, C.byref(m),
                               None) == seer.ERR_INVALID_ARG


def test_attn_launches_rejects_bad_args():
    """The launch-count query validates like the calls it mirrors (it needs a GPU
    only for the occupancy of the batched launches, so its counts are checked in
    the GPU tests)."""
    L = seer.lib()
    d = _desc()
    assert L.seer_attn_launches(None, 64, 1, 1, None, 0) == -1
    assert L.seer_attn_launches(C.byref(d), 64, 3, 1, None, 0) == -1      # mask kind 0, 1 or 2
    assert L.seer_attn_launches(C.byref(d), 96, 1, 1, None, 0) == -1      # 64- or 128-token blocks
    bad = seer.AttnOpts(split=5)
    assert L.seer_attn_launches(C.byref(d), 64, 1, 1, C.byref(bad), 0) == -1


def test_attention_ws_rejects_bad_args():
    L = seer.lib()
    d = _desc()
    m = seer.BlockMaskStruct()
    m.n_blocks, m.count, m.idx, m.dense = 16, FAKE, FAKE, None
    args = (FAKE, FAKE, FAKE, FAKE, None)
    assert L.seer_bsattn_ws(C.byref(d), 64, None, 1, 0.0, *args, FAKE * 16, 1 << 30, None, None) == \
        seer.ERR_INVALID_ARG
    for bad in (seer.AttnOpts(heads_per_wg=3), seer.AttnOpts(walk_classes=3), seer.AttnOpts(walk_classes=32),
                seer.AttnOpts(walk_classes=-1)):
        assert L.seer_bsattn_ws(C.byref(d), 64, C.byref(m), 1, 0.0, *args, None, 0, C.byref(bad), None) == \
            seer.ERR_INVALID_ARG
    assert L.seer_bsattn_ws(C.byref(d), 64, C.byref(m), 1, 0.0, *args, FAKE * 16 + 8, 1 << 30, None, None) == \
        seer.ERR_INVALID_ARG                                               # misaligned workspace
    assert L.seer_dense_attn_ws(C.byref(d), 1, float("inf"), *args, FAKE * 16, 1 << 30, None, None) == \
        seer.ERR_INVALID_ARG


def test_block_128_gate_and_mask_validation():
    L = seer.lib()
    d = _desc(B=1, Hq=4, Hkv=2, S=1088, D=128)   # 1088 = 8.5 x 128: 9 blocks, the last partial
    assert _call_gate(d, _gate(block=128), mask_nb=8) == seer.ERR_INVALID_ARG
    assert L.seer_mask_idx_elems(C.byref(d), 128) == 4 * 9 * 9
    d = _desc(B=1, Hq=4, Hkv=2, S=1024, D=128)
    assert _call_gate(d, _gate(block=128), mask_nb=16) == seer.ERR_INVALID_ARG  # mask must have 8 blocks
    g = _gate(block=128)
    need = L.seer_gate_workspace_bytes(C.byref(d), C.byref(g), 1)
    up = lambda x: (x + 255) // 256 * 256
    assert need == up(4 * _sr(8) * 3 * 128 * 2) + up(2 * _sr(8) * 3 * 128 * 2) + up(4 * 8 * 8 * 4)
    m = seer.BlockMaskStruct()
    m.n_blocks, m.count, m.idx, m.dense = 16, FAKE, FAKE, None
    assert L.seer_mask_from_dense(C.byref(d), 128, FAKE, C.byref(m), None) == seer.ERR_INVALID_ARG


def test_partial_last_block_sizes():
    """Sequences that are not a multiple of 64: ceil(S / block) blocks everywhere."""
    L = seer.lib()
    d, g = _desc(B=1, Hq=4, Hkv=2, S=1000, D=128), _gate()
    up = lambda x: (x + 255) // 256 * 256
    nb = 16  # ceil(1000 / 64)
    assert L.seer_mask_idx_elems(C.byref(d), 64) == 4 * nb * nb
    assert L.seer_gate_workspace_bytes(C.byref(d), C.byref(g), 0) == (
        up(4 * _sr(nb) * 3 * 128 * 2) + up(2 * _sr(nb) * 3 * 128 * 2))
    assert L.seer_attn_gt_workspace_bytes(C.byref(d), 64, 0) == 4 * nb * nb * 64 * 4
    assert _call_gate(d, g, mask_nb=15) == seer.ERR_INVALID_ARG


def test_kv_shared_flags_are_validated():
    """The shared-mask variant: the gate's and the mask's kv_shared flags must
    agree and be 0 or 1; the distillation step is per head only."""
    L = seer.lib()
    d = _desc()
    m = seer.BlockMaskStruct()
    m.n_blocks, m.count, m.idx, m.dense = 16, FAKE, FAKE, None
    m.kv_shared = 0
    g = _gate(kv_shared=1)  # mask rows per KV head requested, mask says per query head
    assert L.seer_gate(C.byref(d), C.byref(g), FAKE, FAKE, FAKE, FAKE, C.byref(m), None, FAKE * 16,
                       1 << 40, None) == seer.ERR_INVALID_ARG
    assert _call_gate(_desc(), _gate(kv_shared=2)) == seer.ERR_INVALID_ARG
    m.kv_shared = 2
    args = (FAKE, FAKE, FAKE, FAKE, None, None)
    assert L.seer_bsattn(C.byref(d), 64, C.byref(m), 1, 0.0, *args) == seer.ERR_INVALID_ARG
    assert L.seer_mask_from_dense(C.byref(d), 64, FAKE, C.byref(m), None) == seer.ERR_INVALID_ARG
    gt = _gate(kv_shared=1)
    assert L.seer_gate_distill(C.byref(d), C.byref(gt), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                               FAKE * 16, 1 << 40, None, None) == seer.ERR_UNSUPPORTED


def test_varlen_rejects_bad_offsets_and_sizes_the_mask():
    L = seer.lib()
    d = _desc(B=3, Hq=4, Hkv=2, S=300)
    good = (C.c_int32 * 4)(0, 100, 100, 300)  # one empty sequence
    n_count = C.c_size_t(0)
    # nb = 2, 0, 4 blocks of 64: count 4 * (2 + 0 + 4), idx 4 * (4 + 0 + 16)
    assert L.seer_varlen_mask_elems(C.byref(d), good, 64, 0, C.byref(n_count)) == 80
    assert n_count.value == 24
    assert L.seer_varlen_mask_elems(C.byref(d), good, 64, 1, C.byref(n_count)) == 40  # per KV head
    m = seer.BlockMaskStruct()
    m.n_blocks, m.count, m.idx, m.dense, m.kv_shared = 0, FAKE, FAKE, None, 0
    g = _gate()
    args = (FAKE, FAKE, FAKE, FAKE, None, None)
    for bad in ((1, 100, 100, 300), (0, 200, 100, 300), (0, 100, 100, 299)):
        cu = (C.c_int32 * 4)(*bad)
        assert L.seer_varlen_mask_elems(C.byref(d), cu, 64, 0, None) == 0
        assert L.seer_gate_varlen(C.byref(d), cu, C.byref(g), FAKE, FAKE, FAKE, FAKE, C.byref(m), FAKE * 16,
                                  1 << 40, None) == seer.ERR_INVALID_ARG
        assert L.seer_bsattn_varlen(C.byref(d), cu, 64, C.byref(m), 1, 0.0, *args) == seer.ERR_INVALID_ARG
    assert L.seer_bsattn_varlen(C.byref(d), good, 96, C.byref(m), 1, 0.0, *args) == seer.ERR_UNSUPPORTED
    assert L.seer_gate_varlen(C.byref(d), good, C.byref(g), FAKE, FAKE, FAKE, FAKE, C.byref(m), None, 0,
                              None) == seer.ERR_WORKSPACE
