// seer_api.cpp -- the C ABI of libseer.so (declared in include/seer.h).
//
// Every entry point validates its arguments on the host before launching
// anything, then enqueues kernels on the caller's stream and returns without
// synchronising.  The library owns no memory and keeps no state.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "launch.h"
#include "seer.h"

namespace {

constexpr size_t kAlign = 256;

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t elem_size(int32_t dtype) { return dtype == SEER_F32 ? 4 : 2; }

// 64-token attention tiles covering seq_len (the last one may be partial).
int64_t tiles(int seq_len) { return (seq_len + SEER_BLOCK - 1) / SEER_BLOCK; }

// Checks shared by every call that takes a seer_attn_desc.  `tensors` selects
// which stride triples are used: bit 0 q, 1 k, 2 v, 3 o.
seer_status check_desc(const seer_attn_desc* d, int tensors) {
  if (!d) return SEER_ERR_INVALID_ARG;
  if (d->batch <= 0 || d->heads_q <= 0 || d->heads_kv <= 0 || d->seq_len <= 0 || d->head_dim <= 0)
    return SEER_ERR_INVALID_ARG;
  if (d->heads_q % d->heads_kv != 0) return SEER_ERR_INVALID_ARG;
  if (d->dtype != SEER_BF16 && d->dtype != SEER_F32) return SEER_ERR_INVALID_ARG;
  if (d->head_dim != 64 && d->head_dim != 128) return SEER_ERR_UNSUPPORTED;
  const int64_t vec = 16 / (int64_t)elem_size(d->dtype);  // elements per 16-byte access
  const int64_t* st[4] = {d->q_stride, d->k_stride, d->v_stride, d->o_stride};
  for (int t = 0; t < 4; ++t) {
    if (!(tensors & (1 << t))) continue;
    for (int e = 0; e < 3; ++e)
      if (st[t][e] < 0 || st[t][e] % vec != 0) return SEER_ERR_UNSUPPORTED;
    if (st[t][2] < d->head_dim) return SEER_ERR_INVALID_ARG;  // rows may not overlap
  }
  const int64_t tasks = (int64_t)d->batch * d->heads_q * tiles(d->seq_len);
  if (tasks > INT32_MAX / 2) return SEER_ERR_UNSUPPORTED;
  return SEER_OK;
}

seer::TensorView view(const void* p, const int64_t* st) { return {p, st[0], st[1], st[2]}; }

// Blocks of `block` tokens covering seq_len (the last one may be partial).
int blocks_of(int seq_len, int block) { return (seq_len + block - 1) / block; }

// Checks of the gate shape and weights (shared by seer_gate and seer_gate_distill).
seer_status check_gate_common(const seer_attn_desc* d, const seer_gate_desc* g) {
  seer_status s = check_desc(d, 0x3);
  if (s != SEER_OK) return s;
  if (!g) return SEER_ERR_INVALID_ARG;
  if (g->block != 64 && g->block != 128) return SEER_ERR_UNSUPPORTED;
  if (g->gate_dim != 32 && g->gate_dim != 64 && g->gate_dim != 128) return SEER_ERR_UNSUPPORTED;
  if (blocks_of(d->seq_len, g->block) > 4096) return SEER_ERR_UNSUPPORTED;
  if (!(g->rope_theta >= 0.0) || std::isinf(g->rope_theta)) return SEER_ERR_INVALID_ARG;
  if (g->kv_shared != 0 && g->kv_shared != 1) return SEER_ERR_INVALID_ARG;
  return SEER_OK;
}

seer_status check_gate(const seer_attn_desc* d, const seer_gate_desc* g) {
  seer_status s = check_gate_common(d, g);
  if (s != SEER_OK) return s;
  switch (g->mode) {
    case SEER_TOPK_RATIO:
      if (!(g->topk_ratio > 0.0 && g->topk_ratio <= 1.0)) return SEER_ERR_INVALID_ARG;
      break;
    case SEER_TOPK_FIXED:
      if (g->topk_k < 1) return SEER_ERR_INVALID_ARG;
      break;
    case SEER_THRESHOLD:
      if (!g->head_thresholds && std::isnan(g->threshold)) return SEER_ERR_INVALID_ARG;
      break;
    default:
      return SEER_ERR_INVALID_ARG;
  }
  return SEER_OK;
}

// Gate workspace: the projected rows Qg, Kg, then the logits when they live in
// the workspace.  The rows are fp32 for the fused kernel, or three bf16 parts
// per element for the logits kernel; one call uses one of the two forms, so
// they share the region (split = false: the fp32 form only).
struct GateLayout {
  size_t qg, kg, qs, ks, logits, total;
};

GateLayout gate_layout(const seer_attn_desc* d, const seer_gate_desc* g, bool logits_in_ws, bool split = true) {
  const size_t nb = (size_t)blocks_of(d->seq_len, g->block);
  const size_t Dg = g->gate_dim;
  const size_t ns = (size_t)seer::split_rows((int)nb);
  GateLayout L;
  L.qg = 0;
  L.kg = round_up((size_t)d->batch * d->heads_q * nb * Dg * 4);
  size_t rows_end = L.kg + round_up((size_t)d->batch * d->heads_kv * nb * Dg * 4);
  L.qs = 0;
  L.ks = round_up((size_t)d->batch * d->heads_q * ns * 3 * Dg * 2);
  if (split) rows_end = std::max(rows_end, L.ks + round_up((size_t)d->batch * d->heads_kv * ns * 3 * Dg * 2));
  L.logits = rows_end;
  L.total = L.logits + (logits_in_ws ? round_up((size_t)d->batch * d->heads_q * nb * nb * 4) : 0);
  return L;
}

// The four backward products of seer_gate_distill (pointers may be null when
// only the shapes are wanted):
//   dQg[b,h] = dL[b,h] Kg[b,g] / sqrt(Dg)                       (dL lower triangular)
//   dKg[b,g][j] = sum over the group's heads h and rows i of dL[b,h][i][j] Qg[b,h][i] / sqrt(Dg)
//   dWq[h] = sum over b, i of Qp[b,h,i]^T dQg[b,h,i]           (shared weights: also over h)
//   dWk[g] = sum over b, j of Kp[b,g,j]^T dKg[b,g,j]
struct DistillGemms {
  seer::GemmArgs dqg, dkg, dwq, dwk;
};

DistillGemms distill_gemms(int B, int Hq, int Hkv, int D, int Dg, int nb, bool ph, int min_chunks, int tile_n,
                           const float* dl, const float* qg, const float* kg, const float* qp, const float* kp,
                           float* dqg, float* dkg, float* dwq, float* dwk, float* part) {
  const int G = Hq / Hkv;
  const int64_t nn = (int64_t)nb * nb;
  const float rsqrt_dg = (float)(1.0 / std::sqrt((double)Dg));
  DistillGemms r;
  seer::GemmArgs g{};
  g.A = dl; g.B = kg; g.C = dqg;
  g.M = nb; g.N = Dg; g.K1 = 1; g.K2 = nb; g.Z = B * Hq; g.bdiv = G; g.tri = 1;
  g.sam = nb; g.sak1 = 0; g.sak2 = 1; g.saz = nn;
  g.sbk1 = 0; g.sbk2 = Dg; g.sbn = 1; g.sbz = (int64_t)nb * Dg;
  g.scm = Dg; g.scz = (int64_t)nb * Dg;
  g.alpha = rsqrt_dg;
  g.part = part;
  r.dqg = g;

  g = seer::GemmArgs{};
  g.A = dl; g.B = qg; g.C = dkg;
  g.M = nb; g.N = Dg; g.K1 = G; g.K2 = nb; g.Z = B * Hkv; g.bdiv = 1; g.tri = 2;
  g.sam = 1; g.sak1 = nn; g.sak2 = nb; g.saz = G * nn;
  g.sbk1 = (int64_t)nb * Dg; g.sbk2 = Dg; g.sbn = 1; g.sbz = (int64_t)G * nb * Dg;
  g.scm = Dg; g.scz = (int64_t)nb * Dg;
  g.alpha = rsqrt_dg;
  g.part = part;
  r.dkg = g;

  g = seer::GemmArgs{};
  g.A = qp; g.B = dqg; g.C = dwq;
  g.M = D; g.N = Dg; g.K2 = nb; g.bdiv = 1; g.tri = 0;
  g.sam = 1; g.sak2 = D;
  g.sbk2 = Dg; g.sbn = 1;
  g.scm = Dg; g.scz = (int64_t)D * Dg;
  g.alpha = 1.0f;
  g.part = part;
  if (ph) {
    g.Z = Hq; g.K1 = B;
    g.saz = (int64_t)nb * D; g.sak1 = (int64_t)Hq * nb * D;
    g.sbz = (int64_t)nb * Dg; g.sbk1 = (int64_t)Hq * nb * Dg;
  } else {
    g.Z = 1; g.K1 = B * Hq;
    g.saz = 0; g.sak1 = (int64_t)nb * D;
    g.sbz = 0; g.sbk1 = (int64_t)nb * Dg;
  }
  r.dwq = g;

  g = seer::GemmArgs{};
  g.A = kp; g.B = dkg; g.C = dwk;
  g.M = 3 * D; g.N = Dg; g.K2 = nb; g.bdiv = 1; g.tri = 0;
  g.sam = 1; g.sak2 = 3 * D;
  g.sbk2 = Dg; g.sbn = 1;
  g.scm = Dg; g.scz = (int64_t)3 * D * Dg;
  g.alpha = 1.0f;
  g.part = part;
  if (ph) {
    g.Z = Hkv; g.K1 = B;
    g.saz = (int64_t)nb * 3 * D; g.sak1 = (int64_t)Hkv * nb * 3 * D;
    g.sbz = (int64_t)nb * Dg; g.sbk1 = (int64_t)Hkv * nb * Dg;
  } else {
    g.Z = 1; g.K1 = B * Hkv;
    g.saz = 0; g.sak1 = (int64_t)nb * 3 * D;
    g.sbz = 0; g.sbk1 = (int64_t)nb * Dg;
  }
  r.dwk = g;
  for (seer::GemmArgs* x : {&r.dqg, &r.dkg, &r.dwq, &r.dwk}) {
    x->min_chunks = min_chunks;
    x->tile_n = tile_n;
  }
  return r;
}

// Workspace of seer_gate_distill: projected rows, pooled rows, logits (then
// their gradient), projected-row gradients, per-row losses, and the split
// products of the backward GEMMs (run one after another, so one buffer).
struct DistillLayout {
  size_t qg, kg, qs, ks, qp, kp, logits, dqg, dkg, row_loss, part, total;
};

DistillLayout distill_layout(const seer_attn_desc* d, const seer_gate_desc* g, int min_chunks, int tile_n) {
  const size_t nb = (size_t)blocks_of(d->seq_len, g->block);
  const size_t B = d->batch, Hq = d->heads_q, Hkv = d->heads_kv, D = d->head_dim, Dg = g->gate_dim;
  DistillLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += round_up(bytes);
    return at;
  };
  L.qg = take(B * Hq * nb * Dg * 4);
  L.kg = take(B * Hkv * nb * Dg * 4);
  L.qs = take(B * Hq * seer::split_rows((int)nb) * 3 * Dg * 2);
  L.ks = take(B * Hkv * seer::split_rows((int)nb) * 3 * Dg * 2);
  L.qp = take(B * Hq * nb * D * 4);
  L.kp = take(B * Hkv * nb * 3 * D * 4);
  L.logits = take(B * Hq * nb * nb * 4);
  L.dqg = take(B * Hq * nb * Dg * 4);
  L.dkg = take(B * Hkv * nb * Dg * 4);
  L.row_loss = take((B * Hq * nb + seer::kLossParts) * 8);
  const DistillGemms gm = distill_gemms((int)B, (int)Hq, (int)Hkv, (int)D, (int)Dg, (int)nb, g->w_per_head != 0,
                                        min_chunks, tile_n, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                        nullptr, nullptr, nullptr);
  int64_t part = 0;
  for (const seer::GemmArgs* a : {&gm.dqg, &gm.dkg, &gm.dwq, &gm.dwk})
    part = std::max(part, seer::gemm_partial_elems(*a));
  L.part = take((size_t)part * 4);
  L.total = off;
  return L;
}

seer_status from_hip(hipError_t e) { return e == hipSuccess ? SEER_OK : SEER_ERR_HIP; }

seer_status check_attn(const seer_attn_desc* desc, float sm_scale, const void* q,
                              const void* k, const void* v, const void* o) {
  seer_status s = check_desc(desc, 0xF);
  if (s != SEER_OK) return s;
  if (!q || !k || !v || !o) return SEER_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)) return SEER_ERR_INVALID_ARG;
  if (std::isnan(sm_scale) || std::isinf(sm_scale)) return SEER_ERR_INVALID_ARG;
  return SEER_OK;
}

seer::AttnArgs attn_args(const seer_attn_desc* desc, int32_t causal, float sm_scale,
                                const void* q, const void* k, const void* v, void* o, float* lse) {
  seer::AttnArgs a;
  a.q = view(q, desc->q_stride);
  a.k = view(k, desc->k_stride);
  a.v = view(v, desc->v_stride);
  a.o = o;
  a.osb = desc->o_stride[0];
  a.osh = desc->o_stride[1];
  a.oss = desc->o_stride[2];
  a.lse = lse;
  a.batch = desc->batch;
  a.heads_q = desc->heads_q;
  a.heads_kv = desc->heads_kv;
  a.n_blocks = blocks_of(desc->seq_len, SEER_BLOCK);
  a.seq_len = desc->seq_len;
  a.mask_blocks = 0;
  a.head_dim = desc->head_dim;
  a.bf16 = desc->dtype == SEER_BF16;
  a.causal = causal != 0;
  a.scale = sm_scale > 0.f ? sm_scale : (float)(1.0 / std::sqrt((double)desc->head_dim));
  a.count = nullptr;
  a.idx = nullptr;
  a.mask_shift = 0;
  a.mask_kv = false;
  a.pool_r = nullptr;
  a.gt = nullptr;
  a.split_parts = 0;
  a.split_w = 0;
  a.split_slots = 0;
  a.split_bounds = nullptr;
  a.split_tickets = nullptr;
  a.heads_per_wg = 2;
  a.batch_min_blocks = 2048;
  a.batch_wgs = 0;
  a.walk_classes = 4;  // measured: 131072 tokens 17.1 -> 14.4-14.7 ms, 65536 (GQA 7:1) 7.56 -> 7.25 ms
  a.part_lse = nullptr;
  a.part_o = nullptr;
  return a;
}

// Workspace of the key-range split: per-row records [rows][P + 3] int32 (range
// list offsets, non-empty range count, arrival counter), the task-queue tickets
// [8] int32, then the partial log-sum-exps [slots][64] fp32 and outputs
// [slots][64][D] bf16.
struct SplitLayout {
  int parts, w;
  int64_t slots;  // per (batch, head)
  size_t bounds, tickets, lse, o, total;
};

SplitLayout split_layout(const seer_attn_desc* d, int w) {
  SplitLayout L{};
  const int nb = blocks_of(d->seq_len, SEER_BLOCK);
  if (w <= 0) return L;
  L.w = w;
  L.parts = (nb + w - 1) / w;
  L.slots = seer::split_slots_per_head(nb, L.w);
  const size_t bh = (size_t)d->batch * d->heads_q;
  L.bounds = 0;
  L.tickets = round_up(bh * nb * (L.parts + 3) * sizeof(int32_t));
  L.lse = L.tickets + round_up(8 * sizeof(int32_t));
  L.o = L.lse + round_up(bh * L.slots * 64 * sizeof(float));
  L.total = L.o + round_up(bh * L.slots * 64 * d->head_dim * sizeof(uint16_t));
  return L;
}

int split_width_for(const seer_attn_desc* d, int32_t causal, const seer_attn_opts* o) {
  return seer::split_width(blocks_of(d->seq_len, SEER_BLOCK), d->head_dim, causal != 0, d->dtype == SEER_BF16,
                           o && o->split == 1, o ? o->split_width : 0);
}

// The launch options with their defaults resolved (NULL or zero fields: defaults).
void apply_opts(seer::AttnArgs& a, const seer_attn_opts* o) {
  if (!o) return;
  if (o->heads_per_wg > 0) a.heads_per_wg = o->heads_per_wg;
  if (o->batch_min_blocks < 0) a.batch_min_blocks = 0;
  else if (o->batch_min_blocks > 0) a.batch_min_blocks = o->batch_min_blocks;
  if (o->batch_wgs > 0) a.batch_wgs = o->batch_wgs;
  if (o->walk_classes > 0) a.walk_classes = o->walk_classes;
}

seer_status check_opts(const seer_attn_opts* o) {
  if (!o) return SEER_OK;
  if ((o->split != 0 && o->split != 1) || (o->heads_per_wg > 0 && o->heads_per_wg != 1 && o->heads_per_wg != 2 &&
                                           o->heads_per_wg != 4) ||
      o->walk_classes < 0 || o->walk_classes > 16 || (o->walk_classes & (o->walk_classes - 1)) != 0)
    return SEER_ERR_INVALID_ARG;
  return SEER_OK;
}

// Bytes of row-max workspace per query head: nb key tiles x 64 queries per query block.
size_t gt_head_bytes(const seer_attn_desc* d) {
  const size_t nb = (size_t)blocks_of(d->seq_len, SEER_BLOCK);
  return nb * nb * 64 * sizeof(float);
}

}  // namespace

extern "C" {

int seer_abi_version(void) { return SEER_ABI_VERSION; }

const char* seer_status_str(int status) {
  switch (status) {
    case SEER_OK: return "SEER_OK";
    case SEER_ERR_INVALID_ARG: return "SEER_ERR_INVALID_ARG";
    case SEER_ERR_UNSUPPORTED: return "SEER_ERR_UNSUPPORTED";
    case SEER_ERR_WORKSPACE: return "SEER_ERR_WORKSPACE";
    case SEER_ERR_HIP: return "SEER_ERR_HIP";
    default: return "SEER_ERR_UNKNOWN";
  }
}

size_t seer_gate_workspace_bytes(const seer_attn_desc* desc, const seer_gate_desc* gate,
                                 int32_t logits_in_workspace) {
  if (check_gate(desc, gate) != SEER_OK) return 0;
  return gate_layout(desc, gate, logits_in_workspace != 0).total;
}

size_t seer_mask_idx_elems(const seer_attn_desc* desc, int32_t block) {
  if (!desc || (block != 64 && block != 128) || desc->batch <= 0 || desc->heads_q <= 0 ||
      desc->seq_len <= 0)
    return 0;
  const size_t nb = (size_t)blocks_of(desc->seq_len, block);
  return (size_t)desc->batch * desc->heads_q * nb * nb;
}

// Longest gate rows (in blocks) that seer_gate selects with the fused kernel.
constexpr int kFusedGateMaxBlocks = 128;

// The gate after argument checks.  fused: the logits are formed and selected
// in one kernel (gate_fused_kernel) and never leave on-chip memory, so the
// workspace holds only the projected rows; otherwise the logits kernel writes
// them to logits_out or the workspace and the selection kernel reads them.
static seer_status gate_run(const seer_attn_desc* desc, const seer_gate_desc* gate, const void* q, const void* k,
                            const float* wq, const float* wk, seer_block_mask* out, float* logits_out,
                            void* workspace, bool fused, hipStream_t st) {
  seer_status s;
  const int nb = blocks_of(desc->seq_len, gate->block);
  const bool logits_in_ws = logits_out == nullptr && !fused;
  const GateLayout L = gate_layout(desc, gate, logits_in_ws, !fused);
  char* ws = static_cast<char*>(workspace);
  float* qg = reinterpret_cast<float*>(ws + L.qg);
  float* kg = reinterpret_cast<float*>(ws + L.kg);
  uint16_t* qs = fused ? nullptr : reinterpret_cast<uint16_t*>(ws + L.qs);
  uint16_t* ks = fused ? nullptr : reinterpret_cast<uint16_t*>(ws + L.ks);
  float* logits = logits_in_ws ? reinterpret_cast<float*>(ws + L.logits) : logits_out;
  const int D = desc->head_dim, Dg = gate->gate_dim;

  seer::PoolProjArgs pa;
  pa.q = view(q, desc->q_stride);
  pa.k = view(k, desc->k_stride);
  pa.batch = desc->batch;
  pa.heads_q = desc->heads_q;
  pa.heads_kv = desc->heads_kv;
  pa.n_blocks = nb;
  pa.head_dim = D;
  pa.gate_dim = Dg;
  pa.bf16 = desc->dtype == SEER_BF16;
  pa.wq = wq;
  pa.wk = wk;
  pa.wq_head_stride = gate->w_per_head ? (int64_t)D * Dg : 0;
  pa.wk_head_stride = gate->w_per_head ? (int64_t)3 * D * Dg : 0;
  // the fused kernel reads the fp32 rows, the logits kernel only their parts
  pa.qg = fused ? qg : nullptr;
  pa.kg = fused ? kg : nullptr;
  pa.rope_base = gate->rope_theta > 0.0 ? gate->rope_theta / gate->block : 0.0;
  pa.qp = nullptr;
  pa.kp = nullptr;
  pa.qs = qs;
  pa.ks = ks;
  pa.block = gate->block;
  pa.seq_len = desc->seq_len;
  if ((s = from_hip(seer::launch_pool_proj(pa, st))) != SEER_OK) return s;

  const float scale = (float)(1.0 / std::sqrt((double)Dg));
  if (!fused) {
    seer::GateLogitsArgs la;
    la.qs = qs;
    la.ks = ks;
    la.batch = desc->batch;
    la.heads_q = desc->heads_q;
    la.heads_kv = desc->heads_kv;
    la.n_blocks = nb;
    la.gate_dim = Dg;
    la.scale = scale;
    la.logits = logits;
    if ((s = from_hip(seer::launch_gate_logits(la, st))) != SEER_OK) return s;
  }

  seer::SelectArgs sa;
  sa.logits = fused ? nullptr : logits;
  sa.batch = desc->batch;
  sa.heads_q = desc->heads_q;
  sa.n_blocks = nb;
  sa.mode = gate->mode;
  sa.topk_ratio = gate->topk_ratio;
  sa.topk_k = gate->topk_k;
  sa.threshold = gate->threshold;
  sa.head_thresholds = gate->mode == SEER_THRESHOLD ? gate->head_thresholds : nullptr;
  sa.keep_first = gate->keep_first ? 1 : 0;
  sa.keep_diag = gate->keep_diag ? 1 : 0;
  sa.group = gate->kv_shared ? desc->heads_q / desc->heads_kv : 0;
  sa.count = out->count;
  sa.idx = out->idx;
  sa.dense = out->dense;
  if (fused) {
    seer::GateFusedArgs fa;
    fa.qg = qg;
    fa.kg = kg;
    fa.heads_kv = desc->heads_kv;
    fa.gate_dim = Dg;
    fa.scale = scale;
    fa.sel = sa;
    return from_hip(seer::launch_gate_fused(fa, st));
  }
  return from_hip(seer::launch_select(sa, st));
}

seer_status seer_gate(const seer_attn_desc* desc, const seer_gate_desc* gate, const void* q,
                      const void* k, const float* wq, const float* wk, seer_block_mask* out,
                      float* logits_out, void* workspace, size_t workspace_bytes, void* stream) {
  seer_status s = check_gate(desc, gate);
  if (s != SEER_OK) return s;
  if (!q || !k || !wq || !wk || !out || !out->count || !out->idx) return SEER_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(wq) || !aligned16(wk)) return SEER_ERR_INVALID_ARG;
  const int nb = blocks_of(desc->seq_len, gate->block);
  if (out->n_blocks != nb || out->kv_shared != gate->kv_shared) return SEER_ERR_INVALID_ARG;
  const GateLayout L = gate_layout(desc, gate, logits_out == nullptr);
  if (!workspace || workspace_bytes < L.total) return SEER_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return SEER_ERR_INVALID_ARG;
  // Short rows take the fused score + select kernel, whose logits never leave
  // LDS (16 rows per workgroup; at up to 128 blocks several workgroups share a
  // CU).  Longer rows fill 64-128 KiB of LDS per workgroup, which leaves one
  // workgroup per CU and no overlap of its MFMA and selection phases: measured
  // gate 0.059 against 0.067 ms at 8192 tokens (32 query / 8 KV heads), but
  // 0.173 against 0.143 ms at 32768 and 0.92 against 0.76 ms at 131072.
  const bool fused = logits_out == nullptr && !gate->kv_shared && nb <= kFusedGateMaxBlocks &&
                     seer::gate_fused_supported(nb, gate->gate_dim);
  return gate_run(desc, gate, q, k, wq, wk, out, logits_out, workspace, fused, static_cast<hipStream_t>(stream));
}

seer_status seer_gate_noalloc(const seer_attn_desc* desc, const seer_gate_desc* gate, const void* q,
                              const void* k, const float* wq, const float* wk, seer_block_mask* out,
                              void* stream) {
  seer_status s = check_gate(desc, gate);
  if (s != SEER_OK) return s;
  if (!q || !k || !wq || !wk || !out || !out->count || !out->idx) return SEER_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(wq) || !aligned16(wk)) return SEER_ERR_INVALID_ARG;
  const int nb = blocks_of(desc->seq_len, gate->block);
  if (out->n_blocks != nb || out->kv_shared != gate->kv_shared) return SEER_ERR_INVALID_ARG;
  if (gate->kv_shared || !seer::gate_fused_supported(nb, gate->gate_dim)) return SEER_ERR_UNSUPPORTED;
  const GateLayout L = gate_layout(desc, gate, false, false);
  if (L.total > seer::kGateScratchBytes) return SEER_ERR_WORKSPACE;  // beyond the static scratch
  void* scratch = seer::gate_scratch();
  if (!scratch) return SEER_ERR_HIP;
  return gate_run(desc, gate, q, k, wq, wk, out, nullptr, scratch, true, static_cast<hipStream_t>(stream));
}

size_t seer_gate_noalloc_max_bytes(void) { return seer::kGateScratchBytes; }

// block: tokens per mask block (64 or 128; ignored without a mask).
static seer_status attn_common(const seer_attn_desc* desc, int32_t block, const seer_block_mask* mask,
                               int32_t causal, float sm_scale, const void* q, const void* k,
                               const void* v, void* o, float* lse, void* workspace,
                               size_t workspace_bytes, const seer_attn_opts* opts, void* stream,
                               int* count = nullptr) {
  seer_status s = check_attn(desc, sm_scale, q, k, v, o);
  if (s != SEER_OK) return s;
  if ((s = check_opts(opts)) != SEER_OK) return s;
  if (mask) {
    if (block != 64 && block != 128) return SEER_ERR_UNSUPPORTED;
    const int nbm = blocks_of(desc->seq_len, block);
    if (!mask->count || !mask->idx || mask->n_blocks != nbm) return SEER_ERR_INVALID_ARG;
    if (mask->kv_shared != 0 && mask->kv_shared != 1) return SEER_ERR_INVALID_ARG;
    if (nbm > 65536) return SEER_ERR_UNSUPPORTED;
  }
  seer::AttnArgs a = attn_args(desc, causal, sm_scale, q, k, v, o, lse);
  a.count = mask ? mask->count : nullptr;
  a.idx = mask ? mask->idx : nullptr;
  a.mask_shift = (mask && block == 128) ? 1 : 0;
  a.mask_blocks = mask ? mask->n_blocks : 0;
  a.mask_kv = mask && mask->kv_shared;
  apply_opts(a, opts);
  if (workspace && a.mask_shift == 0 && !a.mask_kv) {  // the split runs on per-head 64-token masks
    if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return SEER_ERR_INVALID_ARG;
    const SplitLayout L = split_layout(desc, split_width_for(desc, causal, opts));
    if (L.w > 0 && workspace_bytes >= L.total) {  // key-range split
      char* ws = static_cast<char*>(workspace);
      a.split_parts = L.parts;
      a.split_w = L.w;
      a.split_slots = L.slots;
      a.split_bounds = reinterpret_cast<int32_t*>(ws + L.bounds);
      a.split_tickets = reinterpret_cast<int32_t*>(ws + L.tickets);
      a.part_lse = reinterpret_cast<float*>(ws + L.lse);
      a.part_o = reinterpret_cast<uint16_t*>(ws + L.o);
    }
  }
  return from_hip(seer::launch_attn(a, static_cast<hipStream_t>(stream), count));
}

seer_status seer_bsattn(const seer_attn_desc* desc, int32_t block, const seer_block_mask* mask,
                        int32_t causal, float sm_scale, const void* q, const void* k,
                        const void* v, void* o, float* lse, void* stream) {
  if (!mask || !desc) return SEER_ERR_INVALID_ARG;
  return attn_common(desc, block, mask, causal, sm_scale, q, k, v, o, lse, nullptr, 0, nullptr, stream);
}

seer_status seer_dense_attn(const seer_attn_desc* desc, int32_t causal, float sm_scale,
                            const void* q, const void* k, const void* v, void* o, float* lse,
                            void* stream) {
  return attn_common(desc, SEER_BLOCK, nullptr, causal, sm_scale, q, k, v, o, lse, nullptr, 0, nullptr, stream);
}

size_t seer_attn_workspace_bytes(const seer_attn_desc* desc, int32_t block, int32_t causal,
                                 const seer_attn_opts* opts) {
  if (block != SEER_BLOCK || check_desc(desc, 0xF) != SEER_OK || check_opts(opts) != SEER_OK) return 0;
  return split_layout(desc, split_width_for(desc, causal, opts)).total;
}

seer_status seer_bsattn_ws(const seer_attn_desc* desc, int32_t block, const seer_block_mask* mask,
                           int32_t causal, float sm_scale, const void* q, const void* k, const void* v,
                           void* o, float* lse, void* workspace, size_t workspace_bytes,
                           const seer_attn_opts* opts, void* stream) {
  if (!mask || !desc) return SEER_ERR_INVALID_ARG;
  return attn_common(desc, block, mask, causal, sm_scale, q, k, v, o, lse, workspace, workspace_bytes, opts,
                     stream);
}

seer_status seer_dense_attn_ws(const seer_attn_desc* desc, int32_t causal, float sm_scale,
                               const void* q, const void* k, const void* v, void* o, float* lse,
                               void* workspace, size_t workspace_bytes, const seer_attn_opts* opts,
                               void* stream) {
  return attn_common(desc, SEER_BLOCK, nullptr, causal, sm_scale, q, k, v, o, lse, workspace,
                     workspace_bytes, opts, stream);
}

int32_t seer_attn_launches(const seer_attn_desc* desc, int32_t block, int32_t mask_kind, int32_t causal,
                           const seer_attn_opts* opts, size_t workspace_bytes) {
  if (!desc || mask_kind < 0 || mask_kind > 2) return -1;
  // stand-in pointers: nothing is dereferenced or launched when counting
  char* fake = reinterpret_cast<char*>(kAlign);
  seer_block_mask m{};
  if (mask_kind > 0) {
    if (block != 64 && block != 128) return -1;
    m.n_blocks = blocks_of(desc->seq_len, block);
    m.count = reinterpret_cast<int32_t*>(fake);
    m.idx = reinterpret_cast<uint16_t*>(fake);
    m.kv_shared = mask_kind == 2;
  }
  int count = 0;
  const seer_status s = attn_common(desc, mask_kind > 0 ? block : SEER_BLOCK, mask_kind > 0 ? &m : nullptr, causal,
                                    0.f, fake, fake, fake, fake, nullptr, workspace_bytes ? fake : nullptr,
                                    workspace_bytes, opts, nullptr, &count);
  return s == SEER_OK ? count : -1;
}

seer_status seer_mask_from_dense(const seer_attn_desc* desc, int32_t block, const uint8_t* dense,
                                 seer_block_mask* out, void* stream) {
  if (!desc || !dense || !out || !out->count || !out->idx) return SEER_ERR_INVALID_ARG;
  if (desc->batch <= 0 || desc->heads_q <= 0 || desc->seq_len <= 0) return SEER_ERR_INVALID_ARG;
  if (block != 64 && block != 128) return SEER_ERR_UNSUPPORTED;
  const int nb = blocks_of(desc->seq_len, block);
  if (out->n_blocks != nb) return SEER_ERR_INVALID_ARG;
  if (out->kv_shared != 0 && out->kv_shared != 1) return SEER_ERR_INVALID_ARG;
  if (out->kv_shared && (desc->heads_kv <= 0 || desc->heads_q % desc->heads_kv != 0)) return SEER_ERR_INVALID_ARG;
  if (nb > 4096) return SEER_ERR_UNSUPPORTED;
  seer::MaskFromDenseArgs a;
  a.dense = dense;
  a.rows = (int64_t)desc->batch * (out->kv_shared ? desc->heads_kv : desc->heads_q) * nb;
  a.n_blocks = nb;
  a.count = out->count;
  a.idx = out->idx;
  return from_hip(seer::launch_mask_from_dense(a, static_cast<hipStream_t>(stream)));
}

size_t seer_attn_gt_workspace_bytes(const seer_attn_desc* desc, int32_t block, int32_t kv_groups) {
  if (block != SEER_BLOCK || check_desc(desc, 0xF) != SEER_OK) return 0;
  const int64_t groups = (int64_t)desc->batch * desc->heads_kv;
  const int64_t use = (kv_groups <= 0 || kv_groups >= groups) ? groups : kv_groups;
  const int G = desc->heads_q / desc->heads_kv;
  return (size_t)use * G * gt_head_bytes(desc);
}

seer_status seer_attn_gt(const seer_attn_desc* desc, int32_t block, int32_t causal, float sm_scale,
                         const void* q, const void* k, const void* v, void* o, float* lse,
                         float* gt, void* workspace, size_t workspace_bytes, const seer_attn_opts* opts,
                         void* stream) {
  if (block != SEER_BLOCK) return desc ? SEER_ERR_UNSUPPORTED : SEER_ERR_INVALID_ARG;
  seer_status s = check_attn(desc, sm_scale, q, k, v, o);
  if (s != SEER_OK) return s;
  if ((s = check_opts(opts)) != SEER_OK) return s;
  if (!gt) return SEER_ERR_INVALID_ARG;
  const int G = desc->heads_q / desc->heads_kv;
  const size_t group_bytes = (size_t)G * gt_head_bytes(desc);
  if (!workspace || workspace_bytes < group_bytes) return SEER_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return SEER_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t nb = blocks_of(desc->seq_len, SEER_BLOCK);
  const int64_t all = (int64_t)desc->batch * desc->heads_kv;
  seer::AttnArgs a = attn_args(desc, causal, sm_scale, q, k, v, o, lse);
  apply_opts(a, opts);
  a.pool_r = static_cast<float*>(workspace);
  if (workspace_bytes / group_bytes >= (size_t)all) {  // every head in one launch
    a.gt = gt;
    return from_hip(seer::launch_attn(a, st));
  }
  // otherwise: runs of KV groups of one batch entry per launch
  const int per = (int)(workspace_bytes / group_bytes);
  const size_t qe = desc->dtype == SEER_F32 ? 4 : 2;
  for (int b = 0; b < desc->batch; ++b)
    for (int g0 = 0; g0 < desc->heads_kv; g0 += per) {
      const int ng = std::min(per, desc->heads_kv - g0);
      const int h0 = g0 * G;
      seer::AttnArgs c = a;
      c.batch = 1;
      c.heads_kv = ng;
      c.heads_q = ng * G;
      c.q.ptr = static_cast<const char*>(q) + qe * (b * desc->q_stride[0] + h0 * desc->q_stride[1]);
      c.k.ptr = static_cast<const char*>(k) + qe * (b * desc->k_stride[0] + g0 * desc->k_stride[1]);
      c.v.ptr = static_cast<const char*>(v) + qe * (b * desc->v_stride[0] + g0 * desc->v_stride[1]);
      c.o = static_cast<char*>(o) + qe * (b * desc->o_stride[0] + h0 * desc->o_stride[1]);
      const int64_t hrow = (int64_t)b * desc->heads_q + h0;  // first query head of the run
      c.lse = lse ? lse + hrow * desc->seq_len : nullptr;
      c.gt = gt + hrow * nb * nb;
      if ((s = from_hip(seer::launch_attn(c, st))) != SEER_OK) return s;
    }
  return SEER_OK;
}

static int distill_min_chunks(const seer_distill_opts* opts) {
  return (opts && opts->gemm_min_chunks >= 1) ? opts->gemm_min_chunks : 8;
}

// 0 (chosen from the shape), 64 or 128; -1: invalid
static int distill_tile_n(const seer_distill_opts* opts) {
  const int t = opts ? opts->gemm_tile_n : 0;
  return (t == 0 || t == 64 || t == 128) ? t : -1;
}

size_t seer_gate_distill_workspace_bytes(const seer_attn_desc* desc, const seer_gate_desc* gate,
                                         const seer_distill_opts* opts) {
  if (check_gate_common(desc, gate) != SEER_OK) return 0;
  const int tile_n = distill_tile_n(opts);
  if (tile_n < 0) return 0;
  return distill_layout(desc, gate, distill_min_chunks(opts), tile_n).total;
}

seer_status seer_gate_distill(const seer_attn_desc* desc, const seer_gate_desc* gate, const void* q,
                              const void* k, const float* wq, const float* wk, const float* gt,
                              float* loss, float* dwq, float* dwk, void* workspace,
                              size_t workspace_bytes, const seer_distill_opts* opts, void* stream) {
  seer_status s = check_gate_common(desc, gate);
  if (s != SEER_OK) return s;
  if (gate->kv_shared) return SEER_ERR_UNSUPPORTED;  // the distillation target is per query head
  if (!q || !k || !wq || !wk || !gt || !loss || !dwq || !dwk) return SEER_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(wq) || !aligned16(wk)) return SEER_ERR_INVALID_ARG;
  const int min_chunks = distill_min_chunks(opts);
  const int tile_n = distill_tile_n(opts);
  if (tile_n < 0) return SEER_ERR_INVALID_ARG;
  const DistillLayout W = distill_layout(desc, gate, min_chunks, tile_n);
  if (!workspace || workspace_bytes < W.total) return SEER_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return SEER_ERR_INVALID_ARG;

  char* ws = static_cast<char*>(workspace);
  float* qg = reinterpret_cast<float*>(ws + W.qg);
  float* kg = reinterpret_cast<float*>(ws + W.kg);
  uint16_t* qs = reinterpret_cast<uint16_t*>(ws + W.qs);
  uint16_t* ks = reinterpret_cast<uint16_t*>(ws + W.ks);
  float* qp = reinterpret_cast<float*>(ws + W.qp);
  float* kp = reinterpret_cast<float*>(ws + W.kp);
  float* dl = reinterpret_cast<float*>(ws + W.logits);
  float* dqg = reinterpret_cast<float*>(ws + W.dqg);
  float* dkg = reinterpret_cast<float*>(ws + W.dkg);
  double* row_loss = reinterpret_cast<double*>(ws + W.row_loss);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int B = desc->batch, Hq = desc->heads_q, Hkv = desc->heads_kv, D = desc->head_dim;
  const int Dg = gate->gate_dim;
  const int nb = blocks_of(desc->seq_len, gate->block);
  const double rope_base = gate->rope_theta > 0.0 ? gate->rope_theta / gate->block : 0.0;
  const float rsqrt_dg = (float)(1.0 / std::sqrt((double)Dg));

  // forward: pooled rows (kept), projected rows, logits
  seer::PoolProjArgs pa;
  pa.q = view(q, desc->q_stride);
  pa.k = view(k, desc->k_stride);
  pa.batch = B;
  pa.heads_q = Hq;
  pa.heads_kv = Hkv;
  pa.n_blocks = nb;
  pa.head_dim = D;
  pa.gate_dim = Dg;
  pa.bf16 = desc->dtype == SEER_BF16;
  pa.wq = wq;
  pa.wk = wk;
  pa.wq_head_stride = gate->w_per_head ? (int64_t)D * Dg : 0;
  pa.wk_head_stride = gate->w_per_head ? (int64_t)3 * D * Dg : 0;
  pa.qg = qg;
  pa.kg = kg;
  pa.rope_base = rope_base;
  pa.qp = qp;
  pa.kp = kp;
  pa.qs = qs;
  pa.ks = ks;
  pa.block = gate->block;
  pa.seq_len = desc->seq_len;
  if ((s = from_hip(seer::launch_pool_proj(pa, st))) != SEER_OK) return s;

  seer::GateLogitsArgs la;
  la.qs = qs;
  la.ks = ks;
  la.batch = B;
  la.heads_q = Hq;
  la.heads_kv = Hkv;
  la.n_blocks = nb;
  la.gate_dim = Dg;
  la.scale = rsqrt_dg;
  la.logits = dl;
  if ((s = from_hip(seer::launch_gate_logits(la, st))) != SEER_OK) return s;

  // loss and logit gradient
  seer::KlArgs ka;
  ka.logits = dl;
  ka.gt = gt;
  ka.rows = (int64_t)B * Hq * nb;
  ka.n_blocks = nb;
  ka.inv_rows = (float)(1.0 / (double)ka.rows);
  ka.row_loss = row_loss;
  ka.loss = loss;
  if ((s = from_hip(seer::launch_kl_rows(ka, st))) != SEER_OK) return s;

  const DistillGemms gm = distill_gemms(B, Hq, Hkv, D, Dg, nb, gate->w_per_head != 0, min_chunks, tile_n, dl, qg, kg, qp,
                                        kp, dqg, dkg, dwq, dwk, reinterpret_cast<float*>(ws + W.part));
  if ((s = from_hip(seer::launch_gemm_f32(gm.dqg, st))) != SEER_OK) return s;
  if ((s = from_hip(seer::launch_gemm_f32(gm.dkg, st))) != SEER_OK) return s;
  if (rope_base > 0.0) {  // back through the block-level RoPE
    seer::RopeArgs ra{dqg, (int64_t)B * Hq, nb, Dg, rope_base};
    if ((s = from_hip(seer::launch_rope_inverse(ra, st))) != SEER_OK) return s;
    ra = seer::RopeArgs{dkg, (int64_t)B * Hkv, nb, Dg, rope_base};
    if ((s = from_hip(seer::launch_rope_inverse(ra, st))) != SEER_OK) return s;
  }
  if ((s = from_hip(seer::launch_gemm_f32(gm.dwq, st))) != SEER_OK) return s;
  return from_hip(seer::launch_gemm_f32(gm.dwk, st));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// packed variable-length batches: one batch-1 pass per sequence on the stream
// ---------------------------------------------------------------------------

namespace {

// Checks cu_seqlens and builds the batch-1 descriptor of sequence b (strides of
// the packed layout; tokens [cu[b], cu[b+1])).
seer_status check_cu(const seer_attn_desc* d, const int32_t* cu) {
  if (!d || !cu || d->batch <= 0) return SEER_ERR_INVALID_ARG;
  if (cu[0] != 0) return SEER_ERR_INVALID_ARG;
  for (int b = 0; b < d->batch; ++b)
    if (cu[b + 1] < cu[b]) return SEER_ERR_INVALID_ARG;
  if (cu[d->batch] != d->seq_len) return SEER_ERR_INVALID_ARG;
  return SEER_OK;
}

seer_attn_desc seq_desc(const seer_attn_desc* d, const int32_t* cu, int b) {
  seer_attn_desc s = *d;
  s.batch = 1;
  s.seq_len = cu[b + 1] - cu[b];
  s.q_stride[0] = s.k_stride[0] = s.v_stride[0] = s.o_stride[0] = 0;
  return s;
}

const void* at_token(const void* p, const int64_t* st, int64_t t, size_t es) {
  return p ? static_cast<const char*>(p) + (size_t)(t * st[2]) * es : nullptr;
}

struct VarlenMaskOffsets {
  int64_t count, idx;
};

// Offsets of sequence b's rows in a packed variable-length mask: count rows
// [H][nb_b] and idx rows [H][nb_b][nb_b] of the sequences before it.
VarlenMaskOffsets varlen_mask_offsets(const int32_t* cu, int b, int heads, int block) {
  VarlenMaskOffsets o{0, 0};
  for (int s = 0; s < b; ++s) {
    const int64_t nb = blocks_of(cu[s + 1] - cu[s], block);
    o.count += heads * nb;
    o.idx += heads * nb * nb;
  }
  return o;
}

}  // namespace

extern "C" {

size_t seer_varlen_mask_elems(const seer_attn_desc* desc, const int32_t* cu_seqlens_host, int32_t block,
                              int32_t kv_shared, size_t* count_elems) {
  if (check_cu(desc, cu_seqlens_host) != SEER_OK || (block != 64 && block != 128) || desc->heads_q <= 0 ||
      desc->heads_kv <= 0 || desc->heads_q % desc->heads_kv != 0)
    return 0;
  const int heads = kv_shared ? desc->heads_kv : desc->heads_q;
  const VarlenMaskOffsets o = varlen_mask_offsets(cu_seqlens_host, desc->batch, heads, block);
  if (count_elems) *count_elems = (size_t)o.count;
  return (size_t)o.idx;
}

size_t seer_gate_varlen_workspace_bytes(const seer_attn_desc* desc, const int32_t* cu_seqlens_host,
                                        const seer_gate_desc* gate) {
  if (check_cu(desc, cu_seqlens_host) != SEER_OK) return 0;
  size_t need = 0;
  for (int b = 0; b < desc->batch; ++b) {
    const seer_attn_desc sd = seq_desc(desc, cu_seqlens_host, b);
    if (sd.seq_len == 0) continue;
    if (check_gate(&sd, gate) != SEER_OK) return 0;
    need = std::max(need, gate_layout(&sd, gate, true).total);
  }
  return need;
}

seer_status seer_gate_varlen(const seer_attn_desc* desc, const int32_t* cu_seqlens_host,
                             const seer_gate_desc* gate, const void* q, const void* k, const float* wq,
                             const float* wk, seer_block_mask* out, void* workspace, size_t workspace_bytes,
                             void* stream) {
  seer_status s = check_cu(desc, cu_seqlens_host);
  if (s != SEER_OK) return s;
  if (!gate || !out || !out->count || !out->idx || !q || !k) return SEER_ERR_INVALID_ARG;
  if (out->kv_shared != gate->kv_shared) return SEER_ERR_INVALID_ARG;
  const size_t es = elem_size(desc->dtype);
  const int heads = gate->kv_shared ? desc->heads_kv : desc->heads_q;
  // validate every sequence before launching anything
  for (int b = 0; b < desc->batch; ++b) {
    const seer_attn_desc sd = seq_desc(desc, cu_seqlens_host, b);
    if (sd.seq_len == 0) continue;
    if ((s = check_gate(&sd, gate)) != SEER_OK) return s;
    if (workspace_bytes < gate_layout(&sd, gate, true).total || !workspace) return SEER_ERR_WORKSPACE;
    if (!aligned16(at_token(q, desc->q_stride, cu_seqlens_host[b], es)) ||
        !aligned16(at_token(k, desc->k_stride, cu_seqlens_host[b], es)))
      return SEER_ERR_INVALID_ARG;
  }
  for (int b = 0; b < desc->batch; ++b) {
    const seer_attn_desc sd = seq_desc(desc, cu_seqlens_host, b);
    if (sd.seq_len == 0) continue;
    const VarlenMaskOffsets o = varlen_mask_offsets(cu_seqlens_host, b, heads, gate->block);
    seer_block_mask m = *out;
    m.n_blocks = blocks_of(sd.seq_len, gate->block);
    m.count = out->count + o.count;
    m.idx = out->idx + o.idx;
    m.dense = out->dense ? out->dense + o.idx : nullptr;
    s = seer_gate(&sd, gate, at_token(q, desc->q_stride, cu_seqlens_host[b], es),
                  at_token(k, desc->k_stride, cu_seqlens_host[b], es), wq, wk, &m, nullptr, workspace,
                  workspace_bytes, stream);
    if (s != SEER_OK) return s;
  }
  return SEER_OK;
}

seer_status seer_bsattn_varlen(const seer_attn_desc* desc, const int32_t* cu_seqlens_host, int32_t block,
                               const seer_block_mask* mask, int32_t causal, float sm_scale, const void* q,
                               const void* k, const void* v, void* o, float* lse, void* stream) {
  seer_status s = check_cu(desc, cu_seqlens_host);
  if (s != SEER_OK) return s;
  if (!mask || !mask->count || !mask->idx) return SEER_ERR_INVALID_ARG;
  if (block != 64 && block != 128) return SEER_ERR_UNSUPPORTED;
  if (mask->kv_shared != 0 && mask->kv_shared != 1) return SEER_ERR_INVALID_ARG;
  const size_t es = elem_size(desc->dtype);
  const int heads = mask->kv_shared ? desc->heads_kv : desc->heads_q;
  for (int b = 0; b < desc->batch; ++b) {
    const seer_attn_desc sd = seq_desc(desc, cu_seqlens_host, b);
    if (sd.seq_len == 0) continue;
    if ((s = check_attn(&sd, sm_scale, at_token(q, desc->q_stride, cu_seqlens_host[b], es),
                        at_token(k, desc->k_stride, cu_seqlens_host[b], es),
                        at_token(v, desc->v_stride, cu_seqlens_host[b], es),
                        at_token(o, desc->o_stride, cu_seqlens_host[b], es))) != SEER_OK)
      return s;
    if (blocks_of(sd.seq_len, block) > 65536) return SEER_ERR_UNSUPPORTED;
  }
  for (int b = 0; b < desc->batch; ++b) {
    const seer_attn_desc sd = seq_desc(desc, cu_seqlens_host, b);
    if (sd.seq_len == 0) continue;
    const VarlenMaskOffsets mo = varlen_mask_offsets(cu_seqlens_host, b, heads, block);
    seer_block_mask m = *mask;
    m.n_blocks = blocks_of(sd.seq_len, block);
    m.count = mask->count + mo.count;
    m.idx = mask->idx + mo.idx;
    m.dense = nullptr;
    float* lb = lse ? lse + (int64_t)desc->heads_q * cu_seqlens_host[b] : nullptr;  // [Hq][len_b] per sequence
    s = attn_common(&sd, block, &m, causal, sm_scale, at_token(q, desc->q_stride, cu_seqlens_host[b], es),
                    at_token(k, desc->k_stride, cu_seqlens_host[b], es),
                    at_token(v, desc->v_stride, cu_seqlens_host[b], es),
                    const_cast<void*>(at_token(o, desc->o_stride, cu_seqlens_host[b], es)), lb, nullptr, 0,
                    nullptr, stream);
    if (s != SEER_OK) return s;
  }
  return SEER_OK;
}

}  // extern "C"
