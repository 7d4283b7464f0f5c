// launch.h -- internal (C++) launchers behind the C ABI in include/seer.h.
// Arguments are validated by the ABI layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace seer {

struct TensorView {  // [batch][heads][seq][dim], element strides of (batch, head, seq)
  const void* ptr;
  int64_t sb, sh, ss;
};

// Rows of one head's split gate rows: nb rounded up to whole 32-row groups.
__host__ __device__ __forceinline__ int split_rows(int nb) { return (nb + 31) / 32 * 32; }

struct PoolProjArgs {
  TensorView q, k;
  int batch, heads_q, heads_kv, n_blocks, head_dim, gate_dim;
  bool bf16;
  const float* wq;
  const float* wk;
  int64_t wq_head_stride, wk_head_stride;  // 0 when one matrix is shared by all heads
  float* qg;  // [B][Hq][nb][Dg] (nullptr: not stored)
  float* kg;  // [B][Hkv][nb][Dg] (nullptr: not stored)
  double rope_base;  // > 0: block-level RoPE with this base (model base / block)
  float* qp;  // optional pooled Q [B][Hq][nb][D] (nullptr: not stored)
  float* kp;  // optional pooled K [B][Hkv][nb][3D]
  // optional split rows for the bf16 logits kernel: Qg, Kg as three bf16 parts
  // (hi, mid, lo) per element, [B][H][split_rows(nb)][3][Dg] elements in the
  // lane order of the kernel's MFMA operands (nullptr: not stored)
  uint16_t* qs;
  uint16_t* ks;
  int block;  // tokens per gate block: 64 or 128
  int seq_len;  // tokens; the last block holds seq_len - (n_blocks - 1) block of them
};

struct GateLogitsArgs {
  const uint16_t* qs;  // Qg split in three bf16 parts (PoolProjArgs::qs)
  const uint16_t* ks;  // Kg split in three bf16 parts (PoolProjArgs::ks)
  int batch, heads_q, heads_kv, n_blocks, gate_dim;
  float scale;   // 1/sqrt(Dg)
  float* logits; // [B][Hq][nb][nb]
};

struct SelectArgs {
  const float* logits;  // [B][Hq][nb][nb], entries j <= i of each row are read
  int batch, heads_q, n_blocks;
  int mode;             // 0 topk ratio, 1 topk fixed, 2 threshold
  double topk_ratio;
  int topk_k;
  float threshold;
  const float* head_thresholds;  // device [Hq] ([Hkv] when group > 0) or nullptr
  int group;            // 0: one row per query head; G: one row per KV head, scored by
                        // the mean of its G query heads' probabilities
  int keep_first, keep_diag;
  int32_t* count;
  uint16_t* idx;
  uint8_t* dense;  // optional
};

// Fused gate score and selection (per-query-head masks): the logits of the
// projected rows qg, kg are formed in LDS and selected there (sel.logits unused).
struct GateFusedArgs {
  const float* qg;  // [B][Hq][nb][Dg]
  const float* kg;  // [B][Hkv][nb][Dg]
  int heads_kv, gate_dim;
  float scale;      // 1/sqrt(Dg)
  SelectArgs sel;
};
// Whether the fused path serves this shape (row length and gate width).
bool gate_fused_supported(int n_blocks, int gate_dim);

// The gate's static device scratch (seer_gate_noalloc): kGateScratchBytes per
// device, held until the process ends.  gate_scratch() returns this device's
// copy (its address looked up once per device), or nullptr on a HIP error.
constexpr size_t kGateScratchBytes = (size_t)64 << 20;
void* gate_scratch();

struct MaskFromDenseArgs {
  const uint8_t* dense;
  int64_t rows;
  int n_blocks;
  int32_t* count;
  uint16_t* idx;
};

struct AttnArgs {
  TensorView q, k, v;
  void* o;
  int64_t osb, osh, oss;
  float* lse;  // [B][Hq][S] or nullptr
  int batch, heads_q, heads_kv, n_blocks, head_dim;  // n_blocks: 64-token tiles, ceil(S / 64)
  int seq_len;       // S; rows past it in the last tile are padding (clamped reads, no writes)
  int mask_blocks;   // blocks of the mask (ceil(S / 64) or ceil(S / 128)), 0 when dense
  bool bf16;
  bool causal;
  float scale;
  const int32_t* count;  // nullptr: dense (every causal block)
  const uint16_t* idx;
  int mask_shift;        // 0: mask of 64-token blocks; 1: of 128-token blocks, each
                         // entry standing for two 64-key tiles
  bool mask_kv;          // the mask has one row set per KV head, shared by the
                         // group's query heads (count [B][Hkv][nb], idx [B][Hkv][nb][nb])
  // ground-truth mode (dense only): per-tile row maxima [rows][nb][64] and the
  // 2D max-pooled probability map [B][Hq][nb][nb]; both nullptr otherwise
  float* pool_r;
  float* gt;
  // key-range split (causal, bf16): each row is cut into ranges of split_w key
  // blocks, computed as separate tasks into partial slots and merged by each
  // row's last task; split_w == 0 disables it
  int split_parts;              // ceil(n_blocks / split_w)
  int split_w;
  int64_t split_slots;          // partial slots per (batch, head)
  int32_t* split_bounds;        // [rows][split_parts + 3]: range list offsets, non-empty
                                // range count, arrival counter (split_bounds_kernel)
  int32_t* split_tickets;       // [8] task-queue tickets (zeroed by split_bounds_kernel)
  // launch options (seer_attn_opts with its defaults resolved)
  int heads_per_wg;             // cap on query heads per workgroup for shared rows (1, 2, 4)
  int batch_min_blocks;         // batched launches of sparse rows from this many blocks (0: never)
  int batch_wgs;                // workgroups per batch (0: the resident capacity)
  int walk_classes;             // unsplit sparse rows walk their blocks by residue classes
                                // mod this (a power of two up to 16; 1: ascending)
  float* part_lse;              // [slots][64] log2-domain log-sum-exp of each partial
  uint16_t* part_o;             // [slots][64][D] bf16 partial outputs, normalised
};

// Gate distillation (Eq. 2): row-wise KL between the renormalised ground truth
// and the gate softmax, and the logit gradient written over the logits.
// The gradient is written for j < min(nb, 64 (i / 64 + 1)): entries j > i up to
// the end of the row's 64-row tile are 0, and entries beyond are never read
// (the backward products skip them by causality at 64-row tile granularity).
constexpr int kKlTile = 64;
constexpr int kLossParts = 64;  // first-level partial sums of the row losses
struct KlArgs {
  float* logits;       // [rows][nb] in: logits (j <= i), out: dloss/dlogit (see above)
  const float* gt;     // [rows][nb] ground truth (j <= i read)
  int64_t rows;
  int n_blocks;
  float inv_rows;      // 1 / rows: the loss is the mean over rows
  double* row_loss;    // [rows + kLossParts]: per-row losses, then the partial sums
  float* loss;         // device scalar: mean of the row losses
};

// C[z][m][n] = alpha * sum_{k1 < K1, k2 < K2} A(z, m, k1, k2) * B(z / bdiv, k1, k2, n), fp32,
// with element strides; tri = 1: A vanishes for k2 > m, tri = 2: for k2 < m.
// When gemm_splits() > 1 the (k1, k2) range is cut into that many parts whose
// products go to `part` ([Z][splits][M][N], gemm_partial_elems() floats) and
// are summed in a fixed order by a second kernel.
struct GemmArgs {
  const float* A;
  const float* B;
  float* C;
  int M, N, K1, K2, Z, bdiv, tri;
  int64_t sam, sak1, sak2, saz;
  int64_t sbk1, sbk2, sbn, sbz;
  int64_t scm, scz;
  float alpha;
  float* part;
  int min_chunks;  // K chunks per part at least (seer_distill_opts.gemm_min_chunks; 8 by default)
  int tile_n;      // output tile columns: 64, 128, or 0 (chosen from the shape)
};
int gemm_splits(const GemmArgs& a);
int64_t gemm_partial_elems(const GemmArgs& a);

struct RopeArgs {  // inverse block-level RoPE of rows [rows][nb][Dg], in place
  float* x;
  int64_t rows;
  int n_blocks, gate_dim;
  double base;
};

hipError_t launch_pool_proj(const PoolProjArgs& a, hipStream_t s);
hipError_t launch_kl_rows(const KlArgs& a, hipStream_t s);
hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s);
hipError_t launch_rope_inverse(const RopeArgs& a, hipStream_t s);
hipError_t launch_gate_logits(const GateLogitsArgs& a, hipStream_t s);
hipError_t launch_select(const SelectArgs& a, hipStream_t s);
hipError_t launch_gate_fused(const GateFusedArgs& a, hipStream_t s);
hipError_t launch_mask_from_dense(const MaskFromDenseArgs& a, hipStream_t s);
// With a non-null `count` nothing is launched: the attention-kernel launches
// the call would make are counted into *count.
hipError_t launch_attn(const AttnArgs& a, hipStream_t s, int* count = nullptr);
// Split geometry: the key-range width in blocks for a launch (0 when the shape
// does not split) and the partial slots per (batch, head) for a range width.
int split_width(int n_blocks, int head_dim, bool causal, bool bf16, bool want, int width);
int64_t split_slots_per_head(int n_blocks, int w);

}  // namespace seer
