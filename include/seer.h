/*
 * seer.h -- C ABI of the MI355X (gfx950) SeerAttention prefill library, libseer.so.
 *
 * SeerAttention (arXiv 2410.13276) adds an attention gate (AttnGate) that
 * predicts, per attention head, which 64x64 tiles of the causal attention map
 * matter; a block-sparse FlashAttention forward then computes only those tiles.
 * This library provides both halves plus a dense comparison path:
 *
 *   seer_gate        pooled-Q/K gate scores and the block mask they select
 *                    (section 3.1, Eq. 1; Eq. 3 TopK; Eq. 4 threshold)
 *   seer_bsattn      block-sparse causal attention over the active tiles (section 3.3)
 *   seer_dense_attn  the same kernel over every causal tile (the dense baseline
 *                    the paper compares against in section 4.2)
 *   seer_bsattn_ws, seer_dense_attn_ws  the same with a workspace that lets
 *                    long rows be split into key ranges for L2 locality
 *   seer_mask_from_dense  compaction of a caller-made 0/1 block mask into the
 *                    index-list form seer_bsattn reads
 *   seer_attn_gt     dense attention that also returns the 2D max-pooled
 *                    attention map, the gate's distillation target (Eq. 2,
 *                    appendix A.1)
 *   seer_gate_distill  the gate's distillation step (section 3.2, Eq. 2):
 *                    KL(ground truth || gate score) and its weight gradients
 *   seer_gate_varlen, seer_bsattn_varlen  the gate and block-sparse attention
 *                    of a packed batch of variable-length sequences
 *
 * Conventions shared by every entry point:
 *  - Pointers to tensors are DEVICE pointers (HIP device memory of the current
 *    device) unless a name ends in _host.  The caller allocates and owns every
 *    buffer; the library allocates nothing and keeps no state between calls.
 *  - Every call is asynchronous on `stream` (a hipStream_t passed as void*;
 *    NULL is the default stream) and never synchronises the host.  The caller
 *    synchronises before reading results.
 *  - Arguments are validated on the host before anything is launched.  On a
 *    validation error the call returns a non-zero seer_status, launches
 *    nothing and leaves every output untouched.  A launch failure reported by
 *    the HIP runtime returns SEER_ERR_HIP.  No C++ exception crosses the ABI.
 *  - Calls on different streams touching different outputs may overlap; the
 *    library has no global state, so every entry point is reentrant.
 *  - Q/K/V/O are [batch][heads][seq][head_dim] with element strides given per
 *    (batch, head, seq) and head_dim contiguous.  Query head h reads KV head
 *    h / (heads_q / heads_kv) (grouped-query attention, contiguous groups).
 *  - "Causal" means aligned prefill: query t sees key s iff s <= t.
 *  - seq_len need not be a multiple of the block: nb = ceil(seq_len / block),
 *    and the last block is partial (the gate pools it over the tokens it
 *    holds; attention neither reads past the end of Q/K/V nor writes past the
 *    end of O/LSE).
 */
#ifndef SEER_H
#define SEER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SEER_ABI_VERSION 5
#define SEER_BLOCK 64 /* the attention tile edge and the default gate block (section 4); gate
                        blocks and masks of 128 tokens are the other size the paper names */

typedef enum {
  SEER_OK = 0,
  SEER_ERR_INVALID_ARG = 1, /* NULL pointer, non-positive size, inconsistent shape */
  SEER_ERR_UNSUPPORTED = 2, /* valid request outside what is built (see each call) */
  SEER_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required */
  SEER_ERR_HIP = 4          /* the HIP runtime reported an error at launch */
} seer_status;

typedef enum { SEER_BF16 = 0, SEER_F32 = 1 } seer_dtype;

typedef enum {
  SEER_TOPK_RATIO = 0, /* keep ceil(topk_ratio * (i + 1)) of the i + 1 causal blocks of row i */
  SEER_TOPK_FIXED = 1, /* keep topk_k blocks per row (capped at i + 1) */
  SEER_THRESHOLD = 2   /* keep blocks whose gate probability is strictly above the threshold */
} seer_select_mode;

/* Shape and layout of Q, K, V and O (shared by the gate and attention). */
typedef struct {
  int32_t batch;
  int32_t heads_q;
  int32_t heads_kv;  /* heads_q % heads_kv == 0 */
  int32_t seq_len;   /* any length >= 1 (the last block may be partial) */
  int32_t head_dim;  /* 64 or 128 */
  int32_t dtype;     /* seer_dtype of Q, K, V and O */
  int64_t q_stride[3]; /* element strides of (batch, head, seq); head_dim stride is 1 */
  int64_t k_stride[3];
  int64_t v_stride[3];
  int64_t o_stride[3];
} seer_attn_desc;

/* AttnGate parameters (section 3.1, Eq. 1; selection per Eq. 3 / Eq. 4). */
typedef struct {
  int32_t block;       /* pooling kernel = stride = mask block: 64 or 128 tokens (the two block
                          sizes section 3.3 gives for the sparse kernel); the last block may be
                          partial (see the conventions above) */
  int32_t gate_dim;    /* Dg, output width of the gate linear layers: 32, 64 or 128 */
  int32_t w_per_head;  /* 1: wq [heads_q][D][Dg], wk [heads_kv][3D][Dg];
                          0: one wq [D][Dg] and one wk [3D][Dg] shared by all heads */
  int32_t mode;        /* seer_select_mode */
  double topk_ratio;   /* SEER_TOPK_RATIO: in (0, 1]; the product with i + 1 is formed in double */
  int32_t topk_k;      /* SEER_TOPK_FIXED: >= 1 */
  float threshold;     /* SEER_THRESHOLD: global threshold, used when head_thresholds is NULL */
  const float* head_thresholds; /* SEER_THRESHOLD: device [heads_q] per-head thresholds, or NULL */
  int32_t keep_first;  /* 1: block 0 is always kept */
  int32_t keep_diag;   /* 1: the diagonal block i is always kept (no empty row) */
  double rope_theta;   /* > 0: block-level RoPE in the gate (section 3.1): q and k are
                          taken before the model's RoPE, and the projected rows Qg, Kg
                          are rotated at their block positions with base rope_theta /
                          block (rope_theta is the model's RoPE base; rotate-half
                          pairing (d, d + Dg/2)).  0 disables it. */
  int32_t kv_shared;   /* 1: one mask per KV group instead of per query head (a
                          variant, not the paper's per-head gate): block j of query
                          block i is scored by the mean over the group's query heads
                          of their probabilities P[h][i][j], and TopK / threshold
                          select on that score; head_thresholds then has heads_kv
                          entries and out->kv_shared must be 1.  0: per head. */
} seer_gate_desc;

/* Block mask in compacted form: for row r = (b, h, i), idx[r][0 .. count[r]-1]
 * are the active key blocks j in strictly ascending order.  Caller-owned.
 * With kv_shared = 1 the rows are per KV head (h = KV head; heads = heads_kv
 * below) and row (b, g, i) applies to every query head of group g: attention
 * then loads each K/V tile once for several query heads of the group. */
typedef struct {
  int32_t n_blocks;  /* nb = ceil(seq_len / block), block 64 or 128 */
  int32_t* count;    /* device [batch][heads][nb], heads = heads_q (or heads_kv) */
  uint16_t* idx;     /* device [batch][heads][nb][nb] */
  uint8_t* dense;    /* optional device [batch][heads][nb][nb] 0/1 copy, or NULL */
  int32_t kv_shared; /* 0: rows per query head; 1: rows per KV head (see above) */
} seer_block_mask;

/* Launch options of the attention calls.  They choose how the work is
 * scheduled, never what is computed (apart from the split's bf16 rounding of
 * its partial outputs).  A NULL pointer or a zero field selects the default. */
typedef struct {
  int32_t split;            /* 1: cut long causal bf16 rows into key ranges (seer_bsattn_ws /
                               seer_dense_attn_ws with a workspace of seer_attn_workspace_bytes);
                               0: never (default) */
  int32_t split_width;      /* key blocks per range; <= 0: sized so that a range's K and V fill
                               an XCD's 4 MB L2 (128 blocks at head_dim 128) */
  int32_t heads_per_wg;     /* cap on the query heads one workgroup serves where the heads of a
                               KV group share their rows (dense attention, the ground truth, a
                               kv_shared mask): 1, 2 or 4; 0: 2 */
  int32_t batch_min_blocks; /* per-head sparse rows of at least this many 64-token blocks launch
                               the heaviest quarter of their tasks in batches of resident workgroups;
                               0: 2048; < 0: never */
  int32_t batch_wgs;        /* workgroups per such batch (rounded down to a multiple of 8);
                               0: as many as the GPU holds at once */
  int32_t walk_classes;     /* sparse rows of 64-token masks (unsplit, at most 2048 entries)
                               visit their blocks j = S q + c in the order (c, q): one column
                               order common to every row, which keeps the rows running at once
                               on K/V tiles near each other even where a mask selects runs of
                               adjacent blocks.  S = walk_classes: 1 (ascending), 2, 4, 8 or 16;
                               0: 4.  Changes only the order in which a row's tiles are summed */
} seer_attn_opts;

/* Options of seer_gate_distill (NULL or zero fields: defaults). */
typedef struct {
  int32_t gemm_min_chunks;  /* the backward products split their reduction into parts of at
                               least this many 32-wide chunks; 0: 8 */
  int32_t gemm_tile_n;      /* output tile width of the backward products, 64 or 128 columns
                               (any other value: SEER_ERR_INVALID_ARG); 0: 128 when gate_dim
                               is 128 and the rows hold at least 1024 blocks, else 64.
                               Changes only how the products are tiled and split */
} seer_distill_opts;

/* ABI version (SEER_ABI_VERSION of the built library). */
int seer_abi_version(void);

/* Static, human-readable name of a status code. */
const char* seer_status_str(int status);

/* Bytes of device workspace seer_gate needs for this shape (0 on invalid
 * arguments): the pooled-and-projected Q and K, (heads_q + heads_kv) nb
 * gate_dim values per batch entry, held as three bf16 parts each for the
 * logits kernel (6 bytes per value with nb rounded up to a multiple of 32;
 * 60 MiB for 32 + 8 heads of 2048 blocks at gate_dim 128; the fused kernel of
 * short rows keeps them as fp32 in the same region) and, when
 * logits_in_workspace is set (seer_gate called with logits_out NULL), the fp32
 * gate logits [batch][heads_q][nb][nb]. */
size_t seer_gate_workspace_bytes(const seer_attn_desc* desc, const seer_gate_desc* gate,
                                 int32_t logits_in_workspace);

/* Elements of the idx array of a per-query-head seer_block_mask for this shape
 * (B*Hq*nb*nb; a kv_shared mask needs B*Hkv*nb*nb). */
size_t seer_mask_idx_elems(const seer_attn_desc* desc, int32_t block);

/*
 * AttnGate (section 3.1, Eq. 1) and block selection (Eq. 3 / Eq. 4).
 *   Qp = average of each 64-token block of Q            [B][Hq][nb][D]
 *   Kp = max | min | average of each block of K         [B][Hkv][nb][3D]
 *   Qg = Qp Wq, Kg = Kp Wk (no bias)                    fp32
 *   optional block-level RoPE of Qg[i], Kg[j] at block positions i, j
 *   L[i][j] = Qg[i] . Kg[g][j] / sqrt(Dg) for j <= i    (block-causal)
 *   P = softmax over j of L[i][.]
 *   TopK: the forced blocks ({0} if keep_first, {i} if keep_diag) plus the best
 *         remaining causal blocks by L, ties to the smaller j, k_i blocks in all
 *         with k_i = min(i + 1, max(#forced, k)).
 *   Threshold: the forced blocks plus every causal j with P[i][j] > threshold.
 *   With gate->kv_shared the rows are per KV group and P above is replaced by
 *   the mean of P over the group's query heads.
 * Inputs q, k follow desc (bf16 or fp32); wq, wk are fp32 (layout in
 * seer_gate_desc).  Writes out->count, out->idx and, when non-NULL, out->dense.
 * logits_out (device float [B][Hq][nb][nb], or NULL) receives L for j <= i
 * (entries above the diagonal unspecified); when NULL, L lives in the
 * workspace between the logits kernel and the selection kernel, except for
 * per-query-head masks of at most 128 blocks, where one kernel forms and
 * selects the logits in on-chip memory (that part of the workspace then stays
 * unused).
 * workspace: device memory of at least seer_gate_workspace_bytes(desc, gate,
 * logits_out == NULL) bytes, 256-byte aligned.
 * Unsupported: gate->block not in {64, 128}, head_dim not in {64, 128},
 * gate_dim not in {32, 64, 128}, nb > 4096.
 */
seer_status seer_gate(const seer_attn_desc* desc, const seer_gate_desc* gate,
                      const void* q, const void* k, const float* wq, const float* wk,
                      seer_block_mask* out, float* logits_out,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * seer_gate for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): no
 * workspace argument and no allocation.  Its scratch (the projected rows Qg,
 * Kg) is a static device array of seer_gate_noalloc_max_bytes() bytes per
 * device (64 MiB; each device the library runs on holds it until the process
 * ends), and the logits are formed and selected in one kernel, never leaving
 * on-chip memory.  Masks equal seer_gate's except where a logit lies within
 * rounding of the selection cut (the two form the logits in a different
 * summation order).  Every call on a device shares that device's scratch:
 * calls that overlap on one device (concurrent streams, or host threads)
 * race, so serialise them.
 * Errors: as seer_gate; SEER_ERR_UNSUPPORTED for a kv_shared gate or rows of
 * more than 2048 blocks; SEER_ERR_WORKSPACE when the projected rows,
 * (heads_q + heads_kv) nb gate_dim fp32 per batch entry, exceed the scratch.
 */
seer_status seer_gate_noalloc(const seer_attn_desc* desc, const seer_gate_desc* gate,
                              const void* q, const void* k, const float* wq, const float* wk,
                              seer_block_mask* out, void* stream);

/* Size of seer_gate_noalloc's static scratch, in bytes. */
size_t seer_gate_noalloc_max_bytes(void);

/*
 * Block-sparse FlashAttention forward (section 3.3): for each query block i of
 * (b, h) and each active key block j of mask row (b, h, i) -- row (b, g, i),
 * g = h / (heads_q / heads_kv), of a kv_shared mask -- (blocks of `block`
 * tokens, 64 or 128; a 128-token mask is run as its 64-token tiles),
 *   O_i = softmax(sm_scale * Q_i K^T) V over the keys of the active blocks,
 * with the causal mask applied inside the diagonal block when causal != 0.
 * sm_scale <= 0 selects 1/sqrt(head_dim).  o follows desc (same dtype as q);
 * lse (device float [B][Hq][seq], or NULL) receives the natural-log
 * log-sum-exp of each query's scaled scores.  A row with no active block
 * yields O = 0 and LSE = -inf.  When causal, list entries j > i end the row;
 * entries j >= nb always end it, and count is clamped to nb, so a malformed
 * mask cannot make the kernel read out of bounds.
 * Unsupported: block not in {64, 128}, head_dim not in {64, 128}.
 */
seer_status seer_bsattn(const seer_attn_desc* desc, int32_t block, const seer_block_mask* mask,
                        int32_t causal, float sm_scale, const void* q, const void* k,
                        const void* v, void* o, float* lse, void* stream);

/*
 * Dense attention (the comparison path): seer_bsattn with every block active
 * (j <= i when causal, every j otherwise), without reading a mask.
 */
seer_status seer_dense_attn(const seer_attn_desc* desc, int32_t causal, float sm_scale,
                            const void* q, const void* k, const void* v, void* o, float* lse,
                            void* stream);

/*
 * Workspace bytes that let seer_bsattn_ws / seer_dense_attn_ws run the
 * key-range split for this shape and options, or 0 when the call does not
 * split (then it needs no workspace).  The split is opt-in (opts->split = 1;
 * the unsplit kernels measured faster on this hardware at the workloads here)
 * and applies to causal bf16 attention when a row can reach more than one
 * range of w key blocks (w = opts->split_width, or 128 at head_dim 128 and 256
 * at head_dim 64).  With P = ceil(nb / w) ranges: (P + 3) ints per query block,
 * 32 bytes of task-queue tickets, and (256 + 128 head_dim) bytes per partial
 * slot; a query head has sum over i of (floor(i / w) + 1) slots (8.6 GB for 32
 * heads of 131072 tokens at head_dim 128).  0 on invalid arguments.
 */
size_t seer_attn_workspace_bytes(const seer_attn_desc* desc, int32_t block, int32_t causal,
                                 const seer_attn_opts* opts);

/*
 * seer_bsattn / seer_dense_attn with launch options and a workspace for the
 * key-range split (section 3.3's kernel, scheduled for L2 locality): each
 * causal row is cut into ranges of w key blocks computed as separate tasks by
 * persistent workgroups that take the tasks in (KV group, range, query block)
 * order, so that every XCD reads one range's K and V at a time; a task writes
 * its normalised partial output (bf16) and log-sum-exp to the workspace, and a
 * row's last task merges them in a fixed order (results are reproducible bit
 * for bit).  O may differ from the unsplit call by the rounding of the
 * partials (well inside the bf16 output tolerance).  With opts NULL or
 * opts->split = 0, workspace NULL or smaller than seer_attn_workspace_bytes,
 * or a shape that does not split, the call is the unsplit one with the other
 * options applied.  workspace: device memory, 256-byte aligned; contents on
 * return unspecified.  SEER_ERR_INVALID_ARG for an option outside its range.
 */
seer_status seer_bsattn_ws(const seer_attn_desc* desc, int32_t block, const seer_block_mask* mask,
                           int32_t causal, float sm_scale, const void* q, const void* k,
                           const void* v, void* o, float* lse, void* workspace,
                           size_t workspace_bytes, const seer_attn_opts* opts, void* stream);
seer_status seer_dense_attn_ws(const seer_attn_desc* desc, int32_t causal, float sm_scale,
                               const void* q, const void* k, const void* v, void* o, float* lse,
                               void* workspace, size_t workspace_bytes, const seer_attn_opts* opts,
                               void* stream);

/*
 * Number of attention-kernel launches one seer_bsattn_ws / seer_dense_attn_ws
 * call with these arguments makes (mask_kind 0: dense, 1: a per-query-head
 * mask of `block`-token blocks, 2: a kv_shared mask), on the current device;
 * -1 on invalid arguments.  Launches nothing.  (Long sparse rows launch in
 * batches and a KV group at a time, so one call can be tens of launches.)
 */
int32_t seer_attn_launches(const seer_attn_desc* desc, int32_t block, int32_t mask_kind, int32_t causal,
                           const seer_attn_opts* opts, size_t workspace_bytes);

/*
 * Compacts a 0/1 block mask dense (device uint8 [B][heads][nb][nb], heads =
 * heads_kv when out->kv_shared, else heads_q; any non-zero byte is active)
 * into out->count / out->idx (ascending).  out->dense is ignored.
 */
seer_status seer_mask_from_dense(const seer_attn_desc* desc, int32_t block, const uint8_t* dense,
                                 seer_block_mask* out, void* stream);

/*
 * Workspace bytes of seer_attn_gt when it processes `kv_groups` KV groups per
 * launch (a KV group is one KV head and its heads_q / heads_kv query heads of
 * one batch entry); kv_groups <= 0 or >= batch * heads_kv means all of them
 * (one launch).  The workspace holds, per query head, the raw-score maximum of
 * every query over every key tile: fp32 [heads][nb][nb][64], 16 nb^2 KiB per
 * query head (1 GiB per head at seq_len 131072).  0 on invalid arguments.
 */
size_t seer_attn_gt_workspace_bytes(const seer_attn_desc* desc, int32_t block, int32_t kv_groups);

/*
 * Dense attention with the 2D max-pooled attention map (Eq. 2; computed as in
 * appendix A.1, Eq. 5-6).  Computes o and lse exactly as seer_dense_attn, and
 *   gt[b][h][i][j] = max over queries t of block i and keys s of block j of
 *                    softmax_s(sm_scale q_t . k_s)  (s <= t when causal),
 * 0 where block j holds no key visible to block i (j > i when causal).
 * gt: device float [batch][heads_q][nb][nb], caller-owned.  lse may be NULL.
 * workspace: device memory, 256-byte aligned, of at least
 * seer_attn_gt_workspace_bytes(desc, block, 1) bytes; the call runs as many KV
 * groups per launch as it holds (all at once with
 * seer_attn_gt_workspace_bytes(desc, block, 0)), several launches on `stream`
 * otherwise.  Its contents on return are unspecified.
 * opts (may be NULL): heads_per_wg applies; the split does not.
 * Errors: as seer_dense_attn; SEER_ERR_WORKSPACE if the workspace is missing
 * or smaller than one KV group needs.
 */
seer_status seer_attn_gt(const seer_attn_desc* desc, int32_t block, int32_t causal, float sm_scale,
                         const void* q, const void* k, const void* v, void* o, float* lse,
                         float* gt, void* workspace, size_t workspace_bytes, const seer_attn_opts* opts,
                         void* stream);

/* Bytes of device workspace seer_gate_distill needs for this shape and options
 * (0 on invalid arguments). */
size_t seer_gate_distill_workspace_bytes(const seer_attn_desc* desc, const seer_gate_desc* gate,
                                         const seer_distill_opts* opts);

/*
 * One distillation step of the gate (section 3.2, Eq. 2): the forward of
 * seer_gate up to the block-causal softmax P (pooling, linear layers, the
 * optional block-level RoPE, logits), then, with T the ground-truth row
 * gt[b][h][i][0..i] renormalised to sum 1 (a row summing to 0 gives T = 0),
 *   *loss = mean over the batch * heads_q * nb rows of KL(T || P)
 *         = sum_j T_j (log T_j - log P_j) / rows,   0 log 0 = 0,
 * and its gradients with respect to the gate weights:
 *   dwq, dwk: device fp32, the layout of wq, wk (per head or shared, as
 *   gate->w_per_head), overwritten (not accumulated).
 * gt: device fp32 [batch][heads_q][nb][nb] (seer_attn_gt's output; entries
 * j > i are not read).  loss: device fp32 scalar.  q, k, wq, wk as seer_gate.
 * Of gate, only block, gate_dim, w_per_head and rope_theta are used.
 * workspace: device memory of at least seer_gate_distill_workspace_bytes(desc,
 * gate, opts) bytes, 256-byte aligned (opts may be NULL).  No atomics: results
 * are identical run to run.
 * Errors: as seer_gate; SEER_ERR_INVALID_ARG for a NULL gt, loss, dwq or dwk.
 */
seer_status seer_gate_distill(const seer_attn_desc* desc, const seer_gate_desc* gate,
                              const void* q, const void* k, const float* wq, const float* wk,
                              const float* gt, float* loss, float* dwq, float* dwk,
                              void* workspace, size_t workspace_bytes, const seer_distill_opts* opts,
                              void* stream);

/*
 * Packed variable-length batches (the prefill layout of a serving batch):
 * desc->batch sequences, sequence b holding tokens [cu_seqlens_host[b],
 * cu_seqlens_host[b + 1]) of packed Q/K/V/O.  cu_seqlens_host is a host array
 * of batch + 1 non-decreasing offsets with cu[0] = 0 and cu[batch] =
 * desc->seq_len (the total token count); a sequence may be empty.  Strides come
 * from desc: q_stride[2] is the token stride and q_stride[1] the head stride
 * (q_stride[0] is ignored), e.g. [T][H][D] packing.  Every sequence is its own
 * causal (or non-causal) problem: no attention or pooling crosses a boundary,
 * and each has nb_b = ceil(len_b / block) blocks.  The calls run one batch-1
 * pass per sequence on `stream`, through the same kernels as seer_gate /
 * seer_bsattn (so results equal separate per-sequence calls bit for bit);
 * arguments of every sequence are validated before anything is launched.
 *
 * Mask layout: the sequences' row sets back to back.  Sequence b's count rows
 * [H][nb_b] start at element sum_{b'<b} H nb_b' of mask->count, and its idx
 * rows [H][nb_b][nb_b] at element sum_{b'<b} H nb_b'^2 of mask->idx (and of
 * mask->dense when present); H = heads_q, or heads_kv when kv_shared.
 * mask->n_blocks is ignored.  LSE (optional) is stored per sequence as
 * [heads_q][len_b] starting at element heads_q * cu[b].
 */

/* Elements of the idx array of a packed variable-length mask (0 on invalid
 * arguments); *count_elems (if not NULL) receives the elements of count. */
size_t seer_varlen_mask_elems(const seer_attn_desc* desc, const int32_t* cu_seqlens_host, int32_t block,
                              int32_t kv_shared, size_t* count_elems);

/* Workspace bytes of seer_gate_varlen: the largest sequence's seer_gate workspace
 * with the logits in the workspace (0 on invalid arguments). */
size_t seer_gate_varlen_workspace_bytes(const seer_attn_desc* desc, const int32_t* cu_seqlens_host,
                                        const seer_gate_desc* gate);

/* seer_gate over every sequence of a packed batch (section 3.1, Eq. 1, Eq. 3 / 4
 * per sequence); the workspace is reused by the sequences in stream order. */
seer_status seer_gate_varlen(const seer_attn_desc* desc, const int32_t* cu_seqlens_host,
                             const seer_gate_desc* gate, const void* q, const void* k, const float* wq,
                             const float* wk, seer_block_mask* out, void* workspace, size_t workspace_bytes,
                             void* stream);

/* seer_bsattn over every sequence of a packed batch (section 3.3 per sequence). */
seer_status seer_bsattn_varlen(const seer_attn_desc* desc, const int32_t* cu_seqlens_host, int32_t block,
                               const seer_block_mask* mask, int32_t causal, float sm_scale, const void* q,
                               const void* k, const void* v, void* o, float* lse, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SEER_H */
