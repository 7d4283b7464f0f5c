/*
 * seer_oracle.c -- plain fp64 CPU oracle for the SeerAttention prefill path
 * (arXiv 2410.13276).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the independent checker for the HIP
 * library in paper_2410_13276_amd/.  It shares no source, header, table or
 * helper with that library and must never be linked into it.  Only tests/,
 * __graft_entry__.smoke() and the cpu_baseline leg of bench.py may call it.
 *
 * Every step is written the slow, obvious way, in double precision, in the
 * order the paper states it:
 *
 *   orc_pool          -- section 3.1 ("Attention Gate Design" and "Pooling
 *                        Method Selection"): non-overlapping pooling along the
 *                        sequence with kernel = stride = B; Q uses average
 *                        pooling, K uses max, min and average pooling whose
 *                        results are concatenated along the hidden dimension
 *                        (order: max | min | avg).
 *   orc_linear        -- Eq. 1: the learnable linear layers W_q, W_k applied to
 *                        the pooled tensors (no bias term appears in Eq. 1).
 *   orc_block_rope    -- section 3.1 "Block-level RoPE in AttnGate": the gate is
 *                        fed pre-RoPE Q and K and rotates the projected rows at
 *                        their block positions with the reduced base theta / B
 *                        (rotate-half pairing (d, d + Dg/2) as in Llama).
 *   orc_gate_logits   -- Eq. 1: (W_q P_q(Q)) . (W_k P_k(K))^T / sqrt(d), with d
 *                        the contracted (gate) dimension, block-causal.
 *   orc_gate_logscore -- Eq. 1: the row softmax, returned in log form
 *                        ell = L - logsumexp(L) so that probabilities too small
 *                        for a double are still ordered exactly.
 *   orc_select        -- Eq. 3 (TopK) and Eq. 4 (threshold) with the always-kept
 *                        first and diagonal blocks.
 *   orc_group_logscore -- the shared-mask variant's score: the mean over a KV
 *                        group's query heads of their gate probabilities.
 *   orc_attn          -- softmax(Q K^T / sqrt(d)) V restricted to the keys whose
 *                        64-token block is active in the block mask (section 3.3
 *                        "Block Sparse Flash-Attn Kernel"); an all-ones mask is
 *                        plain causal attention (the dense comparison path).
 *   orc_maxpool_gt    -- Eq. 2: MaxPool2D over blocks of the full (causal or
 *                        not) attention probability map, the distillation
 *                        ground truth; all rows or a subset of query blocks.
 *
 * Sequences need not be a multiple of the block: the last block is then
 * partial (pooled over the tokens it holds; its rows past the end are not
 * queries and come back as NaN from orc_attn).
 *
 * Inputs arrive in the element type the GPU receives (fp32, or bf16 given as
 * raw 16-bit patterns) and are widened to double exactly before any arithmetic.
 * Strides are in elements, in the order (batch, head, sequence); the head
 * dimension is contiguous.
 *
 * Parity status of each function is recorded in the tests that pin it; no
 * function here is "parity unpinned".
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_F32 = 0, ORC_BF16 = 1 };
enum { ORC_POOL_AVG = 0, ORC_POOL_MAX_MIN_AVG = 1 };
enum { ORC_TOPK_RATIO = 0, ORC_TOPK_FIXED = 1, ORC_THRESHOLD = 2 };

/* Widen one stored element to double (exact for both fp32 and bf16). */
static double elem(const void *base, int dtype, int64_t off) {
  if (dtype == ORC_F32) return (double)((const float *)base)[off];
  uint32_t u = ((uint32_t)((const uint16_t *)base)[off]) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

int orc_version(void) { return 1; }

int orc_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
  return omp_get_max_threads();
#else
  (void)n;
  return 1;
#endif
}

/*
 * Pooling along the sequence (section 3.1).  x is [B][H][S][D] with strides
 * st[0..2]; block is the pooling kernel and stride.  kind selects
 *   ORC_POOL_AVG          -> out [B][H][nb][D]      (Q side)
 *   ORC_POOL_MAX_MIN_AVG  -> out [B][H][nb][3*D]    (K side: max | min | avg)
 * with nb = ceil(S / block): a partial last block is pooled over the rows it
 * holds (its mean divides by that count).  Returns 0, or -1 for a non-positive
 * block or length.
 */
int orc_pool(const void *x, int dtype, int B, int H, int S, int D,
             const int64_t *st, int block, int kind, double *out) {
  if (block <= 0 || S <= 0) return -1;
  const int nb = (S + block - 1) / block; /* the last block may be partial */
  const int width = (kind == ORC_POOL_AVG) ? D : 3 * D;
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < H; ++h)
      for (int i = 0; i < nb; ++i) {
        double *o = out + (((int64_t)b * H + h) * nb + i) * width;
        for (int d = 0; d < D; ++d) {
          double sum = 0.0, mx = -INFINITY, mn = INFINITY;
          const int t_end = (i + 1) * block < S ? (i + 1) * block : S;
          for (int t = i * block; t < t_end; ++t) {
            double v = elem(x, dtype, b * st[0] + h * st[1] + t * st[2] + d);
            sum += v;
            if (v > mx) mx = v;
            if (v < mn) mn = v;
          }
          double avg = sum / (t_end - i * block);
          if (kind == ORC_POOL_AVG) {
            o[d] = avg;
          } else {
            o[d] = mx;
            o[D + d] = mn;
            o[2 * D + d] = avg;
          }
        }
      }
  return 0;
}

/*
 * Gate linear layer (Eq. 1): out[b][h][i][j] = sum_c in[b][h][i][c] * W[h'][c][j]
 * with h' = h when w_per_head, else 0 (one matrix shared by all heads).
 * in is [B][H][nb][din] (double), W is [H or 1][din][dout] (fp32), out is
 * [B][H][nb][dout].  No bias.
 */
void orc_linear(const double *in, int B, int H, int nb, int din,
                const float *W, int w_per_head, int dout, double *out) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < H; ++h) {
      const float *w = W + (w_per_head ? (int64_t)h * din * dout : 0);
      for (int i = 0; i < nb; ++i) {
        const double *p = in + (((int64_t)b * H + h) * nb + i) * din;
        double *o = out + (((int64_t)b * H + h) * nb + i) * dout;
        for (int j = 0; j < dout; ++j) {
          double acc = 0.0;
          for (int c = 0; c < din; ++c) acc += p[c] * (double)w[(int64_t)c * dout + j];
          o[j] = acc;
        }
      }
    }
}

/*
 * Block-level RoPE (section 3.1): row i of x [rows][nb][Dg] (in place) is the
 * gate feature vector of block i; it is rotated by angle i * w_d in each plane
 * (d, d + Dg/2), d < Dg/2, with w_d = (theta / block)^(-2d/Dg).  theta is the
 * model's RoPE base; block is the pooling block size B.
 */
void orc_block_rope(double *x, int64_t rows, int nb, int Dg, double theta, int block) {
  const int half = Dg / 2;
  const double base = theta / block;
  for (int64_t r = 0; r < rows; ++r)
    for (int i = 0; i < nb; ++i) {
      double *v = x + (r * nb + i) * Dg;
      for (int d = 0; d < half; ++d) {
        const double w = pow(base, -2.0 * d / Dg);
        const double ang = (double)i * w;
        const double c = cos(ang), s = sin(ang);
        const double a = v[d], b = v[d + half];
        v[d] = a * c - b * s;
        v[d + half] = a * s + b * c;
      }
    }
}

/*
 * Gate logits (Eq. 1), block-causal: for query head h the key side comes from
 * KV head g = h / (Hq/Hkv).  L[b][h][i][j] = Qg[b][h][i] . Kg[b][g][j] / sqrt(Dg)
 * for j <= i and -inf for j > i.  L is [B][Hq][nb][nb].
 */
void orc_gate_logits(const double *Qg, const double *Kg, int B, int Hq, int Hkv,
                     int nb, int Dg, double *L) {
  const int G = Hq / Hkv;
  const double inv_sqrt = 1.0 / sqrt((double)Dg);
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < Hq; ++h) {
      const int g = h / G;
      for (int i = 0; i < nb; ++i) {
        const double *q = Qg + (((int64_t)b * Hq + h) * nb + i) * Dg;
        double *row = L + (((int64_t)b * Hq + h) * nb + i) * nb;
        for (int j = 0; j < nb; ++j) {
          if (j > i) {
            row[j] = -INFINITY;
            continue;
          }
          const double *k = Kg + (((int64_t)b * Hkv + g) * nb + j) * Dg;
          double acc = 0.0;
          for (int c = 0; c < Dg; ++c) acc += q[c] * k[c];
          row[j] = acc * inv_sqrt;
        }
      }
    }
}

/*
 * Row softmax of the gate logits in log form (Eq. 1):
 * ell[r][j] = L[r][j] - log(sum_{j'} exp(L[r][j'])), with -inf kept as -inf.
 * rows = B*Hq*nb rows of length nb.
 */
void orc_gate_logscore(const double *L, int64_t rows, int nb, double *ell) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    const double *l = L + r * nb;
    double *e = ell + r * nb;
    double m = -INFINITY;
    for (int j = 0; j < nb; ++j)
      if (l[j] > m) m = l[j];
    double s = 0.0;
    for (int j = 0; j < nb; ++j)
      if (l[j] != -INFINITY) s += exp(l[j] - m);
    const double lse = m + log(s);
    for (int j = 0; j < nb; ++j) e[j] = (l[j] == -INFINITY) ? -INFINITY : l[j] - lse;
  }
}

/*
 * Shared-mask variant (a mask per KV group instead of per query head; the
 * paper's gate is per head, section 3.1): the group's score of block j for
 * query block i is the mean over its G = Hq / Hkv query heads h of the gate
 * probabilities P[h][i][j] = exp(ell[h][i][j]).  Returned in log form,
 *   ellg[b][g][i][j] = log( (1/G) sum_h exp(ell[b][h][i][j]) ),
 * formed as a log-sum-exp over the heads so that tiny probabilities keep their
 * order; entries that are -inf for every head stay -inf.
 */
void orc_group_logscore(const double *ell, int B, int Hq, int Hkv, int nb, double *ellg) {
  const int G = Hq / Hkv;
  const int64_t rows = (int64_t)B * Hkv * nb;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    const int i = (int)(r % nb);
    const int g = (int)((r / nb) % Hkv);
    const int b = (int)(r / ((int64_t)nb * Hkv));
    double *out = ellg + r * nb;
    for (int j = 0; j < nb; ++j) {
      double m = -INFINITY;
      for (int h = 0; h < G; ++h) {
        const double x = ell[(((int64_t)b * Hq + (int64_t)g * G + h) * nb + i) * nb + j];
        if (x > m) m = x;
      }
      if (m == -INFINITY) {
        out[j] = -INFINITY;
        continue;
      }
      double s = 0.0;
      for (int h = 0; h < G; ++h)
        s += exp(ell[(((int64_t)b * Hq + (int64_t)g * G + h) * nb + i) * nb + j] - m);
      out[j] = m + log(s / (double)G);
    }
  }
}

/* Candidate ordering for TopK: larger log-score first, smaller block index on ties. */
typedef struct {
  double v;
  int j;
} cand_t;

static int cand_cmp(const void *a, const void *b) {
  const cand_t *x = (const cand_t *)a, *y = (const cand_t *)b;
  if (x->v > y->v) return -1;
  if (x->v < y->v) return 1;
  return (x->j < y->j) ? -1 : (x->j > y->j);
}

/*
 * Per-row k for the TopK modes.  Ratio mode keeps ceil(rho * (i + 1)) of the
 * i + 1 causal blocks of row i (the product is formed in double), never fewer
 * than the forced blocks and never more than the row holds.
 */
int orc_topk_k(int mode, int i, double rho, int k_fixed, int n_forced) {
  int k;
  if (mode == ORC_TOPK_RATIO)
    k = (int)ceil(rho * (double)(i + 1));
  else
    k = k_fixed;
  if (k < n_forced) k = n_forced;
  if (k > i + 1) k = i + 1;
  return k;
}

/*
 * Block selection (Eq. 3 / Eq. 4) on the log-scores ell [B][Hq][nb][nb].
 * Forced set F_i = {0 if keep_first} U {i if keep_diag}.
 *   TopK modes: F_i plus the (k_i - |F_i|) best non-forced causal blocks by
 *     ell, ties to the smaller block index.  cut[r] = ell of the last block so
 *     taken (NAN if none was taken, i.e. the row is decided by F_i alone or
 *     takes every candidate).
 *   Threshold: F_i plus {j <= i : exp(ell[i][j]) > thr_h}, compared in double
 *     against the fp32 threshold widened to double; thr has n_thr = 1 (global)
 *     or Hq (per head) entries.  cut[r] = log(thr_h).
 * Outputs (any may be NULL): mask [B][Hq][nb][nb] 0/1, count [B][Hq][nb],
 * idx [B][Hq][nb][nb] ascending (first count entries valid), cut [B][Hq][nb].
 */
int orc_select(const double *ell, int B, int Hq, int nb, int mode, double rho,
               int k_fixed, const float *thr, int n_thr, int keep_first,
               int keep_diag, uint8_t *mask, int32_t *count, uint16_t *idx,
               double *cut) {
  if (mode == ORC_THRESHOLD && !(n_thr == 1 || n_thr == Hq)) return -1;
  const int64_t rows = (int64_t)B * Hq * nb;
  int bad = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : bad)
  for (int64_t r = 0; r < rows; ++r) {
    const int i = (int)(r % nb);
    const int h = (int)((r / nb) % Hq);
    const double *e = ell + r * nb;
    uint8_t *sel = (uint8_t *)calloc((size_t)nb, 1);
    cand_t *c = (cand_t *)malloc(sizeof(cand_t) * (size_t)(i + 1));
    if (!sel || !c) {
      bad = 1;
      free(sel);
      free(c);
      continue;
    }
    int n_forced = 0;
    if (keep_first) { sel[0] = 1; ++n_forced; }
    if (keep_diag && !sel[i]) { sel[i] = 1; ++n_forced; }
    double row_cut = NAN;
    if (mode == ORC_THRESHOLD) {
      const double t = (double)thr[n_thr == 1 ? 0 : h];
      for (int j = 0; j <= i; ++j)
        if (exp(e[j]) > t) sel[j] = 1;
      row_cut = log(t);
    } else {
      const int k = orc_topk_k(mode, i, rho, k_fixed, n_forced);
      int nc = 0;
      for (int j = 0; j <= i; ++j)
        if (!sel[j]) { c[nc].v = e[j]; c[nc].j = j; ++nc; }
      qsort(c, (size_t)nc, sizeof(cand_t), cand_cmp);
      const int take = k - n_forced;
      for (int t = 0; t < take; ++t) sel[c[t].j] = 1;
      if (take > 0 && take < nc) row_cut = c[take - 1].v;
    }
    int n = 0;
    for (int j = 0; j < nb; ++j) {
      if (mask) mask[r * nb + j] = sel[j];
      if (sel[j]) {
        if (idx) idx[r * nb + n] = (uint16_t)j;
        ++n;
      }
    }
    if (count) count[r] = n;
    if (cut) cut[r] = row_cut;
    free(sel);
    free(c);
  }
  return bad ? -2 : 0;
}

/*
 * Masked causal attention (section 3.3, and the attention map of Eq. 2).
 * For query t in q-block i of (b, h), with KV head g = h / (Hq/Hkv), the key
 * set is A(t) = { s : (s <= t or not causal) and mask[b][h][i][s/block] != 0 };
 * mask == NULL means every block is active (dense attention).
 *   O[t]   = sum_{s in A(t)} softmax_s(scale * q_t . k_s) v_s
 *   LSE[t] = log sum_{s in A(t)} exp(scale * q_t . k_s)
 * An empty A(t) gives O = 0 and LSE = -inf.
 * rows lists n_rows q-block tasks as int32 triples (b, h, i); rows == NULL means
 * every (b, h, i) in that order.  O is [n_rows][block][D] and LSE is
 * [n_rows][block] (both may be NULL-free only; LSE may be NULL).
 */
int orc_attn(const void *q, const void *k, const void *v, int dtype, int B,
             int Hq, int Hkv, int S, int D, const int64_t *qs, const int64_t *ks,
             const int64_t *vs, int block, int causal, double scale,
             const uint8_t *mask, const int32_t *rows, int n_rows, double *O,
             double *LSE) {
  if (block <= 0 || S <= 0 || Hkv <= 0 || Hq % Hkv != 0) return -1;
  const int nb = (S + block - 1) / block; /* the last block may be partial */
  const int G = Hq / Hkv;
  const int64_t total = rows ? n_rows : (int64_t)B * Hq * nb;
  int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
  for (int64_t r = 0; r < total; ++r) {
    int b, h, i;
    if (rows) {
      b = rows[3 * r];
      h = rows[3 * r + 1];
      i = rows[3 * r + 2];
    } else {
      b = (int)(r / ((int64_t)Hq * nb));
      h = (int)((r / nb) % Hq);
      i = (int)(r % nb);
    }
    const int g = h / G;
    double *score = (double *)malloc(sizeof(double) * (size_t)S);
    double *qv = (double *)malloc(sizeof(double) * (size_t)D);
    if (!score || !qv) {
      bad = 1;
      free(score);
      free(qv);
      continue;
    }
    const uint8_t *mrow = mask ? mask + (((int64_t)b * Hq + h) * nb + i) * nb : NULL;
    for (int tt = 0; tt < block; ++tt) {
      const int t = i * block + tt;
      double *o = O + (r * block + tt) * D;
      if (t >= S) { /* past the end of a partial last block: no query */
        for (int d = 0; d < D; ++d) o[d] = NAN;
        if (LSE) LSE[r * block + tt] = NAN;
        continue;
      }
      for (int d = 0; d < D; ++d) qv[d] = elem(q, dtype, b * qs[0] + h * qs[1] + (int64_t)t * qs[2] + d);
      double m = -INFINITY;
      for (int s = 0; s < S; ++s) {
        const int active = (!causal || s <= t) && (!mrow || mrow[s / block]);
        if (!active) {
          score[s] = NAN; /* marks "not in A(t)" */
          continue;
        }
        double acc = 0.0;
        for (int d = 0; d < D; ++d)
          acc += qv[d] * elem(k, dtype, b * ks[0] + g * ks[1] + (int64_t)s * ks[2] + d);
        score[s] = scale * acc;
        if (score[s] > m) m = score[s];
      }
      for (int d = 0; d < D; ++d) o[d] = 0.0;
      if (m == -INFINITY) {
        if (LSE) LSE[r * block + tt] = -INFINITY;
        continue;
      }
      double l = 0.0;
      for (int s = 0; s < S; ++s) {
        if (isnan(score[s])) continue;
        const double p = exp(score[s] - m);
        l += p;
        for (int d = 0; d < D; ++d)
          o[d] += p * elem(v, dtype, b * vs[0] + g * vs[1] + (int64_t)s * vs[2] + d);
      }
      for (int d = 0; d < D; ++d) o[d] /= l;
      if (LSE) LSE[r * block + tt] = m + log(l);
    }
    free(score);
    free(qv);
  }
  return bad ? -2 : 0;
}

/*
 * Distillation ground truth (Eq. 2): gt[i][j] = max over the block-sized tile
 * (i, j) of the attention probabilities softmax(scale * Q K^T), keys s <= t
 * when causal.  Tiles with no visible key (j > i, causal) hold 0.
 * rows: int32 [n_rows][3] of (b, h, i) query-block rows, or NULL for all rows
 * in (b, h, i) order; gt is [n][nb] with n = n_rows or B * Hq * nb.
 */
int orc_maxpool_gt(const void *q, const void *k, int dtype, int B, int Hq,
                   int Hkv, int S, int D, const int64_t *qs, const int64_t *ks,
                   int block, int causal, double scale, const int32_t *rows,
                   int64_t n_rows, double *gt) {
  if (block <= 0 || S <= 0 || Hkv <= 0 || Hq % Hkv != 0) return -1;
  const int nb = (S + block - 1) / block; /* the last block may be partial */
  const int G = Hq / Hkv;
  const int64_t n = rows ? n_rows : (int64_t)B * Hq * nb;
  int bad = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : bad)
  for (int64_t r = 0; r < n; ++r) {
    int b, h, i;
    if (rows) {
      b = rows[3 * r];
      h = rows[3 * r + 1];
      i = rows[3 * r + 2];
      if (b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= nb) {
        bad = 1;
        continue;
      }
    } else {
      b = (int)(r / ((int64_t)Hq * nb));
      h = (int)((r / nb) % Hq);
      i = (int)(r % nb);
    }
    const int g = h / G;
    double *score = (double *)malloc(sizeof(double) * (size_t)S);
    if (!score) {
      bad = 1;
      continue;
    }
    double *out = gt + r * nb;
    for (int j = 0; j < nb; ++j) out[j] = 0.0;
    const int t_end = (i + 1) * block < S ? (i + 1) * block : S;
    for (int t = i * block; t < t_end; ++t) {
      const int last = causal ? t : S - 1; /* keys 0..last are visible */
      double m = -INFINITY;
      for (int s = 0; s <= last; ++s) {
        double acc = 0.0;
        for (int d = 0; d < D; ++d)
          acc += elem(q, dtype, b * qs[0] + h * qs[1] + (int64_t)t * qs[2] + d) *
                 elem(k, dtype, b * ks[0] + g * ks[1] + (int64_t)s * ks[2] + d);
        score[s] = scale * acc;
        if (score[s] > m) m = score[s];
      }
      double l = 0.0;
      for (int s = 0; s <= last; ++s) l += exp(score[s] - m);
      for (int s = 0; s <= last; ++s) {
        const double p = exp(score[s] - m) / l;
        if (p > out[s / block]) out[s / block] = p;
      }
    }
    free(score);
  }
  return bad ? -2 : 0;
}
