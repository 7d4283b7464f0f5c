// gate_kernels.hip -- AttnGate kernels for gfx950 (SeerAttention, arXiv 2410.13276).
//
//   pool_proj_kernel    section 3.1 + Eq. 1: average-pool Q and max|min|avg-pool K
//                       over each 64- or 128-token block, then the gate linear layers and,
//                       optionally, the block-level RoPE of section 3.1.
//                       HBM-bound: streams Q and K once with 16-byte loads; the
//                       GEMV reuses each weight element for every block of the
//                       workgroup.
//   gate_logits_kernel  Eq. 1: Qg Kg^T / sqrt(Dg) on the block-causal lower
//                       triangle, 128x128 tiles on bf16 MFMA
//                       (v_mfma_f32_32x32x16_bf16) from Qg, Kg split in three
//                       bf16 parts each (fp32-accurate products).
//   select_kernel       Eq. 3 (TopK by an exact select: one pass over 256
//                       equal-width value buckets, then, inside the target
//                       bucket, ranks of its gathered keys (at most 64) or
//                       8-bit digits of order-preserving keys, each from a
//                       per-wavefront LDS histogram; ties to the smaller
//                       block index) or Eq. 4 (strict
//                       threshold on the row softmax), plus the always-kept first
//                       and diagonal blocks; one wavefront per query-block row,
//                       writing the ascending index list by ballot compaction.
//   gate_fused_kernel   the logits of 16 query-block rows on fp32 MFMA into LDS,
//                       then select_kernel's selection of each row from LDS; no
//                       logits buffer, so it serves the no-allocation gate.
//   mask_from_dense_kernel  the same compaction for caller-made 0/1 masks.
#include <mutex>

#include "device_common.h"
#include "launch.h"

namespace seer {

// ---------------------------------------------------------------------------
// pooling + gate linear layers
// ---------------------------------------------------------------------------

template <typename T>
struct Load16;
template <>
struct Load16<float> {
  static constexpr int N = 4;
  __device__ static void get(const float* p, float* out) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
    for (int e = 0; e < 4; ++e) out[e] = v[e];
  }
};
template <>
struct Load16<uint16_t> {
  static constexpr int N = 8;
  __device__ static void get(const uint16_t* p, float* out) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      out[2 * e] = __uint_as_float(v[e] << 16);
      out[2 * e + 1] = __uint_as_float(v[e] & 0xFFFF0000u);
    }
  }
};

// x as the sum of three bf16 values hi + mid + lo (each rounded to nearest
// even from what the previous parts leave; both differences are exact in fp32
// because each part is within a factor of two of the remainder it rounds).
// hi + mid + lo reproduces x to about 2^-27 relative, so products of the parts
// summed in fp32 (the bf16 logits kernel) stay as accurate as an fp32 product.
//
// The parts are stored in the order the logits kernel's MFMA operands consume
// them: per 32-row group rb, 16-feature step c and part p, one 1 KiB run of 64
// lanes x 8 features, lane hf 32 + rl holding features 16c + 8hf .. +7 of row
// 32 rb + rl, so that every operand load of a wavefront reads 1 KiB of
// contiguous memory.  A head holds ceil(nb / 32) groups (split_rows(nb) rows).
__host__ __device__ __forceinline__ int64_t split_index(int r, int f, int part, int dg) {
  const int rb = r / 32, rl = r % 32, c = f / 16, hf = (f / 8) % 2, e = f % 8;
  return ((((int64_t)rb * (dg / 16) + c) * 3 + part) * 64 + (hf * 32 + rl)) * 8 + e;
}

__device__ __forceinline__ void store_split(uint16_t* head, int r, int f, int dg, float x) {
  const __bf16 hi = (__bf16)x;
  const float r1 = x - (float)hi;
  const __bf16 mid = (__bf16)r1;
  const __bf16 lo = (__bf16)(r1 - (float)mid);
  head[split_index(r, f, 0, dg)] = __builtin_bit_cast(uint16_t, hi);
  head[split_index(r, f, 1, dg)] = __builtin_bit_cast(uint16_t, mid);
  head[split_index(r, f, 2, dg)] = __builtin_bit_cast(uint16_t, lo);
}

// One workgroup of 256 threads pools R consecutive 64-token blocks of one head
// and then projects the R pooled rows through the head's gate weights.  Each
// thread owns one 16-byte column chunk of one block and walks its rows: all
// of them (RS = 1), or one of RS equal row ranges (short sequences, whose
// RS = 1 grid would hold too few workgroups to keep enough loads in flight),
// the ranges' partial sums, maxima and minima then combined through LDS.
template <typename T, int D, int DG, int RS>
struct PoolTiling {
  static constexpr int EPL = Load16<T>::N;  // elements per 16-byte load
  static constexpr int TPR = D / EPL;       // threads per block row
  static constexpr int R = 256 / (TPR * RS);  // blocks per workgroup
  static constexpr bool ok = R >= 1 && R * TPR * RS == 256 && R * DG >= 256 && (R * DG) % 256 == 0;
};

template <typename T, int D, int DG, bool IS_K, int BLK, int RS>
__device__ __forceinline__ void pool_proj_head(const T* __restrict__ x, int64_t ss, int nb, int seq_len,
                                               const float* __restrict__ W,
                                               float* __restrict__ out, float* smem,
                                               float* srot, double rope_base,
                                               float* __restrict__ pooled_out, uint16_t* __restrict__ split) {
  using Til = PoolTiling<T, D, DG, RS>;
  constexpr int EPL = Til::EPL;
  constexpr int TPR = Til::TPR;
  constexpr int R = Til::R;
  constexpr int WIDTH = IS_K ? 3 * D : D;
  constexpr int RPT = R * DG / 256;  // output rows per thread in the GEMV
  constexpr int PSTR = RS * WIDTH;   // LDS floats between pooled rows
  static_assert(Til::ok, "bad tiling");

  const int t = threadIdx.x;
  const int c = t % TPR;
  const int rs = (t / TPR) % RS;  // this thread's row range
  const int r = t / (TPR * RS);
  const int blk = blockIdx.x * R + r;

  if (blk < nb) {
    float sum[EPL], mx[EPL], mn[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      sum[e] = 0.f;
      mx[e] = -INFINITY;
      mn[e] = INFINITY;
    }
    const T* base = x + (int64_t)blk * BLK * ss + c * EPL;
    const int nrow = min(BLK, seq_len - blk * BLK);  // the last block may be partial
    const int row_end = min(nrow, (rs + 1) * (BLK / RS));
#pragma unroll 8
    for (int row = rs * (BLK / RS); row < row_end; ++row) {
      float v[EPL];
      Load16<T>::get(base + row * ss, v);
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        sum[e] += v[e];
        if (IS_K) {
          mx[e] = fmaxf(mx[e], v[e]);
          mn[e] = fminf(mn[e], v[e]);
        }
      }
    }
    // RS = 1: the pooled row; otherwise the range's raw sum, maximum, minimum
    float* prow = smem + (r * RS + rs) * WIDTH + c * EPL;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      const float avg = RS == 1 ? sum[e] / (float)nrow : sum[e];
      if (IS_K) {
        prow[e] = mx[e];
        prow[D + e] = mn[e];
        prow[2 * D + e] = avg;
      } else {
        prow[e] = avg;
      }
    }
    if (RS == 1 && pooled_out) {  // the pooled row itself (kept for the gate's weight gradients)
      float* po = pooled_out + (int64_t)blk * WIDTH + c * EPL;
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        po[e] = prow[e];
        if (IS_K) {
          po[D + e] = prow[D + e];
          po[2 * D + e] = prow[2 * D + e];
        }
      }
    }
  }
  __syncthreads();
  if constexpr (RS > 1) {
    // combine the ranges in range order into the first range's slot: maxima,
    // minima, and the sums divided by the block's row count
    for (int idx = t; idx < R * WIDTH; idx += 256) {
      const int rr = idx / WIDTH, col = idx % WIDTH;
      const int bb = blockIdx.x * R + rr;
      if (bb >= nb) continue;
      float* p = smem + rr * PSTR + col;
      float v = p[0];
      const int kind = IS_K ? col / D : 2;  // 0 max, 1 min, 2 mean
#pragma unroll
      for (int q = 1; q < RS; ++q) {
        const float u = p[q * WIDTH];
        v = kind == 0 ? fmaxf(v, u) : (kind == 1 ? fminf(v, u) : v + u);
      }
      if (kind == 2) v /= (float)min(BLK, seq_len - bb * BLK);
      p[0] = v;
      if (pooled_out) pooled_out[(int64_t)bb * WIDTH + col] = v;
    }
    __syncthreads();
  }

  // GEMV: out[r][j] = sum_c pooled[r][c] * W[c][j]
  const int j = t % DG;
  const int r0 = t / DG;  // rows r0, r0 + 256/DG, ...
  constexpr int RSTEP = 256 / DG;
  float acc[RPT];
#pragma unroll
  for (int q = 0; q < RPT; ++q) acc[q] = 0.f;
#pragma unroll 2
  for (int cc = 0; cc < WIDTH; cc += 4) {
    float w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = W[(int64_t)(cc + e) * DG + j];
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      const f32x4 p = *reinterpret_cast<const f32x4*>(smem + (r0 + q * RSTEP) * PSTR + cc);
      acc[q] = fmaf(p[0], w[0], acc[q]);
      acc[q] = fmaf(p[1], w[1], acc[q]);
      acc[q] = fmaf(p[2], w[2], acc[q]);
      acc[q] = fmaf(p[3], w[3], acc[q]);
    }
  }
  if (rope_base > 0.0) {
    // Block-level RoPE (section 3.1): rotate plane (d, d + DG/2) of the row of
    // block bb by angle bb * base^(-2d/DG); the angle is formed in double.
#pragma unroll
    for (int q = 0; q < RPT; ++q) srot[(r0 + q * RSTEP) * DG + j] = acc[q];
    __syncthreads();
    constexpr int HALF = DG / 2;
    const int d = j % HALF;
    const double w = pow(rope_base, -2.0 * d / DG);
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      const int rr = r0 + q * RSTEP;
      const int bb = blockIdx.x * R + rr;
      const double ang = (double)bb * w;
      const float cs = (float)cos(ang), sn = (float)sin(ang);
      const float a = srot[rr * DG + d], b = srot[rr * DG + d + HALF];
      acc[q] = (j < HALF) ? (a * cs - b * sn) : (a * sn + b * cs);
    }
  }
#pragma unroll
  for (int q = 0; q < RPT; ++q) {
    const int bb = blockIdx.x * R + r0 + q * RSTEP;
    if (bb < nb) {
      if (out) out[(int64_t)bb * DG + j] = acc[q];
      if (split) store_split(split, bb, j, DG, acc[q]);
    }
  }
}

template <typename T, int D, int DG, int BLK, int RS>
__global__ __launch_bounds__(256) void pool_proj_kernel(PoolProjArgs a) {
  constexpr int R = PoolTiling<T, D, DG, RS>::R;
  __shared__ __attribute__((aligned(16))) float smem[R * RS * 3 * D];
  __shared__ float srot[R * DG];
  const int b = blockIdx.z;
  // the K heads' workgroups (max | min | avg pooling, a GEMV three times as
  // wide) are dispatched first, so that the lighter Q heads' fill the end
  const int slot = (blockIdx.y + a.heads_q) % (a.heads_q + a.heads_kv);
  if (slot < a.heads_q) {
    const int h = slot;
    const T* x = static_cast<const T*>(a.q.ptr) + b * a.q.sb + h * a.q.sh;
    float* out = a.qg ? a.qg + ((int64_t)b * a.heads_q + h) * a.n_blocks * DG : nullptr;
    float* po = a.qp ? a.qp + ((int64_t)b * a.heads_q + h) * a.n_blocks * D : nullptr;
    uint16_t* sp = a.qs ? a.qs + ((int64_t)b * a.heads_q + h) * split_rows(a.n_blocks) * 3 * DG : nullptr;
    pool_proj_head<T, D, DG, false, BLK, RS>(x, a.q.ss, a.n_blocks, a.seq_len, a.wq + h * a.wq_head_stride, out, smem, srot,
                                    a.rope_base, po, sp);
  } else {
    const int g = slot - a.heads_q;
    const T* x = static_cast<const T*>(a.k.ptr) + b * a.k.sb + g * a.k.sh;
    float* out = a.kg ? a.kg + ((int64_t)b * a.heads_kv + g) * a.n_blocks * DG : nullptr;
    float* po = a.kp ? a.kp + ((int64_t)b * a.heads_kv + g) * a.n_blocks * 3 * D : nullptr;
    uint16_t* sp = a.ks ? a.ks + ((int64_t)b * a.heads_kv + g) * split_rows(a.n_blocks) * 3 * DG : nullptr;
    pool_proj_head<T, D, DG, true, BLK, RS>(x, a.k.ss, a.n_blocks, a.seq_len, a.wk + g * a.wk_head_stride, out, smem, srot,
                                   a.rope_base, po, sp);
  }
}

// Row ranges per block: 4 when the grid of whole-block threads would hold fewer
// than kPoolSplitWgs workgroups (and the tiling allows it), else 1.
constexpr int kPoolSplitWgs = 512;

template <typename T, int D, int DG, int RS>
static hipError_t pool_proj_launch_rs(const PoolProjArgs& a, hipStream_t s) {
  constexpr int R = PoolTiling<T, D, DG, RS>::R;
  dim3 grid((a.n_blocks + R - 1) / R, a.heads_q + a.heads_kv, a.batch);
  if (a.block == 64) hipLaunchKernelGGL((pool_proj_kernel<T, D, DG, 64, RS>), grid, dim3(256), 0, s, a);
  else if (a.block == 128) hipLaunchKernelGGL((pool_proj_kernel<T, D, DG, 128, RS>), grid, dim3(256), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

template <typename T, int D, int DG>
static hipError_t pool_proj_launch(const PoolProjArgs& a, hipStream_t s) {
  constexpr int R1 = PoolTiling<T, D, DG, 1>::R;
  const int64_t wgs = (int64_t)((a.n_blocks + R1 - 1) / R1) * (a.heads_q + a.heads_kv) * a.batch;
  if constexpr (PoolTiling<T, D, DG, 4>::ok) {
    if (wgs < kPoolSplitWgs) return pool_proj_launch_rs<T, D, DG, 4>(a, s);
  }
  return pool_proj_launch_rs<T, D, DG, 1>(a, s);
}

template <typename T, int D>
static hipError_t pool_proj_dg(const PoolProjArgs& a, hipStream_t s) {
  switch (a.gate_dim) {
    case 32: return pool_proj_launch<T, D, 32>(a, s);
    case 64: return pool_proj_launch<T, D, 64>(a, s);
    case 128: return pool_proj_launch<T, D, 128>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_pool_proj(const PoolProjArgs& a, hipStream_t s) {
  if (a.bf16) {
    if (a.head_dim == 64) return pool_proj_dg<uint16_t, 64>(a, s);
    if (a.head_dim == 128) return pool_proj_dg<uint16_t, 128>(a, s);
  } else {
    if (a.head_dim == 64) return pool_proj_dg<float, 64>(a, s);
    if (a.head_dim == 128) return pool_proj_dg<float, 128>(a, s);
  }
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// gate logits: L = Qg Kg^T * scale on 64x64 lower-triangular tiles
// ---------------------------------------------------------------------------

// Each of the 4 wavefronts computes a 64x64 sub-tile of a 128x128 tile as 2x2
// blocks of 32x32 on bf16 MFMA (v_mfma_f32_32x32x16_bf16), from Qg and Kg held
// as three bf16 parts each (store_split): of the nine part products the six
// down to 2^-18 of the leading one (hi.hi, hi.mid, mid.hi, hi.lo, lo.hi,
// mid.mid) are summed in fp32, which keeps the logits as accurate as fp32
// products (the dropped ones and the split's remainder lie near 2^-26 of it) at 6 bf16 MFMAs (192
// cycles) per 32x32x16 step instead of 8 fp32 MFMAs (512 cycles).  Operand
// lanes: A (rows i of Qg) and B (rows j of Kg) both hold, in lane half hf =
// lane/32 and feature step c, the gate features 16c + 8hf .. +7, so the
// contraction pairs identical features (the parts are stored in exactly this
// lane order, split_index).  Output lane holds column j = lane%32 and rows
// 8*(e/4) + 4*hf + e%4 of a 32x32 block (e = accumulator index).  Blocks
// entirely above the diagonal are computed (a per-MFMA branch broke the
// MFMA stream into small blocks) but not stored.  The next feature step's operands
// load while the current one multiplies (two steps in flight measured no
// faster).
template <int DG>
__global__ __launch_bounds__(256) void gate_logits_kernel(GateLogitsArgs a) {
  const int nb = a.n_blocks;
  // Workgroup -> (batch x head, tile): workgroups are dealt to the 8 XCDs in
  // turn, so with a multiple of 8 (batch, head) pairs, pair p's tiles all go
  // to XCD p % 8, which then holds one head's rows and its KV head's in its
  // L2 at a time; otherwise the pairs follow each other.
  const int T = (nb + 127) / 128;
  const int tiles = T * (T + 1) / 2;
  const int pairs = a.batch * a.heads_q;
  const int wg = blockIdx.x;
  int pair, x;
  if (pairs % 8 == 0) {
    const int k = wg / 8;
    pair = (k / tiles) * 8 + wg % 8;
    x = k % tiles;
  } else {
    pair = wg / tiles;
    x = wg % tiles;
  }
  const int h = pair % a.heads_q;
  const int b = pair / a.heads_q;
  // decode the linear lower-triangular tile index
  int I = (int)((sqrtf(8.0f * x + 1.0f) - 1.0f) * 0.5f);
  while ((I + 1) * (I + 2) / 2 <= x) ++I;
  while (I * (I + 1) / 2 > x) --I;
  const int J = x - I * (I + 1) / 2;
  const int g = h / (a.heads_q / a.heads_kv);

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int wi = wave / 2, wj = wave % 2;
  if (I == J && wj > wi) return;  // sub-tile entirely above the diagonal
  const int i0 = I * 128 + wi * 64;
  const int j0 = J * 128 + wj * 64;
  if (i0 >= nb || j0 >= nb) return;
  const bool diag = I == J && wi == wj;  // block (0, 1) of this sub-tile lies above the diagonal
  const int hf = lane / 32;
  // operand runs (split_index): row group rb, step c, part p at
  // ((rb DG/16 + c) 3 + p) 512 elements; groups past the last hold only rows
  // past nb, whose logits are never stored, so a clamped group serves them
  const int nrb = split_rows(nb) / 32;
  const uint16_t* qhead = a.qs + ((int64_t)b * a.heads_q + h) * split_rows(nb) * 3 * DG + 8 * lane;
  const uint16_t* khead = a.ks + ((int64_t)b * a.heads_kv + g) * split_rows(nb) * 3 * DG + 8 * lane;
  const uint16_t* qrow[2];
  const uint16_t* krow[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    qrow[s] = qhead + (int64_t)min(i0 / 32 + s, nrb - 1) * (DG / 16) * 3 * 512;
    krow[s] = khead + (int64_t)min(j0 / 32 + s, nrb - 1) * (DG / 16) * 3 * 512;
  }

  f32x16 acc[2][2];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[r][c][e] = 0.f;
  // operands of feature step c: part p of row block s
  bf16x8 qn[2][3], kn[2][3];
  auto load = [&](int c, bf16x8 (&qo)[2][3], bf16x8 (&ko)[2][3]) {
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int p = 0; p < 3; ++p) {
        qo[s][p] = *reinterpret_cast<const bf16x8*>(qrow[s] + (3 * c + p) * 512);
        ko[s][p] = *reinterpret_cast<const bf16x8*>(krow[s] + (3 * c + p) * 512);
      }
  };
  load(0, qn, kn);
  // part pairs (Q part, K part) in the order they are summed
  constexpr int PQ[6] = {0, 0, 1, 0, 2, 1};
  constexpr int PK[6] = {0, 1, 0, 2, 0, 1};
#pragma unroll
  for (int c = 0; c < DG / 16; ++c) {
    bf16x8 qa[2][3], kb[2][3];
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int p = 0; p < 3; ++p) {
        qa[s][p] = qn[s][p];
        kb[s][p] = kn[s][p];
      }
    if (c + 1 < DG / 16) load(c + 1, qn, kn);
#pragma unroll
    for (int t = 0; t < 6; ++t)
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int cc = 0; cc < 2; ++cc)  // (diagonal sub-tiles compute their upper block too: no branch here)
          acc[r][cc] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[r][PQ[t]], kb[cc][PK[t]], acc[r][cc], 0, 0, 0);
  }
  float* out = a.logits + ((int64_t)b * a.heads_q + h) * nb * nb;
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      if (diag && c > r) continue;
      const int jcol = j0 + 32 * c + lane % 32;
      if (jcol >= nb) continue;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int irow = i0 + 32 * r + 8 * (e / 4) + 4 * hf + (e % 4);
        if (irow < nb) out[(int64_t)irow * nb + jcol] = acc[r][c][e] * a.scale;
      }
    }
}

hipError_t launch_gate_logits(const GateLogitsArgs& a, hipStream_t s) {
  const int T = (a.n_blocks + 127) / 128;
  const int64_t wgs = (int64_t)T * (T + 1) / 2 * a.heads_q * a.batch;
  if (wgs > INT32_MAX) return hipErrorInvalidValue;
  dim3 grid((unsigned)wgs);
  switch (a.gate_dim) {
    case 32: hipLaunchKernelGGL(gate_logits_kernel<32>, grid, dim3(256), 0, s, a); break;
    case 64: hipLaunchKernelGGL(gate_logits_kernel<64>, grid, dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL(gate_logits_kernel<128>, grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// block selection: one wavefront per query-block row
// ---------------------------------------------------------------------------

// Writes the ascending index list (and optional 0/1 row) of a row whose
// selection bit for block j = 64m + lane is bit m of sel.
template <int MAXM>
__device__ __forceinline__ void emit_row(uint64_t sel, int nb, int64_t row, int32_t* count,
                                         uint16_t* idx, uint8_t* dense) {
  const int lane = threadIdx.x % kWave;
  const uint64_t lt = lanemask_lt();
  int base = 0;
#pragma unroll
  for (int m = 0; m < MAXM; ++m) {
    const int j = 64 * m + lane;
    const bool s = ((sel >> m) & 1) && j < nb;
    const uint64_t bal = __ballot(s);
    if (s) idx[row * nb + base + __popcll(bal & lt)] = (uint16_t)j;
    if (dense && j < nb) dense[row * nb + j] = s ? 1 : 0;
    base += __popcll(bal);
  }
  if (lane == 0) count[row] = base;
}

// A wave-uniform float (equal in every lane) as a scalar.
__device__ __forceinline__ float uniform_f(float x) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}

// A copy of a wave-uniform int that the compiler cannot merge with other uses
// of the same value.  The word loops below each compare it with their
// constant word index: merged across loops, those per-word conditions would
// stay live as 64-bit lane masks for the whole selection and spill.
__device__ __forceinline__ int opaque_sgpr(int x) {
  asm volatile("" : "+s"(x));
  return x;
}

// Block selection of one query-block row i of mask head h from its values v
// (v[m] of a lane: block j = 64 m + lane; -inf for j > i), written straight
// to the row's index list (and optional 0/1 row): the forced blocks, plus
// either the strict threshold on the row softmax (Eq. 4) or the TopK of the
// remaining causal blocks (Eq. 3, ties to the smaller block index).  `hist`:
// this wavefront's 256-word LDS histogram.  One wavefront.
//
// TopK finds the cut without sorting.  A first pass counts the candidates in
// 256 equal-width buckets of their value range (the bucket index never
// decreases with the value, so the bucket holding the take-th largest value
// is found from the counts); the candidates of that bucket (usually a few) are
// gathered one per lane and the cut T is read off their ranks.  A bucket of
// more than 64 candidates (heavy ties) is resolved by bisection over the keys.
// Every block then takes one test: above the bucket, or in it and at or above
// T, with ties at T going to the smaller indices.  State is kept per block in
// registers (bucket indices, no bit masks), so the passes are straight-line
// code.
template <int MAXM>
__device__ __forceinline__ void select_emit(const SelectArgs& a, const float (&v)[MAXM], int i, int h,
                                            int64_t row, uint32_t* hist) {
  const int lane = threadIdx.x % kWave;
  const int nb = a.n_blocks;
  const int M = i / 64 + 1;  // words holding the causal blocks j <= i (wave-uniform)
  const uint64_t lt = lanemask_lt();
  const int f0 = a.keep_first ? 0 : -1;  // forced blocks (-1: none)
  const int f1 = a.keep_diag ? i : -1;
  // Words 1 .. M-2 are full: every block in them is a causal candidate (the
  // forced blocks lie in words 0 and M-1, blocks past the diagonal only in
  // M-1), so they take no per-block state tests; the two edge words do.
  auto edge = [&](int m) { return m == 0 || m == opaque_sgpr(M) - 1; };
  // b[m]: -2 forced, -1 past the diagonal, otherwise a candidate (0; for TopK
  // its value bucket below).  All later tests read b, so no per-block
  // condition has to stay live across the passes.
  int b[MAXM];
#pragma unroll
  for (int m = 0; m < MAXM; ++m) {
    b[m] = -1;
    if (m < opaque_sgpr(M)) {
      b[m] = 0;
      if (edge(m)) {
        const int j = 64 * m + lane;
        b[m] = j > i ? -1 : (((j == f0) | (j == f1)) ? -2 : 0);
      }
    }
  }

  // selection rule, filled in below: a causal block is taken if forced, or
  // (threshold) v - lse > lthr, or (TopK) its bucket > bstar, or == bstar and
  // (all_in || key > T || (key == T && tie rank < need))
  const bool thr_mode = a.mode == 2;
  float lse = 0.f, lthr = -INFINITY;
  int bstar = -1;
  bool all_in = true;
  uint32_t T = 0u;
  int need = -1;  // < 0: no tie at T to break

  if (thr_mode) {  // threshold on the softmax probability (Eq. 4, strict)
    float mx = -INFINITY;
#pragma unroll
    for (int m = 0; m < MAXM; ++m)
      if (m < opaque_sgpr(M)) mx = fmaxf(mx, v[m]);
    mx = uniform_f(wave_max(mx));
    float sum = 0.f;
#pragma unroll
    for (int m = 0; m < MAXM; ++m)
      if (m < opaque_sgpr(M)) sum += __expf(v[m] - mx);  // exp(-inf) = 0 past the diagonal
    sum = uniform_f(wave_sum(sum));
    lse = mx + __logf(sum);
    const float t = a.head_thresholds ? a.head_thresholds[h] : a.threshold;
    lthr = t <= 0.f ? -INFINITY : __logf(t);
  } else {  // TopK (Eq. 3) over the non-forced causal blocks
    const int nf = (a.keep_first ? 1 : 0) + ((a.keep_diag && !(a.keep_first && i == 0)) ? 1 : 0);
    int kk = (a.mode == 0) ? (int)ceil(a.topk_ratio * (double)(i + 1)) : a.topk_k;
    kk = min(i + 1, max(nf, kk));
    const int take = kk - nf;
    const int ncand = i + 1 - nf;
    if (take >= ncand) {
      bstar = -1;  // every candidate
    } else if (take <= 0) {
      bstar = 256;  // none
    } else {
      // value range of the causal blocks (the forced ones included: a range
      // that covers every candidate keeps the bucket index monotone); v is -inf
      // past the diagonal, which only word M-1 holds
      float cmx = -INFINITY, cmn = INFINITY;
#pragma unroll
      for (int m = 0; m < MAXM; ++m)
        if (m < opaque_sgpr(M)) {
          cmx = fmaxf(cmx, v[m]);
          if (m == opaque_sgpr(M) - 1) cmn = fminf(cmn, 64 * m + lane <= i ? v[m] : INFINITY);
          else cmn = fminf(cmn, v[m]);
        }
      cmx = uniform_f(wave_max(cmx));
      cmn = uniform_f(-wave_max(-cmn));
      const float span = cmx - cmn;
      const float scale = (span > 0.f && span < INFINITY) ? 256.f / span : 0.f;
      // bucket pass
      *reinterpret_cast<u32x4*>(hist + 4 * lane) = u32x4{0u, 0u, 0u, 0u};
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int m = 0; m < MAXM; ++m) {
        if (m < opaque_sgpr(M)) {
          const int bk = min(255, max(0, (int)((v[m] - cmn) * scale)));
          if (edge(m)) {
            b[m] = b[m] == 0 ? bk : b[m];
            if (b[m] >= 0) atomicAdd(hist + b[m], 1u);
          } else {
            b[m] = bk;
            atomicAdd(hist + bk, 1u);
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
      const u32x4 cnt4 = *reinterpret_cast<const u32x4*>(hist + 4 * lane);  // bins 4 lane .. +3
      const int local = (int)(cnt4[0] + cnt4[1] + cnt4[2] + cnt4[3]);
      int incl = local;  // candidates in the bins of this lane and every higher lane
#pragma unroll
      for (int off = 1; off < kWave; off <<= 1) {
        const int t = __shfl_down(incl, off);
        if (lane + off < kWave) incl += t;
      }
      // the target bin: the highest b with #{bucket >= b} >= take
      int run = incl - local, found = -1, ab = 0, cc = 0;
#pragma unroll
      for (int e = 3; e >= 0; --e) {
        if (found < 0 && run < take && run + (int)cnt4[e] >= take) {
          found = e;
          ab = run;
          cc = (int)cnt4[e];
        }
        run += (int)cnt4[e];
      }
      const uint64_t hit = __ballot(found >= 0);  // exactly one lane: bins are monotone
      const int src = __builtin_ctzll(hit);
      bstar = 4 * src + __builtin_amdgcn_readlane(found, src);
      const int above = __builtin_amdgcn_readlane(ab, src);
      const int cb = __builtin_amdgcn_readlane(cc, src);
      const int want = take - above;  // 1 <= want <= cb
      if (want < cb) {
        all_in = false;
        int gt = 0, ge = 0;  // bucket candidates with key > T, >= T
        if (cb <= kWave) {
          // gather the bucket's keys one per lane (words without one are
          // skipped on their ballot), then T = the key of rank want
          __builtin_amdgcn_wave_barrier();
          int n = 0;
#pragma unroll
          for (int m = 0; m < MAXM; ++m) {
            if (m < opaque_sgpr(M)) {
              const bool in_b = b[m] == bstar;
              const uint64_t bal = __ballot(in_b);
              if (bal != 0) {
                if (in_b) hist[n + __popcll(bal & lt)] = ordered_key(v[m]);
                n += __popcll(bal);
              }
            }
          }
          __builtin_amdgcn_wave_barrier();
          const uint32_t key = lane < cb ? hist[lane] : 0u;
          int g = 0, eqc = 0;
          for (int t = 0; t < cb; ++t) {
            const uint32_t kt = hist[t];
            g += kt > key ? 1 : 0;
            eqc += kt == key ? 1 : 0;
          }
          const uint64_t hit2 = __ballot(lane < cb && g < want && g + eqc >= want);
          const int s2 = __builtin_ctzll(hit2);
          T = (uint32_t)__builtin_amdgcn_readlane((int)key, s2);
          gt = __builtin_amdgcn_readlane(g, s2);
          ge = gt + __builtin_amdgcn_readlane(eqc, s2);
        } else {
          // heavy ties: bisection over the keys of the bucket,
          // count(key >= lo) >= want > count(key >= hi + 1)
          auto count_ge = [&](uint32_t x) -> int {
            int c = 0;
#pragma unroll
            for (int m = 0; m < MAXM; ++m)
              if (m < opaque_sgpr(M)) c += __popcll(__ballot(b[m] == bstar && ordered_key(v[m]) >= x));
            return c;
          };
          uint32_t klo = 0xFFFFFFFFu, khi = 0u;
#pragma unroll
          for (int m = 0; m < MAXM; ++m)
            if (m < opaque_sgpr(M)) {
              const uint32_t k = ordered_key(v[m]);
              klo = min(klo, b[m] == bstar ? k : 0xFFFFFFFFu);
              khi = max(khi, b[m] == bstar ? k : 0u);
            }
          klo = (uint32_t)__builtin_amdgcn_readfirstlane((int)wave_min_u32(klo));
          khi = (uint32_t)__builtin_amdgcn_readfirstlane((int)wave_max_u32(khi));
          uint32_t lo = klo, hi = khi;
          while (lo < hi) {
            const uint32_t mid = lo + ((hi - lo) >> 1) + 1;  // in (lo, hi]
            if (count_ge(mid) >= want) lo = mid;
            else hi = mid - 1;
          }
          T = lo;
          ge = count_ge(T);
          gt = T < khi ? count_ge(T + 1) : 0;
        }
        need = (ge == want) ? -1 : want - gt;  // ties at T straddle the cut: take the first `need`
      }
    }
  }

  // emit: ascending index list by ballot compaction.  The rule reduces to
  // compares against scalars: taken if forced, or bucket > bstar, or bucket ==
  // bstar and (the whole bucket is in, or key >= kcut, or tied at T with rank
  // < need).  The key tests run only in words that hold the cut bucket.
  const bool in_rule = !thr_mode && bstar >= 0 && bstar < 256;  // bucket bstar is split by keys
  const bool by_key = in_rule && !all_in;
  const bool tie = by_key && need >= 0;
  const uint32_t kcut = tie ? T + 1u : T;
  const bool key_in = !(tie && T == 0xFFFFFFFFu);  // (no key lies above the largest)
  const int bmin = (in_rule && !by_key) ? bstar : bstar + 1;  // buckets taken whole
  uint16_t* const idx_row = a.idx + row * nb;
  uint8_t* const dense_row = a.dense ? a.dense + row * nb : nullptr;
  int base = 0, before = 0;
#pragma unroll
  for (int m = 0; m < MAXM; ++m) {
    const int j = 64 * m + lane;
    if (m < opaque_sgpr(M)) {
      const int bm = b[m];
      bool s;
      if (thr_mode) {
        s = (bm == -2) | ((bm == 0) & (v[m] - lse > lthr));
      } else {
        s = (bm == -2) | (bm >= bmin);
        if (by_key) {
          const bool in_b = bm == bstar;
          if (__ballot(in_b) != 0) {
            const uint32_t key = ordered_key(v[m]);
            s = s | (in_b & (key >= kcut) & key_in);
            if (tie) {  // the smallest-index candidates tied at T
              const bool eq = in_b & (key == T);
              const uint64_t bal_eq = __ballot(eq);
              s = s | (eq & (before + (int)__popcll(bal_eq & lt) < need));
              before += __popcll(bal_eq);
            }
          }
        }
      }
      const uint64_t bal = __ballot(s);
      if (s) idx_row[base + (int)__popcll(bal & lt)] = (uint16_t)j;
      base += __popcll(bal);
      if (dense_row && j < nb) dense_row[j] = s ? 1 : 0;
    } else if (dense_row && j < nb) {
      dense_row[j] = 0;
    }
  }
  if (lane == 0) a.count[row] = base;
}

// GROUP: rows of a mask shared by a KV group (a separate instantiation, so the
// per-head kernel keeps its register budget and occupancy).
template <int MAXM, bool GROUP>
__device__ __forceinline__ void select_rows(const SelectArgs& a) {
  __shared__ __attribute__((aligned(16))) uint32_t s_hist[4][256];  // per-wavefront digit histogram
  const int lane = threadIdx.x % kWave;
  // the wavefront index is uniform: readfirstlane makes row, i and the word
  // count M scalars, so the per-word guards below are scalar branches
  // grid: (query-block rows / 4, mask heads, batch), heaviest rows first
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int nb = a.n_blocks;
  const int G = GROUP ? a.group : 0;  // > 0: rows of a mask shared by the G query heads of a KV group
  const int mheads = G > 0 ? a.heads_q / G : a.heads_q;  // heads of the mask
  const int i = nb - 1 - ((int)blockIdx.x * 4 + wv);
  if (i < 0) return;
  const int h = blockIdx.y;  // query head, or KV head when shared
  const int64_t row = ((int64_t)blockIdx.z * mheads + h) * nb + i;
  const int M = i / 64 + 1;  // words holding the causal blocks j <= i (wave-uniform)

  // v[m]: block j = 64 m + lane, -inf past the diagonal
  float v[MAXM];
  if constexpr (!GROUP) {
    const float* L = a.logits + row * nb;
#pragma unroll
    for (int m = 0; m < MAXM; ++m) {
      v[m] = -INFINITY;
      if (m < M && 64 * m + lane <= i) v[m] = L[64 * m + lane];
    }
  } else {
    // the group's score of block j: the mean over its query heads of their gate
    // probabilities, held as its logarithm so that TopK (by value) and the
    // threshold test (against the log of the row sum, 1) below apply unchanged
    float sc[MAXM];
#pragma unroll
    for (int m = 0; m < MAXM; ++m) sc[m] = 0.f;
    const int64_t b = blockIdx.z;
    for (int hh = 0; hh < G; ++hh) {
      const float* L = a.logits + (((b * a.heads_q) + (int64_t)h * G + hh) * nb + i) * nb;
#pragma unroll
      for (int m = 0; m < MAXM; ++m) v[m] = (m < M && 64 * m + lane <= i) ? L[64 * m + lane] : -INFINITY;
      float mx = -INFINITY;
#pragma unroll
      for (int m = 0; m < MAXM; ++m)
        if (m < M) mx = fmaxf(mx, v[m]);
      mx = wave_max(mx);
      float s = 0.f;
#pragma unroll
      for (int m = 0; m < MAXM; ++m)
        if (m < M) s += __expf(v[m] - mx);
      const float lse = mx + __logf(wave_sum(s));
#pragma unroll
      for (int m = 0; m < MAXM; ++m)
        if (m < M) sc[m] += __expf(v[m] - lse);
    }
    const float inv_g = 1.0f / (float)G;
#pragma unroll
    for (int m = 0; m < MAXM; ++m) v[m] = (m < M && 64 * m + lane <= i) ? __logf(sc[m] * inv_g) : -INFINITY;
  }
  select_emit<MAXM>(a, v, i, h, row, s_hist[wv]);
}

template <int MAXM, bool GROUP>
__global__ __launch_bounds__(256) void select_kernel(SelectArgs a) {
  select_rows<MAXM, GROUP>(a);
}

// Rows of 1025 to 2048 blocks: the selection is latency bound (one wavefront
// walks a row through dependent passes), so occupancy pays: held to 96 VGPRs
// for a fifth wavefront per SIMD (the compiler's choice is 103, four), at a
// spill of 11 words per lane.  Measured at 131072 tokens: selection 0.215-0.221
// -> 0.190-0.193 ms; six wavefronts (80 VGPRs, 40 spilled) 0.189-0.190 ms.
// (The shorter-row instantiations keep five wavefronts per SIMD without a hint.)
template <bool GROUP>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(5))) void select_kernel_m32(SelectArgs a) {
  select_rows<32, GROUP>(a);
}

// ---------------------------------------------------------------------------
// fused gate score + select: the logits never leave LDS
// ---------------------------------------------------------------------------
//
// One workgroup of 16 wavefronts per (batch, head, 16 consecutive query-block
// rows).  Phase 1 computes the rows' block-causal logits (Eq. 1) on fp32 MFMA
// (v_mfma_f32_16x16x4_f32) into LDS: wavefront w takes the 16-column tiles
// w, w + 16, ...; lane l supplies row / column l % 16 and the contiguous run
// of Dg / 4 gate features starting at (l / 16) Dg / 4, so A and B pair
// identical features.  Phase 2: wavefront w selects row i0 + w from LDS with
// the select of select_kernel.  Kg of a KV head (nb Dg fp32, 1 MiB at 2048
// blocks) stays in L2 for the head's workgroups.  LDS: 16 rows of 64 MAXM + 4
// floats (the pad puts rows 4 apart on different banks): 128 KiB at 2048
// blocks, the largest row length served here, 64 KiB at 1024 (two workgroups
// per CU).  Once every wavefront holds its row in registers the same LDS holds
// the wavefronts' 1 KiB selection histograms.
constexpr int kFusedRows = 16;
constexpr int kFusedMaxBlocks = 2048;

template <int MAXM, int DG>
__global__ __launch_bounds__(1024) void gate_fused_kernel(GateFusedArgs a) {
  constexpr int LDL = 64 * MAXM + 4;
  constexpr int WORDS = kFusedRows * LDL > kFusedRows * 256 ? kFusedRows * LDL : kFusedRows * 256;
  __shared__ __attribute__((aligned(16))) float sL[WORDS];
  const int nb = a.sel.n_blocks;
  const int chunks = (nb + kFusedRows - 1) / kFusedRows;
  // 1-D grid, heaviest rows first over the whole launch (head by head, the
  // last heads' heavy rows would run alone at the end: measured 0.93 -> 0.86 ms
  // at 131072 tokens, 0.178 -> 0.153 ms at 32768)
  const int nbh = a.sel.batch * a.sel.heads_q;
  const int chunk = chunks - 1 - (int)blockIdx.x / nbh;
  const int h = (int)blockIdx.x % nbh % a.sel.heads_q, b = (int)blockIdx.x % nbh / a.sel.heads_q;
  const int g = h / (a.sel.heads_q / a.heads_kv);
  const int i0 = kFusedRows * chunk;
  const int ncols = min(nb, i0 + kFusedRows);  // block-causal: columns j <= i0 + 15
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
  const int r16 = lane % 16, kq = lane / 16;
  constexpr int KS = DG / 4;  // MFMA steps: this lane's features kq KS .. kq KS + KS - 1

  // phase 1: logits of rows i0 .. i0 + 15 (rows past nb repeat the last one)
  float qa[KS];
  {
    const float* qrow = a.qg + (((int64_t)b * a.sel.heads_q + h) * nb + min(i0 + r16, nb - 1)) * DG + kq * KS;
#pragma unroll
    for (int u = 0; u < KS / 4; ++u) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(qrow + 4 * u);
#pragma unroll
      for (int e = 0; e < 4; ++e) qa[4 * u + e] = x[e];
    }
  }
  const float* kbase = a.kg + ((int64_t)b * a.heads_kv + g) * nb * DG + kq * KS;
  // the next column tile's operands load while the current one multiplies
  auto load_k = [&](int ct, f32x4 (&kb)[KS / 4]) {
    const float* krow = kbase + (int64_t)min(16 * ct + r16, nb - 1) * DG;
#pragma unroll
    for (int u = 0; u < KS / 4; ++u) kb[u] = *reinterpret_cast<const f32x4*>(krow + 4 * u);
  };
  f32x4 kn[KS / 4];
  if (wave * 16 < ncols) load_k(wave, kn);
  for (int ct = wave; ct * 16 < ncols; ct += kFusedRows) {
    f32x4 kb[KS / 4];
#pragma unroll
    for (int u = 0; u < KS / 4; ++u) kb[u] = kn[u];
    if ((ct + kFusedRows) * 16 < ncols) load_k(ct + kFusedRows, kn);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < KS; ++st) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[st], kb[st / 4][st % 4], acc, 0, 0, 0);
    // accumulator e of lane l: row 4 (l / 16) + e, column 16 ct + l % 16
#pragma unroll
    for (int e = 0; e < 4; ++e) sL[(4 * kq + e) * LDL + 16 * ct + r16] = acc[e] * a.scale;
  }
  __syncthreads();

  // phase 2: wavefront w selects row i0 + w (rows past nb take no part)
  const int i = i0 + wave;
  const int M = i / 64 + 1;
  const float* L = sL + wave * LDL;
  float v[MAXM];
#pragma unroll
  for (int m = 0; m < MAXM; ++m) {
    v[m] = -INFINITY;
    if (m < M && i < nb && 64 * m + lane <= i) v[m] = L[64 * m + lane];
  }
  __syncthreads();  // every row is in registers: the LDS now holds the histograms
  if (i >= nb) return;
  const int64_t row = ((int64_t)b * a.sel.heads_q + h) * nb + i;
  select_emit<MAXM>(a.sel, v, i, h, row, reinterpret_cast<uint32_t*>(sL) + 256 * wave);
}

// Static scratch of seer_gate_noalloc: the projected rows Qg and Kg (the fused
// kernel needs no logits buffer).  Every call on a device shares that device's
// copy.  In host code `scratch` names a host-side stand-in, never the device
// memory: the device address comes from hipGetSymbolAddress, once per device
// with that device current.
static __device__ __align__(256) char scratch[kGateScratchBytes];

void* gate_scratch() {
  constexpr int kMaxDevices = 64;
  static std::once_flag once[kMaxDevices];
  static void* ptr[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::call_once(once[dev], [dev]() {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess) ptr[dev] = p;
  });
  return ptr[dev];
}

bool gate_fused_supported(int n_blocks, int gate_dim) {
  return n_blocks >= 1 && n_blocks <= kFusedMaxBlocks && (gate_dim == 32 || gate_dim == 64 || gate_dim == 128);
}

template <int MAXM>
static hipError_t gate_fused_dg(const GateFusedArgs& a, hipStream_t s) {
  const int chunks = (a.sel.n_blocks + kFusedRows - 1) / kFusedRows;
  const int64_t wgs = (int64_t)chunks * a.sel.heads_q * a.sel.batch;
  if (wgs > INT32_MAX) return hipErrorInvalidValue;
  const dim3 grid((unsigned)wgs);
  switch (a.gate_dim) {
    case 32: hipLaunchKernelGGL((gate_fused_kernel<MAXM, 32>), grid, dim3(1024), 0, s, a); break;
    case 64: hipLaunchKernelGGL((gate_fused_kernel<MAXM, 64>), grid, dim3(1024), 0, s, a); break;
    case 128: hipLaunchKernelGGL((gate_fused_kernel<MAXM, 128>), grid, dim3(1024), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gate_fused(const GateFusedArgs& a, hipStream_t s) {
  if (!gate_fused_supported(a.sel.n_blocks, a.gate_dim) || a.sel.group > 0) return hipErrorInvalidValue;
  const int m = (a.sel.n_blocks + 63) / 64;
  if (m <= 1) return gate_fused_dg<1>(a, s);
  if (m <= 2) return gate_fused_dg<2>(a, s);
  if (m <= 4) return gate_fused_dg<4>(a, s);
  if (m <= 8) return gate_fused_dg<8>(a, s);
  if (m <= 16) return gate_fused_dg<16>(a, s);
  return gate_fused_dg<32>(a, s);
}

template <int MAXM>
static hipError_t select_launch(const SelectArgs& a, hipStream_t s) {
  const dim3 grid((unsigned)((a.n_blocks + 3) / 4), (unsigned)(a.group > 0 ? a.heads_q / a.group : a.heads_q),
                  (unsigned)a.batch);
  if constexpr (MAXM == 32) {
    if (a.group > 0) hipLaunchKernelGGL((select_kernel_m32<true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((select_kernel_m32<false>), grid, dim3(256), 0, s, a);
  } else {
    if (a.group > 0) hipLaunchKernelGGL((select_kernel<MAXM, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((select_kernel<MAXM, false>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  const int m = (a.n_blocks + 63) / 64;
  if (m <= 1) return select_launch<1>(a, s);
  if (m <= 2) return select_launch<2>(a, s);
  if (m <= 4) return select_launch<4>(a, s);
  if (m <= 8) return select_launch<8>(a, s);
  if (m <= 16) return select_launch<16>(a, s);
  if (m <= 32) return select_launch<32>(a, s);
  if (m <= 64) return select_launch<64>(a, s);
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// dense 0/1 mask -> ascending index lists
// ---------------------------------------------------------------------------

template <int MAXM>
__global__ __launch_bounds__(256) void mask_from_dense_kernel(MaskFromDenseArgs a) {
  const int lane = threadIdx.x % kWave;
  const int64_t row = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (row >= a.rows) return;
  uint64_t sel = 0;
#pragma unroll
  for (int m = 0; m < MAXM; ++m) {
    const int j = 64 * m + lane;
    sel |= (uint64_t)(j < a.n_blocks && a.dense[row * a.n_blocks + j] != 0) << m;
  }
  emit_row<MAXM>(sel, a.n_blocks, row, a.count, a.idx, nullptr);
}

template <int MAXM>
static hipError_t mfd_launch(const MaskFromDenseArgs& a, hipStream_t s) {
  dim3 grid((unsigned)((a.rows + 3) / 4));
  hipLaunchKernelGGL(mask_from_dense_kernel<MAXM>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mask_from_dense(const MaskFromDenseArgs& a, hipStream_t s) {
  const int m = (a.n_blocks + 63) / 64;
  if (m <= 1) return mfd_launch<1>(a, s);
  if (m <= 4) return mfd_launch<4>(a, s);
  if (m <= 16) return mfd_launch<16>(a, s);
  if (m <= 64) return mfd_launch<64>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace seer
