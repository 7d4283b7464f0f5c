// distill_kernels.hip -- the gate's distillation step for gfx950 (SeerAttention
// section 3.2, Eq. 2): KL(ground truth || gate score) and its gradients with
// respect to the gate weights.
//
//   kl_rows_kernel      one wavefront per query-block row (kl_rows_staged_kernel:
//                       the row held in registers): the row's softmax of
//                       the gate logits, the ground-truth row renormalised to a
//                       distribution T, the row's KL(T || P) and the logit
//                       gradient (P sum(T) - T) / rows written over the logits.
//   loss_part_kernel,   the mean of the row losses in a fixed order (two
//   loss_mean_kernel    levels of workgroup sums in double: run-to-run
//                       identical).
//   gemm_f32_kernel     fp32 strided batched products for the backward pass
//                       (dQg = dL Kg, dKg = dL^T Qg, dW = pooled^T dG), 64x64
//                       LDS tiles of the operands split in three bf16 parts on
//                       bf16 MFMA (fp32-accurate), triangular skipping of the
//                       causal zeros, K split over several workgroups when
//                       the output tiles are few.
//   gemm_reduce_kernel  sums the split parts in a fixed order.
//   rope_inverse_kernel rotates gradient rows back through the block-level
//                       RoPE (the transpose of the forward rotation).
#include <algorithm>
#include <cstdlib>

#include "device_common.h"
#include "launch.h"

namespace seer {

namespace {

constexpr int kRowsPerBlock = 4;  // wavefronts (rows) per workgroup

// V consecutive entries per lane (V = 4: 16-byte loads; needs nb % 4 == 0 and
// 16-byte aligned rows).  Two passes over the row: an online max / sum of the
// exponentials with the target's sum, then the loss and the gradient.
template <int V>
__global__ __launch_bounds__(256) void kl_rows_kernel(KlArgs a) {
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + wave;
  if (r >= a.rows) return;
  const int nb = a.n_blocks;
  const int i = (int)(r % nb);
  const int M = i + 1;                                  // causal entries j <= i
  const int Mz = min(nb, (i / kKlTile + 1) * kKlTile);  // entries the gradient covers
  float* Lr = a.logits + r * nb;
  const float* gr = a.gt + r * nb;
  auto load = [&](const float* p, int j0, float (&x)[V]) {
    if constexpr (V == 4) {
      const f32x4 u = *reinterpret_cast<const f32x4*>(p + j0);
#pragma unroll
      for (int e = 0; e < 4; ++e) x[e] = u[e];
    } else {
      x[0] = p[j0];
    }
  };

  float mx = -INFINITY, es = 0.f, gs = 0.f;
  for (int j0 = V * lane; j0 < M; j0 += V * kWave) {
    float l[V], g[V];
    load(Lr, j0, l);
    load(gr, j0, g);
#pragma unroll
    for (int e = 0; e < V; ++e)
      if (j0 + e < M) {
        if (l[e] > mx) {
          es = es * __expf(mx - l[e]) + 1.f;
          mx = l[e];
        } else {
          es += __expf(l[e] - mx);
        }
        gs += g[e];
      }
  }
  const float mw = wave_max(mx);
  es = wave_sum(mx == -INFINITY ? 0.f : es * __expf(mx - mw));
  gs = wave_sum(gs);
  const float lse = mw + __logf(es);
  const float inv_gs = gs > 0.f ? 1.0f / gs : 0.f;
  const float tsum = gs > 0.f ? 1.0f : 0.f;  // sum of T
  const float log_gs = gs > 0.f ? __logf(gs) : 0.f;
  float loss = 0.f;
  for (int j0 = V * lane; j0 < Mz; j0 += V * kWave) {
    float l[V], g[V], d[V];
    if (j0 < M) {
      load(Lr, j0, l);
      load(gr, j0, g);
    }
#pragma unroll
    for (int e = 0; e < V; ++e) {
      d[e] = 0.f;
      if (j0 + e < M) {
        const float logp = l[e] - lse;
        const float t = g[e] * inv_gs;
        if (t > 0.f) loss += t * ((__logf(g[e]) - log_gs) - logp);
        d[e] = (__expf(logp) * tsum - t) * a.inv_rows;
      }
    }
    if constexpr (V == 4) {
      *reinterpret_cast<f32x4*>(Lr + j0) = f32x4{d[0], d[1], d[2], d[3]};
    } else {
      Lr[j0] = d[0];
    }
  }
  double dl = (double)loss;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) dl += __shfl_xor(dl, off);
  if (lane == 0) a.row_loss[r] = dl;
}

// The same row computation with the row held in registers (16-byte chunks u =
// 0 .. NW-1 of a lane: entries 4 (lane + 64 u) .. +3), every load issued before
// any is used: the streaming loop above waits for each chunk in turn (its
// online maximum depends on the previous one).  Needs nb % 4 == 0, 16-byte
// aligned rows and nb <= 256 NW.
template <int NW>
__global__ __launch_bounds__(256) void kl_rows_staged_kernel(KlArgs a) {
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + wave;
  if (r >= a.rows) return;
  const int nb = a.n_blocks;
  const int i = (int)(r % nb);
  const int M = i + 1;                                  // causal entries j <= i
  const int Mz = min(nb, (i / kKlTile + 1) * kKlTile);  // entries the gradient covers
  float* Lr = a.logits + r * nb;
  const float* gr = a.gt + r * nb;
  // entries past the diagonal (and chunks past the row) read as logit -inf and
  // target 0, which takes them out of every sum below
  f32x4 l[NW], g[NW];
#pragma unroll
  for (int u = 0; u < NW; ++u) {
    const int j0 = 4 * (lane + 64 * u);
    f32x4 lu = {-INFINITY, -INFINITY, -INFINITY, -INFINITY}, gu = {0.f, 0.f, 0.f, 0.f};
    if (j0 < M) {
      lu = *reinterpret_cast<const f32x4*>(Lr + j0);
      gu = *reinterpret_cast<const f32x4*>(gr + j0);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool ok = j0 + e < M;
      l[u][e] = ok ? lu[e] : -INFINITY;
      g[u][e] = ok ? gu[e] : 0.f;
    }
  }
  float mx = -INFINITY, gs = 0.f;
#pragma unroll
  for (int u = 0; u < NW; ++u)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      mx = fmaxf(mx, l[u][e]);
      gs += g[u][e];
    }
  const float mw = wave_max(mx);
  float es = 0.f;
#pragma unroll
  for (int u = 0; u < NW; ++u)
#pragma unroll
    for (int e = 0; e < 4; ++e) es += __expf(l[u][e] - mw);  // exp(-inf) = 0
  es = wave_sum(es);
  gs = wave_sum(gs);
  const float lse = mw + __logf(es);
  const float inv_gs = gs > 0.f ? 1.0f / gs : 0.f;
  const float tsum = gs > 0.f ? 1.0f : 0.f;  // sum of T
  const float log_gs = gs > 0.f ? __logf(gs) : 0.f;
  float loss = 0.f;
#pragma unroll
  for (int u = 0; u < NW; ++u) {
    const int j0 = 4 * (lane + 64 * u);
    f32x4 d;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float logp = l[u][e] - lse;
      const float t = g[u][e] * inv_gs;
      if (t > 0.f) loss += t * ((__logf(g[u][e]) - log_gs) - logp);
      d[e] = (__expf(logp) * tsum - t) * a.inv_rows;  // 0 past the diagonal
    }
    if (j0 < Mz) *reinterpret_cast<f32x4*>(Lr + j0) = d;
  }
  double dl = (double)loss;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) dl += __shfl_xor(dl, off);
  if (lane == 0) a.row_loss[r] = dl;
}

// The mean of the row losses in a fixed order (double accumulation: identical
// run to run): kLossParts workgroups sum contiguous ranges of rows, then one
// workgroup sums their results.
__device__ __forceinline__ double block_sum_256(double s, double* part) {
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  return part[0];
}

__global__ __launch_bounds__(256) void loss_part_kernel(const double* __restrict__ row_loss, int64_t rows,
                                                         double* __restrict__ parts) {
  __shared__ double part[256];
  const int64_t lo = rows * blockIdx.x / kLossParts, hi = rows * (blockIdx.x + 1) / kLossParts;
  double s = 0.0;
  for (int64_t r = lo + threadIdx.x; r < hi; r += 256) s += row_loss[r];
  s = block_sum_256(s, part);
  if (threadIdx.x == 0) parts[blockIdx.x] = s;
}

__global__ __launch_bounds__(256) void loss_mean_kernel(const double* __restrict__ parts, int64_t rows,
                                                         float* __restrict__ loss) {
  __shared__ double part[256];
  const double s = block_sum_256((int)threadIdx.x < kLossParts ? parts[threadIdx.x] : 0.0, part);
  if (threadIdx.x == 0) loss[0] = (float)(s / (double)rows);
}

// 64 x 64 NB output tile per 256-thread workgroup (NB 32x32 blocks per
// wavefront, sharing its A operand), K in chunks of 32 staged through two LDS buffers: the next chunk's global loads
// are in flight in registers while the current chunk's MFMAs run, one barrier
// per chunk.  Each fp32 operand value is written to LDS as three bf16 parts
// (hi = RNE(x), mid = RNE(x - hi), lo = RNE(x - hi - mid); both differences
// are exact), and the products of the parts down to 2^-18 of the leading one
// (hi.hi, hi.mid, mid.hi, hi.lo, lo.hi, mid.mid) are summed in fp32 by
// v_mfma_f32_32x32x16_bf16: fp32-accurate products at 6 MFMAs of 32 cycles
// per 32x32x16 step instead of 8 fp32 MFMAs (v_mfma_f32_32x32x2_f32) of 64.
// The LDS tiles are [part][row][k] bf16 with k contiguous in rows of 64 bytes,
// their four 16-byte chunks XOR-swizzled by (row / 4) % 4 so that 16 lanes
// reading 16 rows hit 16 distinct bank groups (48 KiB for the two buffers at
// NB = 1: three workgroups per CU; 72 KiB at NB = 2: two), and a lane reads the 8 k values of one MFMA
// operand (k = 16 s + 8 hf .. +7 of its row or column at step s) with one
// 16-byte read per part.  Operand tiles are read from global memory along
// whichever index has unit stride, so that loads coalesce for every layout
// used here.  A workgroup computes part s of its tile's (k1, k2) chunks; with
// splits > 1 the part's product goes to g.part.
constexpr int kT = 64;
constexpr int kKc = 32;
constexpr int kKb = kKc;                // LDS row stride (bf16 elements)
constexpr int kLoads = kT * kKc / 256;  // elements of each operand per thread and chunk
static_assert(kT == kKlTile, "the logit gradient is written up to the end of each row's GEMM tile");
static_assert(kT == 64 && kKc == 32 && kLoads == 8, "the element mapping of fetch and stash");

// Element offset within an LDS row of k (a multiple of 8: one 16-byte chunk).
__device__ __forceinline__ int swz(int row, int k) { return (((k >> 3) ^ ((row >> 2) & 3)) << 3) | (k & 7); }

// The three bf16 parts of x.
__device__ __forceinline__ void split3(float x, __bf16& hi, __bf16& mid, __bf16& lo) {
  hi = (__bf16)x;
  const float r = x - (float)hi;
  mid = (__bf16)r;
  lo = (__bf16)(r - (float)mid);
}

// Tiles are dispatched heaviest first over the whole launch (a 1-D grid):
// the row-tile index outermost, in the order of decreasing work for the
// triangular products (tri 1: rows near the end contract the longest k range;
// tri 2: rows near the start), then the batch index and split part, then the
// column tile.  Launched batch by batch instead, each batch's heavy tiles
// would come last and the final batches' would run alone at the end.
template <int NB>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs g, int splits) {
  constexpr int TN = kT * NB;  // output tile columns
  __shared__ __attribute__((aligned(16))) __bf16 sA[2][3][kT][kKb];
  __shared__ __attribute__((aligned(16))) __bf16 sB[2][3][TN][kKb];
  const int t = threadIdx.x;
  const int ntn = (g.N + TN - 1) / TN, ntm = (g.M + kT - 1) / kT, nzs = g.Z * splits;
  const int lin = blockIdx.x;
  const int tn = lin % ntn;
  const int zs = (lin / ntn) % nzs;
  const int tq = lin / ntn / nzs;  // position in the row-tile order
  const int tm = g.tri == 1 ? ntm - 1 - tq : tq;
  const int m0 = tm * kT, n0 = tn * TN;
  const int z = zs / splits, sp = zs % splits;
  const float* A = g.A + (int64_t)z * g.saz;
  const float* B = g.B + (int64_t)(z / g.bdiv) * g.sbz;
  const int wave = t / kWave, lane = t % kWave;
  const int wm = wave / 2, wn = wave % 2;
  const int hf = lane / 32, col = lane % 32;
  f32x16 acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[b][e] = 0.f;

  // k2 range that can hold non-zero A entries for this row tile
  int k2lo = 0, k2hi = g.K2;
  if (g.tri == 1) k2hi = min(g.K2, m0 + kT);
  if (g.tri == 2) k2lo = min(g.K2, m0);
  const bool a_mfast = g.sam == 1;
  const bool b_nfast = g.sbn == 1;
  const int nck = (k2hi - k2lo + kKc - 1) / kKc;  // chunks per k1
  const int64_t total = (int64_t)g.K1 * nck;
  const int64_t c0 = total * sp / splits, c1 = total * (sp + 1) / splits;

  // Element u of this thread's share of a chunk.  Row index fast in memory:
  // row = t % 64, k = 8 (t / 64) + u (the thread's 8 values are contiguous in
  // the LDS row: one 16-byte write per part).  k fast: row = t / 32 + 8u,
  // k = t % 32.  Either way one offset per operand plus u times a uniform
  // stride addresses every element.
  const int ar = a_mfast ? t % 64 : t / 32, ak = a_mfast ? 8 * (t / 64) : t % 32;
  const int br = b_nfast ? t % 64 : t / 32, bk = b_nfast ? 8 * (t / 64) : t % 32;
  const int64_t a_off = (int64_t)(m0 + ar) * g.sam + (int64_t)ak * g.sak2;
  const int64_t b_off = (int64_t)(n0 + br) * g.sbn + (int64_t)bk * g.sbk2;
  const int64_t a_du = a_mfast ? g.sak2 : 8 * g.sam;  // offset step per u
  const int64_t b_du = b_nfast ? g.sbk2 : 8 * g.sbn;
  const bool full_mn = m0 + kT <= g.M && n0 + TN <= g.N;

  // B is fetched and stashed as NB column halves of 64, each mapped as A is
  float ra[kLoads], rb[NB][kLoads];
  int k1 = 0, kc = 0;  // the chunk being fetched: K1 index, chunk within the k2 range
  if (c0 < c1) {
    k1 = (int)(c0 / nck);
    kc = (int)(c0 % nck);
  }
  auto fetch = [&]() {
    const int kk = k2lo + kc * kKc;
    const float* Ak = A + (int64_t)k1 * g.sak1 + (int64_t)kk * g.sak2 + a_off;
    const float* Bk = B + (int64_t)k1 * g.sbk1 + (int64_t)kk * g.sbk2 + b_off;
    const int kmax = k2hi - kk;  // k of this chunk below kmax hold data
    if (full_mn && kmax >= kKc) {
#pragma unroll
      for (int u = 0; u < kLoads; ++u) ra[u] = Ak[u * a_du];
#pragma unroll
      for (int h = 0; h < NB; ++h)
#pragma unroll
        for (int u = 0; u < kLoads; ++u) rb[h][u] = Bk[(int64_t)(kT * h) * g.sbn + u * b_du];
    } else {
#pragma unroll
      for (int u = 0; u < kLoads; ++u) {
        const bool aok = a_mfast ? (m0 + ar < g.M && ak + u < kmax) : (m0 + ar + 8 * u < g.M && ak < kmax);
        ra[u] = aok ? Ak[u * a_du] : 0.f;
      }
#pragma unroll
      for (int h = 0; h < NB; ++h) {
        const int nh = n0 + kT * h + br;
#pragma unroll
        for (int u = 0; u < kLoads; ++u) {
          const bool bok = b_nfast ? (nh < g.N && bk + u < kmax) : (nh + 8 * u < g.N && bk < kmax);
          rb[h][u] = bok ? Bk[(int64_t)(kT * h) * g.sbn + u * b_du] : 0.f;
        }
      }
    }
    if (++kc == nck) {
      kc = 0;
      ++k1;
    }
  };
  // the 8 values of one operand into its LDS tile, split in three parts
  auto stash_one = [&](auto& s, const float (&r)[kLoads], bool fast, int row, int k) {
    if (fast) {  // one row, k .. k + 7
      bf16x8 h, m, l;
#pragma unroll
      for (int u = 0; u < kLoads; ++u) {
        __bf16 a, b, c;
        split3(r[u], a, b, c);
        h[u] = a;
        m[u] = b;
        l[u] = c;
      }
      const int kw = swz(row, k);
      *reinterpret_cast<bf16x8*>(&s[0][row][kw]) = h;
      *reinterpret_cast<bf16x8*>(&s[1][row][kw]) = m;
      *reinterpret_cast<bf16x8*>(&s[2][row][kw]) = l;
    } else {  // rows row + 8u, one k
#pragma unroll
      for (int u = 0; u < kLoads; ++u) {
        const int rw = row + 8 * u, kw = swz(rw, k);
        split3(r[u], s[0][rw][kw], s[1][rw][kw], s[2][rw][kw]);
      }
    }
  };
  auto stash = [&](int buf) {
    stash_one(sA[buf], ra, a_mfast, ar, ak);
#pragma unroll
    for (int h = 0; h < NB; ++h) stash_one(sB[buf], rb[h], b_nfast, kT * h + br, bk);
  };
  if (c0 < c1) {
    fetch();
    stash(0);
  }
  __syncthreads();
  // part pairs (A part, B part) in the order they are summed
  constexpr int PA[6] = {0, 0, 1, 0, 2, 1};
  constexpr int PB[6] = {0, 1, 0, 2, 0, 1};
  int buf = 0;
  for (int64_t c = c0; c < c1; ++c) {
    const bool more = c + 1 < c1;
    if (more) fetch();
    // wavefront (wm, wn) accumulates the NB 32x32 blocks at rows 32 wm,
    // columns 32 (NB wn + b) of the tile; lane (hf, col) supplies k = 16 st +
    // 8 hf .. +7 of its row (A) and column (B) to MFMA step st
#pragma unroll
    for (int st = 0; st < kKc / 16; ++st) {
      bf16x8 av[3];
#pragma unroll
      for (int p = 0; p < 3; ++p)
        av[p] = *reinterpret_cast<const bf16x8*>(&sA[buf][p][32 * wm + col][swz(32 * wm + col, 16 * st + 8 * hf)]);
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int bn = 32 * (NB * wn + b) + col;
        bf16x8 bv[3];
#pragma unroll
        for (int p = 0; p < 3; ++p)
          bv[p] = *reinterpret_cast<const bf16x8*>(&sB[buf][p][bn][swz(bn, 16 * st + 8 * hf)]);
#pragma unroll
        for (int q = 0; q < 6; ++q)
          acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[PA[q]], bv[PB[q]], acc[b], 0, 0, 0);
      }
    }
    if (more) stash(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int n = n0 + 32 * (NB * wn + b) + col;
    if (n >= g.N) continue;
    if (splits == 1) {
      float* C = g.C + (int64_t)z * g.scz;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0 + 32 * wm + 8 * (e / 4) + 4 * hf + (e % 4);
        if (m < g.M) C[(int64_t)m * g.scm + n] = g.alpha * acc[b][e];
      }
    } else {
      float* P = g.part + ((int64_t)z * splits + sp) * g.M * g.N;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0 + 32 * wm + 8 * (e / 4) + 4 * hf + (e % 4);
        if (m < g.M) P[(int64_t)m * g.N + n] = acc[b][e];
      }
    }
  }
}

// C = alpha * (sum of the parts in order s = 0, 1, ...): identical run to run.
__global__ __launch_bounds__(256) void gemm_reduce_kernel(GemmArgs g, int splits) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t mn = (int64_t)g.M * g.N;
  if (idx >= (int64_t)g.Z * mn) return;
  const int64_t z = idx / mn, r = idx % mn;
  const float* P = g.part + z * splits * mn + r;
  float s = 0.f;
  for (int p = 0; p < splits; ++p) s += P[p * mn];
  g.C[z * g.scz + (r / g.N) * g.scm + r % g.N] = g.alpha * s;
}

// Inverse block-level RoPE: plane (d, d + Dg/2) of row i rotates by
// -i * base^(-2d/Dg) (the angle formed in double, as in the forward).
__global__ __launch_bounds__(256) void rope_inverse_kernel(RopeArgs a) {
  const int half = a.gate_dim / 2;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = a.rows * a.n_blocks * half;
  if (idx >= total) return;
  const int d = (int)(idx % half);
  const int64_t ri = idx / half;  // (row, i)
  const int i = (int)(ri % a.n_blocks);
  const double ang = (double)i * pow(a.base, -2.0 * d / a.gate_dim);
  const float cs = (float)cos(ang), sn = (float)sin(ang);
  float* v = a.x + ri * a.gate_dim;
  const float x0 = v[d], x1 = v[d + half];
  v[d] = x0 * cs + x1 * sn;
  v[d + half] = -x0 * sn + x1 * cs;
}

}  // namespace

hipError_t launch_kl_rows(const KlArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  const int64_t blocks = (a.rows + kRowsPerBlock - 1) / kRowsPerBlock;
  const bool vec = a.n_blocks % 4 == 0 && reinterpret_cast<uintptr_t>(a.logits) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(a.gt) % 16 == 0;
  const dim3 grid((unsigned)blocks);
  if (vec && a.n_blocks <= 256) hipLaunchKernelGGL(kl_rows_staged_kernel<1>, grid, dim3(256), 0, s, a);
  else if (vec && a.n_blocks <= 512) hipLaunchKernelGGL(kl_rows_staged_kernel<2>, grid, dim3(256), 0, s, a);
  else if (vec && a.n_blocks <= 1024) hipLaunchKernelGGL(kl_rows_staged_kernel<4>, grid, dim3(256), 0, s, a);
  else if (vec && a.n_blocks <= 2048) hipLaunchKernelGGL(kl_rows_staged_kernel<8>, grid, dim3(256), 0, s, a);
  else if (vec) hipLaunchKernelGGL(kl_rows_kernel<4>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(kl_rows_kernel<1>, grid, dim3(256), 0, s, a);
  double* parts = a.row_loss + a.rows;
  hipLaunchKernelGGL(loss_part_kernel, dim3(kLossParts), dim3(256), 0, s, a.row_loss, a.rows, parts);
  hipLaunchKernelGGL(loss_mean_kernel, dim3(1), dim3(256), 0, s, parts, a.rows, a.loss);
  return hipGetLastError();
}

// Output tile width.  128 columns (each A chunk is then split into parts once
// per 128 columns instead of once per 64, and every barrier covers twice the
// MFMAs, at two workgroups per CU instead of three) when the product has that
// many and a long contraction: measured with their split sums at 2048 blocks
// (32 query / 8 KV heads, gate_dim 128) 0.50 -> 0.43 ms, at 1024 blocks (28 /
// 4 heads) 0.164 -> 0.158 ms, but at 512 blocks 0.090 -> 0.098 ms (too few
// tiles).
static int gemm_tile_n(const GemmArgs& a) {
  if (a.tile_n == kT || a.tile_n == 2 * kT) return a.tile_n;
  return (a.N >= 2 * kT && a.K2 >= 32 * kKc) ? 2 * kT : kT;
}

// Parts per output tile: enough workgroups to fill the chip (about 2048 of
// 64-column tiles, 1024 of 128-column ones) when the tiles alone are fewer,
// but at least a.min_chunks chunks of K per part on the longest tile (8 by
// default; a smaller value lets tests split small products).
int gemm_splits(const GemmArgs& a) {
  if (a.M <= 0 || a.N <= 0 || a.Z <= 0) return 1;
  const int min_chunks = a.min_chunks >= 1 ? a.min_chunks : 8;
  const int tn = gemm_tile_n(a);
  const int64_t tiles = (int64_t)((a.N + tn - 1) / tn) * ((a.M + kT - 1) / kT) * a.Z;
  const int64_t chunks = (int64_t)a.K1 * ((a.K2 + kKc - 1) / kKc);
  const int64_t target = 2048 * kT / tn;  // workgroups (the same output area in flight)
  int64_t sp = (target + tiles - 1) / tiles;
  sp = std::min<int64_t>(sp, chunks / min_chunks);
  sp = std::min<int64_t>(sp, 64);
  return (int)std::max<int64_t>(sp, 1);
}

int64_t gemm_partial_elems(const GemmArgs& a) {
  const int sp = gemm_splits(a);
  return sp > 1 ? (int64_t)a.Z * sp * a.M * a.N : 0;
}

hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0 || a.Z <= 0) return hipSuccess;
  const int sp = gemm_splits(a);
  if (sp > 1 && a.part == nullptr) return hipErrorInvalidValue;
  const int tn = gemm_tile_n(a);
  const int64_t tiles = (int64_t)((a.N + tn - 1) / tn) * ((a.M + kT - 1) / kT) * a.Z * sp;
  if (tiles > INT32_MAX) return hipErrorInvalidValue;
  if (tn == 2 * kT) hipLaunchKernelGGL(gemm_f32_kernel<2>, dim3((unsigned)tiles), dim3(256), 0, s, a, sp);
  else hipLaunchKernelGGL(gemm_f32_kernel<1>, dim3((unsigned)tiles), dim3(256), 0, s, a, sp);
  if (sp > 1) {
    const int64_t n = (int64_t)a.Z * a.M * a.N;
    hipLaunchKernelGGL(gemm_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a, sp);
  }
  return hipGetLastError();
}

hipError_t launch_rope_inverse(const RopeArgs& a, hipStream_t s) {
  const int64_t total = a.rows * a.n_blocks * (a.gate_dim / 2);
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_inverse_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace seer
