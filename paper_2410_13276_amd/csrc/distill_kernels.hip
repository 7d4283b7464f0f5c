// distill_kernels.hip -- the gate's distillation step for gfx950 (SeerAttention
// section 3.2, Eq. 2): KL(ground truth || gate score) and its gradients with
// respect to the gate weights.
//
//   kl_rows_kernel      one wavefront per query-block row: the row's softmax of
//                       the gate logits, the ground-truth row renormalised to a
//                       distribution T, the row's KL(T || P) and the logit
//                       gradient (P sum(T) - T) / rows written over the logits.
//   loss_mean_kernel    the mean of the row losses in a fixed order (one
//                       workgroup, double accumulation: run-to-run identical).
//   gemm_f32_kernel     fp32 strided batched products for the backward pass
//                       (dQg = dL Kg, dKg = dL^T Qg, dW = pooled^T dG), 64x64
//                       LDS tiles on fp32 MFMA, triangular skipping of the
//                       causal zeros.
//   rope_inverse_kernel rotates gradient rows back through the block-level
//                       RoPE (the transpose of the forward rotation).
#include "device_common.h"
#include "launch.h"

namespace seer {

namespace {

constexpr int kRowsPerBlock = 4;  // wavefronts (rows) per workgroup

__global__ __launch_bounds__(256) void kl_rows_kernel(KlArgs a) {
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + wave;
  if (r >= a.rows) return;
  const int nb = a.n_blocks;
  const int i = (int)(r % nb);
  const int M = i + 1;  // causal entries j <= i
  float* Lr = a.logits + r * nb;
  const float* gr = a.gt + r * nb;

  float mx = -INFINITY, gs = 0.f;
  for (int j = lane; j < M; j += kWave) {
    mx = fmaxf(mx, Lr[j]);
    gs += gr[j];
  }
  mx = wave_max(mx);
  gs = wave_sum(gs);
  float es = 0.f;
  for (int j = lane; j < M; j += kWave) es += __expf(Lr[j] - mx);
  es = wave_sum(es);
  const float lse = mx + __logf(es);
  const float inv_gs = gs > 0.f ? 1.0f / gs : 0.f;
  const float tsum = gs > 0.f ? 1.0f : 0.f;  // sum of T
  const float log_gs = gs > 0.f ? __logf(gs) : 0.f;
  float loss = 0.f;
  for (int j = lane; j < nb; j += kWave) {
    float d = 0.f;
    if (j < M) {
      const float l = Lr[j];
      const float g = gr[j];
      const float logp = l - lse;
      const float t = g * inv_gs;
      if (t > 0.f) loss += t * ((__logf(g) - log_gs) - logp);
      d = (__expf(logp) * tsum - t) * a.inv_rows;
    }
    Lr[j] = d;
  }
  double dl = (double)loss;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) dl += __shfl_xor(dl, off);
  if (lane == 0) a.row_loss[r] = dl;
}

__global__ __launch_bounds__(256) void loss_mean_kernel(const double* __restrict__ row_loss,
                                                         int64_t rows, float* __restrict__ loss) {
  __shared__ double part[256];
  double s = 0.0;
  for (int64_t r = threadIdx.x; r < rows; r += 256) s += row_loss[r];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = (float)(part[0] / (double)rows);
}

// 64x64 output tile per 256-thread workgroup (a 32x32 fp32-MFMA block per
// wavefront, v_mfma_f32_32x32x2_f32), K in chunks of 16 staged through LDS.  Operand tiles are read along whichever
// index has unit stride, so that loads coalesce for every layout used here.
constexpr int kT = 64;
constexpr int kKc = 16;

__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs g) {
  __shared__ float sA[kKc][kT + 4];
  __shared__ float sB[kKc][kT + 4];
  const int t = threadIdx.x;
  const int m0 = blockIdx.y * kT, n0 = blockIdx.x * kT;
  const int z = blockIdx.z;
  const float* A = g.A + (int64_t)z * g.saz;
  const float* B = g.B + (int64_t)(z / g.bdiv) * g.sbz;
  const int wave = t / kWave, lane = t % kWave;
  const int wm = wave / 2, wn = wave % 2;
  const int hf = lane / 32, col = lane % 32;
  f32x16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;

  // k2 range that can hold non-zero A entries for this row tile
  int k2lo = 0, k2hi = g.K2;
  if (g.tri == 1) k2hi = min(g.K2, m0 + kT);
  if (g.tri == 2) k2lo = min(g.K2, m0);
  const bool a_mfast = g.sam == 1;
  const bool b_nfast = g.sbn == 1;

  for (int k1 = 0; k1 < g.K1; ++k1) {
    const float* Ak = A + (int64_t)k1 * g.sak1;
    const float* Bk = B + (int64_t)k1 * g.sbk1;
    for (int kk = k2lo; kk < k2hi; kk += kKc) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = t + 256 * u;
        const int m = a_mfast ? e % kT : e / kKc;
        const int k = a_mfast ? e / kT : e % kKc;
        const int gm = m0 + m, gk = kk + k;
        sA[k][m] = (gm < g.M && gk < k2hi) ? Ak[(int64_t)gm * g.sam + (int64_t)gk * g.sak2] : 0.f;
        const int n = b_nfast ? e % kT : e / kKc;
        const int kb = b_nfast ? e / kT : e % kKc;
        const int gn = n0 + n, gkb = kk + kb;
        sB[kb][n] = (gn < g.N && gkb < k2hi) ? Bk[(int64_t)gkb * g.sbk2 + (int64_t)gn * g.sbn] : 0.f;
      }
      __syncthreads();
      // wavefront (wm, wn) accumulates the 32x32 block at rows 32 wm, columns 32 wn
      // of the tile; each MFMA contracts the two k of one step, lane half hf
      // supplying k = 2 s + hf of row (or column) lane % 32
#pragma unroll
      for (int st = 0; st < kKc / 2; ++st)
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(sA[2 * st + hf][32 * wm + col], sB[2 * st + hf][32 * wn + col],
                                                   acc, 0, 0, 0);
      __syncthreads();
    }
  }
  float* C = g.C + (int64_t)z * g.scz;
  const int n = n0 + 32 * wn + col;
  if (n < g.N) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int m = m0 + 32 * wm + 8 * (e / 4) + 4 * hf + (e % 4);
      if (m < g.M) C[(int64_t)m * g.scm + n] = g.alpha * acc[e];
    }
  }
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
  hipLaunchKernelGGL(kl_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a);
  hipLaunchKernelGGL(loss_mean_kernel, dim3(1), dim3(256), 0, s, a.row_loss, a.rows, a.loss);
  return hipGetLastError();
}

hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0 || a.Z <= 0) return hipSuccess;
  dim3 grid((a.N + kT - 1) / kT, (a.M + kT - 1) / kT, a.Z);
  hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rope_inverse(const RopeArgs& a, hipStream_t s) {
  const int64_t total = a.rows * a.n_blocks * (a.gate_dim / 2);
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_inverse_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace seer
