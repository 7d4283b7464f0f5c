// attn_kernels.hip -- block-sparse / dense causal FlashAttention forward for gfx950.
//
// SeerAttention section 3.3: the gate's block mask selects which 64x64 tiles of
// the causal attention map are computed; inactive tiles cost neither loads nor
// MFMA work.  The dense comparison path is the same kernel walking every causal
// tile.  Precision: bf16 operands, fp32 accumulation and softmax; P is rounded
// to bf16 before the PV product; O is stored by round-to-nearest-even.
//
// Work decomposition.  One workgroup (2 wavefronts) owns one (batch, head,
// query block) row of the block mask: 64 queries, 32 per wavefront.  It walks
// the row's ascending list of active key blocks; per key block it stages the
// K tile (row-major) and the V tile (transposed, key-contiguous) in LDS, while
// the next tile's global loads are already in flight in registers.
//
// Transposed formulation.  Each wavefront computes S^T = K Q^T and O^T = V^T P^T
// with v_mfma_f32_32x32x16_bf16, so that the MFMA output column -- one lane
// (and its partner lane + 32) -- is one query.  The softmax row statistics
// (running max m, partial sum l, rescale factor) are then per-lane scalars: the
// row max needs one cross-lane exchange per tile instead of a 32-lane reduction,
// and rescaling O needs no broadcast.
//
// MFMA 32x32 output layout used throughout: accumulator e of lane L holds
// row 8*(e/4) + 4*(L/32) + e%4, column L%32.  Operand k-slots only need to agree
// between A and B (lane half + slot), which every product below guarantees.
#include "device_common.h"
#include "launch.h"

namespace seer {

namespace {

struct Task {
  int b, h, i;
};

// Task order: query-block rows heaviest first (i descending), the query heads
// of one KV head adjacent, and each KV-head group kept on one XCD (workgroups
// are dispatched round-robin over the 8 XCDs, each with its own L2), so the
// K/V tiles of a group are shared through one L2.  Groups are split over
// several XCDs by row residue when there are fewer than 8.
struct TaskMap {
  int batch, heads_q, heads_kv, nb;
  int R;        // XCDs per KV group (row residue classes); 0 selects linear order
  int lanes_x;  // (group, residue) lanes per XCD
  int per_xcd;  // tasks per XCD
};

__device__ __forceinline__ Task decode_task(const TaskMap& m, int wg) {
  const int G = m.heads_q / m.heads_kv;
  Task t;
  if (m.R > 0) {
    const int x = wg % 8;
    const int u = wg / 8;
    const int hh = u % G;
    const int lam_l = (u / G) % m.lanes_x;
    const int nu = u / (G * m.lanes_x);
    const int lam = x * m.lanes_x + lam_l;
    const int s = lam / m.R;
    const int rho = lam % m.R;
    t.i = m.nb - 1 - (nu * m.R + rho);
    t.b = s / m.heads_kv;
    t.h = (s % m.heads_kv) * G + hh;
  } else {
    const int bh = m.batch * m.heads_q;
    const int nu = wg / bh;
    const int rem = wg % bh;
    t.b = rem / m.heads_q;
    t.h = rem % m.heads_q;
    t.i = m.nb - 1 - nu;
  }
  return t;
}

struct KernelArgs {
  AttnArgs a;
  TaskMap map;
  float scale_log2;  // scale * log2(e)
};

// Iterates the active key blocks of a row: the compacted list for the sparse
// kernel, 0..i (causal) or 0..nb-1 for the dense one.  Entries that are out of
// range (>= nb, or > i when causal) end the row.
template <bool SPARSE>
struct RowList {
  const uint16_t* idx;
  int n, nb, i;
  bool causal;
  __device__ __forceinline__ int at(int p) const { return SPARSE ? (int)idx[p] : p; }
  __device__ __forceinline__ bool ok(int j) const { return j < nb && (!causal || j <= i); }
};

template <bool SPARSE>
__device__ __forceinline__ RowList<SPARSE> make_list(const AttnArgs& a, const Task& t) {
  RowList<SPARSE> L;
  L.nb = a.n_blocks;
  L.i = t.i;
  L.causal = a.causal;
  const int64_t row = ((int64_t)t.b * a.heads_q + t.h) * a.n_blocks + t.i;
  if (SPARSE) {
    L.idx = a.idx + row * a.n_blocks;
    L.n = min(max(a.count[row], 0), a.n_blocks);
  } else {
    L.idx = nullptr;
    L.n = a.causal ? t.i + 1 : a.n_blocks;
  }
  return L;
}

// Online-softmax update of one 64-key tile held as S^T in s[0..1] (32 keys each);
// converts s in place to unnormalised probabilities and returns the factor by
// which the running output must be rescaled.
__device__ __forceinline__ float softmax_tile(f32x16 (&s)[2], float& m_run, float& l_run,
                                              float c) {
  float mloc = -INFINITY;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) mloc = fmaxf(mloc, s[mt][e]);
  mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
  const float m_new = fmaxf(m_run, mloc);
  const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
  const float alpha = exp2f((m_run - m_use) * c);
  const float mc = m_use * c;
  float psum = 0.f;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float p = exp2f(fmaf(s[mt][e], c, -mc));
      s[mt][e] = p;
      psum += p;
    }
  l_run = l_run * alpha + psum;
  m_run = m_new;
  return alpha;
}

// ---------------------------------------------------------------------------
// bf16 kernel
// ---------------------------------------------------------------------------

template <int D>
struct Bf16Layout {
  static constexpr int KSTR = D + 8;   // LDS row stride of K (bf16 elements), conflict-free b128 reads
  static constexpr int VSTR = 64 + 4;  // LDS row stride of V^T (one row per feature d)
  static constexpr int OSTR = D + 8;   // LDS row stride of the output staging tile
  static constexpr int K_BYTES = 64 * KSTR * 2;
  static constexpr int V_BYTES = D * VSTR * 2;
  static constexpr int VBL = D / 64;   // (4 keys x 8 features) V blocks per thread per tile
  static_assert(64 * OSTR * 2 <= K_BYTES + V_BYTES, "output staging must fit");
};

// One thread's share of a K or V tile in flight (16-byte chunks; 128 threads).
template <int D>
struct StageRegs {
  static constexpr int N = D / 16;  // == 4 * VBL as well
  u32x4 r[N];
};

template <int D>
__device__ __forceinline__ void load_k(StageRegs<D>& st, const uint16_t* __restrict__ kp,
                                       int64_t kss, int j, int tid) {
  constexpr int CPR = D / 8;  // 16-byte chunks per row
#pragma unroll
  for (int e = 0; e < StageRegs<D>::N; ++e) {
    const int q = tid + 128 * e;
    const int key = q / CPR, c = q % CPR;
    st.r[e] = *reinterpret_cast<const u32x4*>(kp + (int64_t)(64 * j + key) * kss + 8 * c);
  }
}

template <int D>
__device__ __forceinline__ void store_k(const StageRegs<D>& st, uint16_t* sK, int tid) {
  using Lay = Bf16Layout<D>;
  constexpr int CPR = D / 8;
#pragma unroll
  for (int e = 0; e < StageRegs<D>::N; ++e) {
    const int q = tid + 128 * e;
    const int key = q / CPR, c = q % CPR;
    *reinterpret_cast<u32x4*>(sK + key * Lay::KSTR + 8 * c) = st.r[e];
  }
}

// V is loaded as blocks of 4 consecutive keys x 8 features (four 16-byte rows)
template <int D>
__device__ __forceinline__ void load_v(StageRegs<D>& st, const uint16_t* __restrict__ vp,
                                       int64_t vss, int j, int tid) {
  constexpr int CPR = D / 8;
#pragma unroll
  for (int e = 0; e < Bf16Layout<D>::VBL; ++e) {
    const int bq = tid + 128 * e;
    const int kq = bq / CPR, c = bq % CPR;
#pragma unroll
    for (int rr = 0; rr < 4; ++rr)
      st.r[4 * e + rr] =
          *reinterpret_cast<const u32x4*>(vp + (int64_t)(64 * j + 4 * kq + rr) * vss + 8 * c);
  }
}

// V^T in LDS: feature row d = 8c + f holds keys 4kq..4kq+3 as one 8-byte store
template <int D>
__device__ __forceinline__ void store_v(const StageRegs<D>& st, uint16_t* sVt, int tid) {
  using Lay = Bf16Layout<D>;
  constexpr int CPR = D / 8;
#pragma unroll
  for (int e = 0; e < Lay::VBL; ++e) {
    const int bq = tid + 128 * e;
    const int kq = bq / CPR, c = bq % CPR;
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      const uint32_t sel = (f & 1) ? 0x07060302u : 0x05040100u;
      const int w = f >> 1;
      u32x2 pk;
      pk[0] = __builtin_amdgcn_perm(st.r[4 * e + 1][w], st.r[4 * e + 0][w], sel);
      pk[1] = __builtin_amdgcn_perm(st.r[4 * e + 3][w], st.r[4 * e + 2][w], sel);
      *reinterpret_cast<u32x2*>(sVt + (8 * c + f) * Lay::VSTR + 4 * kq) = pk;
    }
  }
}

// Two workgroups' worth of wavefronts per SIMD (<= 256 registers per lane) so
// that one wavefront's softmax overlaps another's MFMA work.
//
// Pipeline per key tile n (single LDS buffer, two barriers):
//   S = K_n Q^T from LDS                    (K_{n+1} loads in flight)
//   barrier A -> store K_{n+1}; issue V_{n+1} loads
//   softmax, O += V_n^T P^T from LDS
//   barrier B -> store V_{n+1}; issue K_{n+2} loads
// K_{n+1} becomes visible to S_{n+1} through barrier B, V_{n+1} to PV_{n+1}
// through the next barrier A; K and V staging share one set of registers.
template <int D, bool SPARSE>
__global__ __launch_bounds__(128) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_fwd_bf16_kernel(KernelArgs ka) {
  using Lay = Bf16Layout<D>;
  __shared__ __attribute__((aligned(16))) uint16_t smem[(Lay::K_BYTES + Lay::V_BYTES) / 2];
  uint16_t* sK = smem;
  uint16_t* sVt = smem + Lay::K_BYTES / 2;

  const AttnArgs& a = ka.a;
  const Task t = decode_task(ka.map, blockIdx.x);
  const int tid = threadIdx.x;
  const int wave = tid / 64;
  const int lane = tid % 64;
  const int hf = lane / 32;
  const int col = lane % 32;
  const int G = a.heads_q / a.heads_kv;
  const int g = t.h / G;

  const uint16_t* qp = static_cast<const uint16_t*>(a.q.ptr) + t.b * a.q.sb + t.h * a.q.sh;
  const uint16_t* kp = static_cast<const uint16_t*>(a.k.ptr) + t.b * a.k.sb + g * a.k.sh;
  const uint16_t* vp = static_cast<const uint16_t*>(a.v.ptr) + t.b * a.v.sb + g * a.v.sh;

  // Q^T operand: lane holds query q0 + col, features 16ks + 8hf .. +7
  const int qrow = 64 * t.i + 32 * wave + col;
  bf16x8 qf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
    qf[ks] = *reinterpret_cast<const bf16x8*>(qp + (int64_t)qrow * a.q.ss + 16 * ks + 8 * hf);

  f32x16 acc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[dt][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float c = ka.scale_log2;

  // key blocks are read one step ahead; the first out-of-range entry ends the row
  const RowList<SPARSE> list = make_list<SPARSE>(a, t);
  auto next_j = [&](int p) -> int {
    if (p >= list.n) return -1;
    const int j = list.at(p);
    return list.ok(j) ? j : -1;
  };
  int j = next_j(0);
  int jn = (j >= 0) ? next_j(1) : -1;

  StageRegs<D> st;
  if (j >= 0) {
    load_k<D>(st, kp, a.k.ss, j, tid);
    store_k<D>(st, sK, tid);
    load_v<D>(st, vp, a.v.ss, j, tid);
    store_v<D>(st, sVt, tid);
    if (jn >= 0) load_k<D>(st, kp, a.k.ss, jn, tid);
  }
  __syncthreads();

  for (int n = 0; j >= 0; ++n) {
    const int jnn = (jn >= 0) ? next_j(n + 2) : -1;

    // S^T = K Q^T: two 32-key halves of the tile
    f32x16 s[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s[mt][e] = 0.f;
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        const bf16x8 kf =
            *reinterpret_cast<const bf16x8*>(sK + (32 * mt + col) * Lay::KSTR + 16 * ks + 8 * hf);
        s[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[mt], 0, 0, 0);
      }
    }
    __syncthreads();  // A: K_n fully consumed
    if (jn >= 0) {
      store_k<D>(st, sK, tid);
      load_v<D>(st, vp, a.v.ss, jn, tid);
    }

    if (a.causal && j == t.i) {  // diagonal tile: key kl visible to query ql iff kl <= ql
      const int ql = 32 * wave + col;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kl = 32 * mt + 8 * (e / 4) + 4 * hf + (e % 4);
          if (kl > ql) s[mt][e] = -INFINITY;
        }
    }
    const float alpha = softmax_tile(s, m_run, l_run, c);
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[dt][e] *= alpha;

    // P^T operand: k-step kt covers keys 32*(kt/2) + 16*(kt%2) + {4hf+0..3, 8+4hf+0..3},
    // exactly accumulators 8*(kt%2) .. +7 of half kt/2
    bf16x8 pb[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int e = 0; e < 8; ++e) pb[kt][e] = (__bf16)s[kt / 2][8 * (kt % 2) + e];

    // O^T += V^T P^T; the V^T operand row is feature d = 32dt + col with the same keys
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const uint16_t* vr = sVt + (32 * dt + col) * Lay::VSTR + 32 * (kt / 2) + 16 * (kt % 2) + 4 * hf;
        const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vr);
        const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vr + 8);
        const bf16x8 vf = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[kt], acc[dt], 0, 0, 0);
      }
    __syncthreads();  // B: V_n fully consumed, K_{n+1} visible
    if (jn >= 0) {
      store_v<D>(st, sVt, tid);
      if (jnn >= 0) load_k<D>(st, kp, a.k.ss, jnn, tid);
    }
    j = jn;
    jn = jnn;
  }

  // epilogue: normalise, stage through LDS, store rows with 16-byte writes
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = (l_tot > 0.f) ? 1.0f / l_tot : 0.f;
  __syncthreads();
  uint16_t* sO = smem;
  const int ql = 32 * wave + col;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      bf16x4 o4;
#pragma unroll
      for (int r = 0; r < 4; ++r) o4[r] = (__bf16)(acc[dt][4 * jj + r] * inv);
      *reinterpret_cast<bf16x4*>(sO + ql * Lay::OSTR + 32 * dt + 8 * jj + 4 * hf) = o4;
    }
  __syncthreads();
  uint16_t* op = static_cast<uint16_t*>(a.o) + t.b * a.osb + t.h * a.osh;
  constexpr int CPR = D / 8;
#pragma unroll
  for (int e = 0; e < 64 * CPR / 128; ++e) {
    const int q = tid + 128 * e;
    const int r = q / CPR, cc = q % CPR;
    *reinterpret_cast<u32x4*>(op + (int64_t)(64 * t.i + r) * a.oss + 8 * cc) =
        *reinterpret_cast<const u32x4*>(sO + r * Lay::OSTR + 8 * cc);
  }
  if (a.lse && hf == 0) {
    const float lse = (l_tot > 0.f) ? m_run * a.scale + __logf(l_tot) : -INFINITY;
    a.lse[((int64_t)t.b * a.heads_q + t.h) * (int64_t)a.n_blocks * 64 + qrow] = lse;
  }
}

// ---------------------------------------------------------------------------
// fp32 kernel (v_mfma_f32_32x32x2_f32): same structure, no prefetch
// ---------------------------------------------------------------------------

template <int D>
__global__ __launch_bounds__(128) void attn_fwd_f32_kernel(KernelArgs ka, int sparse) {
  constexpr int KS = D + 4;  // LDS row stride of K (floats)
  constexpr int VS = D;      // LDS row stride of V (floats)
  __shared__ __attribute__((aligned(16))) float sK[64 * KS];
  __shared__ __attribute__((aligned(16))) float sV[64 * VS];

  const AttnArgs& a = ka.a;
  const Task t = decode_task(ka.map, blockIdx.x);
  const int tid = threadIdx.x;
  const int wave = tid / 64;
  const int lane = tid % 64;
  const int hf = lane / 32;
  const int col = lane % 32;
  const int g = t.h / (a.heads_q / a.heads_kv);

  const float* qp = static_cast<const float*>(a.q.ptr) + t.b * a.q.sb + t.h * a.q.sh;
  const float* kp = static_cast<const float*>(a.k.ptr) + t.b * a.k.sb + g * a.k.sh;
  const float* vp = static_cast<const float*>(a.v.ptr) + t.b * a.v.sb + g * a.v.sh;

  const int qrow = 64 * t.i + 32 * wave + col;
  f32x4 qf[D / 8];  // features 8u + 4hf .. +3 of this lane's query
#pragma unroll
  for (int u = 0; u < D / 8; ++u)
    qf[u] = *reinterpret_cast<const f32x4*>(qp + (int64_t)qrow * a.q.ss + 8 * u + 4 * hf);

  f32x16 acc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[dt][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float c = ka.scale_log2;

  RowList<true> sl;
  RowList<false> dl;
  int n_tiles;
  if (sparse) {
    sl = make_list<true>(a, t);
    n_tiles = sl.n;
  } else {
    dl = make_list<false>(a, t);
    n_tiles = dl.n;
  }
  for (int n = 0; n < n_tiles; ++n) {
    const int j = sparse ? sl.at(n) : dl.at(n);
    if (!(sparse ? sl.ok(j) : dl.ok(j))) break;
    __syncthreads();
    constexpr int CPR = D / 4;
#pragma unroll
    for (int e = 0; e < 64 * CPR / 128; ++e) {
      const int q = tid + 128 * e;
      const int key = q / CPR, cc = q % CPR;
      *reinterpret_cast<f32x4*>(sK + key * KS + 4 * cc) =
          *reinterpret_cast<const f32x4*>(kp + (int64_t)(64 * j + key) * a.k.ss + 4 * cc);
      *reinterpret_cast<f32x4*>(sV + key * VS + 4 * cc) =
          *reinterpret_cast<const f32x4*>(vp + (int64_t)(64 * j + key) * a.v.ss + 4 * cc);
    }
    __syncthreads();

    f32x16 s[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s[mt][e] = 0.f;
#pragma unroll
      for (int u = 0; u < D / 8; ++u) {
        const f32x4 kf = *reinterpret_cast<const f32x4*>(sK + (32 * mt + col) * KS + 8 * u + 4 * hf);
#pragma unroll
        for (int vv = 0; vv < 4; ++vv)
          s[mt] = __builtin_amdgcn_mfma_f32_32x32x2f32(kf[vv], qf[u][vv], s[mt], 0, 0, 0);
      }
    }
    if (a.causal && j == t.i) {
      const int ql = 32 * wave + col;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kl = 32 * mt + 8 * (e / 4) + 4 * hf + (e % 4);
          if (kl > ql) s[mt][e] = -INFINITY;
        }
    }
    const float alpha = softmax_tile(s, m_run, l_run, c);
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[dt][e] *= alpha;
    // O^T += V^T P^T one key pair per MFMA: lane half hf supplies key
    // 32mt + 8(e/4) + 4hf + e%4, whose probability this lane already holds
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = 32 * mt + 8 * (e / 4) + 4 * hf + (e % 4);
          acc[dt] = __builtin_amdgcn_mfma_f32_32x32x2f32(sV[key * VS + 32 * dt + col], s[mt][e],
                                                         acc[dt], 0, 0, 0);
        }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = (l_tot > 0.f) ? 1.0f / l_tot : 0.f;
  float* op = static_cast<float*>(a.o) + t.b * a.osb + t.h * a.osh + (int64_t)qrow * a.oss;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      f32x4 o4;
#pragma unroll
      for (int r = 0; r < 4; ++r) o4[r] = acc[dt][4 * jj + r] * inv;
      *reinterpret_cast<f32x4*>(op + 32 * dt + 8 * jj + 4 * hf) = o4;
    }
  if (a.lse && hf == 0) {
    const float lse = (l_tot > 0.f) ? m_run * a.scale + __logf(l_tot) : -INFINITY;
    a.lse[((int64_t)t.b * a.heads_q + t.h) * (int64_t)a.n_blocks * 64 + qrow] = lse;
  }
}

static int gcd_int(int x, int y) {
  while (y) {
    const int r = x % y;
    x = y;
    y = r;
  }
  return x;
}

static TaskMap make_map(const AttnArgs& a) {
  TaskMap m;
  m.batch = a.batch;
  m.heads_q = a.heads_q;
  m.heads_kv = a.heads_kv;
  m.nb = a.n_blocks;
  const int slices = a.batch * a.heads_kv;
  const int R = 8 / gcd_int(slices, 8);
  const int64_t total = (int64_t)a.batch * a.heads_q * a.n_blocks;
  if (a.n_blocks % R == 0 && total % 8 == 0) {
    m.R = R;
    m.lanes_x = slices * R / 8;
    m.per_xcd = (int)(total / 8);
  } else {
    m.R = 0;
    m.lanes_x = 0;
    m.per_xcd = 0;
  }
  return m;
}

}  // namespace

hipError_t launch_attn(const AttnArgs& a, hipStream_t s) {
  KernelArgs ka;
  ka.a = a;
  ka.map = make_map(a);
  ka.scale_log2 = a.scale * kLog2e;
  const int64_t total = (int64_t)a.batch * a.heads_q * a.n_blocks;
  if (total == 0) return hipSuccess;
  dim3 grid((unsigned)total), block(128);
  const bool sparse = a.count != nullptr;
  if (a.bf16) {
    if (a.head_dim == 128) {
      if (sparse) hipLaunchKernelGGL((attn_fwd_bf16_kernel<128, true>), grid, block, 0, s, ka);
      else hipLaunchKernelGGL((attn_fwd_bf16_kernel<128, false>), grid, block, 0, s, ka);
    } else if (a.head_dim == 64) {
      if (sparse) hipLaunchKernelGGL((attn_fwd_bf16_kernel<64, true>), grid, block, 0, s, ka);
      else hipLaunchKernelGGL((attn_fwd_bf16_kernel<64, false>), grid, block, 0, s, ka);
    } else {
      return hipErrorInvalidValue;
    }
  } else {
    if (a.head_dim == 128) hipLaunchKernelGGL(attn_fwd_f32_kernel<128>, grid, block, 0, s, ka, (int)sparse);
    else if (a.head_dim == 64) hipLaunchKernelGGL(attn_fwd_f32_kernel<64>, grid, block, 0, s, ka, (int)sparse);
    else return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace seer
