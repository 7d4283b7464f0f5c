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
// the row's ascending list of active key blocks; per key block the K and V
// tiles reach LDS by direct loads (row-major, swizzled), the next tile's loads
// in flight while the current one is consumed.  Where every query head of a
// KV group walks the same row (a mask shared by the group, and dense rows), one
// workgroup holds 2 (or 4) query heads of the group for the same query block
// and each K/V tile load serves all of them.
//
// Ground-truth mode (appendix A.1, Eq. 5-6; the distillation target of Eq. 2):
// the dense kernel also stores, per query and key tile, the tile row maximum of
// the raw scores r, which online softmax forms anyway; once the row's final
// max and denominator are known, the workgroup rescales its stored maxima into
// probabilities and takes the column max over its 64 queries, giving the 2D
// max-pooled attention map without ever holding a probability matrix.
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
#include <algorithm>
#include <cstdlib>
#include <mutex>

#include "device_common.h"
#include "launch.h"

namespace seer {

namespace {

struct Task {
  int b, h, i;
  int p;  // key range of a split task (0 otherwise)
};

// Task order.  Workgroups are dispatched round-robin over the 8 XCDs (each
// with its own L2), so workgroup w runs on XCD w % 8 and is that XCD's
// (w / 8)-th task.  The order keeps the K/V working set of each L2 small:
//  - the KV-head groups (batch x KV head) are processed in phases of `gpp`
//    groups whose K and V fit the Infinity Cache together;
//  - in a phase each group owns R = 8 / gpp XCDs, split by query-block residue
//    i % R, so one group's K/V tiles are shared through those XCDs' L2;
//  - within an XCD, query-block rows run heaviest first (i descending) with
//    the query heads of the group adjacent (they read the same K/V).
// Shapes that do not fit this scheme use the plain heaviest-first order.
struct TaskMap {
  int batch, heads_q, heads_kv, nb;
  int R;    // XCDs per group; 0 selects the plain order
  int gpp;  // groups per phase (R * gpp == 8)
  int tpp;  // tasks per XCD per phase = (nb / R) * G
};

__device__ __forceinline__ Task decode_task(const TaskMap& m, int wg) {
  const int G = m.heads_q / m.heads_kv;
  Task t;
  if (m.R > 0) {
    const int x = wg % 8;
    const int u = wg / 8;
    const int ph = u / m.tpp;
    const int rem = u % m.tpp;
    const int nu = rem / G;
    const int hh = rem % G;
    const int slot = ph * m.gpp + x / m.R;
    const int rho = x % m.R;
    t.i = m.nb - 1 - (nu * m.R + rho);
    t.b = slot / m.heads_kv;
    t.h = (slot % m.heads_kv) * G + hh;
  } else {
    const int bh = m.batch * m.heads_q;
    const int nu = wg / bh;
    const int rem = wg % bh;
    t.b = rem / m.heads_q;
    t.h = rem % m.heads_q;
    t.i = m.nb - 1 - nu;
  }
  t.p = 0;
  return t;
}

// Key-range split.  Each causal row i is cut into ranges of w key blocks:
// range r holds blocks [r w, r w + w), and row i reaches ranges 0 .. i / w.  A
// task is one (batch, head, query block, range).  Tasks are ordered by KV group
// (batch x KV head), then by range, then by query block (heaviest first), then
// by query head.  The resident workgroups take tasks in that order from nq
// queues (queue x holds tasks x, x + nq, x + 2 nq, ...; workgroup g draws from
// queue g % nq by an atomic ticket, so with nq = 8 each XCD drains its own
// queue): the tasks running at any moment are a window of consecutive tasks,
// and every XCD reads the K and V of one range of one group -- w blocks, sized
// so that their K and V fit an XCD's 4 MB L2.  (A fixed stride of tasks per
// workgroup lets the workgroups drift apart by several ranges over a call, as
// task lengths vary: measured L2 hit rate 0.31 against 0.78.)
struct SplitMap {
  int heads_q, heads_kv, nb, w, parts;  // parts = ceil(nb / w)
  int64_t per_group;                    // tasks of one group: G sum_r (nb - r w)
  int64_t total;                        // per_group * groups
  int nq;                               // task queues: min(8, grid)
};

__device__ __forceinline__ Task decode_split(const SplitMap& m, int64_t task) {
  const int G = m.heads_q / m.heads_kv;
  const int grp = (int)(task / m.per_group);
  int u = (int)(task % m.per_group);
  int r = 0;
  for (; r < m.parts - 1; ++r) {  // uniform: the range whose tasks hold u
    const int c = G * (m.nb - r * m.w);
    if (u < c) break;
    u -= c;
  }
  Task t;
  t.p = r;
  t.i = m.nb - 1 - u / G;
  t.b = grp / m.heads_kv;
  t.h = (grp % m.heads_kv) * G + u % G;
  return t;
}

// Partial slots of the rows before row i of one (batch, head): row i' owns
// floor(i' / w) + 1 consecutive slots, one per range it reaches.
__device__ __forceinline__ int64_t split_offset(int i, int w) {
  const int64_t q = i / w, r = i % w;
  return i + w * q * (q - 1) / 2 + r * q;
}

// Per-row record of the split (split_bounds_kernel): list offsets of ranges
// 0 .. P, the number of non-empty ranges, and the row's arrival counter.
__host__ __device__ __forceinline__ int split_stride(int parts) { return parts + 3; }

struct KernelArgs {
  AttnArgs a;
  TaskMap map;
  SplitMap split;
  float scale_log2;  // scale * log2(e)
  int task_base;     // first task of this launch (launches in batches, see launch_attn_one)
};

// Iterates the active key blocks of a row: the compacted list for the sparse
// kernel, 0..i (causal) or 0..nb-1 for the dense one.  Entries that are out of
// range (>= nb, or > i when causal) end the row.
// A sparse row's list holds mask entries; with 128-token mask blocks (sh = 1)
// position p of the row is the 64-key tile 2 idx[p / 2] + p % 2, so every
// entry stands for two tiles and n counts tiles.
template <bool SPARSE>
struct RowList {
  const uint16_t* idx;
  int n, nb, i;
  int lo;  // dense: first key block
  int sh;  // sparse: log2(mask block / 64)
  bool causal;
  __device__ __forceinline__ int at(int p) const {
    return SPARSE ? ((int)idx[p >> sh] << sh) + (p & sh) : lo + p;
  }
  __device__ __forceinline__ bool ok(int j) const { return j < nb && (!causal || j <= i); }
};

// The row's list; for a split task only the entries of its key range (for
// sparse rows located by split_bounds_kernel beforehand).
template <bool SPARSE, bool SPLIT = false>
__device__ __forceinline__ RowList<SPARSE> make_list(const AttnArgs& a, const Task& t) {
  RowList<SPARSE> L;
  L.nb = a.n_blocks;
  L.i = t.i;
  L.causal = a.causal;
  L.lo = 0;
  L.sh = 0;
  const int64_t row = ((int64_t)t.b * a.heads_q + t.h) * a.n_blocks + t.i;
  if (SPARSE) {
    const int sh = a.mask_shift;
    const int nbm = a.mask_blocks;  // blocks of the mask
    // a mask shared by a KV group has one row per (batch, KV head, block)
    const int64_t mrow = a.mask_kv ? ((int64_t)t.b * a.heads_kv + t.h / (a.heads_q / a.heads_kv)) * nbm + (t.i >> sh)
                                   : ((int64_t)t.b * a.heads_q + t.h) * nbm + (t.i >> sh);
    L.sh = sh;
    L.idx = a.idx + mrow * nbm;
    L.n = min(max(a.count[mrow], 0), nbm) << sh;
    if (SPLIT) {  // (the split runs on 64-token masks only)
      const int32_t* bd = a.split_bounds + row * split_stride(a.split_parts) + t.p;
      const int s0 = bd[0];
      L.idx += s0;
      L.n = bd[1] - s0;
    }
  } else {
    L.idx = nullptr;
    L.n = a.causal ? t.i + 1 : a.n_blocks;
    if (SPLIT) {
      L.lo = t.p * a.split_w;
      L.n = min(L.lo + a.split_w, t.i + 1) - L.lo;
    }
  }
  return L;
}

// Online-softmax update of one 64-key tile held as S^T in s[0..1] (32 keys each);
// converts s in place to unnormalised probabilities and returns the factor by
// which the running output must be rescaled.
__device__ __forceinline__ float softmax_tile(f32x16 (&s)[2], float& m_run, float& l_run,
                                              float c, float& mloc) {
  mloc = -INFINITY;
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

// Ground-truth epilogue of one query block (appendix A.1, Eq. 6 and the column
// max after it).  rrow[j][t] holds the raw-score maximum of query t over key
// tile j; sL2[t] = m_t c + log2(l_t) is the final softmax normaliser of query t
// in the exp2 domain (c = scale log2 e), so exp2(r c - sL2) is the largest
// probability query t gives a key of tile j.  Tiles j >= n_vis hold no visible
// key and pool to 0.  Thread `tid` of `nthr` handles tiles tid, tid + nthr, ...
__device__ __forceinline__ void pool_epilogue(const float* __restrict__ rrow, const float* sL2,
                                              float c, int n_vis, int nb,
                                              float* __restrict__ gtrow, int tid, int nthr) {
  for (int j = tid; j < nb; j += nthr) {
    float x = -INFINITY;
    if (j < n_vis) {
      const f32x4* rp = reinterpret_cast<const f32x4*>(rrow + (int64_t)j * 64);
#pragma unroll 4
      for (int u = 0; u < 16; ++u) {
        const f32x4 r = rp[u];
        const f32x4 l = *reinterpret_cast<const f32x4*>(sL2 + 4 * u);
#pragma unroll
        for (int e = 0; e < 4; ++e) x = fmaxf(x, fmaf(r[e], c, -l[e]));
      }
    }
    gtrow[j] = __builtin_amdgcn_exp2f(x);
  }
}

// Partial results cross XCDs, and each XCD has its own L2.  They are therefore
// written and read with device-scope accesses (relaxed atomics at agent scope:
// loads and stores that bypass the non-coherent caches), so no cache-wide
// fence is needed: a device-scope fence would write back and invalidate the
// whole L2 of the XCD and, issued once per task, destroy the K/V reuse the
// split exists for (measured: L2 hit rate 0.19 instead of 0.78).
__device__ __forceinline__ void store_dev(void* p, uint64_t v) {
  __hip_atomic_store(static_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_dev(float* p, float v) {
  __hip_atomic_store(reinterpret_cast<uint32_t*>(p), __float_as_uint(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t load_dev(const void* p) {
  return __hip_atomic_load(static_cast<uint64_t*>(const_cast<void*>(p)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_dev(const float* p) {
  return __uint_as_float(__hip_atomic_load(reinterpret_cast<uint32_t*>(const_cast<float*>(p)), __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT));
}

// A split task's partial output is stored straight from the MFMA accumulators
// (no LDS staging): slot element ((wave * D/32 + dt) * 4 + jj) * 256 + 4 lane + r
// holds accumulator 4 jj + r of feature tile dt of that lane, i.e. query
// 32 wave + lane % 32, feature 32 dt + 8 jj + 4 (lane / 32) + r.  Each store
// instruction of a wavefront writes 512 contiguous bytes.
__device__ __forceinline__ int64_t part_index(int D, int wave, int dt, int jj, int lane) {
  return ((int64_t)(wave * (D / 32) + dt) * 4 + jj) * 256 + 4 * lane;
}

// Merge of a split row's partial outputs, run by the row's last task (its two
// wavefronts in the layout above).  Partial p holds O_p normalised within
// range p and lse_p, its log2-domain log-sum-exp, so O = sum_p 2^(lse_p - lse)
// O_p with lse = log2 sum_p 2^lse_p, taken over the row's non-empty ranges in
// ascending p: a fixed order, so the result does not depend on which task
// arrives last.  The loads of two partials are in flight at a time.
template <int D>
__device__ __forceinline__ void merge_row(const AttnArgs& a, int b, int h, int i, const int32_t* bd, int wave,
                                          int lane) {
  const int w = a.split_w;
  const int nparts = i / w + 1;  // the split is causal
  const int64_t slot0 = ((int64_t)b * a.heads_q + h) * a.split_slots + split_offset(i, w);
  const int ql = 32 * wave + lane % 32;
  float mx = -INFINITY;
  for (int p = 0; p < nparts; ++p)
    if (bd[p + 1] > bd[p]) mx = fmaxf(mx, load_dev(a.part_lse + (slot0 + p) * 64 + ql));
  f32x16 acc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[dt][e] = 0.f;
  float sum = 0.f;
  if (mx > -INFINITY) {
    for (int p0 = 0; p0 < nparts; p0 += 2) {
      uint64_t v[2][D / 8];
      float wgt[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int p = p0 + u;
        const bool use = p < nparts && bd[p + 1] > bd[p];
        const float lp = use ? load_dev(a.part_lse + (slot0 + p) * 64 + ql) : -INFINITY;
        wgt[u] = lp == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(lp - mx);
        const uint16_t* src = a.part_o + (slot0 + (use ? p : p0)) * 64 * D;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            v[u][4 * dt + jj] = use ? load_dev(src + part_index(D, wave, dt, jj, lane)) : 0ull;
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        sum += wgt[u];
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const uint64_t x = v[u][4 * dt + jj];
#pragma unroll
            for (int r = 0; r < 4; ++r)
              acc[dt][4 * jj + r] = fmaf(wgt[u], __uint_as_float((uint32_t)(x >> (16 * r)) << 16), acc[dt][4 * jj + r]);
          }
      }
    }
  }
  const int t = 64 * i + ql;
  if (t >= a.seq_len) return;  // padding row of a partial last tile
  const float inv = sum > 0.f ? 1.0f / sum : 0.f;
  uint16_t* dst = static_cast<uint16_t*>(a.o) + b * a.osb + h * a.osh + (int64_t)t * a.oss + 4 * (lane / 32);
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      bf16x4 o4;
#pragma unroll
      for (int r = 0; r < 4; ++r) o4[r] = (__bf16)(acc[dt][4 * jj + r] * inv);
      *reinterpret_cast<bf16x4*>(dst + 32 * dt + 8 * jj) = o4;
    }
  if (a.lse && lane < 32)
    a.lse[((int64_t)b * a.heads_q + h) * a.seq_len + t] =
        sum > 0.f ? (mx + __log2f(sum)) * 0.6931471805599453f : -INFINITY;
}

// ---------------------------------------------------------------------------
// bf16 kernel
// ---------------------------------------------------------------------------
//
// Tiles reach LDS by direct global->LDS loads (global_load_lds_dwordx4: lane l
// of a wavefront writes its 16 bytes at base + 16 l), so no registers stage
// them.  K and V are both kept row-major (one row per key, D features), with
// the 16-byte chunks of each row XOR-swizzled so that every operand read is
// free of LDS bank conflicts on gfx950 (64 banks, 16 lanes per pass); the
// gather permutation is applied on the global side of the load.
//  - K chunk c of row r sits at chunk c ^ fk(r): the S^T operand read (16
//    lanes = 16 consecutive rows, one chunk each) hits 16 distinct bank groups.
//  - V chunk c of row r sits at chunk c ^ fv(r): the V^T operand is read with
//    ds_read_b64_tr_b16, whose 8-byte reads are served 32 lanes per pass: 4
//    consecutive rows x 64 bytes (four 16-byte chunks, 4k .. 4k + 3, of each
//    row).  fv XORs the chunk index with a multiple of 4 that differs for the
//    4 rows (or, at D = 64, for the two 256-byte lines they span), so the pass
//    covers 16 distinct chunk positions = all 64 banks once.  (A 2-way
//    conflict remained with an XOR by 2 (r % 4), which only separates rows
//    within a 16-lane group.)
//
// ds_read_b64_tr_b16 semantics (within each group of 16 lanes): view the 16
// lanes' 8-byte reads as a 16 x 4 matrix C of 16-bit values; lane 4a + b
// receives C[a][b], C[a+4][b], C[a+8][b], C[a+12][b].  With lane 16g + r
// pointing at key row base + r/4, feature 4(r%4) + 16(g%2) + 32dt, output lane
// L receives the four consecutive keys base..base+3 of feature 32dt + L%32 --
// exactly four k-slots of the V^T operand of the 32x32x16 MFMA.

template <int D>
struct Bf16Layout {
  static constexpr int CPR = D / 8;           // 16-byte chunks per row
  static constexpr int RP = 16 / CPR;         // rows per 256 bytes (the 64-bank span)
  static constexpr int TILE = 64 * D;         // bf16 elements per K or V tile
  static constexpr int LOADS = D / 16;        // direct 16-byte loads per thread per tile
  static constexpr int OSTR = D + 8;          // output staging row
  static_assert(64 * OSTR <= 2 * TILE, "output staging must fit");
  __device__ static int fk(int r) { return (r / RP) & (CPR - 1); }
  __device__ static int fv(int r) { return 4 * ((r / RP) & (CPR / 4 - 1)); }
};

// One 16-byte direct global->LDS load per lane (global_load_lds_dwordx4): lane
// l writes LDS bytes [lds_base + 16 l, +16) from global address base + voff.
// Issued through inline assembly so that the compiler does not add
// conservative vmcnt waits in front of every LDS read; the kernel waits for
// its own loads explicitly (wait_loads) before the barrier that publishes them.
__device__ __forceinline__ void dma16(uint32_t lds_base, const void* base, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds_base), "v"(voff), "s"(base)
               : "memory", "m0");
}

__device__ __forceinline__ void wait_loads() {
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this thread's direct loads have landed
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Direct load of one 64-row tile.  Wavefront w, load e covers LDS chunks
// q = 64 (2e + w) + lane: row q / CPR, physical chunk q % CPR, which holds
// global chunk (q % CPR) ^ f(row).  Since 128 e is a multiple of CPR, the row
// is 128e / CPR + (64w + lane) / CPR: the first term is uniform (folded into
// the scalar base) and the swizzle f depends on e only through e & 1, so each
// lane needs two byte offsets per tensor, computed once (dma_offsets).
template <int D, bool IS_V>
__device__ __forceinline__ uint32_t dma_offset(int ss, int wave, int lane, int e_parity) {
  using Lay = Bf16Layout<D>;
  const int ql = 64 * wave + lane;
  const int r = 128 * e_parity / Lay::CPR + ql / Lay::CPR;
  const int pc = ql % Lay::CPR;
  const int gc = pc ^ (IS_V ? Lay::fv(r) : Lay::fk(r));
  return (uint32_t)(((ql / Lay::CPR) * ss + 8 * gc) * 2);
}

template <int D>
__device__ __forceinline__ void load_tile_lds(uint32_t lds, const uint16_t* __restrict__ tile,
                                              int ss, int wave_u, const uint32_t (&off)[2]) {
  using Lay = Bf16Layout<D>;
#pragma unroll
  for (int e = 0; e < Lay::LOADS; ++e)
    dma16(lds + 1024u * (2 * e + wave_u), tile + (int64_t)(128 * e / Lay::CPR) * ss, off[e & 1]);
}

// With NW >= 4 wavefronts sharing the tile, wavefront w issues loads e =
// 0 .. D / (8 NW) - 1, covering LDS chunk ch = NW e + w, i.e. chunks q = 64 ch +
// lane: row q / CPR, physical chunk q % CPR.  The row advances by 64 NW / CPR
// (a multiple of 16) per load, which leaves both swizzles unchanged, so each
// lane needs one byte offset per tensor; the rest is the scalar base.
template <int D, bool IS_V, int NW>
__device__ __forceinline__ uint32_t dma_offset_nw(int ss, int wave, int lane) {
  using Lay = Bf16Layout<D>;
  static_assert(NW >= 4 && (64 * NW / Lay::CPR) % 16 == 0, "swizzle must not depend on the load");
  const int ql = 64 * wave + lane;
  const int r = ql / Lay::CPR;
  const int gc = (ql % Lay::CPR) ^ (IS_V ? Lay::fv(r) : Lay::fk(r));
  return (uint32_t)((r * ss + 8 * gc) * 2);
}

template <int D, int NW>
__device__ __forceinline__ void load_tile_lds_nw(uint32_t lds, const uint16_t* __restrict__ tile, int ss,
                                                 int wave_u, uint32_t off) {
  using Lay = Bf16Layout<D>;
#pragma unroll
  for (int e = 0; e < D / (8 * NW); ++e)
    dma16(lds + 1024u * (NW * e + wave_u), tile + (int64_t)(64 * NW * e / Lay::CPR) * ss, off);
}

// The last tile of a sequence that ends inside it: rows past the end are read
// from the last row instead (finite data, masked or discarded later), so no
// load leaves the tensor.  Row offsets are per lane and per load here.
template <int D, bool IS_V, int NW = 2>
__device__ __forceinline__ void load_tile_lds_clamped(uint32_t lds, const uint16_t* __restrict__ tile,
                                                      int ss, int wave, int wave_u, int lane,
                                                      int rows_valid) {
  using Lay = Bf16Layout<D>;
  const int ql = 64 * wave + lane;
  const int pc = ql % Lay::CPR;
#pragma unroll
  for (int e = 0; e < D / (8 * NW); ++e) {
    const int r = 64 * NW * e / Lay::CPR + ql / Lay::CPR;  // the LDS row this lane fills
    const int gc = pc ^ (IS_V ? Lay::fv(r) : Lay::fk(r));
    const int rr = min(r, rows_valid - 1);
    dma16(lds + 1024u * (NW * e + wave_u), tile, (uint32_t)((rr * ss + 8 * gc) * 2));
  }
}

// Sparse rows read their key-block list through a 256-entry LDS window, so the
// loop issues no vector-memory loads of its own (whose waits would also drain
// the tile loads in flight).
constexpr int kListChunk = 256;
// Unsplit sparse rows hold up to this many list entries in LDS at once (a whole
// row of a 131072-token mask), so that a row can be walked in another order.
constexpr int kListWhole = 2048;

// Two workgroups' worth of wavefronts per SIMD (<= 256 registers per lane) so
// that one wavefront's softmax overlaps another's MFMA work.
//
// Pipeline per key tile n (one K and one V buffer, two barriers):
//   S = K_n Q^T from LDS                  (V_n landing)
//   wait + barrier A -> issue K_{n+1}     (V_n visible; K_n consumed)
//   softmax, O += V_n^T P^T from LDS      (K_{n+1} landing)
//   wait + barrier B -> issue V_{n+1}     (K_{n+1} visible; V_n consumed)
// Operand reads are issued two MFMAs ahead of their use.
//
// Softmax rescaling is lazy: the running max of a query only moves (and O, l
// are only rescaled) when some lane's tile max exceeds it by more than 2^8 in
// the exp2 domain; otherwise probabilities up to 2^8 are accumulated against
// the stale max, which leaves O / l unchanged.
//
// The dense instantiation also serves the ground-truth mode (a.gt set): a
// uniform runtime switch rather than a third instantiation.
//
// With SPLIT the workgroups are persistent: each walks its share of the split
// tasks (see SplitMap), computing one key range of a row per task.  A task
// stores the normalised partial output (bf16) and its log2-domain log-sum-exp
// in the range's partial slot, then counts itself in the row's arrival counter;
// the row's last task merges the partials (merge_row).  A row whose active
// tiles all lie in one range is written directly.
//
// RAGGED: the sequence ends inside its last tile (the clamped loads and the
// key mask past the end exist only in that instantiation).
//
// NH > 1 (rows shared by the query heads of a KV group: a mask shared by the
// group, or dense rows): the workgroup holds NH query heads of one group, two
// wavefronts each, for the same query block; each K/V tile is loaded once into
// LDS for all of them, which divides the K/V loads by NH.  The task map then
// counts head slots of NH heads.
template <int D, bool SPARSE, bool SPLIT, bool RAGGED, int NH = 1>
__global__ __launch_bounds__(128 * NH) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_fwd_bf16_kernel(KernelArgs ka) {
  using Lay = Bf16Layout<D>;
  constexpr int NW = 2 * NH;  // wavefronts
  static_assert(NH == 1 || !SPLIT, "shared-row workgroups serve unsplit rows");
  // K and V tiles in one array: the epilogue stages a query block's output
  // (64 rows of OSTR elements) through both
  __shared__ __attribute__((aligned(16))) uint16_t sKV[2 * Lay::TILE];
  uint16_t* const sK = sKV;
  uint16_t* const sV = sKV + Lay::TILE;
  constexpr int kWin = SPLIT ? kListChunk : kListWhole;  // entries of the LDS list window
  __shared__ uint16_t sList[SPARSE ? kWin : 1];
  __shared__ int sListN;  // entries of a row walked by residue classes
  __shared__ __attribute__((aligned(16))) float sL2[SPARSE ? 1 : 64 * NH];
  __shared__ int sLast;    // SPLIT: this task completed its row
  __shared__ int sTicket;  // SPLIT: the workgroup's next ticket of its queue

  const AttnArgs& a = ka.a;
  const int queue = SPLIT ? (int)(blockIdx.x % ka.split.nq) : 0;
  if constexpr (SPLIT) {
    if (threadIdx.x == 0) sTicket = __hip_atomic_fetch_add(a.split_tickets + queue, 1, __ATOMIC_RELAXED,
                                                           __HIP_MEMORY_SCOPE_AGENT);
  }
  // SPLIT: the next non-empty task of the workgroup's queue (false at the end).
  // Uniform: every thread takes the same path through its barriers.
  auto next_split_task = [&](Task& out) -> bool {
    for (;;) {
      __syncthreads();  // sTicket is set
      const int64_t task = (int64_t)sTicket * ka.split.nq + queue;
      __syncthreads();  // every thread has read the ticket before it is replaced
      if (task >= ka.split.total) return false;
      if (threadIdx.x == 0)  // the following task's ticket, drawn one task ahead
        sTicket = __hip_atomic_fetch_add(a.split_tickets + queue, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      out = decode_split(ka.split, task);
      const int32_t* bd = a.split_bounds + (((int64_t)out.b * a.heads_q + out.h) * a.n_blocks + out.i) *
                                               split_stride(a.split_parts);
      if (bd[out.p + 1] > bd[out.p]) return true;  // (a range without active tiles is no task)
    }
  };
  // SPLIT: a task is prefetched during the previous task's epilogue: its Q in
  // qf, its first list window in sList and its first K/V tile in sK / sV
  bf16x8 qf[D / 16];
  Task t_next;
  bool prefetched = false;
  for (;;) {  // SPLIT: tasks drawn from the queue; otherwise a single pass
  Task t;
  if constexpr (SPLIT) {
    if (prefetched) t = t_next;
    else if (!next_split_task(t)) break;
  } else {
    t = decode_task(ka.map, blockIdx.x + ka.task_base);
  }
  const bool pre = SPLIT && prefetched;
  const int tid = threadIdx.x;
  const int wave_all = tid / 64;                       // 0 .. NW - 1
  const int wave_u = __builtin_amdgcn_readfirstlane(wave_all);
  const int wave = wave_all % 2;                       // the query half of this wavefront's head
  const int h0 = t.h * NH;                             // first query head of the workgroup
  t.h = h0;                                            // (uniform: mask row and K/V group)
  const int hq = h0 + wave_all / 2;                    // this wavefront's query head
  const int lane = tid % 64;
  const int hf = lane / 32;
  const int col = lane % 32;
  const int G = a.heads_q / a.heads_kv;
  const int g = t.h / G;
  const int kss = (int)a.k.ss, vss = (int)a.v.ss;
  const uint32_t sK_a = lds_addr(sK), sV_a = lds_addr(sV);
  uint32_t koffd[2], voffd[2];
  if constexpr (NH == 1) {
    koffd[0] = dma_offset<D, false>(kss, wave, lane, 0);
    koffd[1] = dma_offset<D, false>(kss, wave, lane, 1);
    voffd[0] = dma_offset<D, true>(vss, wave, lane, 0);
    voffd[1] = dma_offset<D, true>(vss, wave, lane, 1);
  } else {
    koffd[0] = koffd[1] = dma_offset_nw<D, false, NW>(kss, wave_all, lane);
    voffd[0] = voffd[1] = dma_offset_nw<D, true, NW>(vss, wave_all, lane);
  }

  const uint16_t* qp = static_cast<const uint16_t*>(a.q.ptr) + t.b * a.q.sb + hq * a.q.sh;
  const uint16_t* kp = static_cast<const uint16_t*>(a.k.ptr) + t.b * a.k.sb + g * a.k.sh;
  const uint16_t* vp = static_cast<const uint16_t*>(a.v.ptr) + t.b * a.v.sb + g * a.v.sh;
  const int64_t ktile = 64 * a.k.ss, vtile = 64 * a.v.ss;

  // Q^T operand: lane holds query q0 + col, features 16ks + 8hf .. +7 (rows past
  // the end of the sequence read its last row and are never stored)
  const int S = a.seq_len;
  const int qrow = 64 * t.i + 32 * wave + col;
  const int qrow_c = min(qrow, S - 1);
  const int n_last = S - 64 * (a.n_blocks - 1);  // rows of the last tile
  constexpr bool ragged = RAGGED;
  if (!pre) {
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks)
      qf[ks] = *reinterpret_cast<const bf16x8*>(qp + (int64_t)qrow_c * a.q.ss + 16 * ks + 8 * hf);
  }

  f32x16 acc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[dt][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  float mc = 0.f;  // m_run * c, 0 while m_run is -inf (formed when m_run moves)
  const float c = ka.scale_log2;

  // Per-lane LDS element offsets of the operand reads.  K: row 32mt + col, chunk
  // 2ks + hf (the swizzle depends on col only; mt adds 32 rows).  V (transposed
  // read): rows 32(kt/2) + 16(kt%2) + {0, 8} + 4hf + r4, features 32dt + d0; the
  // swizzle depends on the lane only, the rest are immediate offsets.
  int koff[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) koff[ks] = col * D + 8 * ((2 * ks + hf) ^ Lay::fk(col));
  const int r16 = lane % 16;
  const int r4 = r16 / 4;
  const int d0 = 4 * (r16 % 4) + 16 * ((lane / 16) % 2);
  const int vrow = 4 * hf + r4;
  const int fvl = Lay::fv(vrow);
  int voff[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt) voff[dt] = vrow * D + 8 * ((4 * dt + d0 / 8) ^ fvl) + d0 % 8;

  // row list
  const RowList<SPARSE> list = make_list<SPARSE, SPLIT>(a, t);
  const bool pool = !SPARSE && !SPLIT && a.gt != nullptr;  // ground-truth mode
  const int64_t trow = ((int64_t)t.b * a.heads_q + hq) * a.n_blocks + t.i;  // this wavefront's head
  float* const rrow = pool ? a.pool_r + trow * a.n_blocks * 64 : nullptr;
  auto fetch_chunk = [&](int base) {  // mask entries [base, base + kWin) of the row, ascending
    if (SPARSE) {
      const int ne = list.n >> list.sh;
#pragma unroll
      for (int p = tid; p < kWin; p += 128 * NH)
        if (base + p < ne) sList[p] = list.idx[base + p];
    }
  };
  // last valid key block: j <= i when causal, j < nb always (i < nb); a dense
  // list is valid by construction
  const int jmax = a.causal ? t.i : a.n_blocks - 1;
  // Walk by residue classes (a.walk_classes = S > 1; unsplit rows of 64-token
  // masks held whole in LDS): the row visits its blocks j = S q + c in the order
  // (c, q), i.e. every row follows one common column order, in which runs of
  // adjacent blocks are spread apart.  Wavefront 0 partitions the ascending
  // list into the S classes, stable within each class (ballot ranks: the order,
  // and so every result, is deterministic); entries past jmax, the ascending
  // list's tail, are dropped.
  const int wcls = (SPARSE && !SPLIT && list.sh == 0 && list.n <= kWin && a.walk_classes > 1) ? a.walk_classes : 1;
  auto fetch_classes = [&]() {
    if (wave_all == 0) {
      const uint64_t lt = lanemask_lt();
      const int msk = wcls - 1;
      int cnt[16];
#pragma unroll
      for (int c = 0; c < 16; ++c) cnt[c] = 0;
      for (int k0 = 0; k0 < list.n; k0 += 64) {
        const int e = k0 + lane;
        const int v = e < list.n ? (int)list.idx[e] : 0;
        const bool ok = e < list.n && v <= jmax;
        const int cl = v & msk;
#pragma unroll
        for (int c = 0; c < 16; ++c)
          if (c < wcls) cnt[c] += __popcll(__ballot(ok && cl == c));
      }
      int run = 0;
#pragma unroll
      for (int c = 0; c < 16; ++c) {
        const int t0 = cnt[c];
        cnt[c] = run;  // first walk position of class c
        if (c < wcls) run += t0;
      }
      for (int k0 = 0; k0 < list.n; k0 += 64) {
        const int e = k0 + lane;
        const int v = e < list.n ? (int)list.idx[e] : 0;
        const bool ok = e < list.n && v <= jmax;
        const int cl = v & msk;
#pragma unroll
        for (int c = 0; c < 16; ++c) {
          if (c < wcls) {
            const uint64_t bal = __ballot(ok && cl == c);
            if (ok && cl == c) sList[cnt[c] + __popcll(bal & lt)] = (uint16_t)v;
            cnt[c] += __popcll(bal);
          }
        }
      }
      if (lane == 0) sListN = run;
    }
  };
  if (!pre) {
    if (wcls > 1) fetch_classes();
    else fetch_chunk(0);
  }
  __syncthreads();
  const int list_n = wcls > 1 ? sListN : list.n;  // tiles this row walks
  auto entry = [&](int p) -> int {  // p must lie in the current LDS window
    if (p >= list_n) return -1;
    if (!SPARSE) return list.lo + p;
    const int jj = ((int)sList[(p >> list.sh) % kWin] << list.sh) + (p & list.sh);
    return jj <= jmax ? jj : -1;
  };
  int j = entry(0);
  int jn = (j >= 0) ? entry(1) : -1;
  int n = 0;

  // S^T = K Q^T for the tile in sK (two 32-key halves).  With `interleave`,
  // the reads and MFMAs are issued in the same scheduling region as the
  // softmax VALU work of the previous tile (see below).
  constexpr int NS = 2 * (D / 16);
  auto s_product = [&](f32x16 (&sn)[2]) {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int e = 0; e < 16; ++e) sn[mt][e] = 0.f;
    // the two 32-key halves alternate, so consecutive MFMAs are independent
    bf16x8 kf[NS];
#pragma unroll
    for (int st = 0; st < NS; ++st)
      kf[st] = *reinterpret_cast<const bf16x8*>(sK + 32 * (st % 2) * D + koff[st / 2]);
#pragma unroll
    for (int st = 0; st < NS; ++st) {
      const int mt = st % 2, ks = st / 2;
      sn[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st], qf[ks], sn[mt], 0, 0, 0);
    }
  };

  auto load_k = [&](int jt) {
    if (RAGGED && jt == a.n_blocks - 1)
      load_tile_lds_clamped<D, false, NW>(sK_a, kp + jt * ktile, kss, wave_all, wave_u, lane, n_last);
    else if constexpr (NH == 1)
      load_tile_lds<D>(sK_a, kp + jt * ktile, kss, wave_u, koffd);
    else
      load_tile_lds_nw<D, NW>(sK_a, kp + jt * ktile, kss, wave_u, koffd[0]);
  };
  auto load_v = [&](int jt) {
    if (RAGGED && jt == a.n_blocks - 1)
      load_tile_lds_clamped<D, true, NW>(sV_a, vp + jt * vtile, vss, wave_all, wave_u, lane, n_last);
    else if constexpr (NH == 1)
      load_tile_lds<D>(sV_a, vp + jt * vtile, vss, wave_u, voffd);
    else
      load_tile_lds_nw<D, NW>(sV_a, vp + jt * vtile, vss, wave_u, voffd[0]);
  };

  // diagonal tile: key kl visible to query ql iff kl <= ql.  Without causality
  // the last tile of a sequence ending inside it hides its keys past the end
  // (with causality they are already hidden from every real query).
  auto mask_tile = [&](f32x16 (&s)[2], int jt) {
    const bool diag = a.causal && jt == t.i;
    const bool tail = ragged && !a.causal && jt == a.n_blocks - 1;
    if (diag || tail) {
      const int ql = 32 * wave + col;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kl = 32 * mt + 8 * (e / 4) + 4 * hf + (e % 4);
          if ((diag && kl > ql) || (tail && kl >= n_last)) s[mt][e] = -INFINITY;
        }
    }
  };
  // the row max of a tile per query: the two lane halves hold the two 32-key
  // halves of a query's tile row, exchanged in registers by v_permlane32_swap
  auto row_max = [&](const f32x16 (&s)[2]) -> float {
    float mx2[2] = {-INFINITY, -INFINITY};  // two independent max chains
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx2[mt] = fmaxf(mx2[mt], s[mt][e]);
    const float m = fmaxf(mx2[0], mx2[1]);
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
    return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
  };

  f32x16 sA[2], sB[2];
  float mloc = -INFINITY;  // row max of the tile in the current S buffer
  bool resc = false;       // whether that tile moves the running max
  if (j >= 0 && !pre) {
    load_k(j);
    load_v(j);
  }
  wait_loads();  // also retires the Q loads: nothing the loop body waits on is pending
  __syncthreads();
  if (j >= 0) {
    s_product(sA);
    mask_tile(sA, j);
    mloc = row_max(sA);
    resc = __ballot((mloc - m_run) * c > 8.0f) != 0;
  }
  __syncthreads();  // K_j consumed
  if (jn >= 0) load_k(jn);
  wait_loads();
  __syncthreads();  // K_jn (and V_j) visible

  // One tile j.  On entry: sc holds S for tile j, sK holds K_jn, sV holds V_j
  // (its load may still be in flight), a load of nothing else is pending.
  //   softmax(S_j) on VALU || S_jn = K_jn Q^T on MFMA      (one scheduling region)
  //   wait + barrier M -> issue K_jnn                       (V_j visible; K_jn consumed)
  //   O += V_j^T P_j^T
  //   wait + barrier E -> issue V_jn                        (K_jnn visible; V_j consumed)
  auto tile = [&](f32x16 (&sc)[2], f32x16 (&sn)[2]) {
    int jnn = -1;
    if (jn >= 0) {
      if (SPARSE && ((n + 2) & ((kWin << list.sh) - 1)) == 0 && n + 2 < list_n) {
        fetch_chunk((n + 2) >> list.sh);  // every thread has read entry n + 1 already
        wait_loads();
        __syncthreads();
      }
      jnn = entry(n + 2);
    }
    // online softmax (lazy rescale); tile j's masked row max and the rescale
    // decision were formed under the previous tile's P.V product
    if (resc) {
      const float m_new = fmaxf(m_run, mloc);
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c);
      m_run = m_new;
      mc = (m_run == -INFINITY) ? 0.f : m_run * c;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[dt][e] *= alpha;
    }

    // S for the next tile (harmless junk when there is none)
    s_product(sn);
    // P^T operand of k-step kt: accumulators 8(kt%2)..+7 of half kt/2, i.e. keys
    // 32(kt/2) + 16(kt%2) + {4hf + 0..3, 8 + 4hf + 0..3}
    bf16x8 pb[4];
    float ps[4];  // four independent partial sums, each started with its first term (the
                  // compiler keeps 0 + p as an add: p might be -0, which exp2 never returns)
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sc[kt / 2][8 * (kt % 2) + e], c, -mc));
        ps[kt] = e == 0 ? p : ps[kt] + p;
        pb[kt][e] = (__bf16)p;
      }
    l_run += (ps[0] + ps[1]) + (ps[2] + ps[3]);
    // schedule: four K reads ahead, then each MFMA of the next tile's S with
    // seven VALU instructions of this tile's softmax
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int st = 0; st < NS - 4; ++st) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 7, 0);
    }
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 7, 0);
    }
    // keep the softmax and the next S in this region: arithmetic is otherwise
    // free to sink past the barrier into the P.V region
    asm volatile("" ::"v"(pb[0]), "v"(pb[1]), "v"(pb[2]), "v"(pb[3]), "v"(l_run), "v"(sn[0]), "v"(sn[1]));
    wait_loads();
    __syncthreads();  // M: V_j visible, K_jn consumed
    // the P.V product runs at raised wave priority: of the two wavefronts sharing
    // a SIMD, the one feeding the matrix core issues first (measured: sparse
    // 128k 19.8 -> 18.3 ms, dense split -1%)
    __builtin_amdgcn_s_setprio(2);
    if (jnn >= 0) load_k(jnn);
    // ground truth: this tile's row max (Eq. 5), completed with the K load by barrier E
    if (pool && hf == 0) rrow[(int64_t)j * 64 + 32 * wave + col] = mloc;

    // O^T += V^T P^T; V^T operand: feature 32dt + col, the same keys as pb[kt]
    // feature tiles dt alternate, so consecutive MFMAs are independent
    auto vread = [&](int st) -> bf16x8 {
      const int dt = st % (D / 32), kt = st / (D / 32);
      const int rows = 32 * (kt / 2) + 16 * (kt % 2);
      const uint16_t* base = sV + rows * D + voff[dt];
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)base);
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4*)(base + 8 * D));
      return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    };
    if (jn >= 0) mask_tile(sn, jn);
    constexpr int NV = 4 * (D / 32);
    bf16x8 vf0 = vread(0), vf1 = vread(1);
#pragma unroll
    for (int st = 0; st < NV; ++st) {
      bf16x8 vf2;
      if (st + 2 < NV) vf2 = vread(st + 2);
      acc[st % (D / 32)] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf0, pb[st / (D / 32)], acc[st % (D / 32)], 0, 0, 0);
      vf0 = vf1;
      vf1 = vf2;
    }
    const float mloc_n = row_max(sn);
    // schedule: transposed V reads run two MFMAs ahead, the next tile's row max
    // fills VALU slots between the MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int st = 0; st < NV - 2; ++st) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    resc = __ballot((mloc_n - m_run) * c > 8.0f) != 0;
    wait_loads();
    __builtin_amdgcn_s_setprio(0);
    __syncthreads();  // E: V_j consumed, K_jnn visible
    if (jn >= 0) load_v(jn);
    mloc = mloc_n;
    j = jn;
    jn = jnn;
    ++n;
  };

  // unrolled twice so that the two S buffers swap roles without copies
  while (j >= 0) {
    tile(sA, sB);
    if (j < 0) break;
    tile(sB, sA);
  }

  // epilogue: normalise, stage through LDS, store rows with 16-byte writes
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = (l_tot > 0.f) ? 1.0f / l_tot : 0.f;
  if constexpr (SPLIT) {
    // The next task first: its Q, first list window and first K/V tile load
    // while this task writes its output and counts itself in its row (qf, sK
    // and sV are free: every tile of this task has been consumed).
    Task nx;
    prefetched = next_split_task(nx);
    uint16_t lw[kListChunk / 128];  // this thread's entries of the next list window
    if (prefetched) {
      t_next = nx;
      const int gx = nx.h / G;
      const int64_t xrow = ((int64_t)nx.b * a.heads_q + nx.h) * a.n_blocks + nx.i;
      const int32_t* bx = a.split_bounds + xrow * split_stride(a.split_parts) + nx.p;
      int j0;
      if constexpr (SPARSE) {
        const int s0 = bx[0], cnt = bx[1] - s0;
        const uint16_t* li = a.idx + xrow * a.n_blocks + s0;  // (the split runs on per-head 64-token masks)
#pragma unroll
        for (int u = 0; u < kListChunk / 128; ++u) {
          const int e = tid + 128 * u;
          lw[u] = e < cnt ? li[e] : (uint16_t)0;
        }
        j0 = li[0];
      } else {
        j0 = nx.p * a.split_w;
      }
      const uint16_t* qx = static_cast<const uint16_t*>(a.q.ptr) + nx.b * a.q.sb + nx.h * a.q.sh;
      const int qr = min(64 * nx.i + 32 * wave + col, S - 1);
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks)
        qf[ks] = *reinterpret_cast<const bf16x8*>(qx + (int64_t)qr * a.q.ss + 16 * ks + 8 * hf);
      if (j0 <= nx.i) {  // a valid first block (the task's list re-checks every entry)
        const uint16_t* kx = static_cast<const uint16_t*>(a.k.ptr) + nx.b * a.k.sb + gx * a.k.sh + j0 * ktile;
        const uint16_t* vx = static_cast<const uint16_t*>(a.v.ptr) + nx.b * a.v.sb + gx * a.v.sh + j0 * vtile;
        if (RAGGED && j0 == a.n_blocks - 1) {
          load_tile_lds_clamped<D, false, NW>(sK_a, kx, kss, wave_all, wave_u, lane, n_last);
          load_tile_lds_clamped<D, true, NW>(sV_a, vx, vss, wave_all, wave_u, lane, n_last);
        } else {
          load_tile_lds<D>(sK_a, kx, kss, wave_u, koffd);
          load_tile_lds<D>(sV_a, vx, vss, wave_u, voffd);
        }
      }
    }
    // this task's output, straight from the accumulators: the row's output (a
    // row whose active tiles all lie in one range) or the task's partial
    const int32_t* bd = a.split_bounds + trow * split_stride(a.split_parts);
    const int nne = bd[a.split_parts + 1];
    const int ql = 32 * wave + col;
    if (nne == 1) {
      if (qrow < S) {
        uint16_t* dst = static_cast<uint16_t*>(a.o) + t.b * a.osb + t.h * a.osh + (int64_t)qrow * a.oss + 4 * hf;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            bf16x4 o4;
#pragma unroll
            for (int r = 0; r < 4; ++r) o4[r] = (__bf16)(acc[dt][4 * jj + r] * inv);
            *reinterpret_cast<bf16x4*>(dst + 32 * dt + 8 * jj) = o4;
          }
        if (a.lse && hf == 0)
          a.lse[((int64_t)t.b * a.heads_q + t.h) * (int64_t)S + qrow] =
              (l_tot > 0.f) ? m_run * a.scale + __logf(l_tot) : -INFINITY;
      }
    } else {
      const int64_t slot = ((int64_t)t.b * a.heads_q + t.h) * a.split_slots + split_offset(t.i, a.split_w) + t.p;
      uint16_t* dst = a.part_o + slot * 64 * D;
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          bf16x4 o4;
#pragma unroll
          for (int r = 0; r < 4; ++r) o4[r] = (__bf16)(acc[dt][4 * jj + r] * inv);
          store_dev(dst + part_index(D, wave, dt, jj, lane), __builtin_bit_cast(uint64_t, o4));
        }
      if (hf == 0) store_dev(a.part_lse + slot * 64 + ql, (l_tot > 0.f) ? m_run * c + __log2f(l_tot) : -INFINITY);
      // every thread's partial stores have completed (device scope) before the
      // task counts itself in the row; the row's last task merges (no task ever
      // waits for another)
      wait_loads();
      __syncthreads();
      if (tid == 0) {
        int32_t* cnt = const_cast<int32_t*>(bd) + a.split_parts + 2;
        sLast = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nne - 1;
      }
      __syncthreads();
      if (sLast) merge_row<D>(a, t.b, t.h, t.i, bd, wave, lane);
    }
    if (!prefetched) break;
    if constexpr (SPARSE) {
      wait_loads();  // the list entries have arrived (the next task's first barrier publishes them)
#pragma unroll
      for (int u = 0; u < kListChunk / 128; ++u) sList[tid + 128 * u] = lw[u];
    }
    continue;  // the next task
  }
  wait_loads();
  uint16_t* sO = sKV;  // 2 tiles of staging room
  const int ql = 32 * wave + col;
  const int rows_out = !RAGGED ? 64 : min(64, S - 64 * t.i);  // rows past the end are not stored
  // the workgroup's heads take turns with the staging room (one query block each)
#pragma unroll
  for (int hs = 0; hs < NH; ++hs) {
    __syncthreads();
    if (wave_all / 2 == hs) {
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          bf16x4 o4;
#pragma unroll
          for (int r = 0; r < 4; ++r) o4[r] = (__bf16)(acc[dt][4 * jj + r] * inv);
          *reinterpret_cast<bf16x4*>(sO + ql * Lay::OSTR + 32 * dt + 8 * jj + 4 * hf) = o4;
        }
    }
    __syncthreads();
    uint16_t* op = static_cast<uint16_t*>(a.o) + t.b * a.osb + (h0 + hs) * a.osh + (int64_t)64 * t.i * a.oss;
#pragma unroll
    for (int e = 0; e < 64 * Lay::CPR / (128 * NH); ++e) {
      const int q = tid + 128 * NH * e;
      const int r = q / Lay::CPR, cc = q % Lay::CPR;
      if (r < rows_out)
        *reinterpret_cast<u32x4*>(op + (int64_t)r * a.oss + 8 * cc) =
            *reinterpret_cast<const u32x4*>(sO + r * Lay::OSTR + 8 * cc);
    }
  }
  if (a.lse && hf == 0 && qrow < S) {
    const float lse = (l_tot > 0.f) ? m_run * a.scale + __logf(l_tot) : -INFINITY;
    a.lse[((int64_t)t.b * a.heads_q + hq) * (int64_t)S + qrow] = lse;
  }
  if (pool) {
    // padding rows take no part in the column max
    if (hf == 0) sL2[64 * (wave_all / 2) + ql] = (l_tot > 0.f && qrow < S) ? m_run * c + __log2f(l_tot) : INFINITY;
    wait_loads();  // the row-max stores of this workgroup have completed
    __syncthreads();
#pragma unroll
    for (int hs = 0; hs < NH; ++hs) {
      const int64_t hrow = ((int64_t)t.b * a.heads_q + h0 + hs) * a.n_blocks + t.i;
      pool_epilogue(a.pool_r + hrow * a.n_blocks * 64, sL2 + 64 * hs, c, list.n, a.n_blocks,
                    a.gt + hrow * a.n_blocks, tid, 128 * NH);
    }
  }
  if constexpr (!SPLIT) {
    break;
  }
  }  // task loop
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
  __shared__ __attribute__((aligned(16))) float sL2[64];

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

  const int S = a.seq_len;
  const int qrow = 64 * t.i + 32 * wave + col;
  const int qrow_c = min(qrow, S - 1);  // rows past the end read the last row, never stored
  const int n_last = S - 64 * (a.n_blocks - 1);
  const bool ragged = n_last < 64;
  f32x4 qf[D / 8];  // features 8u + 4hf .. +3 of this lane's query
#pragma unroll
  for (int u = 0; u < D / 8; ++u)
    qf[u] = *reinterpret_cast<const f32x4*>(qp + (int64_t)qrow_c * a.q.ss + 8 * u + 4 * hf);

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
  const bool pool = a.gt != nullptr;  // the launcher enables it for dense rows only
  const int64_t trow = ((int64_t)t.b * a.heads_q + t.h) * a.n_blocks + t.i;
  float* const rrow = pool ? a.pool_r + trow * a.n_blocks * 64 : nullptr;
  for (int n = 0; n < n_tiles; ++n) {
    const int j = sparse ? sl.at(n) : dl.at(n);
    if (!(sparse ? sl.ok(j) : dl.ok(j))) break;
    __syncthreads();
    constexpr int CPR = D / 4;
#pragma unroll
    for (int e = 0; e < 64 * CPR / 128; ++e) {
      const int q = tid + 128 * e;
      const int key = q / CPR, cc = q % CPR;
      const int krow = min(64 * j + key, S - 1);  // clamped inside the last tile
      *reinterpret_cast<f32x4*>(sK + key * KS + 4 * cc) =
          *reinterpret_cast<const f32x4*>(kp + (int64_t)krow * a.k.ss + 4 * cc);
      *reinterpret_cast<f32x4*>(sV + key * VS + 4 * cc) =
          *reinterpret_cast<const f32x4*>(vp + (int64_t)krow * a.v.ss + 4 * cc);
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
    const bool diag = a.causal && j == t.i;
    const bool tail = ragged && !a.causal && j == a.n_blocks - 1;
    if (diag || tail) {
      const int ql = 32 * wave + col;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kl = 32 * mt + 8 * (e / 4) + 4 * hf + (e % 4);
          if ((diag && kl > ql) || (tail && kl >= n_last)) s[mt][e] = -INFINITY;
        }
    }
    float rmax;
    const float alpha = softmax_tile(s, m_run, l_run, c, rmax);
    if (pool && hf == 0) rrow[(int64_t)j * 64 + 32 * wave + col] = rmax;  // Eq. 5
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
  if (qrow < S) {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        f32x4 o4;
#pragma unroll
        for (int r = 0; r < 4; ++r) o4[r] = acc[dt][4 * jj + r] * inv;
        *reinterpret_cast<f32x4*>(op + 32 * dt + 8 * jj + 4 * hf) = o4;
      }
  }
  if (a.lse && hf == 0 && qrow < S) {
    const float lse = (l_tot > 0.f) ? m_run * a.scale + __logf(l_tot) : -INFINITY;
    a.lse[((int64_t)t.b * a.heads_q + t.h) * (int64_t)S + qrow] = lse;
  }
  if (pool) {
    if (hf == 0) sL2[32 * wave + col] = (l_tot > 0.f && qrow < S) ? m_run * c + __log2f(l_tot) : INFINITY;
    __threadfence_block();
    __syncthreads();
    pool_epilogue(rrow, sL2, c, n_tiles, a.n_blocks, a.gt + trow * a.n_blocks, tid, 128);
  }
}

// ---------------------------------------------------------------------------
// key-range split: list bounds and the merge of partial results
// ---------------------------------------------------------------------------

// One wavefront per row (batch, head, query block) of a split launch.  Writes
// the row's record (split_stride(P) ints): bounds[p], p = 0 .. P, the list
// position of range p's first entry (ranges hold blocks [p w, p w + w); a list
// is ascending, and its valid entries are those below limit: i + 1 when
// causal, nb otherwise), then the number of non-empty ranges, then a zeroed
// arrival counter.  Dense rows record key blocks (position j is block j).  A
// row without any active block gets O = 0 and LSE = -inf here: no task writes
// it.
template <int D>
__global__ __launch_bounds__(256) void split_bounds_kernel(AttnArgs a) {
  const int wave = threadIdx.x / 64;
  const int lane = threadIdx.x % 64;
  const int64_t rows = (int64_t)a.batch * a.heads_q * a.n_blocks;
  const int64_t row = (int64_t)blockIdx.x * 4 + wave;
  if (row >= rows) return;
  const int nb = a.n_blocks;
  const int i = (int)(row % nb);
  const int w = a.split_w;
  const int P = a.split_parts;
  const int limit = a.causal ? i + 1 : nb;
  const bool sparse = a.count != nullptr;  // the split runs on per-head 64-token masks
  const int n = sparse ? min(max(a.count[row], 0), nb) : 0;
  const uint16_t* L = sparse ? a.idx + row * nb : nullptr;
  auto lower = [&](int key) -> int {  // list entries below key (key <= limit)
    if (!sparse) return key;
    int lo = 0, hi = n;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if ((int)L[mid] < key) lo = mid + 1;
      else hi = mid;
    }
    return lo;
  };
  int32_t* rec = a.split_bounds + row * split_stride(P);
  if (row == 0 && lane < 8) a.split_tickets[lane] = 0;  // the task queues start empty
  int nne = 0;
  for (int p0 = 0; p0 <= P; p0 += 64) {
    const int p = p0 + lane;
    int bp = 0, bn = 0;
    if (p <= P) {
      bp = lower(min(p * w, limit));
      rec[p] = bp;
    }
    if (p < P) bn = lower(min((p + 1) * w, limit));
    nne += __popcll(__ballot(p < P && bn > bp));
  }
  if (lane == 0) {
    rec[P + 1] = nne;
    rec[P + 2] = 0;
  }
  if (nne == 0) {
    const int b = (int)(row / ((int64_t)a.heads_q * nb)), h = (int)(row / nb % a.heads_q);
    const int t = 64 * i + lane;
    if (t < a.seq_len) {
      uint16_t* op = static_cast<uint16_t*>(a.o) + b * a.osb + h * a.osh + (int64_t)t * a.oss;
#pragma unroll
      for (int u = 0; u < D / 8; ++u) *reinterpret_cast<u32x4*>(op + 8 * u) = u32x4{0u, 0u, 0u, 0u};
      if (a.lse) a.lse[((int64_t)b * a.heads_q + h) * a.seq_len + t] = -INFINITY;
    }
  }
}

// Groups per phase: the largest power of two whose K + V stay within 32 MiB;
// each group is then spread over R = 8 / gpp XCDs.  Measured at 131072 tokens
// (64 MiB of K + V per group): one group at a time over all 8 XCDs beat one
// group per XCD by 11% (sparse) and 7% (dense).  At 65536 tokens with 7 query
// heads per KV group and per-head densities of 5-40% (32 MiB per group), one
// group at a time over all 8 XCDs beat two groups on 4 XCDs each by 17%: the
// groups' unequal work no longer leaves half the XCDs idle at the end; 8k and
// 32k shapes (4 and 16 MiB per group) ran the same with budgets of 32 and 64 MiB,
// and slower with 16 or less.
#ifndef SEER_KV_PHASE_BUDGET_MB
#define SEER_KV_PHASE_BUDGET_MB 32
#endif
static TaskMap make_map(const AttnArgs& a) {
  TaskMap m;
  m.batch = a.batch;
  m.heads_q = a.heads_q;
  m.heads_kv = a.heads_kv;
  m.nb = a.n_blocks;
  m.R = 0;
  m.gpp = 0;
  m.tpp = 0;
  const int slices = a.batch * a.heads_kv;
  const int G = a.heads_q / a.heads_kv;
  const double kv_bytes = 2.0 * a.n_blocks * 64.0 * a.head_dim * (a.bf16 ? 2 : 4);
  const double budget = SEER_KV_PHASE_BUDGET_MB * 1024.0 * 1024.0;
  for (int gpp = 8; gpp >= 1; gpp /= 2) {
    const int R = 8 / gpp;
    if (slices % gpp != 0 || a.n_blocks % R != 0) continue;
    if (gpp > 1 && gpp * kv_bytes > budget) continue;
    m.R = R;
    m.gpp = gpp;
    m.tpp = (a.n_blocks / R) * G;
    break;
  }
  return m;
}

}  // namespace

// Width of a split range in key blocks: the K and V of one range fill at most
// an XCD's L2 (4 MB), i.e. 128 blocks at head_dim 128 in bf16 and 256 at head
// dim 64, unless `width` (> 0) sets it.  Rows are split only when asked
// (`want`) and only when a row can reach more than one range.  0: no split.
constexpr int64_t kL2Bytes = 4 << 20;
int split_width(int n_blocks, int head_dim, bool causal, bool bf16, bool want, int width) {
  if (!want || !causal || !bf16) return 0;
  const int w = width > 0 ? width : (int)(kL2Bytes / (2 * 64 * (int64_t)head_dim * 2));
  return n_blocks > w ? w : 0;
}

int64_t split_slots_per_head(int n_blocks, int w) {
  const int64_t q = n_blocks / w, r = n_blocks % w;
  return n_blocks + w * q * (q - 1) / 2 + r * q;
}

// Workgroups of a kernel that the GPU holds at once (compute units x
// occupancy), queried once per device and kernel and kept for the process.
static int resident_capacity(const void* fn, int threads) {
  struct Entry {
    const void* fn;
    int dev, value;
  };
  static std::mutex mu;
  static Entry cache[64];
  static int used = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  {
    std::lock_guard<std::mutex> lk(mu);
    for (int k = 0; k < used; ++k)
      if (cache[k].fn == fn && cache[k].dev == dev) return cache[k].value;
  }
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, 0) != hipSuccess)
    return 0;
  const int value = cus * per_cu;
  std::lock_guard<std::mutex> lk(mu);
  if (used < 64) cache[used++] = Entry{fn, dev, value};
  return value;
}

// Launch helper: with a non-null `count` the launch is only counted (the
// launch-count query), otherwise it is issued on the stream.
#define SEER_LAUNCH(kernel, grid, block, stream, count, ...)                      \
  do {                                                                            \
    if (count) ++*(count);                                                        \
    else hipLaunchKernelGGL(kernel, grid, block, 0, stream, __VA_ARGS__);         \
  } while (0)

template <int D, bool RAGGED>
static hipError_t launch_split(const KernelArgs& ka, bool sparse, hipStream_t s, int* count) {
  const AttnArgs& a = ka.a;
  const int64_t rows = (int64_t)a.batch * a.heads_q * a.n_blocks;
  if (!count) hipLaunchKernelGGL(split_bounds_kernel<D>, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, a);
  const void* fn = sparse ? reinterpret_cast<const void*>(attn_fwd_bf16_kernel<D, true, true, RAGGED>)
                          : reinterpret_cast<const void*>(attn_fwd_bf16_kernel<D, false, true, RAGGED>);
  int64_t grid = resident_capacity(fn, 128);
  if (grid <= 0) grid = 1024;
  grid = std::min<int64_t>(grid, ka.split.total);
  KernelArgs kq = ka;
  kq.split.nq = (int)std::min<int64_t>(8, grid);
  if (sparse) SEER_LAUNCH((attn_fwd_bf16_kernel<D, true, true, RAGGED>), dim3((unsigned)grid), dim3(128), s, count, kq);
  else SEER_LAUNCH((attn_fwd_bf16_kernel<D, false, true, RAGGED>), dim3((unsigned)grid), dim3(128), s, count, kq);
  return count ? hipSuccess : hipGetLastError();
}

static hipError_t launch_attn_one(const AttnArgs& a, hipStream_t s, int* count);

// One launch per KV group when a phase of the task order holds a single group
// (its K and V alone fill the phase's cache budget): the launch boundary keeps
// every XCD on the same group's K and V.  Measured at 131072 tokens (sparse):
// 8 launches 17.8 ms, one launch 18.1 ms.  Not for the split or pooling modes.
hipError_t launch_attn(const AttnArgs& a, hipStream_t s, int* count) {
  const int groups = a.batch * a.heads_kv;
  if (a.split_w > 0 || a.gt != nullptr || groups <= 1 || make_map(a).gpp != 1)
    return launch_attn_one(a, s, count);
  const int G = a.heads_q / a.heads_kv;
  const int64_t es = a.bf16 ? 2 : 4;
  const int nbm = a.mask_blocks;
  for (int b = 0; b < a.batch; ++b)
    for (int g = 0; g < a.heads_kv; ++g) {
      const int h0 = g * G;
      AttnArgs c = a;
      c.batch = 1;
      c.heads_kv = 1;
      c.heads_q = G;
      c.q.ptr = static_cast<const char*>(a.q.ptr) + es * (b * a.q.sb + h0 * a.q.sh);
      c.k.ptr = static_cast<const char*>(a.k.ptr) + es * (b * a.k.sb + g * a.k.sh);
      c.v.ptr = static_cast<const char*>(a.v.ptr) + es * (b * a.v.sb + g * a.v.sh);
      c.o = static_cast<char*>(a.o) + es * (b * a.osb + h0 * a.osh);
      const int64_t hrow = (int64_t)b * a.heads_q + h0;  // first query head of the group
      if (a.lse) c.lse = a.lse + hrow * a.seq_len;
      if (a.count) {
        const int64_t mrow = a.mask_kv ? (int64_t)b * a.heads_kv + g : hrow;  // first mask row set
        c.count = a.count + mrow * nbm;
        c.idx = a.idx + mrow * nbm * nbm;
      }
      const hipError_t e = launch_attn_one(c, s, count);
      if (e != hipSuccess) return e;
    }
  return hipSuccess;
}

// Query heads per workgroup for rows shared by the query heads of a KV group
// (a mask shared by the group, or dense rows): the largest of 4, 2 that divides
// the group and is at most a.heads_per_wg (the option's cap, 2 by default),
// else 1.  Measured at 131072 tokens, 32 query / 8 KV heads, TopK 0.1: per-head
// rows 17.3 ms; shared rows with 1, 2 and 4 heads per workgroup 14.3, 13.0 and
// 13.1 ms (two 4-wavefront workgroups per CU keep their phases independent;
// one 8-wavefront workgroup moves in lockstep).
static int kv_heads_per_wg(const AttnArgs& a) {
  const bool shared_rows = a.count ? a.mask_kv : true;
  if (!shared_rows || !a.bf16 || a.split_w > 0) return 1;
  const int G = a.heads_q / a.heads_kv;
  for (int nh = 4; nh >= 2; nh /= 2)
    if (nh <= a.heads_per_wg && G % nh == 0) return nh;
  return 1;
}

template <int D, bool SPARSE, bool RAGGED>
static void launch_nh(const KernelArgs& ka, int nh, dim3 grid, hipStream_t s, int* count) {
  if (nh == 4) SEER_LAUNCH((attn_fwd_bf16_kernel<D, SPARSE, false, RAGGED, 4>), grid, dim3(512), s, count, ka);
  else SEER_LAUNCH((attn_fwd_bf16_kernel<D, SPARSE, false, RAGGED, 2>), grid, dim3(256), s, count, ka);
}

template <int D>
static void launch_nh_d(const KernelArgs& ka, int nh, bool sparse, bool ragged, dim3 grid, hipStream_t s,
                        int* count) {
  if (sparse) {
    if (ragged) launch_nh<D, true, true>(ka, nh, grid, s, count);
    else launch_nh<D, true, false>(ka, nh, grid, s, count);
  } else {
    if (ragged) launch_nh<D, false, true>(ka, nh, grid, s, count);
    else launch_nh<D, false, false>(ka, nh, grid, s, count);
  }
}

// Sparse rows of long sequences launch in batches of exactly the workgroups the
// GPU holds at once (4 per CU), so that the rows of a batch start together and
// walk their ascending lists roughly in step: concurrent rows then share more
// of their K/V tiles in L2.  Within a batch the order is the usual one (task
// ids continue across batches), so every output is unchanged.  Only the
// heaviest quarter of the tasks is batched: the later batches' shorter rows
// leave too much idle time at their ends.  Measured at 131072 tokens (32 q / 8
// KV heads, TopK 0.1), walking ascending: 17.29 ms unbatched, 16.92 ms with
// every task batched, 16.65 ms with the heavier half batched; with the walk by
// residue classes (one GPU, back to back; batched fraction none / 1/8 / 1/4 / 3/8 / 1/2 /
// 3/4 / all): 14.47-14.53, 14.33-14.36, 14.24-14.33, 14.30-14.35, 14.41-14.51,
// 14.67, 14.83 ms; 48.9 -> 48.2 ms (all batched) with per-head
// densities spread over 5-40%; at 32768 tokens the batch ends' idle time
// outweighed the gain (1.84 -> 2.06 ms; at 65536 tokens with 7 heads of 5-40%
// density 7.6 -> 10.6 ms), hence the size threshold (a.batch_min_blocks, 2048
// blocks by default).  a.batch_wgs > 0 sets the batch size instead.
static int batch_size(const AttnArgs& a, bool ragged) {
  if (a.batch_wgs > 0) return a.batch_wgs / 8 * 8;  // a multiple of 8 keeps the XCD interleave
  const void* fn = a.head_dim == 128
                       ? (ragged ? reinterpret_cast<const void*>(attn_fwd_bf16_kernel<128, true, false, true>)
                                 : reinterpret_cast<const void*>(attn_fwd_bf16_kernel<128, true, false, false>))
                       : (ragged ? reinterpret_cast<const void*>(attn_fwd_bf16_kernel<64, true, false, true>)
                                 : reinterpret_cast<const void*>(attn_fwd_bf16_kernel<64, true, false, false>));
  return resident_capacity(fn, 128) / 8 * 8;
}

static hipError_t launch_attn_one(const AttnArgs& a, hipStream_t s, int* count) {
  KernelArgs ka;
  ka.a = a;
  const int nh = kv_heads_per_wg(a);
  const auto done = [&]() { return count ? hipSuccess : hipGetLastError(); };
  if (nh > 1) {  // tasks over head slots of nh heads: the task order sees heads_q / nh heads
    AttnArgs v = a;
    v.heads_q = a.heads_q / nh;
    ka.map = make_map(v);
    const int64_t total = (int64_t)a.batch * v.heads_q * a.n_blocks;
    if (total == 0) return hipSuccess;
    ka.split = SplitMap{a.heads_q, a.heads_kv, a.n_blocks, 0, 0, 0, 0, 1};
    ka.scale_log2 = a.scale * kLog2e;
    ka.task_base = 0;
    const bool sparse = a.count != nullptr;
    if (a.seq_len <= 0 || (a.n_blocks - 1) * 64 >= a.seq_len || a.n_blocks * 64 < a.seq_len ||
        (a.gt != nullptr && (sparse || !a.pool_r)))
      return hipErrorInvalidValue;
    const bool ragged = a.seq_len % 64 != 0;
    const dim3 grid((unsigned)total);
    if (a.head_dim == 128) launch_nh_d<128>(ka, nh, sparse, ragged, grid, s, count);
    else if (a.head_dim == 64) launch_nh_d<64>(ka, nh, sparse, ragged, grid, s, count);
    else return hipErrorInvalidValue;
    return done();
  }
  ka.map = make_map(a);
  ka.split = SplitMap{a.heads_q, a.heads_kv, a.n_blocks, a.split_w, a.split_parts, 0, 0, 1};
  if (a.split_w > 0) {
    const int64_t G = a.heads_q / a.heads_kv, P = a.split_parts, w = a.split_w;
    ka.split.per_group = G * (P * a.n_blocks - w * P * (P - 1) / 2);
    ka.split.total = ka.split.per_group * a.batch * a.heads_kv;
  }
  ka.scale_log2 = a.scale * kLog2e;
  ka.task_base = 0;
  const int64_t total = (int64_t)a.batch * a.heads_q * a.n_blocks;
  if (total == 0) return hipSuccess;
  dim3 grid((unsigned)total), block(128);
  const bool sparse = a.count != nullptr;
  const bool pool = a.gt != nullptr;
  const bool ragged = a.seq_len % 64 != 0;  // the last tile is partial
  if ((sparse && pool) || (pool && !a.pool_r)) return hipErrorInvalidValue;
  if (a.seq_len <= 0 || (a.n_blocks - 1) * 64 >= a.seq_len || a.n_blocks * 64 < a.seq_len)
    return hipErrorInvalidValue;  // n_blocks must be ceil(seq_len / 64)
  if (a.split_w > 0) {
    // the geometry must be the one split_width chose, with every buffer present
    const int P = a.split_parts;
    if (pool || !a.bf16 || !a.causal || (sparse && (a.mask_shift != 0 || a.mask_kv)) || a.split_w < 1 ||
        P != (a.n_blocks + a.split_w - 1) / a.split_w || P < 2 || !a.part_lse || !a.part_o ||
        !a.split_bounds || !a.split_tickets || a.split_slots != split_slots_per_head(a.n_blocks, a.split_w))
      return hipErrorInvalidValue;
    if (a.head_dim == 128)
      return ragged ? launch_split<128, true>(ka, sparse, s, count) : launch_split<128, false>(ka, sparse, s, count);
    if (a.head_dim == 64)
      return ragged ? launch_split<64, true>(ka, sparse, s, count) : launch_split<64, false>(ka, sparse, s, count);
    return hipErrorInvalidValue;
  }
  if (a.bf16 && sparse && !pool && a.batch_min_blocks > 0 && a.n_blocks >= a.batch_min_blocks) {
    const int E = batch_size(a, ragged);
    if (E > 0 && total > E) {
      // the heaviest quarter of the tasks (the longest rows) in batches, the
      // rest (whose shorter rows would leave batch ends idle) in one launch
      const int64_t batched = (total / 4 + E - 1) / E * E;
      for (int64_t b0 = 0, cnt = 0; b0 < total; b0 += cnt) {
        cnt = b0 < batched ? std::min<int64_t>(E, total - b0) : total - b0;
        ka.task_base = (int)b0;
        const dim3 g((unsigned)cnt);
        if (a.head_dim == 128) {
          if (ragged) SEER_LAUNCH((attn_fwd_bf16_kernel<128, true, false, true>), g, block, s, count, ka);
          else SEER_LAUNCH((attn_fwd_bf16_kernel<128, true, false, false>), g, block, s, count, ka);
        } else {
          if (ragged) SEER_LAUNCH((attn_fwd_bf16_kernel<64, true, false, true>), g, block, s, count, ka);
          else SEER_LAUNCH((attn_fwd_bf16_kernel<64, true, false, false>), g, block, s, count, ka);
        }
      }
      return done();
    }
  }
  if (a.bf16) {
    if (a.head_dim == 128) {
      if (ragged) {
        if (sparse) SEER_LAUNCH((attn_fwd_bf16_kernel<128, true, false, true>), grid, block, s, count, ka);
        else SEER_LAUNCH((attn_fwd_bf16_kernel<128, false, false, true>), grid, block, s, count, ka);
      } else {
        if (sparse) SEER_LAUNCH((attn_fwd_bf16_kernel<128, true, false, false>), grid, block, s, count, ka);
        else SEER_LAUNCH((attn_fwd_bf16_kernel<128, false, false, false>), grid, block, s, count, ka);
      }
    } else if (a.head_dim == 64) {
      if (ragged) {
        if (sparse) SEER_LAUNCH((attn_fwd_bf16_kernel<64, true, false, true>), grid, block, s, count, ka);
        else SEER_LAUNCH((attn_fwd_bf16_kernel<64, false, false, true>), grid, block, s, count, ka);
      } else {
        if (sparse) SEER_LAUNCH((attn_fwd_bf16_kernel<64, true, false, false>), grid, block, s, count, ka);
        else SEER_LAUNCH((attn_fwd_bf16_kernel<64, false, false, false>), grid, block, s, count, ka);
      }
    } else {
      return hipErrorInvalidValue;
    }
  } else {
    if (a.head_dim == 128) SEER_LAUNCH(attn_fwd_f32_kernel<128>, grid, block, s, count, ka, (int)sparse);
    else if (a.head_dim == 64) SEER_LAUNCH(attn_fwd_f32_kernel<64>, grid, block, s, count, ka, (int)sparse);
    else return hipErrorInvalidValue;
  }
  return done();
}

}  // namespace seer
