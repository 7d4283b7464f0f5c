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

// Key-range split.  Each causal row is cut into P ranges of w key blocks
// (P w = nb); range p of row i exists when p w <= i.  Workgroup w runs on XCD
// x = w % 8 as that XCD's (w / 8)-th task, and KV groups (batch x KV head) are
// processed in order.  Every XCD gets the same causal work:
//  - P = 16: within each group, XCD x takes range x and then range 15 - x;
//  - P = 8: groups go in pairs, XCD x taking range x of the first and range
//    7 - x of the second (the XCDs then drift apart by up to a group, whose
//    K and V the Infinity Cache holds).
// Within a range: every query head of the group and every query block that
// reaches the range, heaviest first.  An XCD thus reads w key blocks of K and
// V at a time, which its L2 holds.
struct SplitMap {
  int heads_q, heads_kv, nb, w, parts;
};

__device__ __forceinline__ Task decode_split(const SplitMap& m, int wg) {
  const int G = m.heads_q / m.heads_kv;
  const int x = wg % 8;
  const int u = wg / 8;
  const int pa = x, pb = m.parts - 1 - x;
  const int ta = G * (m.nb - pa * m.w), tb = G * (m.nb - pb * m.w);
  const int unit = u / (ta + tb);  // a group (P = 16) or a pair of groups (P = 8)
  const int rem = u % (ta + tb);
  const bool first = rem < ta;
  int ph;
  if (m.parts == 16) ph = unit;
  else ph = 2 * unit + (first ? 0 : 1);
  const int idx = first ? rem : rem - ta;
  Task t;
  t.p = first ? pa : pb;
  t.i = m.nb - 1 - idx / G;
  t.b = ph / m.heads_kv;
  t.h = (ph % m.heads_kv) * G + idx % G;
  return t;
}

// Partial slots of the rows before row i of one (batch, head): row i' owns
// floor(i' / w) + 1 consecutive slots, one per range it reaches.
__device__ __forceinline__ int64_t split_offset(int i, int w) {
  const int64_t q = i / w, r = i % w;
  return i + w * q * (q - 1) / 2 + r * q;
}

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
      const int32_t* bd = a.split_bounds + row * (a.split_parts + 1) + t.p;
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
// With SPLIT the workgroup computes one key range of its row and stores the
// normalised partial output (bf16) and its log2-domain log-sum-exp in the
// range's partial slot; split_merge_kernel combines the slots afterwards.
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
  __shared__ __attribute__((aligned(16))) uint16_t sK[Lay::TILE];
  __shared__ __attribute__((aligned(16))) uint16_t sV[Lay::TILE];
  __shared__ uint16_t sList[SPARSE ? kListChunk : 1];
  __shared__ __attribute__((aligned(16))) float sL2[SPARSE ? 1 : 64 * NH];

  const AttnArgs& a = ka.a;
  Task t = SPLIT ? decode_split(ka.split, blockIdx.x) : decode_task(ka.map, blockIdx.x + ka.task_base);
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
  bf16x8 qf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
    qf[ks] = *reinterpret_cast<const bf16x8*>(qp + (int64_t)qrow_c * a.q.ss + 16 * ks + 8 * hf);

  f32x16 acc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[dt][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
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
  auto fetch_chunk = [&](int base) {  // mask entries [base, base + kListChunk) of the row
    if (SPARSE) {
      const int ne = list.n >> list.sh;
      for (int p = tid; p < kListChunk; p += 128 * NH)
        if (base + p < ne) sList[p] = list.idx[base + p];
    }
  };
  // last valid key block: j <= i when causal, j < nb always (i < nb); a dense
  // list is valid by construction
  const int jmax = a.causal ? t.i : a.n_blocks - 1;
  auto entry = [&](int p) -> int {  // p must lie in the current LDS window
    if (p >= list.n) return -1;
    if (!SPARSE) return list.lo + p;
    const int jj = ((int)sList[(p >> list.sh) % kListChunk] << list.sh) + (p & list.sh);
    return jj <= jmax ? jj : -1;
  };
  fetch_chunk(0);
  __syncthreads();
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
  if (j >= 0) {
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
      if (SPARSE && ((n + 2) & ((kListChunk << list.sh) - 1)) == 0 && n + 2 < list.n) {
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
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[dt][e] *= alpha;
    }
    const float mc = (m_run == -INFINITY) ? 0.f : m_run * c;

    // S for the next tile (harmless junk when there is none)
    s_product(sn);
    // P^T operand of k-step kt: accumulators 8(kt%2)..+7 of half kt/2, i.e. keys
    // 32(kt/2) + 16(kt%2) + {4hf + 0..3, 8 + 4hf + 0..3}
    bf16x8 pb[4];
    float ps[4] = {0.f, 0.f, 0.f, 0.f};  // four independent partial sums
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sc[kt / 2][8 * (kt % 2) + e], c, -mc));
        ps[kt] += p;
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
  wait_loads();
  uint16_t* sO = sK;  // sK and sV are adjacent: 2 tiles of staging room
  const int ql = 32 * wave + col;
  // destination: the output rows of the query block, or the task's partial slot
  int64_t slot = 0;
  int64_t ors;
  if (SPLIT) {
    slot = ((int64_t)t.b * a.heads_q + t.h) * a.split_slots + split_offset(t.i, a.split_w) + t.p;
    ors = D;
  } else {
    ors = a.oss;
  }
  const int rows_out = (SPLIT || !RAGGED) ? 64 : min(64, S - 64 * t.i);  // rows past the end are not stored
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
    uint16_t* op = SPLIT ? a.part_o + slot * 64 * D
                         : static_cast<uint16_t*>(a.o) + t.b * a.osb + (h0 + hs) * a.osh + (int64_t)64 * t.i * a.oss;
#pragma unroll
    for (int e = 0; e < 64 * Lay::CPR / (128 * NH); ++e) {
      const int q = tid + 128 * NH * e;
      const int r = q / Lay::CPR, cc = q % Lay::CPR;
      if (r < rows_out)
        *reinterpret_cast<u32x4*>(op + (int64_t)r * ors + 8 * cc) =
            *reinterpret_cast<const u32x4*>(sO + r * Lay::OSTR + 8 * cc);
    }
  }
  if (SPLIT) {
    if (hf == 0) a.part_lse[slot * 64 + ql] = (l_tot > 0.f) ? m_run * c + __log2f(l_tot) : -INFINITY;
  } else if (a.lse && hf == 0 && qrow < S) {
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

// One wavefront per sparse row: bounds[p] = number of valid list entries
// (j <= i when causal, j < nb) in key blocks below p w, for p = 0..P.
// Lists are ascending, so range p holds entries [bounds[p], bounds[p + 1]).
__global__ __launch_bounds__(256) void split_bounds_kernel(AttnArgs a) {
  const int wave = threadIdx.x / 64;
  const int lane = threadIdx.x % 64;
  const int64_t rows = (int64_t)a.batch * a.heads_q * a.n_blocks;
  const int64_t row = (int64_t)blockIdx.x * 4 + wave;
  if (row >= rows) return;
  const int nb = a.n_blocks;
  const int i = (int)(row % nb);
  const int w = a.split_w;
  const int n = min(max(a.count[row], 0), nb);
  const uint16_t* L = a.idx + row * nb;
  const int P = a.split_parts;
  int cnt[kMaxSplitParts];
#pragma unroll
  for (int p = 0; p < kMaxSplitParts; ++p) cnt[p] = 0;
  for (int e = lane; e < n; e += 64) {
    const int j = L[e];
    if (j < nb && (!a.causal || j <= i)) {
      const int pj = j / w;
#pragma unroll
      for (int p = 0; p < kMaxSplitParts; ++p) cnt[p] += (pj == p) ? 1 : 0;
    }
  }
  int run = 0;
  int32_t* out = a.split_bounds + row * (P + 1);
#pragma unroll
  for (int p = 0; p < kMaxSplitParts; ++p) {
    if (p == P) break;
    int c = cnt[p];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) c += __shfl_xor(c, off);
    if (lane == p) out[p] = run;
    run += c;
  }
  if (lane == P) out[P] = run;
}

// One workgroup per (batch, head, query block): combines the row's partial
// outputs O_p (normalised within range p) with weights 2^(lse_p - lse), where
// lse = log2 sum_p 2^lse_p, writes O (bf16, round to nearest even) and the
// natural-log LSE.  Thread t handles query t / 4 and a quarter of its features.
template <int D>
__global__ __launch_bounds__(256) void split_merge_kernel(AttnArgs a) {
  constexpr int F = D / 4;  // features per thread
  const int64_t row = blockIdx.x;
  const int nb = a.n_blocks;
  const int i = (int)(row % nb);
  const int64_t bh = row / nb;
  const int b = (int)(bh / a.heads_q), h = (int)(bh % a.heads_q);
  const int w = a.split_w;
  const int nparts = min(a.split_parts, i / w + 1);
  const int64_t slot0 = bh * a.split_slots + split_offset(i, w);
  const int q = threadIdx.x / 4, f0 = (threadIdx.x % 4) * F;
  float mx = -INFINITY;
  for (int p = 0; p < nparts; ++p) mx = fmaxf(mx, a.part_lse[(slot0 + p) * 64 + q]);
  float acc[F];
#pragma unroll
  for (int f = 0; f < F; ++f) acc[f] = 0.f;
  float sum = 0.f;
  if (mx > -INFINITY) {
    for (int p = 0; p < nparts; ++p) {
      const float lp = a.part_lse[(slot0 + p) * 64 + q];
      if (lp == -INFINITY) continue;
      const float wgt = __builtin_amdgcn_exp2f(lp - mx);
      sum += wgt;
      const u32x4* src = reinterpret_cast<const u32x4*>(a.part_o + ((slot0 + p) * 64 + q) * D + f0);
#pragma unroll
      for (int u = 0; u < F / 8; ++u) {
        const u32x4 v = src[u];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[8 * u + 2 * e] = fmaf(wgt, __uint_as_float(v[e] << 16), acc[8 * u + 2 * e]);
          acc[8 * u + 2 * e + 1] = fmaf(wgt, __uint_as_float(v[e] & 0xFFFF0000u), acc[8 * u + 2 * e + 1]);
        }
      }
    }
  }
  const float inv = sum > 0.f ? 1.0f / sum : 0.f;
  if (64 * i + q >= a.seq_len) return;  // padding row of a partial last tile
  uint16_t* dst = static_cast<uint16_t*>(a.o) + b * a.osb + h * a.osh + (int64_t)(64 * i + q) * a.oss + f0;
#pragma unroll
  for (int u = 0; u < F / 8; ++u) {
    bf16x8 o8;
#pragma unroll
    for (int e = 0; e < 8; ++e) o8[e] = (__bf16)(acc[8 * u + e] * inv);
    *reinterpret_cast<bf16x8*>(dst + 8 * u) = o8;
  }
  if (a.lse && threadIdx.x % 4 == 0)
    a.lse[bh * a.seq_len + 64 * i + q] = sum > 0.f ? (mx + __log2f(sum)) * 0.6931471805599453f : -INFINITY;
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

// Ranges narrower than this many key blocks are not worth a split: per-task
// set-up and the partial traffic outweigh the L2 gain.  The environment
// variable SEER_SPLIT_MIN_WIDTH (read on the host at each call) overrides it.
constexpr int kSplitMinWidth = 32;

// Rows are split only on request: the environment variable SEER_SPLIT_DENSE=1
// (dense rows) or SEER_SPLIT_SPARSE=1 (sparse rows), read at each call.  Dense
// rows then take 16 ranges.  Measured at 131072 tokens: the unsplit dense
// kernel with two query heads per workgroup (117 ms) beat 16 ranges (133 ms,
// one head per workgroup, as the split runs); at 32768 tokens 7.4 against
// 9.0 ms, at 8192 equal.  Sparse rows at 10% density: the unsplit kernel
// (18.3 ms) matched 8 ranges (18.7 ms incl. the merge) and beat 16 (20.0 ms),
// the short tasks' set-up and the partial traffic eating the L2 gain; when
// enabled they take 8 ranges if the number of KV groups is even (fewer tasks
// and partials), else 16.
int split_parts(int n_blocks, int kv_groups, bool causal, bool bf16, bool sparse) {
  if (!causal || !bf16) return 0;
  const char* e = getenv(sparse ? "SEER_SPLIT_SPARSE" : "SEER_SPLIT_DENSE");
  if (!e || atoi(e) != 1) return 0;
  int min_w = kSplitMinWidth;
  if (const char* e = getenv("SEER_SPLIT_MIN_WIDTH")) {
    const int v = atoi(e);
    if (v >= 1) min_w = v;
  }
  const int cand[2] = {sparse && kv_groups % 2 == 0 ? 8 : 16, 16};
  for (int P : cand)
    if (n_blocks % P == 0 && n_blocks / P >= min_w) return P;
  return 0;
}

int64_t split_slots_per_head(int n_blocks, int w) {
  const int64_t q = n_blocks / w, r = n_blocks % w;
  return n_blocks + w * q * (q - 1) / 2 + r * q;
}

template <int D, bool RAGGED>
static void launch_split(const KernelArgs& ka, bool sparse, hipStream_t s) {
  const AttnArgs& a = ka.a;
  const int64_t rows = (int64_t)a.batch * a.heads_q * a.n_blocks;
  if (sparse)
    hipLaunchKernelGGL(split_bounds_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, a);
  // per XCD and group (P = 16) or pair of groups (P = 8): G (2 nb - (P - 1) w) tasks
  const int64_t units = a.split_parts == 16 ? (int64_t)a.batch * a.heads_kv : (int64_t)a.batch * a.heads_kv / 2;
  const int64_t tasks = 8 * units * (a.heads_q / a.heads_kv) * (2 * a.n_blocks - (a.split_parts - 1) * a.split_w);
  dim3 grid((unsigned)tasks), block(128);
  if (sparse) hipLaunchKernelGGL((attn_fwd_bf16_kernel<D, true, true, RAGGED>), grid, block, 0, s, ka);
  else hipLaunchKernelGGL((attn_fwd_bf16_kernel<D, false, true, RAGGED>), grid, block, 0, s, ka);
  hipLaunchKernelGGL(split_merge_kernel<D>, dim3((unsigned)rows), dim3(256), 0, s, a);
}

static hipError_t launch_attn_one(const AttnArgs& a, hipStream_t s);

// One launch per KV group when a phase of the task order holds a single group
// (its K and V alone fill the phase's cache budget): the launch boundary keeps
// every XCD on the same group's K and V.  Measured at 131072 tokens (sparse):
// 8 launches 17.8 ms, one launch 18.1 ms.  Not for the split or pooling modes.
hipError_t launch_attn(const AttnArgs& a, hipStream_t s) {
  const int groups = a.batch * a.heads_kv;
  if (a.split_w > 0 || a.gt != nullptr || groups <= 1 || make_map(a).gpp != 1)
    return launch_attn_one(a, s);
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
      const hipError_t e = launch_attn_one(c, s);
      if (e != hipSuccess) return e;
    }
  return hipSuccess;
}

// Query heads per workgroup for rows shared by the query heads of a KV group
// (a mask shared by the group, or dense rows): 2 when the group size allows,
// else 1 (the environment variable SEER_KV_HEADS_PER_WG, read at each call,
// sets the cap: 1, 2 or 4).  Measured at 131072 tokens, 32 query / 8 KV heads,
// TopK 0.1: per-head rows 17.3 ms; shared rows with 1, 2 and 4 heads per
// workgroup 14.3, 13.0 and 13.1 ms (two 4-wavefront workgroups per CU keep
// their phases independent; one 8-wavefront workgroup moves in lockstep).
static int kv_heads_per_wg(const AttnArgs& a) {
  const bool shared_rows = a.count ? a.mask_kv : true;
  if (!shared_rows || !a.bf16 || a.split_w > 0) return 1;
  int cap = 2;
  if (const char* e = getenv("SEER_KV_HEADS_PER_WG")) cap = atoi(e);
  const int G = a.heads_q / a.heads_kv;
  for (int nh = 4; nh >= 2; nh /= 2)
    if (nh <= cap && G % nh == 0) return nh;
  return 1;
}

template <int D, bool SPARSE, bool RAGGED>
static void launch_nh(const KernelArgs& ka, int nh, dim3 grid, hipStream_t s) {
  if (nh == 4) hipLaunchKernelGGL((attn_fwd_bf16_kernel<D, SPARSE, false, RAGGED, 4>), grid, dim3(512), 0, s, ka);
  else hipLaunchKernelGGL((attn_fwd_bf16_kernel<D, SPARSE, false, RAGGED, 2>), grid, dim3(256), 0, s, ka);
}

template <int D>
static void launch_nh_d(const KernelArgs& ka, int nh, bool sparse, bool ragged, dim3 grid, hipStream_t s) {
  if (sparse) {
    if (ragged) launch_nh<D, true, true>(ka, nh, grid, s);
    else launch_nh<D, true, false>(ka, nh, grid, s);
  } else {
    if (ragged) launch_nh<D, false, true>(ka, nh, grid, s);
    else launch_nh<D, false, false>(ka, nh, grid, s);
  }
}

// Sparse rows of long sequences launch in batches of exactly the workgroups the
// GPU holds at once (4 per CU), so that the rows of a batch start together and
// walk their ascending lists roughly in step: concurrent rows then share more
// of their K/V tiles in L2.  Within a batch the order is the usual one (task
// ids continue across batches), so every output is unchanged.  Only the
// heavier half of the tasks is batched: the later batches' short rows leave too
// much idle time at their ends.  Measured at 131072 tokens (32 q / 8 KV heads,
// TopK 0.1): 17.29 ms unbatched, 16.92 ms with every task batched, 16.65 ms
// with the heavier half batched; 48.9 -> 48.2 ms (all batched) with per-head
// densities spread over 5-40%; at 32768 tokens the batch ends' idle time
// outweighed the gain (1.84 -> 2.06 ms; at 65536 tokens with 7 heads of 5-40%
// density 7.6 -> 10.6 ms), hence the size threshold.  The environment variables
// SEER_EPOCH_MIN_BLOCKS (the threshold in 64-token blocks, default 2048) and
// SEER_EPOCH_WGS (the batch size; 0 disables) are read on the host at each
// call.
static int epoch_min_blocks() {
  int v = 2048;
  if (const char* e = getenv("SEER_EPOCH_MIN_BLOCKS")) v = atoi(e);
  return v > 0 ? v : 1;
}

static int resident_workgroups(int head_dim, bool ragged) {
  if (const char* e = getenv("SEER_EPOCH_WGS")) {
    const int v = atoi(e);
    return v > 0 ? v / 8 * 8 : 0;  // a multiple of 8 keeps the XCD interleave of the task order
  }
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  const void* fn = head_dim == 128
                       ? (ragged ? reinterpret_cast<const void*>(attn_fwd_bf16_kernel<128, true, false, true>)
                                 : reinterpret_cast<const void*>(attn_fwd_bf16_kernel<128, true, false, false>))
                       : (ragged ? reinterpret_cast<const void*>(attn_fwd_bf16_kernel<64, true, false, true>)
                                 : reinterpret_cast<const void*>(attn_fwd_bf16_kernel<64, true, false, false>));
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 128, 0) != hipSuccess) return 0;
  return cus * per_cu / 8 * 8;
}

static hipError_t launch_attn_one(const AttnArgs& a, hipStream_t s) {
  KernelArgs ka;
  ka.a = a;
  const int nh = kv_heads_per_wg(a);
  if (nh > 1) {  // tasks over head slots of nh heads: the task order sees heads_q / nh heads
    AttnArgs v = a;
    v.heads_q = a.heads_q / nh;
    ka.map = make_map(v);
    const int64_t total = (int64_t)a.batch * v.heads_q * a.n_blocks;
    if (total == 0) return hipSuccess;
    ka.split = SplitMap{a.heads_q, a.heads_kv, a.n_blocks, 0, 0};
    ka.scale_log2 = a.scale * kLog2e;
    ka.task_base = 0;
    const bool sparse = a.count != nullptr;
    if (a.seq_len <= 0 || (a.n_blocks - 1) * 64 >= a.seq_len || a.n_blocks * 64 < a.seq_len ||
        (a.gt != nullptr && (sparse || !a.pool_r)))
      return hipErrorInvalidValue;
    const bool ragged = a.seq_len % 64 != 0;
    const dim3 grid((unsigned)total);
    if (a.head_dim == 128) launch_nh_d<128>(ka, nh, sparse, ragged, grid, s);
    else if (a.head_dim == 64) launch_nh_d<64>(ka, nh, sparse, ragged, grid, s);
    else return hipErrorInvalidValue;
    return hipGetLastError();
  }
  ka.map = make_map(a);
  ka.split = SplitMap{a.heads_q, a.heads_kv, a.n_blocks, a.split_w, a.split_parts};
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
    // the shape must be the one split_width accepted, with every buffer present
    const int P = a.split_parts;
    if (pool || !a.bf16 || !a.causal || (sparse && a.mask_shift != 0) || (P != 8 && P != 16) ||
        a.split_w * P != a.n_blocks ||
        (P == 8 && (a.batch * a.heads_kv) % 2 != 0) || !a.part_lse || !a.part_o ||
        (sparse && !a.split_bounds) || a.split_slots != split_slots_per_head(a.n_blocks, a.split_w))
      return hipErrorInvalidValue;
    if (a.head_dim == 128) {
      if (ragged) launch_split<128, true>(ka, sparse, s);
      else launch_split<128, false>(ka, sparse, s);
    } else if (a.head_dim == 64) {
      if (ragged) launch_split<64, true>(ka, sparse, s);
      else launch_split<64, false>(ka, sparse, s);
    } else {
      return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  if (a.bf16 && sparse && !pool && a.n_blocks >= epoch_min_blocks()) {
    const int E = resident_workgroups(a.head_dim, ragged);
    if (E > 0 && total > E) {
      // the heavier half of the tasks (the longest rows) in batches, the rest
      // (whose short rows would leave batch ends idle) in one launch
      const int64_t batched = (total / 2 + E - 1) / E * E;
      for (int64_t b0 = 0, cnt = 0; b0 < total; b0 += cnt) {
        cnt = b0 < batched ? std::min<int64_t>(E, total - b0) : total - b0;
        ka.task_base = (int)b0;
        const dim3 g((unsigned)cnt);
        if (a.head_dim == 128) {
          if (ragged) hipLaunchKernelGGL((attn_fwd_bf16_kernel<128, true, false, true>), g, block, 0, s, ka);
          else hipLaunchKernelGGL((attn_fwd_bf16_kernel<128, true, false, false>), g, block, 0, s, ka);
        } else {
          if (ragged) hipLaunchKernelGGL((attn_fwd_bf16_kernel<64, true, false, true>), g, block, 0, s, ka);
          else hipLaunchKernelGGL((attn_fwd_bf16_kernel<64, true, false, false>), g, block, 0, s, ka);
        }
      }
      return hipGetLastError();
    }
  }
  if (a.bf16) {
    if (a.head_dim == 128) {
      if (ragged) {
        if (sparse) hipLaunchKernelGGL((attn_fwd_bf16_kernel<128, true, false, true>), grid, block, 0, s, ka);
        else hipLaunchKernelGGL((attn_fwd_bf16_kernel<128, false, false, true>), grid, block, 0, s, ka);
      } else {
        if (sparse) hipLaunchKernelGGL((attn_fwd_bf16_kernel<128, true, false, false>), grid, block, 0, s, ka);
        else hipLaunchKernelGGL((attn_fwd_bf16_kernel<128, false, false, false>), grid, block, 0, s, ka);
      }
    } else if (a.head_dim == 64) {
      if (ragged) {
        if (sparse) hipLaunchKernelGGL((attn_fwd_bf16_kernel<64, true, false, true>), grid, block, 0, s, ka);
        else hipLaunchKernelGGL((attn_fwd_bf16_kernel<64, false, false, true>), grid, block, 0, s, ka);
      } else {
        if (sparse) hipLaunchKernelGGL((attn_fwd_bf16_kernel<64, true, false, false>), grid, block, 0, s, ka);
        else hipLaunchKernelGGL((attn_fwd_bf16_kernel<64, false, false, false>), grid, block, 0, s, ka);
      }
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
