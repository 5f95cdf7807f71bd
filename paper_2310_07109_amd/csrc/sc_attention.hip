// Sliding-window + global-token sparse attention with exact importance-score
// partials, for gfx950 (SparseCoder, arXiv 2310.07109: Sec. 4.2.1 window,
// Sec. 3.2.1 global tokens, Sec. 5.5 score extraction).
//
// Decomposition of the allowed (query i, key j) pairs of one sequence, both
// valid, into three disjoint regions:
//   R1  i global, any j            -> global-row kernels (dense strip)
//   R2  i not global, j global     -> window kernel, "global key" tiles (and
//                                     band tiles when j lies inside the band)
//   R3  neither global, |i-j| <= r -> window kernel, band tiles
//
// Window kernel, one workgroup (4 waves) per (sequence, head, 64 queries):
//   pass 1  each wave owns 16 queries; K/V tiles of 64 keys are staged in LDS
//           (double-buffered, the next tile's loads in flight during the
//           current tile's math) and S^T = K.Q^T is computed on MFMA so that a
//           lane holds one query and 4 keys of each 16-key sub-tile.  Online
//           softmax in the log2 domain with a lazily raised running max
//           (rescale only when a tile max exceeds it by 8); P is rounded to the
//           storage type and O^T += V^T.P^T runs on MFMA, with the V operand
//           read from the row-major V tile by LDS transpose reads.
//   pass 2  (only when score partials are requested) the same tiles again; each
//           wave owns one 16-key sub-tile for all 64 queries, S = Q.K^T puts a
//           key in each lane and 4 queries per register, P = exp2(S*c - LSE2)
//           is exact, and the column sums are reduced inside the lane, then
//           across the 4 lane groups with permlane swaps.  One float per
//           (block, key) goes to HBM; no atomics, fixed summation order.
#include "sc_device.h"
#include "sc_internal.h"

namespace sc {
namespace {

constexpr int kThreads = 256;
constexpr int kBQ = kQueryBlock;
constexpr int kBK = kKeyTile;
constexpr float kTau = 8.0f;       // lazy-rescale slack in log2 units
constexpr float kNegBig = -1e30f;  // running-max sentinel (finite: avoids inf - inf)
constexpr float kRaiseSum = 256.0f;  // 2^kTau: a lane's sum of P above it triggers a raise

// Minimum resident waves per SIMD the register allocation must allow.
#define SC_OCC(w) __attribute__((amdgpu_waves_per_eu(w)))

// --------------------------------------------------------------- staging ----
// Tiles of 64 rows x 64 head dims move HBM -> registers -> LDS in two steps so
// that the loads of tile t+1 are in flight while tile t is computed.  Each
// thread moves kCpt 16-byte chunks; consecutive threads cover consecutive
// chunks of a row (coalesced loads, conflict-free LDS writes).
template <int DT>
struct Stage {
  using T = typename Tr<DT>::T;
  static constexpr int kEpc = 16 / sizeof(T);        // elements per chunk
  static constexpr int kCpr = kHeadDim / kEpc;       // chunks per row
  static constexpr int kCpt = 64 * kCpr / kThreads;  // chunks per thread
  static constexpr int P = Tr<DT>::kPitch;
  uint4 r[kCpt];

  // rows k0 .. k0+63; rows at or beyond kend are zero (k0 < kend).  The
  // loads are unconditional (row clamped to kend - 1) so that no exec-masked
  // branch separates them from the math they overlap with.
  SC_DEV void load_range(const T* g, long long ld, int k0, int kend) {
#pragma unroll
    for (int i = 0; i < kCpt; ++i) {
      const int c = threadIdx.x + kThreads * i, row = c / kCpr, part = c % kCpr;
      const int k = k0 + row;
      const uint4 v = *reinterpret_cast<const uint4*>(g + (long long)min(k, kend - 1) * ld + part * kEpc);
      r[i] = k < kend ? v : make_uint4(0, 0, 0, 0);
    }
  }
  // row `row` comes from token rowfn(row), or is zero when that is -1
  template <typename RowFn>
  SC_DEV void load_rows(const T* g, long long ld, RowFn rowfn) {
#pragma unroll
    for (int i = 0; i < kCpt; ++i) {
      const int c = threadIdx.x + kThreads * i, row = c / kCpr, part = c % kCpr;
      const int k = rowfn(row);
      r[i] = k >= 0 ? *reinterpret_cast<const uint4*>(g + (long long)k * ld + part * kEpc) : make_uint4(0, 0, 0, 0);
    }
  }
  // into a key / query tile (kValue false) or a value tile (kValue true)
  template <bool kValue = false>
  SC_DEV void store(T* lds) const {
#pragma unroll
    for (int i = 0; i < kCpt; ++i) {
      const int c = threadIdx.x + kThreads * i, row = c / kCpr, part = c % kCpr;
      *reinterpret_cast<uint4*>(lds + (kValue ? Tr<DT>::voff(row, part) : Tr<DT>::off(row, part))) = r[i];
    }
  }
};

// ------------------------------------------------------------ pass 1 tile ---
// One 64-key tile for the 16 queries of a wave.  s[st][i] is the logit of
// (key 16*st + 4g + i, query lr).  ok(st, i) masks keys (kMasked only).
// kHalf >= 0 restricts the tile to its 32 keys 32 kHalf .. 32 kHalf + 31
// (sub-tiles 2 kHalf and 2 kHalf + 1).  The running max m_use is in scaled
// log2 units; softmax_scale >= 0, so the tile max is taken on the raw logits
// and scaled once.
template <int DT, bool kMasked, int kHalf = -1, typename OkFn>
SC_DEV void softmax_tile(const typename Tr<DT>::Frag (&qf)[Tr<DT>::kChunks], const typename Tr<DT>::T* sK,
                         const typename Tr<DT>::T* sV, float c2, int lr, int g, float& m_use, float& l_run,
                         f32x4 (&o)[4], OkFn ok) {
  using TR = Tr<DT>;
  constexpr int kSt0 = kHalf < 0 ? 0 : 2 * kHalf, kNst = kHalf < 0 ? 4 : 2;
  f32x4 s[kNst];
#pragma unroll
  for (int sj = 0; sj < kNst; ++sj) {
    typename TR::Frag kf[TR::kChunks];
    TR::load_frags(sK, 16 * (kSt0 + sj) + lr, g, kf);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < TR::kChunks; ++c) acc = TR::mma(kf[c], qf[c], acc);
    s[sj] = acc;
  }
  bool valid[kNst][4];
  float tmax = -INFINITY;
#pragma unroll
  for (int sj = 0; sj < kNst; ++sj)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      valid[sj][i] = !kMasked || ok(kSt0 + sj, i);
      tmax = vmax(tmax, valid[sj][i] ? s[sj][i] : -INFINITY);
    }
  tmax = group_max(tmax) * c2;
  if (tmax > m_use + kTau) {
    const float f = fast_exp2(m_use - tmax);
    l_run *= f;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) o[dt] *= f;
    m_use = tmax;
  }
  float p[kNst][4];
#pragma unroll
  for (int sj = 0; sj < kNst; ++sj)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float e = fast_exp2(fmaf(s[sj][i], c2, -m_use));
      p[sj][i] = valid[sj][i] ? e : 0.f;
      l_run += p[sj][i];
    }
  if constexpr (DT == 1) {
    // keys of lane group g in MFMA order: 32kc + 4g + (0..3), then 32kc + 16 + 4g + (0..3)
#pragma unroll
    for (int kj = 0; kj < kNst / 2; ++kj) {
      const int kc = kSt0 / 2 + kj;
      bf16x8 pb;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pb[i] = (__bf16)p[2 * kj][i];
        pb[4 + i] = (__bf16)p[2 * kj + 1][i];
      }
      // lane (g, lr) supplies dims 16dt + 4(lr&3) .. +3 of value rows
      // 32kc + 4g + lr/4 and 32kc + 16 + 4g + lr/4
      const int vr = 32 * kc + 4 * g + (lr >> 2), b = (lr >> 1) & 1, e = 4 * (lr & 1);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const i16x4 a0 = lds_read_tr16(sV + TR::voff(vr, 2 * dt + b) + e);
        const i16x4 a1 = lds_read_tr16(sV + TR::voff(vr + 16, 2 * dt + b) + e);
        const i16x8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
        o[dt] = TR::mma(__builtin_bit_cast(bf16x8, a), pb, o[dt]);
      }
    }
  } else {
#pragma unroll
    for (int sj = 0; sj < kNst; ++sj)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
          o[dt] = TR::mma(sV[TR::voff(16 * (kSt0 + sj) + 4 * g + i, 4 * dt + (lr >> 2)) + (lr & 3)], p[sj][i],
                          o[dt]);
  }
}

// ------------------------------------------------------------ column tile ---
// Exact probabilities of the 64 staged queries (rows of sQ, log2-LSE in sL)
// for the 16 keys held in kf, summed per key into this lane's partial.  MFMA
// result register (qst, i) is (query 16*qst + 4g + i, key lr), so the sum over
// queries stays inside the lane; the 4 lane groups are combined once, by the
// caller, after the last tile.  ok(qst, i) masks pairs; emit(q, p) sees every
// probability (used for the paper's band layout).  Bit qst of `live` (wave-
// uniform) says whether query group qst holds a used row; other groups are
// skipped.
template <int DT, bool kMasked, typename OkFn, typename EmitFn>
SC_DEV float col_tile(const typename Tr<DT>::Frag (&kf)[Tr<DT>::kChunks], const typename Tr<DT>::T* sQ,
                      const float* sL, float c2, int lr, int g, OkFn ok, EmitFn emit, unsigned live = 0xFu) {
  using TR = Tr<DT>;
  float cs = 0.f;
#pragma unroll
  for (int qst = 0; qst < 4; ++qst) {
    if (!((live >> qst) & 1u)) continue;  // wave-uniform: no query of this group is used
    typename TR::Frag qf[TR::kChunks];
    TR::load_frags(sQ, 16 * qst + lr, g, qf);
    const f32x4 l2 = *reinterpret_cast<const f32x4*>(sL + 16 * qst + 4 * g);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < TR::kChunks; ++c) acc = TR::mma(qf[c], kf[c], acc);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float p = fast_exp2(fmaf(acc[i], c2, -l2[i]));
      if (kMasked && !ok(qst, i)) p = 0.f;
      emit(16 * qst + 4 * g + i, p);
      cs += p;
    }
  }
  return cs;
}

struct NoEmit {
  SC_DEV void operator()(int, float) const {}
};

template <int DT>
SC_DEV void store_row4(typename Tr<DT>::T* dst, f32x4 v) {
  if constexpr (DT == 1) {
    bf16x4 b;
    b[0] = (__bf16)v[0];
    b[1] = (__bf16)v[1];
    b[2] = (__bf16)v[2];
    b[3] = (__bf16)v[3];
    *reinterpret_cast<bf16x4*>(dst) = b;
  } else {
    *reinterpret_cast<f32x4*>(dst) = v;
  }
}

// LDS shared by all block types of a launch (each block type uses its own
// subset; pointers are handed to the per-type device functions).
// Launch 1 (softmax and P.V): double-buffered K and V tiles.  The query tile
// is staged in b[1] before the pipeline starts: its fragments move to
// registers first, and b[1] is only written after a barrier.
template <int DT>
struct Smem {
  using T = typename Tr<DT>::T;
  static constexpr int P = Tr<DT>::kPitch;
  __attribute__((aligned(16))) T b[2][kBK * P];  // key tiles (query tile first in b[1])
  __attribute__((aligned(16))) T c[2][kBK * Tr<DT>::kPitchV];  // value tiles
  int pos[2][kBK];                                 // positions of gathered rows
  int misc[4];
};
// Launch 2 (column sums): a resident key block, double-buffered query tiles
// with their log2-LSE.
template <int DT>
struct SmemCol {
  using T = typename Tr<DT>::T;
  static constexpr int P = Tr<DT>::kPitch;
  __attribute__((aligned(16))) T a[kBK * P];     // key block
  __attribute__((aligned(16))) T b[2][kBQ * P];  // query tiles (key tiles for the global rows)
  __attribute__((aligned(16))) float l[2][kBQ];  // log2-LSE of staged query rows
  int pos[2][kBK];                                 // positions of gathered rows
  int misc[4];
};

// -------------------------------------------------------- window pass 1 -----
// Geometry of one window block (sequence b, head h, queries q0 .. q0+QB-1) and
// its LDS tables: the global-token bitmask over the key range [kt0, kt1) and
// the list of 64-slot chunks that hold global keys outside that range.
struct WinBlock {
  int qb, bh, h, b, L, q0, kt0, kt1, nkt, nwords, nxc;
};

template <int QB = kBQ>
SC_DEV WinBlock win_block(const AttnArgs& a, int bh, int qb) {
  WinBlock wb;
  wb.bh = bh;
  wb.qb = qb;
  wb.h = wb.bh % a.H;
  wb.b = wb.bh / a.H;
  wb.L = clampi(a.valid_len[wb.b], 0, a.n);
  wb.q0 = wb.qb * QB;
  wb.kt0 = max(0, wb.q0 - a.r);
  wb.kt1 = min(wb.L, wb.q0 + QB + (a.causal ? 0 : a.r));  // causal: no key after the block's last query
  wb.nkt = (wb.kt1 - wb.kt0 + kBK - 1) / kBK;
  wb.nwords = (wb.kt1 - wb.kt0 + 31) >> 5;
  wb.nxc = (a.gpos && a.G > 0) ? (a.G + kBK - 1) / kBK : 0;
  return wb;
}

// Global keys of band tile t as a 64-bit mask (bit j: key kt0 + 64t + j).
SC_DEV unsigned long long tile_gmask(const uint32_t* sBits, int t, int nwords) {
  const unsigned long long lo = sBits[2 * t];
  const unsigned long long hi = 2 * t + 1 < nwords ? sBits[2 * t + 1] : 0u;
  return lo | (hi << 32);
}

// Fills the bitmask and the chunk list; returns the number of tiles (band
// tiles, then global-slot tiles).  Contains barriers; call with q0 < L.
SC_DEV int win_tables(const AttnArgs& a, const WinBlock& wb, uint32_t* sBits, int* sXList, int* sNx) {
  const int tid = threadIdx.x;
  const int* gp = wb.nxc ? a.gpos + (long long)wb.b * a.G : nullptr;
  const int G = gp ? a.G : 0;
  const int p_first = tid < G ? gp[tid] : -1;  // in flight with the caller's loads
  for (int i = tid; i < wb.nwords; i += kThreads) sBits[i] = 0u;
  for (int i = tid; i < wb.nxc; i += kThreads) sXList[i] = 0;
  __syncthreads();
  for (int j = tid; j < G; j += kThreads) {
    const int p = j == tid ? p_first : gp[j];
    if (p >= wb.kt0 && p < wb.kt1)
      atomicOr(&sBits[(p - wb.kt0) >> 5], 1u << ((p - wb.kt0) & 31));
    else if (p >= 0 && p < wb.L && !(a.causal && p >= wb.kt1))  // causal: later keys are never attended
      sXList[j / kBK] = 1;
  }
  __syncthreads();
  if (tid == 0) {
    int m = 0;
    for (int c = 0; c < wb.nxc; ++c)
      if (sXList[c]) sXList[m++] = c;
    *sNx = m;
  }
  __syncthreads();
  return wb.nkt + *sNx;
}

// The same tables when the block has at most 64 global slots, built by wave 0
// alone from one position per lane (p, loaded by the caller): the in-band
// bitmask (zeroed, then or-ed: the LDS operations of one wave take effect in
// program order) and the out-of-band positions compacted in slot order into
// sPos[0 .. *sCnt), with *sNx = 1 when there are any (chunk 0).  One barrier.
SC_DEV int win_tables_small(const AttnArgs& a, const WinBlock& wb, int p, int w, int lane, uint32_t* sBits,
                            int* sXList, int* sNx, int* sPos, int* sCnt) {
  if (w == 0) {
    for (int i = lane; i < wb.nwords; i += 64) sBits[i] = 0u;
    if (p >= wb.kt0 && p < wb.kt1) atomicOr(&sBits[(p - wb.kt0) >> 5], 1u << ((p - wb.kt0) & 31));
    const bool oob = p >= 0 && p < wb.L && (p < wb.kt0 || (!a.causal && p >= wb.kt1));
    const unsigned long long m = __ballot(oob);
    const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    if (oob) sPos[rank] = p;
    if (lane == 0) {
      *sNx = m != 0ull ? 1 : 0;
      *sCnt = __popcll(m);
      sXList[0] = 0;
    }
  }
  __syncthreads();
  return wb.nkt + *sNx;
}

// win_tables for the bf16 window blocks, which also compacts the first
// listed chunk: its out-of-band global positions, in slot order, go to
// sPos[0 .. *sCnt).  The wave whose threads loaded that chunk's slots does it
// from registers (no second load of the positions); a first chunk beyond the
// workgroup's first kThreads slots is loaded again by wave 0.  Contains
// barriers; call with q0 < L.
SC_DEV int win_tables2(const AttnArgs& a, const WinBlock& wb, uint32_t* sBits, int* sXList, int* sNx, int* sPos,
                       int* sCnt) {
  const int tid = threadIdx.x;
  const int* gp = wb.nxc ? a.gpos + (long long)wb.b * a.G : nullptr;
  const int G = gp ? a.G : 0;
  const int p_first = tid < G ? gp[tid] : -1;  // in flight with the caller's loads
  auto out_of_band = [&](int p) { return p >= 0 && p < wb.L && (p < wb.kt0 || (!a.causal && p >= wb.kt1)); };
  for (int i = tid; i < wb.nwords; i += kThreads) sBits[i] = 0u;
  for (int i = tid; i < wb.nxc; i += kThreads) sXList[i] = 0;
  __syncthreads();
  for (int j = tid; j < G; j += kThreads) {
    const int p = j == tid ? p_first : gp[j];
    if (p >= wb.kt0 && p < wb.kt1)
      atomicOr(&sBits[(p - wb.kt0) >> 5], 1u << ((p - wb.kt0) & 31));
    else if (out_of_band(p))  // causal: later keys are never attended
      sXList[j / kBK] = 1;
  }
  __syncthreads();
  if (tid == 0) {
    int m = 0;
    for (int c = 0; c < wb.nxc; ++c)
      if (sXList[c]) sXList[m++] = c;
    *sNx = m;
  }
  __syncthreads();
  const int nx = *sNx;
  if (nx > 0) {
    const int c0 = sXList[0];
    constexpr int kRegChunks = kThreads / kBK;  // chunks whose slots the workgroup's threads loaded
    if ((tid >> 6) == (c0 < kRegChunks ? c0 : 0)) {
      const int j = kBK * c0 + (tid & 63);
      const int p = c0 < kRegChunks ? p_first : (j < G ? gp[j] : -1);  // p_first is gp[j] when c0 < kRegChunks
      const bool use = out_of_band(p);
      const unsigned long long m = __ballot(use);
      const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
      if (use) sPos[rank] = p;
      if ((tid & 63) == 0) *sCnt = __popcll(m);
    }
    __syncthreads();
  }
  return wb.nkt + nx;
}

// Tile loader of pass 1: band tiles are contiguous key ranges, global-slot
// tiles gather the rows of global keys outside the band.
template <int DT>
struct WinLoader {
  using T = typename Tr<DT>::T;
  const AttnArgs& a;
  const WinBlock& wb;
  const int* gp;
  const int* sXList;
  Stage<DT> stk, stv;
  int pos_reg = -1;

  SC_DEV int slot_row(int c, int row) const {
    const int j = kBK * c + row;
    const int p = j < a.G ? gp[j] : -1;
    return (p >= 0 && p < wb.L && (p < wb.kt0 || p >= wb.kt1)) ? p : -1;
  }
  SC_DEV void load(int t, const T* Kg, const T* Vg) {
    if (t < wb.nkt) {
      const int k0 = wb.kt0 + t * kBK;
      stk.load_range(Kg, a.ld_in, k0, wb.kt1);
      stv.load_range(Vg, a.ld_in, k0, wb.kt1);
    } else {
      const int c = sXList[t - wb.nkt];
      stk.load_rows(Kg, a.ld_in, [&](int row) { return slot_row(c, row); });
      stv.load_rows(Vg, a.ld_in, [&](int row) { return slot_row(c, row); });
      if (threadIdx.x < kBK) pos_reg = slot_row(c, threadIdx.x);
    }
  }
  SC_DEV void store(int t, T* sK, T* sV, int* sPos) const {
    stk.store(sK);
    stv.template store<true>(sV);
    if (t >= wb.nkt && threadIdx.x < kBK) sPos[threadIdx.x] = pos_reg;
  }
};

// Pass 1: O, LSE (and the log2 LSE used by the column sums) for the
// non-global queries of the block; zero rows for padding queries.
template <int DT>
SC_DEV void window_fwd_block(const AttnArgs& a, int bh, int qb, Smem<DT>& sm, uint32_t* sDyn) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  using Frag = typename TR::Frag;
  constexpr int P = TR::kPitch;
  const WinBlock wb = win_block(a, bh, qb);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, lr = lane & 15;
  const int n = a.n, r = a.r, L = wb.L, q0 = wb.q0, kt0 = wb.kt0, kt1 = wb.kt1, nkt = wb.nkt;
  const T* Qg = static_cast<const T*>(a.q) + wb.b * a.bs_in + wb.h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + wb.b * a.bs_in + wb.h * kHeadDim;
  const T* Vg = static_cast<const T*>(a.v) + wb.b * a.bs_in + wb.h * kHeadDim;
  T* Og = static_cast<T*>(a.out) + wb.b * a.bs_out + wb.h * kHeadDim;
  float* lseg = a.lse ? a.lse + (long long)wb.bh * n : nullptr;
  float* l2g = a.win_lse2 ? a.win_lse2 + (long long)wb.bh * n : nullptr;

  if (q0 >= L) {  // padding block: zero output rows (unless the caller never reads them)
    constexpr int kEpc = 16 / sizeof(T), kCpr = kHeadDim / kEpc;
    if (!a.skip_pad_out)
      for (int c = tid; c < kBQ * kCpr; c += kThreads) {
        const int q = q0 + c / kCpr;
        if (q < n) zero16(Og + (long long)q * a.ld_out + (c % kCpr) * kEpc);
      }
    for (int i = tid; i < kBQ; i += kThreads)
      if (q0 + i < n) {
        if (lseg) lseg[q0 + i] = -INFINITY;
        if (l2g) l2g[q0 + i] = INFINITY;
      }
    return;
  }
  uint32_t* sBits = sDyn;
  int* sXList = reinterpret_cast<int*>(sDyn + a.rwp / 32 + 2);
  {  // padding query rows are staged as zeros: their (unused) logits stay finite
    Stage<DT> sq;
    sq.load_range(Qg + (long long)q0 * a.ld_in, a.ld_in, 0, L - q0);
    sq.store(sm.b[1]);
  }
  const int ntile = win_tables(a, wb, sBits, sXList, &sm.misc[0]);
  auto gbit = [&](int k) -> bool {
    const int o = k - kt0;
    return (sBits[o >> 5] >> (o & 31)) & 1u;
  };
  WinLoader<DT> ld{a, wb, wb.nxc ? a.gpos + (long long)wb.b * a.G : nullptr, sXList};

  Frag qf[TR::kChunks];
  TR::load_frags(sm.b[1], 16 * w + lr, g, qf);
  const int qa = q0 + 16 * w;
  const int qrow = qa + lr;
  float m_use = kNegBig, l_run = 0.f;
  f32x4 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // band tiles: double-buffered, the next tile's loads overlap this tile's math
  ld.load(0, Kg, Vg);
  ld.store(0, sm.b[0], sm.c[0], sm.pos[0]);
  __syncthreads();  // also: every wave holds its query fragments before b[1] is reused
  for (int t = 0; t < nkt; ++t) {
    const int buf = t & 1;
    if (t + 1 < nkt) ld.load(t + 1, Kg, Vg);
    const int k0 = kt0 + t * kBK;
    const bool near = k0 <= qa + 15 + r && k0 + kBK - 1 >= qa - r;
    if (near || tile_gmask(sBits, t, wb.nwords) != 0ull) {
      const bool interior = k0 + kBK <= kt1 && k0 >= qa + 15 - r && k0 + kBK - 1 <= qa + r;
      if (interior) {
        softmax_tile<DT, false>(qf, sm.b[buf], sm.c[buf], a.c2, lr, g, m_use, l_run, o,
                                [](int, int) { return true; });
      } else {
        // key index inside the tile: 16*st + 4g + i; allowed when it lies in
        // [lo, hi] (window and sequence end) or is a global key of the band.
        // Branch-free: the tile's global keys come as one 64-bit mask (bits
        // beyond kt1 are never set).
        const int lo = qrow - r - k0, hi = min(qrow + r, kt1 - 1) - k0;
        const unsigned long long gm = tile_gmask(sBits, t, wb.nwords) >> (4 * g);
        softmax_tile<DT, true>(qf, sm.b[buf], sm.c[buf], a.c2, lr, g, m_use, l_run, o, [&](int s4, int i) {
          const int kk = 16 * s4 + 4 * g + i;
          return ((kk >= lo) & (kk <= hi)) | (bool)((gm >> (16 * s4 + i)) & 1ull);
        });
      }
    }
    if (t + 1 < nkt) ld.store(t + 1, sm.b[buf ^ 1], sm.c[buf ^ 1], sm.pos[buf ^ 1]);
    __syncthreads();
  }
  // global keys outside the band (few tiles; not pipelined)
  for (int t = nkt; t < ntile; ++t) {
    ld.load(t, Kg, Vg);
    ld.store(t, sm.b[0], sm.c[0], sm.pos[0]);
    __syncthreads();
    const int* sp = sm.pos[0];
    softmax_tile<DT, true>(qf, sm.b[0], sm.c[0], a.c2, lr, g, m_use, l_run, o,
                           [&](int s4, int i) { return sp[16 * s4 + 4 * g + i] >= 0; });
    __syncthreads();
  }

  const float l_row = group_sum(l_run);
  const bool qin = qrow < L;
  const bool qvalid = qin && !gbit(qrow);  // qrow in [q0, L) lies inside [kt0, kt1)
  const float lse2 = m_use + fast_log2(l_row);
  if (qvalid) {
    const float inv = 1.0f / l_row;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) store_row4<DT>(Og + (long long)qrow * a.ld_out + 16 * dt + 4 * g, o[dt] * inv);
    if (g == 0 && lseg) lseg[qrow] = lse2 * kLn2;
  } else if (!qin && qrow < n) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
      store_row4<DT>(Og + (long long)qrow * a.ld_out + 16 * dt + 4 * g, f32x4{0.f, 0.f, 0.f, 0.f});
    if (g == 0 && lseg) lseg[qrow] = -INFINITY;
  }
  // excluded rows (global or padding) get +inf: their column-sum probabilities are 0
  if (g == 0 && l2g && qrow < n) l2g[qrow] = qvalid ? lse2 : INFINITY;
}

// Rows 16w .. 16w+15 of a 64-row bf16 tile (two wave loads of 8 rows); tile
// row R holds global row rowfn(R), which must be a valid row.  Byte offsets
// from the slice base fit in 32 bits (checked by the host).
template <typename RowFn>
SC_DEV void tile_dma(const __bf16* g, unsigned ld_bytes, __bf16* tile, int w, int, RowFn rowfn) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int R0 = 16 * w + 8 * j, R = R0 + (lane >> 3);
    const unsigned u = (lane & 7) ^ (lane >> 3);  // slot (lane & 7) of row R holds unit slot ^ (R & 7)
    // the LDS base is the same for the whole wave; readfirstlane lets the
    // compiler keep it in a scalar register when it derives from a loaded value
    lds_dma16(g, (unsigned)rowfn(R) * ld_bytes + 16u * u,
              __builtin_amdgcn_readfirstlane(lds_addr(tile + R0 * Tr<1>::kPitch)));
  }
}

// ------------------------------------------------------ global rows -------
// Global query rows attend to every valid key: a dense strip, split over key
// ranges of kGlobalKeySpan.  Block = 64 global slots x one key range.
struct GrBlock {
  int kc, gc, h, b, bh;
};
SC_DEV GrBlock gr_block(const AttnArgs& a, int lin) {
  GrBlock r;
  r.kc = lin % a.nkc;
  lin /= a.nkc;
  r.gc = lin % a.ngc;
  lin /= a.ngc;
  r.h = lin % a.H;
  r.b = lin / a.H;
  r.bh = r.b * a.H + r.h;
  return r;
}

// Positions of the block's global slots (-1: unused) into pos[0..63]; returns
// whether any is used.  Contains a barrier.
SC_DEV bool gr_slots(const AttnArgs& a, const GrBlock& blk, int L, int* pos) {
  int valid = 0;
  if (threadIdx.x < kBK) {  // 64 staged rows; those beyond the chunk's slots are unused
    const int j = kGlobalChunk * blk.gc + threadIdx.x;
    const int p = threadIdx.x < kGlobalChunk && j < a.G ? a.gpos[(long long)blk.b * a.G + j] : -1;
    valid = p >= 0 && p < L;
    pos[threadIdx.x] = valid ? p : -1;
  }
  return __syncthreads_or(valid);
}

// Forward of the global rows over one key range: running max, sum and
// unnormalised P.V per row, merged later across ranges.
template <int DT>
SC_DEV void gr_fwd_block(const AttnArgs& a, int lin, Smem<DT>& sm) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  constexpr int P = TR::kPitch;
  const GrBlock blk = gr_block(a, lin);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, lr = lane & 15;
  const int L = clampi(a.valid_len[blk.b], 0, a.n);
  const int kbeg = blk.kc * kGlobalKeySpan;
  if (kbeg >= L) return;
  const int kend = min(L, kbeg + kGlobalKeySpan);
  const T* Qg = static_cast<const T*>(a.q) + blk.b * a.bs_in + blk.h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + blk.b * a.bs_in + blk.h * kHeadDim;
  const T* Vg = static_cast<const T*>(a.v) + blk.b * a.bs_in + blk.h * kHeadDim;
  const int ntile = (kend - kbeg + kBK - 1) / kBK;
  // Round r computes key tiles 2r (buffer 0) and 2r + 1 (buffer 1), one per
  // pair of waves: four round trips to memory per 512 keys instead of eight
  // with one tile per step (the blocks are latency-bound: little math per tile).
  // bf16: the pair goes straight into LDS by direct loads once the previous
  // round has read it (rows past kend repeat the last key; they are masked);
  // fp32: through registers, loaded during the previous round.
  constexpr bool kDma = DT == 1;
  Stage<DT> sk[kDma ? 1 : 2], sv[kDma ? 1 : 2];
  auto load_pair = [&](int t0) {  // fp32
#pragma unroll
    for (int x = 0; x < 2; ++x)
      if (t0 + x < ntile) {
        sk[kDma ? 0 : x].load_range(Kg, a.ld_in, kbeg + (t0 + x) * kBK, kend);
        sv[kDma ? 0 : x].load_range(Vg, a.ld_in, kbeg + (t0 + x) * kBK, kend);
      }
  };
  auto issue_pair = [&](int t0) {  // bf16: direct loads into the tile buffers
    if constexpr (kDma) {
      const unsigned ldb = (unsigned)(2 * a.ld_in);
#pragma unroll
      for (int x = 0; x < 2; ++x)
        if (t0 + x < ntile) {
          const int k0 = kbeg + (t0 + x) * kBK;
          tile_dma(reinterpret_cast<const __bf16*>(Kg), ldb, reinterpret_cast<__bf16*>(sm.b[x]), w, lane,
                   [=](int R) { return min(k0 + R, kend - 1); });
          tile_dma(reinterpret_cast<const __bf16*>(Vg), ldb, reinterpret_cast<__bf16*>(sm.c[x]), w, lane,
                   [=](int R) { return min(k0 + R, kend - 1); });
        }
    }
  };
  auto store_pair = [&](int t0) {  // fp32: registers -> LDS; bf16: direct loads, waited for
    if constexpr (kDma) {
      issue_pair(t0);
      wait_dma();
    } else {
#pragma unroll
      for (int x = 0; x < 2; ++x)
        if (t0 + x < ntile) {
          sk[x].store(sm.b[x]);
          sv[x].template store<true>(sm.c[x]);
        }
    }
  };
  // bf16: the first pair is in flight while the slots and the query rows load
  issue_pair(0);
  if (!gr_slots(a, blk, L, sm.pos[0])) {
    if constexpr (kDma) wait_dma();  // no direct load may land after the block has left
    return;
  }
  // wave w serves the 16 slots of group sg = w & 1 over the tiles of parity
  // kh = w >> 1; the two parities are merged at the end
  const int sg = w & 1, kh = w >> 1;
  const int rowpos = sm.pos[0][16 * sg + lr];                  // the lane's global row (-1: unused)
  const bool wlive = __ballot(rowpos >= 0) != 0ull;            // some slot of the group is used
  typename TR::Frag qf[TR::kChunks];
  if constexpr (kDma) {
    // query fragments straight from memory (the same dims per lane group as
    // the key fragments; unused slots zero)
    const T* qrow = Qg + (long long)max(rowpos, 0) * a.ld_in;
    const bf16x8 z = {};
    qf[0] = rowpos >= 0 ? *reinterpret_cast<const bf16x8*>(qrow + 8 * g) : z;
    qf[1] = rowpos >= 0 ? *reinterpret_cast<const bf16x8*>(qrow + 32 + 8 * g) : z;
    wait_dma();
    __syncthreads();
  } else {
    {
      Stage<DT> sq;
      const int* sp = sm.pos[0];
      sq.load_rows(Qg, a.ld_in, [&](int row) { return sp[row]; });
      load_pair(0);
      sq.store(sm.b[1]);
    }
    __syncthreads();
    TR::load_frags(sm.b[1], 16 * sg + lr, g, qf);
    __syncthreads();  // every wave holds its query fragments before b[1] is reused
    store_pair(0);
    __syncthreads();
  }
  float m_use = kNegBig, l_run = 0.f;
  f32x4 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int t0 = 0; t0 < ntile; t0 += 2) {
    const bool more = t0 + 2 < ntile;
    if (!kDma && more) load_pair(t0 + 2);
    const int t = t0 + kh, k0 = kbeg + t * kBK;
    if (wlive && t < ntile) {
      if (a.causal) {  // the lane's global row attends keys up to its own position
        const int hi = min(kend - 1, rowpos) - k0;
        softmax_tile<DT, true>(qf, sm.b[kh], sm.c[kh], a.c2, lr, g, m_use, l_run, o,
                               [&](int s4, int i) { return 16 * s4 + 4 * g + i <= hi; });
      } else if (k0 + kBK <= kend) {
        softmax_tile<DT, false>(qf, sm.b[kh], sm.c[kh], a.c2, lr, g, m_use, l_run, o, [](int, int) { return true; });
      } else {
        const int hi = kend - 1 - k0;
        softmax_tile<DT, true>(qf, sm.b[kh], sm.c[kh], a.c2, lr, g, m_use, l_run, o,
                               [&](int s4, int i) { return 16 * s4 + 4 * g + i <= hi; });
      }
    }
    if (more) {
      __syncthreads();  // both tiles read before they are overwritten
      store_pair(t0 + 2);
    }
    __syncthreads();
  }
  float l_row = group_sum(l_run);
  // merge the two tile parities of each slot group through LDS (the key tiles
  // are no longer needed): the kh = 1 wave publishes its row state, the
  // kh = 0 wave combines, in that fixed order
  constexpr int kXRow = 68;  // floats per row: 64 dims, max, sum (16-byte aligned rows)
  float* xch = reinterpret_cast<float*>(&sm.b[0][0]);
  float* xrow = xch + (16 * sg + lr) * kXRow;
  if (kh == 1) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) *reinterpret_cast<f32x4*>(xrow + 16 * dt + 4 * g) = o[dt];
    if (g == 0) {
      xrow[64] = m_use;
      xrow[65] = l_row;
    }
  }
  __syncthreads();
  if (kh == 1) return;
  {
    const float m1 = xrow[64], l1 = xrow[65];
    const float m = vmax(m_use, m1);
    const float f0 = fast_exp2(m_use - m), f1 = fast_exp2(m1 - m);
    l_row = l_row * f0 + l1 * f1;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) o[dt] = o[dt] * f0 + *reinterpret_cast<const f32x4*>(xrow + 16 * dt + 4 * g) * f1;
    m_use = m;
  }
  const int slot = kGlobalChunk * blk.gc + 16 * sg + lr;
  const long long idx = ((long long)blk.bh * a.nkc + blk.kc) * a.Gp + slot;
  if (g == 0) {
    a.gr_ml[2 * idx] = m_use;
    a.gr_ml[2 * idx + 1] = l_row;
  }
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) *reinterpret_cast<f32x4*>(a.gr_o + idx * kHeadDim + 16 * dt + 4 * g) = o[dt];
}


// ----------------------------------------------------------- bf16 pass 1 --
// A wave owns kSub1 16-query sub-blocks that share every K fragment and every
// V read.  K/V tiles reach LDS
// through the direct global->LDS loads of gfx950, without staging registers:
// lane i of a wave load fills the 16 bytes at base + 16 i, so the swizzled
// layout is produced by choosing which 16-byte unit of its row lane i fetches.
// 16-query sub-blocks per wave.  Two share every K fragment and V read
// (two MFMAs per LDS read) but need 168 VGPRs (3 waves per SIMD); one needs
// 118 (4 waves per SIMD), which measured 3-5 % faster.
constexpr int kSub1 = 1;
constexpr int kBQ2 = 64 * kSub1;  // queries per block

// One 64-key tile for the query sub-blocks of a wave.  Bit st of `live`
// (wave-uniform) says whether 16-key sub-tile st can hold an allowed pair; in
// masked tiles ok(j, st, i) decides the pair (sub-block j's query, key
// 16 st + 4g + i).  Disallowed logits become -inf, which exp2 maps to 0
// (c2 > 0 is guaranteed by the host).
// S^T = K Q^T of one 64-key tile for both sub-blocks; dead sub-tiles give 0.
// kNst: the tile's first kNst 16-key sub-tiles are computed (4: the whole
// tile; 2: keys 0..31, for gathered global keys that fill half a tile).
template <bool kMasked, int kNst = 4>
SC_DEV void qk_tile2(const bf16x8 (&qf)[kSub1][2], const __bf16* sK, int lr_in, int g_in, unsigned live,
                     f32x4 (&s)[kSub1][4]) {
  using TR = Tr<1>;
  auto is_live = [&](int st) { return !kMasked || ((live >> st) & 1u); };
  const int lr = lr_in, g = g_in;
#pragma unroll
  for (int st = 0; st < kNst; ++st) {
#pragma unroll
    for (int j = 0; j < kSub1; ++j) s[j][st] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (is_live(st)) {
      bf16x8 kf[2];
      TR::load_frags(sK, 16 * st + lr, g, kf);
#pragma unroll
      for (int j = 0; j < kSub1; ++j) {
        s[j][st] = TR::mma(kf[0], qf[j][0], s[j][st]);
        s[j][st] = TR::mma(kf[1], qf[j][1], s[j][st]);
      }
    }
  }
}

// Row maxima of a tile in log2 units (per sub-block).
// Maxima of the lane's own logits of a tile (raw, unscaled), per sub-block.
// (a tree of three-input maxima: 8 for 16 values, 4 for 8)
template <int kNst = 4>
SC_DEV void lane_max2(const f32x4 (&s)[kSub1][4], float (&lmax)[kSub1]) {
  auto max3 = [](float a, float b, float c) { return vmax(vmax(a, b), c); };
#pragma unroll
  for (int j = 0; j < kSub1; ++j) {
    float v[16];
#pragma unroll
    for (int st = 0; st < kNst; ++st)
#pragma unroll
      for (int i = 0; i < 4; ++i) v[4 * st + i] = s[j][st][i];
    if constexpr (kNst == 4) {
      const float r0 = max3(v[0], v[1], v[2]), r1 = max3(v[3], v[4], v[5]), r2 = max3(v[6], v[7], v[8]);
      const float r3 = max3(v[9], v[10], v[11]), r4 = max3(v[12], v[13], v[14]);
      lmax[j] = vmax(max3(r0, r1, r2), max3(r3, r4, v[15]));
    } else {
      lmax[j] = max3(max3(v[0], v[1], v[2]), max3(v[3], v[4], v[5]), vmax(v[6], v[7]));
    }
  }
}

// Raises every running maximum below its tile maximum to it and rescales the
// sums and accumulators (lanes that do not need it scale by 1).  lmax: the
// lanes' own maxima; the tile maximum of a query is taken over its 4 lane
// groups here.
SC_DEV void raise2(const float (&lmax)[kSub1], float c2, float (&m_use)[kSub1], float (&l_run)[kSub1],
                   f32x4 (&o)[kSub1][4]) {
  float tmax[kSub1];
#pragma unroll
  for (int j = 0; j < kSub1; ++j) tmax[j] = group_max(lmax[j]) * c2;
#pragma unroll
  for (int j = 0; j < kSub1; ++j) {
    const bool up = tmax[j] > m_use[j];
    const float f = up ? fast_exp2(m_use[j] - tmax[j]) : 1.0f;
    m_use[j] = up ? tmax[j] : m_use[j];
    l_run[j] *= f;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) o[j][dt] *= f;
  }
}

// P = exp2(S c2 - m) as bf16 MFMA operands, and each query's sum of the
// lane's own P (float32, before rounding).
template <int kNst = 4>
SC_DEV void exp_tile2(const f32x4 (&s)[kSub1][4], float c2, const float (&m_use)[kSub1], bf16x8 (&pb)[kSub1][2],
                      float (&part)[kSub1]) {
#pragma unroll
  for (int j = 0; j < kSub1; ++j) {
    float ps[4];
#pragma unroll
    for (int st = 0; st < kNst; ++st) {
      float p[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) p[i] = fast_exp2(fmaf(s[j][st][i], c2, -m_use[j]));
      ps[st] = (p[0] + p[1]) + (p[2] + p[3]);
#pragma unroll
      for (int i = 0; i < 4; ++i) pb[j][st >> 1][4 * (st & 1) + i] = (__bf16)p[i];
    }
    part[j] = kNst == 4 ? (ps[0] + ps[1]) + (ps[2] + ps[3]) : ps[0] + ps[1];
  }
}

// O^T += V^T P^T for one tile: the V operand comes from transposed reads of
// the row-major tile; lane (g, lr) supplies dims 16dt + 4(lr&3) .. +3 of rows
// 32kc + 4g + lr/4 and 32kc + 16 + 4g + lr/4 (keys in MFMA order)
template <bool kMasked, int kNst = 4>
SC_DEV void pv_tile2(const bf16x8 (&pb)[kSub1][2], const __bf16* sV, f32x4 (&o)[kSub1][4], unsigned live) {
  using TR = Tr<1>;
  auto is_live = [&](int st) { return !kMasked || ((live >> st) & 1u); };
  const int ln = threadIdx.x & 63, lr = ln & 15, g = ln >> 4;
#pragma unroll
  for (int kc = 0; kc < kNst / 2; ++kc) {
    if (!is_live(2 * kc) && !is_live(2 * kc + 1)) continue;
    const int vr = 32 * kc + 4 * g + (lr >> 2), b = (lr >> 1) & 1, e = 4 * (lr & 1);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const i16x4 a0 = lds_read_tr16(sV + TR::off(vr, 2 * dt + b) + e);
      const i16x4 a1 = lds_read_tr16(sV + TR::off(vr + 16, 2 * dt + b) + e);
      const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
      for (int j = 0; j < kSub1; ++j) o[j][dt] = TR::mma(vf, pb[j][kc], o[j][dt]);
    }
  }
}

// One 64-key tile for the query sub-blocks of a wave.  Bit st of `live`
// (wave-uniform) says whether 16-key sub-tile st can hold an allowed pair; in
// masked tiles ok(j, st, i) decides the pair (sub-block j's query, key
// 16 st + 4g + i).  Disallowed logits become -inf, which exp2 maps to 0
// (c2 > 0 is guaranteed by the host).  P is computed with the running max
// first; a logit more than kTau above it makes the lane's sum of P exceed
// 2^kTau, and only then (for the whole wave, when any lane's sum does) are
// the tile maxima taken, the running maxima raised to them and P recomputed.
// So every P stays below 2^kTau, and the maxima are needed only on a raise.
template <bool kMasked, typename OkFn, int kNst = 4>
SC_DEV void softmax_tile2(const bf16x8 (&qf)[kSub1][2], const __bf16* sK, const __bf16* sV, float c2, int lr,
                          int g, float (&m_use)[kSub1], float (&l_run)[kSub1], f32x4 (&o)[kSub1][4], unsigned live,
                          OkFn ok) {
  f32x4 s[kSub1][4];
  qk_tile2<kMasked, kNst>(qf, sK, lr, g, live, s);
  if constexpr (kMasked) {
#pragma unroll
    for (int j = 0; j < kSub1; ++j)
#pragma unroll
      for (int st = 0; st < kNst; ++st)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          s[j][st][i] = (((live >> st) & 1u) && ok(j, st, i)) ? s[j][st][i] : -INFINITY;
  }
  bf16x8 pb[kSub1][2];
  float part[kSub1];
  exp_tile2<kNst>(s, c2, m_use, pb, part);
  bool over = false;
#pragma unroll
  for (int j = 0; j < kSub1; ++j) over |= part[j] > kRaiseSum;
  if (__builtin_amdgcn_ballot_w64(over) != 0ull) {
    float lmax[kSub1];
    lane_max2<kNst>(s, lmax);
    raise2(lmax, c2, m_use, l_run, o);
    exp_tile2<kNst>(s, c2, m_use, pb, part);
  }
#pragma unroll
  for (int j = 0; j < kSub1; ++j) l_run[j] += part[j];
  pv_tile2<kMasked, kNst>(pb, sV, o, live);
}

// Pass 1 for bf16: O, LSE and the log2 LSE of the block's kBQ2 queries.
SC_DEV void window_fwd_v2(const AttnArgs& a, int bh, int qb, Smem<1>& sm, uint32_t* sDyn) {
  using T = __bf16;
  const WinBlock wb = win_block<kBQ2>(a, bh, qb);
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6), g = lane >> 4,
            lr = lane & 15;
  const int n = a.n, r = a.r, L = wb.L, q0 = wb.q0, kt0 = wb.kt0, kt1 = wb.kt1, nkt = wb.nkt;
  // reach of the band after the query: r, or 0 in the causal variant (where a
  // global key after the query is not attended either)
  const bool causal = a.causal != 0;
  const int rh = causal ? 0 : r;
  const long long ld = a.ld_in;
  const unsigned ldb = (unsigned)(2 * a.ld_in);
  const T* Qg = static_cast<const T*>(a.q) + wb.b * a.bs_in + wb.h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + wb.b * a.bs_in + wb.h * kHeadDim;
  const T* Vg = static_cast<const T*>(a.v) + wb.b * a.bs_in + wb.h * kHeadDim;
  T* Og = static_cast<T*>(a.out) + wb.b * a.bs_out + wb.h * kHeadDim;
  float* lseg = a.lse ? a.lse + (long long)wb.bh * n : nullptr;
  float* l2g = a.win_lse2 ? a.win_lse2 + (long long)wb.bh * n : nullptr;

  if (q0 >= L) {  // padding block: zero output rows (unless the caller never reads them)
    if (!a.skip_pad_out)
      for (int c = tid; c < kBQ2 * 8; c += kThreads) {
        const int q = q0 + (c >> 3);
        if (q < n) zero16(Og + (long long)q * a.ld_out + 8 * (c & 7));
      }
    for (int i = tid; i < kBQ2; i += kThreads)
      if (q0 + i < n) {
        if (lseg) lseg[q0 + i] = -INFINITY;
        if (l2g) l2g[q0 + i] = INFINITY;
      }
    return;
  }
  uint32_t* sBits = sDyn;
  int* sXList = reinterpret_cast<int*>(sDyn + a.rwp / 32 + 2);
  auto band_rows = [&](int k0) { return [=](int R) { return min(k0 + R, kt1 - 1); }; };
  // the global positions (up to 64 slots: one per lane of wave 0), the first
  // K/V tile and the query fragments are in flight together
  const bool small_g = a.G <= kBK;
  const int* gpb = wb.nxc ? a.gpos + (long long)wb.b * a.G : nullptr;
  const int p_lane = (small_g && gpb && w == 0 && lane < a.G) ? gpb[lane] : -1;
  tile_dma(Kg, ldb, sm.b[0], w, lane, band_rows(kt0));
  tile_dma(Vg, ldb, sm.c[0], w, lane, band_rows(kt0));
  // query fragments straight from HBM (rows clamped below L; same dims per
  // lane group as the key fragments)
  constexpr int kWQ = 16 * kSub1;  // queries per wave
  const int qa = q0 + kWQ * w;
  bf16x8 qf[kSub1][2];
#pragma unroll
  for (int j = 0; j < kSub1; ++j) {
    const T* qrow = Qg + (long long)min(qa + 16 * j + lr, L - 1) * ld;
    qf[j][0] = *reinterpret_cast<const bf16x8*>(qrow + 8 * g);
    qf[j][1] = *reinterpret_cast<const bf16x8*>(qrow + 32 + 8 * g);
  }
  // bitmask of in-band global keys, the list of 64-slot chunks with keys
  // outside [kt0, kt1), and the first listed chunk compacted into sm.pos[1]
  const int ntile = small_g ? win_tables_small(a, wb, p_lane, w, lane, sBits, sXList, &sm.misc[0], sm.pos[1],
                                               &sm.misc[2])
                            : win_tables2(a, wb, sBits, sXList, &sm.misc[0], sm.pos[1], &sm.misc[2]);
  const int nx = __builtin_amdgcn_readfirstlane(ntile - nkt);  // block-uniform (read from LDS)
  const bool hasg = nx > 0;
  auto gbit = [&](int k) -> bool {
    const int o = k - kt0;
    return (sBits[o >> 5] >> (o & 31)) & 1u;
  };
  // Global keys outside the block's key range, one 64-slot chunk of the
  // global list per tile, compacted (used slots first, in slot order) so that
  // they fill the first rows of the tile.  gather_chunk (further chunks, G >
  // 64) compacts chunk c into sm.pos[buf] (a barrier) and gathers its rows.
  const int* gp = wb.nxc ? a.gpos + (long long)wb.b * a.G : nullptr;
  auto slot_row = [&](int c, int row) {
    const int j = kBK * c + row;
    const int p = j < a.G ? gp[j] : -1;
    return (p >= 0 && p < L && (p < kt0 || (!causal && p >= kt1))) ? p : -1;
  };
  auto gather_rows = [&](int buf, int cnt) {
    auto rows = [&](int R) { return R < cnt ? sm.pos[buf][R] : kt0; };
    tile_dma(Kg, ldb, sm.b[buf], w, lane, rows);
    tile_dma(Vg, ldb, sm.c[buf], w, lane, rows);
  };
  auto gather_chunk = [&](int c, int buf) -> int {
    if (tid < kBK) {  // wave 0: one slot per lane
      const int p = slot_row(c, tid);
      const unsigned long long m = __ballot(p >= 0);
      const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
      if (p >= 0) sm.pos[buf][rank] = p;
      if (tid == 0) sm.misc[1 + buf] = __popcll(m);
    }
    __syncthreads();
    const int cnt = sm.misc[1 + buf];
    gather_rows(buf, cnt);
    return cnt;
  };
  const int gcnt0 = hasg ? sm.misc[2] : 0;
  float m_use[kSub1], l_run[kSub1];
  f32x4 o[kSub1][4];
#pragma unroll
  for (int j = 0; j < kSub1; ++j) {
    m_use[j] = kNegBig;
    l_run[j] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) o[j][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // all vector loads so far (the first tiles, the query fragments) complete
  // here; the compiler-visible wait keeps it from waiting for the query loads
  // inside the tile loop, where the prefetch loads are in flight
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  wait_dma();
  __syncthreads();
  // a gathered chunk: every query of the block attends its first cnt keys
  // (out-of-band global keys; in the causal variant only those before the
  // block are listed); half a tile when they fit in 32 rows
  auto glob_tile = [&](int buf, int cnt) {
    const unsigned live = (cnt > 0 ? 1u : 0u) | (cnt > 16 ? 2u : 0u) | (cnt > 32 ? 4u : 0u) | (cnt > 48 ? 8u : 0u);
    auto ok = [&](int, int st, int i) { return 16 * st + 4 * g + i < cnt; };
    if (cnt <= 32)
      softmax_tile2<true, decltype(ok), 2>(qf, sm.b[buf], sm.c[buf], a.c2, lr, g, m_use, l_run, o, live, ok);
    else
      softmax_tile2<true, decltype(ok), 4>(qf, sm.b[buf], sm.c[buf], a.c2, lr, g, m_use, l_run, o, live, ok);
  };

  // per-lane band bounds of sub-block j relative to a tile start, shifted by
  // the lane group's key offset 4g: key 16st + i of the lane is allowed when
  // it lies in [lo - k0, hi - k0]
  int lo[kSub1], hi[kSub1];
#pragma unroll
  for (int j = 0; j < kSub1; ++j) {
    const int q = qa + 16 * j + lr;
    lo[j] = q - r - 4 * g;
    hi[j] = min(q + rh, kt1 - 1) - 4 * g;
  }
  // Pipeline steps: band tile 0, then (hasg) the first gathered global chunk,
  // then band tiles 1 .. nkt-1; step s computes from buffer s & 1 while the
  // next step's data arrive in the other.  Band tile t therefore lives in
  // buffer t & 1, or (t + 1) & 1 after the global chunk.
  const int par = hasg ? 1 : 0;
  auto bufof = [&](int t) { return (t + (t > 0 ? par : 0)) & 1; };
  auto load_band = [&](int t) {
    const int k1 = kt0 + t * kBK;
    tile_dma(Kg, ldb, sm.b[bufof(t)], w, lane, band_rows(k1));
    tile_dma(Vg, ldb, sm.c[bufof(t)], w, lane, band_rows(k1));
  };
  // every tile step: load the next step's data into the other buffer,
  // compute, wait for the load, barrier (the same sequence in all three
  // phases below; band tile 0 and the global chunk are peeled off)
  auto issue = [&](int t) {
    if (t + 1 < nkt) load_band(t + 1);
  };
  auto finish = [&](int t) {
    if (t + 1 < nkt) wait_dma();
    __syncthreads();
  };
  // tiles that need a mask (band edges, global keys) or are skipped
  auto edge_tile = [&](int t) {
    const int buf = bufof(t), k0 = kt0 + t * kBK;
    const unsigned long long gall = tile_gmask(sBits, t, wb.nwords);
    const bool near = k0 <= qa + kWQ - 1 + rh && k0 + kBK - 1 >= qa - r;
    if (!near && gall == 0ull) return;
    const int wlo = qa - r - k0, whi = min(qa + kWQ - 1 + rh, kt1 - 1) - k0;
    unsigned live = 0u;
#pragma unroll
    for (int st = 0; st < 4; ++st)
      live |= (unsigned)((16 * st + 15 >= wlo && 16 * st <= whi) || ((gall >> (16 * st)) & 0xFFFFull) != 0ull) << st;
    int lt[kSub1], ht[kSub1];
#pragma unroll
    for (int j = 0; j < kSub1; ++j) {
      lt[j] = lo[j] - k0;
      ht[j] = hi[j] - k0;
    }
    // a band edge is one-sided in most tiles: the band starts inside the
    // tile for some query (nlo) or ends inside it (nhi), wave-uniform
    const bool nlo = qa + kWQ - 1 - r - k0 > 0, nhi = min(qa + rh, kt1 - 1) - k0 < kBK - 1;
    if (gall == 0ull && !nhi) {
      softmax_tile2<true>(qf, sm.b[buf], sm.c[buf], a.c2, lr, g, m_use, l_run, o, live,
                          [&](int j, int st, int i) { return 16 * st + i >= lt[j]; });
    } else if (gall == 0ull && !nlo) {
      softmax_tile2<true>(qf, sm.b[buf], sm.c[buf], a.c2, lr, g, m_use, l_run, o, live,
                          [&](int j, int st, int i) { return 16 * st + i <= ht[j]; });
    } else if (gall == 0ull) {
      softmax_tile2<true>(qf, sm.b[buf], sm.c[buf], a.c2, lr, g, m_use, l_run, o, live, [&](int j, int st, int i) {
        const int c = 16 * st + i;
        return (c >= lt[j]) & (c <= ht[j]);
      });
    } else {
      const unsigned long long gm = gall >> (4 * g);
      // a global key is attended by every query, or (causal) by the queries
      // at or after it
      softmax_tile2<true>(qf, sm.b[buf], sm.c[buf], a.c2, lr, g, m_use, l_run, o, live, [&](int j, int st, int i) {
        const int c = 16 * st + i;
        const bool band = (c >= lt[j]) & (c <= ht[j]);
        return band | (((gm >> c) & 1ull) != 0ull && c <= (causal ? ht[j] : 1 << 30));
      });
    }
  };
  // interior tiles [ia, ib) of this wave: every key of the tile lies in the
  // band of all the wave's queries and below kt1 (global keys among them are band
  // keys), so no mask is needed
  const int ia = clampi(-((kt0 - (qa + kWQ - 1 - r)) >> 6), 0, nkt);
  const int ib = clampi(((min(qa + rh, kt1 - 1) - (kBK - 1) - kt0) >> 6) + 1, ia, nkt);
  auto interior_tile = [&](int t) {
    const int buf = bufof(t);
    softmax_tile2<false>(qf, sm.b[buf], sm.c[buf], a.c2, lr, g, m_use, l_run, o, 0xFu,
                         [](int, int, int) { return true; });
  };
  // step 0: band tile 0 (interior for this wave only when ia == 0 < ib)
  // while the global chunk's gather (or band tile 1) arrives
  if (hasg)
    gather_rows(1, gcnt0);
  else
    issue(0);
  if (ia == 0 && ib > 0)
    interior_tile(0);
  else
    edge_tile(0);
  if (hasg || nkt > 1) wait_dma();
  __syncthreads();
  // step 1 (hasg): the gathered global chunk while band tile 1 arrives
  if (hasg) {
    if (nkt > 1) load_band(1);
    glob_tile(1, gcnt0);
    if (nkt > 1) wait_dma();
    __syncthreads();
  }
  int t = 1;
  for (; t < ia; ++t) {
    issue(t);
    edge_tile(t);
    finish(t);
  }
  // interior loop: one variant, no mask
  for (t = max(t, ia); t < ib; ++t) {
    issue(t);
    interior_tile(t);
    finish(t);
  }
  for (; t < nkt; ++t) {
    issue(t);
    edge_tile(t);
    finish(t);
  }
  // further chunks of out-of-band global keys (more than 64 global slots;
  // not pipelined)
  for (int x = 1; x < nx; ++x) {
    const int cnt = gather_chunk(sXList[x], 0);
    wait_dma();
    __syncthreads();
    glob_tile(0, cnt);
    __syncthreads();
  }

#pragma unroll
  for (int j = 0; j < kSub1; ++j) {
    const float l_row = group_sum(l_run[j]);
    const int qrow = qa + 16 * j + lr;
    const bool qin = qrow < L;
    const bool qvalid = qin && !gbit(qrow);  // qrow in [q0, L) lies inside [kt0, kt1)
    const float lse2 = m_use[j] + fast_log2(l_row);
    if (qvalid) {
      const float inv = 1.0f / l_row;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
        store_row4<1>(Og + (long long)qrow * a.ld_out + 16 * dt + 4 * g, o[j][dt] * inv);
      if (g == 0 && lseg) lseg[qrow] = lse2 * kLn2;
    } else if (!qin && qrow < n) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
        store_row4<1>(Og + (long long)qrow * a.ld_out + 16 * dt + 4 * g, f32x4{0.f, 0.f, 0.f, 0.f});
      if (g == 0 && lseg) lseg[qrow] = -INFINITY;
    }
    // excluded rows (global or padding) get +inf: their column-sum probabilities are 0
    if (g == 0 && l2g && qrow < n) l2g[qrow] = qvalid ? lse2 : INFINITY;
  }
}

// Work of launch 1 per (sequence, head) pair and key span: kSpanQB window
// blocks, then the span's global-row blocks (one per 32-slot group).
static_assert(kBQ == kBQ2 && kGlobalKeySpan % kBQ == 0, "window blocks tile the key span");
constexpr int kSpanQB = kGlobalKeySpan / kBQ;
struct FwdSpan {
  int per;  // blocks per span
};

__host__ __device__ inline FwdSpan fwd_span(const AttnArgs& a) { return {kSpanQB + (a.n_gr > 0 ? a.ngc : 0)}; }

// Launch 1: the window pass-1 blocks and the global-row forward blocks (when
// there are global tokens).  Span by span (a.span_major: sequences up to
// kSpanOrderMaxN tokens, and the pruned layers of a stack): a (sequence,
// head) pair's work of key span c (kGlobalKeySpan keys) is the window blocks
// of its queries, then the global-row blocks of its keys, which the window
// blocks just read (they are still in the XCD's L2); the pairs are dealt
// round-robin to the XCDs, a pair's work on one XCD (xcd_span_map).
// Otherwise (longer sequences) the window blocks come first, pair by pair
// (xcd_pair_map), and the global-row blocks last, where they fill the window
// blocks' uneven tail.
template <int DT>
__global__ __launch_bounds__(kThreads) SC_OCC(DT == 1 ? 3 : 2) void k_attn_fwd(AttnArgs a) {
  __shared__ Smem<DT> sm;
  extern __shared__ uint32_t sDyn[];
  if (!a.span_major) {
    const int nwin = a.nqb * a.H * a.B;
    if ((int)blockIdx.x >= nwin) {
      gr_fwd_block<DT>(a, blockIdx.x - nwin, sm);
      return;
    }
    int bh, qb;
    xcd_pair_map(blockIdx.x, a.nqb, a.H * a.B, bh, qb);
    if constexpr (DT == 1)
      window_fwd_v2(a, bh, qb, sm, sDyn);
    else
      window_fwd_block<DT>(a, bh, qb, sm, sDyn);
    return;
  }
  const FwdSpan f = fwd_span(a);
  int bh, c, o;
  xcd_span_map(blockIdx.x, a.nkc, f.per, a.H * a.B, bh, c, o);
  if (o >= kSpanQB) {
    gr_fwd_block<DT>(a, (bh * a.ngc + (o - kSpanQB)) * a.nkc + c, sm);
    return;
  }
  const int qb = c * kSpanQB + o;
  if (qb >= a.nqb) return;  // the last span's missing query blocks
  if constexpr (DT == 1)
    window_fwd_v2(a, bh, qb, sm, sDyn);
  else
    window_fwd_block<DT>(a, bh, qb, sm, sDyn);
}

// -------------------------------------------------------- column sums ------
// Column sums of the exact probabilities, key-outer: a block owns 64 keys,
// keeps their K fragments in registers and walks the query tiles that reach
// them, so every key's sum over queries is finished inside the block.
//   band columns    keys k0..k0+63 of a sequence; queries of their band;
//                   global keys are skipped (their columns are dense)
//   global columns  64 global slots; queries of one 512-query range
// Query rows come with their log2-LSE from pass 1 (+inf for global and
// padding rows, whose own probabilities are counted by the global-row blocks).
template <int DT, bool kBandProbs>
SC_DEV void band_col_block(const AttnArgs& a, int bh, int kb, SmemCol<DT>& sm) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  constexpr int P = TR::kPitch;
  const int h = bh % a.H, b = bh / a.H;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, lr = lane & 15;
  const int n = a.n, r = a.r, G = a.G;
  const int L = clampi(a.valid_len[b], 0, n);
  const int k0 = kb * kBK;
  if (k0 >= L) return;  // the score reduction reads keys below L only
  const int kend = min(L, k0 + kBK);
  const T* Qg = static_cast<const T*>(a.q) + b * a.bs_in + h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + b * a.bs_in + h * kHeadDim;
  const float* l2g = a.win_lse2 + (long long)bh * n;
  const int* gp = (a.gpos && G > 0) ? a.gpos + (long long)b * G : nullptr;
  uint32_t* gmask = reinterpret_cast<uint32_t*>(sm.misc);
  if (tid < 2) gmask[tid] = 0u;
  {
    Stage<DT> sk;
    sk.load_range(Kg + (long long)k0 * a.ld_in, a.ld_in, 0, kend - k0);
    sk.store(sm.a);
  }
  __syncthreads();
  for (int j = tid; j < (gp ? G : 0); j += kThreads) {
    const int p = gp[j];
    if (p >= k0 && p < kend) atomicOr(&gmask[(p - k0) >> 5], 1u << ((p - k0) & 31));
  }
  const int qlo = max(0, k0 - r), qhi = min(L, k0 + kBK + r);
  const int nqt = (qhi - qlo + kBQ - 1) / kBQ;
  Stage<DT> sq;
  float lreg = INFINITY;
  auto load = [&](int t) {
    const int qs = qlo + t * kBQ;
    sq.load_range(Qg, a.ld_in, qs, qhi);
    if (tid < kBQ) lreg = qs + tid < qhi ? l2g[qs + tid] : INFINITY;
  };
  auto store = [&](int buf) {
    sq.store(sm.b[buf]);
    if (tid < kBQ) sm.l[buf][tid] = lreg;
  };
  load(0);
  store(0);
  __syncthreads();
  typename TR::Frag kf[TR::kChunks];
  TR::load_frags(sm.a, 16 * w + lr, g, kf);
  const int key = k0 + 16 * w + lr;
  const bool kuse = key < kend && !((gmask[(key - k0) >> 5] >> ((key - k0) & 31)) & 1u);
  float* bpb = kBandProbs ? a.bp_band + (long long)bh * n * a.bw : nullptr;
  float cs = 0.f;
  for (int t = 0; t < nqt; ++t) {
    const int buf = t & 1;
    if (t + 1 < nqt) load(t + 1);
    const int qs = qlo + t * kBQ;
    // allowed: |q - key| <= r with q = qs + qq, qq = 16*qst + 4g + i
    const int lo = key - r - qs, hi = key + r - qs;
    auto ok = [&](int qst, int i) {
      const int qq = 16 * qst + 4 * g + i;
      return (qq >= lo) & (qq <= hi);
    };
    if constexpr (kBandProbs) {
      cs += col_tile<DT, true>(kf, sm.b[buf], sm.l[buf], a.c2, lr, g, ok, [&](int qq, float p) {
        const int q = qs + qq;
        if (kuse && q < L && p != 0.f && abs(q - key) <= a.rb) bpb[(long long)q * a.bw + (key - q + a.rb)] = p;
      });
    } else {
      const bool interior = qs >= k0 + kBK - 1 - r && qs + kBQ - 1 <= k0 + r;
      cs += interior ? col_tile<DT, false>(kf, sm.b[buf], sm.l[buf], a.c2, lr, g, ok, NoEmit{})
                     : col_tile<DT, true>(kf, sm.b[buf], sm.l[buf], a.c2, lr, g, ok, NoEmit{});
    }
    if (t + 1 < nqt) store(buf ^ 1);
    __syncthreads();
  }
  cs = group_sum(cs);
  if (a.part_band && g == 0 && key < n) a.part_band[(long long)bh * n + key] = kuse ? cs : 0.f;
}


// --------------------------------------- bf16 band columns, 32 keys a wave --
// A block owns 128 keys (4 waves x 32 as two 16-key sub-blocks that share
// every query fragment), keeps their K fragments in registers and walks the
// 64-query tiles that reach them.  Query tiles and their log2-LSE arrive by
// direct global->LDS loads, double-buffered.
constexpr int kBK2 = 128;

// Direct load of 4 bytes per lane: lane i's dword lands at lds + 4 i.
SC_DEV void lds_dma4(const void* base, unsigned voff, unsigned lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :
               : "v"(voff), "s"(base), "s"(lds)
               : "memory", "m0");
}

// One 64-query tile against the wave's two key sub-blocks.  Lane (g, lr) of
// sub-block j holds key lr and queries 16 qst + 4g + i; the query is allowed
// for key j when 16 qst + i >= lo[j] (tested if kLo) and <= hi[j] (if kHi).
template <bool kLo, bool kHi>
SC_DEV void col_tile2(const bf16x8 (&kf)[2][2], const __bf16* sQ, const float* sL, float c2, int lr, int g,
                      f32x4 (&cs)[2], const int (&lo)[2], const int (&hi)[2]) {
  using TR = Tr<1>;
#pragma unroll
  for (int qst = 0; qst < 4; ++qst) {
    bf16x8 qf[2];
    TR::load_frags(sQ, 16 * qst + lr, g, qf);
    const f32x4 l2 = *reinterpret_cast<const f32x4*>(sL + 16 * qst + 4 * g);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = TR::mma(qf[0], kf[j][0], acc);
      acc = TR::mma(qf[1], kf[j][1], acc);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float p = fast_exp2(fmaf(acc[i], c2, -l2[i]));
        const int c = 16 * qst + i;
        if constexpr (kLo && kHi)
          p = (c >= lo[j]) & (c <= hi[j]) ? p : 0.f;
        else if constexpr (kLo)
          p = c >= lo[j] ? p : 0.f;
        else if constexpr (kHi)
          p = c <= hi[j] ? p : 0.f;
        cs[j][i] += p;
      }
    }
  }
}

SC_DEV void band_col_v2(const AttnArgs& a, int bh, int kb, SmemCol<1>& sm) {
  using TR = Tr<1>;
  using T = __bf16;
  const int h = bh % a.H, b = bh / a.H;
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6), g = lane >> 4,
            lr = lane & 15;
  const int n = a.n, r = a.r;
  const int L = clampi(a.valid_len[b], 0, n);
  const int k0 = kb * kBK2;
  if (k0 >= L) return;  // the score reduction reads keys below L only
  const int kend = min(L, k0 + kBK2);
  const long long ld = a.ld_in;
  const unsigned ldb = (unsigned)(2 * a.ld_in);
  const T* Qg = static_cast<const T*>(a.q) + b * a.bs_in + h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + b * a.bs_in + h * kHeadDim;
  const float* l2g = a.win_lse2 + (long long)bh * n;
  // queries before a key reach it through the band by r, or not at all in the
  // causal variant
  const int rl = a.causal ? 0 : r;
  const int qlo = max(0, k0 - rl), qhi = min(L, k0 + kBK2 + r);
  const int nqt = (qhi - qlo + kBQ - 1) / kBQ;
  // query tile t (rows clamped below qhi) and the log2-LSE of its rows
  // (indices clamped below n; rows at or beyond qhi are masked)
  auto issue = [&](int t, int bf) {
    const int qs = qlo + t * kBQ;
    tile_dma(Qg, ldb, sm.b[bf], w, lane, [=](int R) { return min(qs + R, qhi - 1); });
    if (w == 0) lds_dma4(l2g, 4u * (unsigned)min(qs + lane, n - 1), lds_addr(sm.l[bf]));
  };
  issue(0, 0);
  // K fragments of the wave's 32 keys straight from HBM (rows clamped below kend)
  const int kw0 = k0 + 32 * w;
  bf16x8 kf[2][2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const T* krow = Kg + (long long)min(kw0 + 16 * j + lr, kend - 1) * ld;
    kf[j][0] = *reinterpret_cast<const bf16x8*>(krow + 8 * g);
    kf[j][1] = *reinterpret_cast<const bf16x8*>(krow + 32 + 8 * g);
  }
  // global keys of the block: their band columns are not used
  const int* gp = (a.gpos && a.G > 0) ? a.gpos + (long long)b * a.G : nullptr;
  const int G = gp ? a.G : 0;
  const int p_first = tid < G ? gp[tid] : -1;
  uint32_t* gmask = reinterpret_cast<uint32_t*>(sm.misc);
  if (tid < kBK2 / 32) gmask[tid] = 0u;
  __syncthreads();
  for (int j = tid; j < G; j += kThreads) {
    const int p = j == tid ? p_first : gp[j];
    if (p >= k0 && p < kend) atomicOr(&gmask[(p - k0) >> 5], 1u << ((p - k0) & 31));
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): K fragments, positions
  wait_dma();
  __syncthreads();

  // per-lane bounds: query 16 qst + i of the lane (tile start qs) is allowed
  // for key sub-block j when it lies in [lo[j] - qs, hi[j] - qs]
  int lo[2], hi[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int key = kw0 + 16 * j + lr;
    lo[j] = key - rl - 4 * g;
    hi[j] = min(key + r, qhi - 1) - 4 * g;
  }
  f32x4 cs[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  for (int t = 0; t < nqt; ++t) {
    const int buf = t & 1, qs = qlo + t * kBQ;
    if (t + 1 < nqt) issue(t + 1, buf ^ 1);
    if (qs <= kw0 + 31 + r && qs + kBQ - 1 >= kw0 - rl) {
      if (qs >= kw0 + 31 - rl && qs + kBQ - 1 <= kw0 + r && qs + kBQ <= qhi) {
        col_tile2<false, false>(kf, sm.b[buf], sm.l[buf], a.c2, lr, g, cs, lo, hi);
      } else {
        const int l2[2] = {lo[0] - qs, lo[1] - qs}, h2[2] = {hi[0] - qs, hi[1] - qs};
        col_tile2<true, true>(kf, sm.b[buf], sm.l[buf], a.c2, lr, g, cs, l2, h2);
      }
    }
    if (t + 1 < nqt) wait_dma();
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const float c = group_sum((cs[j][0] + cs[j][1]) + (cs[j][2] + cs[j][3]));
    const int key = kw0 + 16 * j + lr;
    const bool kuse = key < kend && !((gmask[(key - k0) >> 5] >> ((key - k0) & 31)) & 1u);
    if (a.part_band && g == 0 && key < n) a.part_band[(long long)bh * n + key] = kuse ? c : 0.f;
  }
}

template <int DT, bool kBandProbs>
SC_DEV void gcol_block(const AttnArgs& a, int lin, SmemCol<DT>& sm) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  constexpr int P = TR::kPitch;
  const int qr = lin % a.nqr;
  lin /= a.nqr;
  const int gc = lin % a.ngc;
  lin /= a.ngc;
  const int h = lin % a.H, b = lin / a.H, bh = b * a.H + h;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, lr = lane & 15;
  const int n = a.n, G = a.G;
  const int L = clampi(a.valid_len[b], 0, n);
  const int qbeg = qr * kGlobalKeySpan;
  if (qbeg >= L) return;  // the score reduction reads ranges below L only
  const int qend = min(L, qbeg + kGlobalKeySpan);
  const T* Qg = static_cast<const T*>(a.q) + b * a.bs_in + h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + b * a.bs_in + h * kHeadDim;
  const float* l2g = a.win_lse2 + (long long)bh * n;
  const int* gp = a.gpos + (long long)b * G;
  int* pos = sm.pos[0];
  if (tid < kBK) {  // 64 staged rows; those beyond the chunk's slots are unused
    const int j = kGlobalChunk * gc + tid;
    const int p = tid < kGlobalChunk && j < G ? gp[j] : -1;
    pos[tid] = (p >= 0 && p < L) ? p : -1;
  }
  __syncthreads();
  {
    Stage<DT> sk;
    sk.load_rows(Kg, a.ld_in, [&](int row) { return pos[row]; });
    sk.store(sm.a);
  }
  const int nqt = (qend - qbeg + kBQ - 1) / kBQ;
  Stage<DT> sq;
  float lreg = INFINITY;
  auto load = [&](int t) {
    const int qs = qbeg + t * kBQ;
    sq.load_range(Qg, a.ld_in, qs, qend);
    if (tid < kBQ) lreg = qs + tid < qend ? l2g[qs + tid] : INFINITY;
  };
  auto store = [&](int buf) {
    sq.store(sm.b[buf]);
    if (tid < kBQ) sm.l[buf][tid] = lreg;
  };
  load(0);
  store(0);
  __syncthreads();
  // wave w serves the 16 global keys of group kg = w & 1 against the query
  // half qh = w >> 1 (16-query groups 2 qh, 2 qh + 1) of every tile; the two
  // halves' sums are added at the end
  const int kg = w & 1, qh = w >> 1;
  const unsigned qlive = qh ? 0xCu : 0x3u;
  typename TR::Frag kf[TR::kChunks];
  TR::load_frags(sm.a, 16 * kg + lr, g, kf);
  const int slot = kGlobalChunk * gc + 16 * kg + lr;
  const bool kuse = pos[16 * kg + lr] >= 0;
  const bool wlive = __ballot(kuse) != 0ull;  // some of the wave's 16 global keys is used
  float* bpc = kBandProbs ? a.bp_gcol + (long long)bh * n * G : nullptr;
  float cs = 0.f;
  for (int t = 0; t < nqt; ++t) {
    const int buf = t & 1;
    if (t + 1 < nqt) load(t + 1);
    const int qs = qbeg + t * kBQ;
    if (!wlive) {
    } else if constexpr (kBandProbs) {
      cs += col_tile<DT, false>(kf, sm.b[buf], sm.l[buf], a.c2, lr, g, [](int, int) { return true; },
                                [&](int qq, float p) {
                                  const int q = qs + qq;
                                  if (kuse && q < L && p != 0.f) bpc[(long long)q * G + slot] = p;
                                }, qlive);
    } else if (a.causal) {  // a global key is attended by the queries at or after it
      const int kp = pos[16 * kg + lr];
      cs += col_tile<DT, true>(kf, sm.b[buf], sm.l[buf], a.c2, lr, g,
                               [&](int qst, int i) { return qs + 16 * qst + 4 * g + i >= kp; }, NoEmit{}, qlive);
    } else {
      cs += col_tile<DT, false>(kf, sm.b[buf], sm.l[buf], a.c2, lr, g, [](int, int) { return true; }, NoEmit{},
                                qlive);
    }
    if (t + 1 < nqt) store(buf ^ 1);
    __syncthreads();
  }
  cs = group_sum(cs);
  // the qh = 1 wave hands its sum to the qh = 0 wave of the same keys (the
  // staged LSE rows are no longer needed)
  float* xs = sm.l[0];
  if (qh == 1 && g == 0) xs[16 * kg + lr] = cs;
  __syncthreads();
  if (qh == 0) {
    cs += xs[16 * kg + lr];
    if (a.part_extra && g == 0 && slot < G) a.part_extra[((long long)bh * a.nqr + qr) * G + slot] = kuse ? cs : 0.f;
  }
}

// Global rows, second half: merge the key-range partials of the block's 64
// rows into their log2-LSE (and, for the first key range, into their output
// rows and natural LSE), then the rows' probabilities summed per key.
template <int DT, bool kBandProbs>
SC_DEV void gr_col_block(const AttnArgs& a, int lin, SmemCol<DT>& sm) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  constexpr int P = TR::kPitch;
  const GrBlock blk = gr_block(a, lin);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, lr = lane & 15;
  const int L = clampi(a.valid_len[blk.b], 0, a.n);
  const int kbeg = blk.kc * kGlobalKeySpan;
  if (kbeg >= L) return;
  const int kend = min(L, kbeg + kGlobalKeySpan);
  float* pg = a.part_grow ? a.part_grow + ((long long)blk.bh * a.ngc + blk.gc) * a.n : nullptr;
  const bool want_cols = a.part_grow || a.bp_grow;
  if (!want_cols && blk.kc != 0) return;  // only the merge of the output rows is needed
  if (!gr_slots(a, blk, L, sm.pos[0])) {
    if (pg)
      for (int k = kbeg + tid; k < kend; k += kThreads) pg[k] = 0.f;
    return;
  }
  const int* pos = sm.pos[0];
  const int nk = (L + kGlobalKeySpan - 1) / kGlobalKeySpan;
  float* sM = sm.l[1];  // per-row max of the merge
  // merge of the key-chunk partials (m, l) of the block's global rows: thread
  // (row, part) combines chunks part, part + 8, ... (a single round of loads
  // for up to 8 chunks), then 32 threads combine the 8 parts
  static_assert(kThreads == 8 * kGlobalChunk, "merge layout: 8 parts of kGlobalChunk rows");
  float* red = reinterpret_cast<float*>(sm.b[1]);  // [2][8][kGlobalChunk]; b[1] is free until the tile loop
  {
    const int row = tid % kGlobalChunk, part = tid / kGlobalChunk;
    const int slot = kGlobalChunk * blk.gc + row;
    float m = kNegBig, l = 0.f;
    if (pos[row] >= 0)
      for (int kc = part; kc < nk; kc += 8) {
        const long long idx = ((long long)blk.bh * a.nkc + kc) * a.Gp + slot;
        const float mk = a.gr_ml[2 * idx], lk = a.gr_ml[2 * idx + 1];
        const float mn = fmaxf(m, mk);
        l = l * fast_exp2(m - mn) + lk * fast_exp2(mk - mn);
        m = mn;
      }
    red[tid] = m;
    red[kThreads + tid] = l;
  }
  __syncthreads();
  if (tid < kGlobalChunk) {
    float m = kNegBig, l = 0.f;
#pragma unroll
    for (int p = 0; p < 8; ++p) m = fmaxf(m, red[p * kGlobalChunk + tid]);
#pragma unroll
    for (int p = 0; p < 8; ++p) l += red[kThreads + p * kGlobalChunk + tid] * fast_exp2(red[p * kGlobalChunk + tid] - m);
    float lse2 = INFINITY;
    if (pos[tid] >= 0) {
      lse2 = m + fast_log2(l);
      if (blk.kc == 0 && a.lse) a.lse[(long long)blk.bh * a.n + pos[tid]] = lse2 * kLn2;
    }
    sm.l[0][tid] = lse2;
    sM[tid] = m;
  }
  __syncthreads();
  if (blk.kc == 0) {  // output rows of the global queries: 8 dims of one row per thread
    const int row = tid >> 3, d0 = 8 * (tid & 7);
    if (pos[row] >= 0) {
      T* Ob = static_cast<T*>(a.out) + blk.b * a.bs_out + blk.h * kHeadDim;
      const int slot = kGlobalChunk * blk.gc + row;
      const float m = sM[row], lse2 = sm.l[0][row];
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      for (int kc0 = 0; kc0 < nk; kc0 += 4) {  // four chunks' loads in flight together
        f32x4 v[4][2];
        float wt[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int kc = min(kc0 + u, nk - 1);
          const long long idx = ((long long)blk.bh * a.nkc + kc) * a.Gp + slot;
          v[u][0] = *reinterpret_cast<const f32x4*>(a.gr_o + idx * kHeadDim + d0);
          v[u][1] = *reinterpret_cast<const f32x4*>(a.gr_o + idx * kHeadDim + d0 + 4);
          wt[u] = kc0 + u < nk ? fast_exp2(a.gr_ml[2 * idx] - m) : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[i] += v[u][i >> 2][i & 3] * wt[u];
      }
      const float sc = fast_exp2(m - lse2);
#pragma unroll
      for (int i = 0; i < 8; ++i) Ob[(long long)pos[row] * a.ld_out + d0 + i] = (T)(acc[i] * sc);
    }
  }
  if (!want_cols) return;
  const T* Qg = static_cast<const T*>(a.q) + blk.b * a.bs_in + blk.h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + blk.b * a.bs_in + blk.h * kHeadDim;
  const int ntile = (kend - kbeg + kBK - 1) / kBK;
  Stage<DT> stk;
  {
    Stage<DT> sq;
    sq.load_rows(Qg, a.ld_in, [&](int row) { return pos[row]; });
    sq.store(sm.a);
  }
  stk.load_range(Kg, a.ld_in, kbeg, kend);
  stk.store(sm.b[0]);
  __syncthreads();
  float* bpr = kBandProbs ? a.bp_grow + (long long)blk.bh * a.G * a.n : nullptr;
  unsigned qlive = 0u;  // 16-slot groups that hold a used global row
#pragma unroll
  for (int qst = 0; qst < 4; ++qst) qlive |= (unsigned)(__ballot(pos[16 * qst + lr] >= 0) != 0ull) << qst;
  for (int t = 0; t < ntile; ++t) {
    const int buf = t & 1, k0 = kbeg + t * kBK;
    if (t + 1 < ntile) stk.load_range(Kg, a.ld_in, k0 + kBK, kend);
    // this wave's 16 keys as the K operand, the 64 global rows as queries
    typename TR::Frag kf[TR::kChunks];
    TR::load_frags(sm.b[buf], 16 * w + lr, g, kf);
    const int key = k0 + 16 * w + lr;
    const bool kin = key < kend;
    float cs;
    if constexpr (kBandProbs) {
      cs = col_tile<DT, false>(kf, sm.a, sm.l[0], a.c2, lr, g, [](int, int) { return true; }, [&](int qq, float p) {
        const int slot = kGlobalChunk * blk.gc + qq;
        if (kin && slot < a.G && p != 0.f) bpr[(long long)slot * a.n + key] = p;
      }, qlive);
    } else if (a.causal) {  // a global row's probabilities reach the keys up to its position
      cs = col_tile<DT, true>(kf, sm.a, sm.l[0], a.c2, lr, g,
                              [&](int qst, int i) { return key <= pos[16 * qst + 4 * g + i]; }, NoEmit{}, qlive);
    } else {
      cs = col_tile<DT, false>(kf, sm.a, sm.l[0], a.c2, lr, g, [](int, int) { return true; }, NoEmit{}, qlive);
    }
    cs = group_sum(cs);
    if (pg && g == 0 && kin) pg[key] = cs;
    if (t + 1 < ntile) stk.store(sm.b[buf ^ 1]);
    __syncthreads();
  }
}

// Work of launch 2 per (sequence, head) pair and key span: nbc band-column
// blocks, ngr global-row blocks, ngcol global-column blocks.
static_assert(kGlobalKeySpan % kBK2 == 0 && kGlobalKeySpan % kBK == 0, "column blocks tile the key span");
struct ColSpan {
  int nbc, ngr, ngcol, per;
};
template <int DT, bool kBandProbs>
__host__ __device__ inline ColSpan col_span(const AttnArgs& a) {
  constexpr int keys = (DT == 1 && !kBandProbs) ? kBK2 : kBK;  // keys per band-column block
  ColSpan f;
  f.nbc = a.n_bcol > 0 ? kGlobalKeySpan / keys : 0;
  f.ngr = a.n_gr > 0 ? a.ngc : 0;
  f.ngcol = a.n_gcol > 0 ? a.ngc : 0;
  f.per = f.nbc + f.ngr + f.ngcol;
  return f;
}

// Launch 2: global-row column blocks, band-column and global-column blocks
// (the last two only when score partials or the band layout are asked for).
// Span by span (a.span_major, as in launch 1): a (sequence, head) pair's work
// of span c (kGlobalKeySpan keys) is the band-column blocks of its keys, the
// global-row blocks of the same keys, then the global-column blocks of its
// queries, the pairs dealt to the XCDs as in launch 1; the global-row and
// global-column blocks find the span's rows in the L2.  Otherwise the
// global-row blocks come first (long; started early they overlap the rest;
// their count padded to a multiple of 8), then the band-column blocks pair
// by pair (xcd_pair_map), then the global-column blocks.
template <int DT, bool kBandProbs>
__global__ __launch_bounds__(kThreads) SC_OCC(kBandProbs ? 2 : 4) void k_attn_cols(AttnArgs a) {
  __shared__ SmemCol<DT> sm;
  if (!a.span_major) {
    const int ngrp = (a.n_gr + 7) & ~7;
    int blk = blockIdx.x;
    if (blk < ngrp) {
      if (blk < a.n_gr) gr_col_block<DT, kBandProbs>(a, blk, sm);
      return;
    }
    blk -= ngrp;
    if (blk < a.n_bcol) {
      int bh, kb;
      xcd_pair_map(blk, a.nkb, a.H * a.B, bh, kb);
      if constexpr (DT == 1 && !kBandProbs)
        band_col_v2(a, bh, kb, sm);
      else
        band_col_block<DT, kBandProbs>(a, bh, kb, sm);
      return;
    }
    gcol_block<DT, kBandProbs>(a, blk - a.n_bcol, sm);
    return;
  }
  const ColSpan f = col_span<DT, kBandProbs>(a);
  int bh, c, o;
  xcd_span_map(blockIdx.x, a.nkc, f.per, a.H * a.B, bh, c, o);
  if (o < f.nbc) {
    const int kb = c * f.nbc + o;
    if (kb >= a.nkb) return;  // the last span's missing key blocks
    if constexpr (DT == 1 && !kBandProbs)
      band_col_v2(a, bh, kb, sm);
    else
      band_col_block<DT, kBandProbs>(a, bh, kb, sm);
    return;
  }
  o -= f.nbc;
  if (o < f.ngr) {
    gr_col_block<DT, kBandProbs>(a, (bh * a.ngc + o) * a.nkc + c, sm);
    return;
  }
  o -= f.ngr;
  gcol_block<DT, kBandProbs>(a, (bh * a.ngc + o) * a.nqr + c, sm);
}

// ------------------------------------------------------ score reduction ----
// scores[b, k] = (sum over heads of: the band column sum of k, its global
// column (summed over query ranges) if k is global, and the global rows'
// column sums) / (H * L).  Workgroup = 64 keys x 4 head groups.  Fixed order
// everywhere; no atomics.
// Score partials of one layer, as the attention kernels write them.
struct ScorePartials {
  const float* band;  // [B, H, n]      band column sums
  const float* gcol;  // [B, H, nqr, G] global-key columns per 512-query range
  const float* grow;  // [B, H, ngc, n] column sums over the global rows
  int n, H, G, ngc, nqr;
};
// the same pieces, written by k_band_keys and k_band_rows
struct ScorePartialsOut {
  float* band;
  float* gcol;
  float* grow;
};

// Attention that key k receives from head bh = b * H + h, in two steps
// applied in this order: score_head_local gives the band column sum plus the
// global-row sums (chunk by chunk), score_head_global then adds, for a global
// key in slot `slot` (-1: not global), its global-column sums over the nqrv
// query ranges in use.  kNgc >= 0 fixes the number of global-row chunks at
// compile time (it must equal sp.ngc; 0, 1 or 2, else -1).
template <int kNgc>
SC_DEV float score_head_local(const ScorePartials& sp, long long bh, int k) {
  float v = sp.band[bh * sp.n + k];
  if constexpr (kNgc >= 0) {
#pragma unroll
    for (int gc = 0; gc < kNgc; ++gc) v += sp.grow[(bh * sp.ngc + gc) * sp.n + k];
  } else {
    for (int gc = 0; gc < sp.ngc; ++gc) v += sp.grow[(bh * sp.ngc + gc) * sp.n + k];
  }
  return v;
}

SC_DEV float score_head_global(const ScorePartials& sp, long long bh, int slot, int nqrv, float v) {
  if (slot >= 0)
    for (int qr = 0; qr < nqrv; ++qr) v += sp.gcol[(bh * sp.nqr + qr) * sp.G + slot];
  return v;
}

constexpr int kScoreKeys = 64;
constexpr int kScoreGroups = 4;
constexpr int kScorePre = 4;  // heads per group whose band / global-row terms are loaded up front

// Thread = key x head group (group j sums heads j, j + 4, ... from 0 up; the
// groups are added in order and the total divided by H * L).  The band and
// global-row terms of the group's first kScorePre heads are loaded before the
// length and the global positions arrive (they need neither), so the
// workgroup waits on memory about once.  kNgc: the number of global-row
// chunks when fixed at compile time (0, 1 or 2), else -1.
template <int kNgc>
__global__ __launch_bounds__(kScoreKeys * kScoreGroups) void k_score_from_partials(ScorePartials sp,
                                                                                    const int* valid_len,
                                                                                    const int* gpos, float* scores) {
  __shared__ int smap[kScoreKeys];
  __shared__ float red[kScoreGroups][kScoreKeys];
  const int n = sp.n, H = sp.H, G = sp.G;
  const int b = blockIdx.y, kb = blockIdx.x * kScoreKeys, tid = threadIdx.x;
  const int lane = tid % kScoreKeys, hg = tid / kScoreKeys, k = kb + lane;
  float pre[kScorePre];
  {
    const int kk = k < n ? k : n - 1;  // clamped key and head: in bounds, unused values are discarded
#pragma unroll
    for (int i = 0; i < kScorePre; ++i)
      pre[i] = score_head_local<kNgc>(sp, (long long)b * H + min(hg + kScoreGroups * i, H - 1), kk);
  }
  const int L = clampi(valid_len[b], 0, n);
  if (tid < kScoreKeys) smap[tid] = -1;
  __syncthreads();
  if (gpos)
    for (int j = tid; j < G; j += blockDim.x) {
      const int p = gpos[(long long)b * G + j];
      if (p >= kb && p < kb + kScoreKeys && p < L) smap[p - kb] = j;
    }
  __syncthreads();
  float acc = 0.f;
  if (k < L) {
    const int slot = smap[lane];
    const int nqrv = (L + kGlobalKeySpan - 1) / kGlobalKeySpan;
    // a global key's column terms of the first kScorePre heads, eight query
    // ranges at a time with all their loads issued together (ranges past
    // nqrv and heads past H read clamped entries that are discarded), added
    // to each head's band / global-row term in range order
    if (slot >= 0)
      for (int q0 = 0; q0 < nqrv; q0 += 8) {
        float t[kScorePre][8];
#pragma unroll
        for (int i = 0; i < kScorePre; ++i) {
          const long long bh = (long long)b * H + min(hg + kScoreGroups * i, H - 1);
#pragma unroll
          for (int u = 0; u < 8; ++u) t[i][u] = sp.gcol[(bh * sp.nqr + min(q0 + u, nqrv - 1)) * sp.G + slot];
        }
#pragma unroll
        for (int i = 0; i < kScorePre; ++i)
#pragma unroll
          for (int u = 0; u < 8; ++u) pre[i] = q0 + u < nqrv ? pre[i] + t[i][u] : pre[i];
      }
#pragma unroll
    for (int i = 0; i < kScorePre; ++i)
      if (hg + kScoreGroups * i < H) acc += pre[i];
    for (int h = hg + kScoreGroups * kScorePre; h < H; h += kScoreGroups) {
      const long long bh = (long long)b * H + h;
      acc += score_head_global(sp, bh, slot, nqrv, score_head_local<kNgc>(sp, bh, k));
    }
  }
  red[hg][lane] = acc;
  __syncthreads();
  if (hg == 0 && k < n) {
    float tot = 0.f;
#pragma unroll
    for (int j = 0; j < kScoreGroups; ++j) tot += red[j][lane];
    scores[(long long)b * n + k] = k < L ? tot / ((float)H * (float)L) : 0.f;
  }
}

// Paper layout -> the score partials of the fused path, so that the final
// reduction is k_score_from_partials.  The score of key k is its band
// sub-diagonal (entries (i, j) with i - r + j = k; zero at global keys), its
// global column (zero at global rows) and its entries of the global rows.
// Entry (i, j) of a head's band sits at i * (2r + 1) + j = 2r * i + k + r, so
// for a fixed row the entries of consecutive keys are consecutive floats.
// Two launches, both in a fixed order with no atomics:
//   k_band_rows    column blocks (sequence, head, 512-row range), dispatched
//                  first: the global-column block of the range summed per
//                  slot, one row group per 32 threads, the row groups added in
//                  order through LDS.  Row blocks (sequence, head, 128 rows):
//                  each block reads its rows once, front to back; the keys
//                  they reach, [i0 - r, i0 + 128 + r), are cut into segments
//                  of 64 * VEC keys, one per wave at a time, and the wave walks
//                  the segment's rows with kU rows in flight, a lane summing
//                  VEC consecutive keys in row order.  VEC = 4 (16-byte loads)
//                  needs r and n multiples of 4 and a 16-byte aligned layout.
//                  Output: one partial sum per (row block, key of its span).
//   k_band_keys    thread = key: the partials of the row blocks that reach it,
//                  in row-block order, then its global-row entries per 32-slot
//                  chunk.
constexpr int kBandRows = 128;
constexpr int kBandUnroll = 16;

int band_segments(int rb, int vec) { return (kBandRows + 2 * rb + 64 * vec - 1) / (64 * vec); }

template <int VEC>
__global__ __launch_bounds__(256) void k_band_rows(const float* bp, const int* valid_len, int B, int n, int H, int G,
                                                   AttnGeom geo, int nseg, float* parts, ScorePartialsOut po) {
  constexpr int kU = 16;  // rows in flight per wave
  constexpr int kSeg = 64 * VEC;
  __shared__ float red[8 * 32];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const long long ncol = G > 0 ? (long long)B * H * geo.nqr : 0;
  const float* band = bp;
  if ((long long)blockIdx.x < ncol) {
    const float* gcol = band + (size_t)B * H * n * geo.bw;
    const int kRG = nthr >> 5;  // row groups (at most 8)
    const int qr = (int)(blockIdx.x % geo.nqr), bh = (int)(blockIdx.x / geo.nqr), b = bh / H;
    const int L = clampi(valid_len[b], 0, n);
    const int rg = tid >> 5, sl = tid & 31;
    const int r0 = qr * kGlobalKeySpan, r1 = min(L, r0 + kGlobalKeySpan);
    for (int s0 = 0; s0 < G; s0 += 32) {
      const int slot = s0 + sl, sc = min(slot, G - 1);  // clamped: in bounds, masked below
      float acc[kBandUnroll] = {};
      int i = r0 + rg;
      for (; i + kRG * (kBandUnroll - 1) < r1; i += kRG * kBandUnroll) {
#pragma unroll
        for (int u = 0; u < kBandUnroll; ++u) acc[u] += gcol[((size_t)bh * n + i + kRG * u) * G + sc];
      }
      for (int u = 0; i < r1; i += kRG, ++u) acc[u] += gcol[((size_t)bh * n + i) * G + sc];
      float t = 0.f;
#pragma unroll
      for (int u = 0; u < kBandUnroll; ++u) t += acc[u];
      red[rg * 32 + sl] = slot < G ? t : 0.f;
      __syncthreads();
      if (rg == 0 && slot < G) {
        float tot = 0.f;
        for (int j = 0; j < kRG; ++j) tot += red[j * 32 + sl];
        po.gcol[((size_t)bh * geo.nqr + qr) * G + slot] = tot;
      }
      __syncthreads();
    }
    return;
  }
  const int np = (n + kBandRows - 1) / kBandRows;
  const long long blk = blockIdx.x - ncol;
  const int p = (int)(blk % np), bh = (int)(blk / np), b = bh / H;
  const int L = clampi(valid_len[b], 0, n);
  const int rb = geo.rb;
  const int i0 = p * kBandRows, i1 = min(L, i0 + kBandRows);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), nw = nthr >> 6;
  const char* head = reinterpret_cast<const char*>(band + (size_t)bh * n * geo.bw);
  const size_t rstride = 8ull * (unsigned)rb;  // bytes per row along a sub-diagonal
  float* out = parts + ((size_t)bh * np + p) * nseg * kSeg;
  for (int seg = wave; seg < nseg; seg += nw) {
    const int kseg = i0 - rb + seg * kSeg;  // first key of the segment (may lie outside [0, n))
    const int kl = kseg + lane * VEC;
    // the segment's rows: those of the block that reach one of its keys
    const int r0 = max(i0, kseg - rb), r1 = min(i1, kseg + kSeg + rb);
    float sum[VEC] = {};
    if (r0 < r1 && kseg < n && kseg + kSeg > 0) {
      // entry (i, key) at 2r * i + key + r lies inside the head's layout for
      // every row i < n and key < n: keys outside [0, n) address a clamped key
      // and are masked, and so are the clamped rows of the last round
      const unsigned loff = (unsigned)(clampi(kl, 0, n - VEC) + rb) * 4u;  // below 8 n
      for (int ib = r0; ib < r1; ib += kU) {
        float v[kU][VEC];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          const char* row = head + rstride * (size_t)min(ib + u, r1 - 1);
          if constexpr (VEC == 4) {
            const f32x4 w = *reinterpret_cast<const f32x4*>(row + loff);
            v[u][0] = w[0], v[u][1] = w[1], v[u][2] = w[2], v[u][3] = w[3];
          } else {
            v[u][0] = *reinterpret_cast<const float*>(row + loff);
          }
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          const int i = ib + u;
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            // entry j = key - i + r of row i exists for 0 <= j <= 2r
            const bool in = i < r1 && (unsigned)(kl + e) < (unsigned)n &&
                            (unsigned)(kl + e - i + rb) <= 2u * (unsigned)rb;
            sum[e] += in ? v[u][e] : 0.f;
          }
        }
      }
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) out[seg * kSeg + lane * VEC + e] = sum[e];
  }
}

__global__ __launch_bounds__(256) void k_band_keys(const float* bp, const int* valid_len, int B, int n, int H, int G,
                                                   AttnGeom geo, int nseg, int seg_keys, const float* parts,
                                                   ScorePartialsOut po) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int bh = blockIdx.y, b = bh / H;
  if (k >= n) return;
  const int L = clampi(valid_len[b], 0, n);
  const int np = (n + kBandRows - 1) / kBandRows, span = nseg * seg_keys, rb = geo.rb;
  float s = 0.f;
  if (k < L) {
    // row blocks holding a row of [k - r, k + r] below L; key k is slot
    // k - (p * 128 - r) < 128 + 2r of block p's span
    const int pa = max(0, k - rb) / kBandRows, pb = min(L - 1, k + rb) / kBandRows;
    for (int p = pa; p <= pb; ++p) s += parts[((size_t)bh * np + p) * span + (k - p * kBandRows + rb)];
  }
  // keys at or beyond L are reached by rows below L only where the entries
  // are zero
  po.band[(size_t)bh * n + k] = k < L ? s : 0.f;
  const float* grow = bp + (size_t)B * H * n * geo.bw + (size_t)B * H * n * G;
  // a chunk's slots loaded together (slots past G read the last slot's row
  // and are dropped), then added in slot order
  for (int c = 0; c < geo.ngc; ++c) {
    float g = 0.f;
    if (k < L) {
      float t[kGlobalChunk];
#pragma unroll
      for (int x = 0; x < kGlobalChunk; ++x)
        t[x] = grow[((size_t)bh * G + min(c * kGlobalChunk + x, G - 1)) * n + k];
#pragma unroll
      for (int x = 0; x < kGlobalChunk; ++x) g = c * kGlobalChunk + x < G ? g + t[x] : g;
    }
    po.grow[((size_t)bh * geo.ngc + c) * n + k] = g;
  }
}

}  // namespace

// ------------------------------------------------------------- host side ---
AttnGeom attn_geom(int n, int window, int G) {
  AttnGeom g;
  g.r = window / 2 < n ? window / 2 : n;
  g.nqb = (n + kBQ - 1) / kBQ;
  const long long rw = (long long)kBQ + 2LL * g.r;
  g.rwp = (int)(rw < n ? rw : n);
  g.ngc = (G + kGlobalChunk - 1) / kGlobalChunk;
  g.Gp = g.ngc * kGlobalChunk;
  g.nkc = (n + kGlobalKeySpan - 1) / kGlobalKeySpan;
  g.nkb = (n + kBK - 1) / kBK;
  g.nqr = (n + kGlobalKeySpan - 1) / kGlobalKeySpan;
  g.rb = window / 2 < n - 1 ? window / 2 : n - 1;
  g.bw = 2 * g.rb + 1;
  return g;
}

size_t partials_floats(int B, int H, int n, const AttnGeom& g, int G) {
  return (size_t)B * H * ((size_t)n + (size_t)g.nqr * G + (size_t)g.ngc * n);
}

size_t band_probs_floats(int B, int H, int n, const AttnGeom& g, int G) {
  return (size_t)B * H * n * ((size_t)g.bw + 2 * (size_t)G);
}

// ------------------------------------------------- benchmark kernel timing
// While enabled, every window-attention call records three events on its
// stream: before launch 1, between the launches, after launch 2.
namespace {
constexpr int kMaxProfiled = 4096;
bool g_prof_on = false;
int g_prof_count = 0;
hipEvent_t g_prof_ev[3 * kMaxProfiled];
bool g_prof_created[3 * kMaxProfiled] = {};

void profile_mark(hipStream_t s, int which) {
  if (!g_prof_on || g_prof_count >= kMaxProfiled) return;
  // (the event of a slot is created on its first use)
  const int i = 3 * g_prof_count + which;
  if (!g_prof_created[i]) g_prof_created[i] = hipEventCreate(&g_prof_ev[i]) == hipSuccess;
  if (g_prof_created[i]) (void)hipEventRecord(g_prof_ev[i], s);
  if (which == 2) ++g_prof_count;
}
}  // namespace

int profile_set(int enable) {
  g_prof_on = enable != 0;
  if (g_prof_on) g_prof_count = 0;
  return 0;
}

int profile_read(double* fwd_ms, double* cols_ms, long long cap, long long* calls) {
  const int cnt = g_prof_count;
  for (int i = 0; i < cnt && i < cap; ++i) {
    for (int j = 0; j < 3; ++j)
      if (!g_prof_created[3 * i + j]) return -1;
    if (hipEventSynchronize(g_prof_ev[3 * i + 2]) != hipSuccess) return -1;
    float a = 0.f, b = 0.f;
    if (hipEventElapsedTime(&a, g_prof_ev[3 * i], g_prof_ev[3 * i + 1]) != hipSuccess) return -1;
    if (hipEventElapsedTime(&b, g_prof_ev[3 * i + 1], g_prof_ev[3 * i + 2]) != hipSuccess) return -1;
    fwd_ms[i] = a;
    cols_ms[i] = b;
  }
  *calls = cnt;
  g_prof_count = 0;
  return 0;
}

// Sequences up to this length are dispatched span by span.  Measured against
// the pair-by-pair order (both launches, bf16, H12 unless noted): as fast or
// faster at every shape up to seq 4096 (B8 n4096 window 512, 32 global
// slots: launch 2 -1 %, HBM traffic 371 -> 245 MB; window 256: launch 2 -6 %;
// 64 slots: -9 %; B64 n1024 window 256 with paper-shaped lengths: -7.5 % and
// -15 %; B8 n1024, B16 n2048: within 1 %), slower at n 8192 (B4 window 512:
// +2 % and +3 %; B2 H16 window 1024 with 64 slots: +5 % and +11 %), where a
// pair's window blocks alone fill an XCD and its K and V stay in that XCD's
// L2 in the pair order.
constexpr int kSpanOrderMaxN = 4096;

template <int DT>
static hipError_t launch_window_t(const AttnArgs& a0, hipStream_t s) {
  AttnArgs a = a0;
  if (a.n <= kSpanOrderMaxN) a.span_major = 1;
  const bool glob = a.G > 0 && a.gpos;
  const bool cols = a.part_band || a.bp_band;
  a.n_gr = glob ? a.nkc * a.ngc * a.H * a.B : 0;
  if (DT == 1 && !a.bp_band) a.nkb = (a.n + kBK2 - 1) / kBK2;  // 128-key column blocks
  a.n_bcol = cols ? a.nkb * a.H * a.B : 0;
  a.n_gcol = (cols && glob) ? a.nqr * a.ngc * a.H * a.B : 0;
  const int nxc = glob ? (a.G + kBK - 1) / kBK : 0;
  if (DT == 1) {  // bf16 pass 1 runs kBQ2-query blocks
    a.nqb = (a.n + kBQ2 - 1) / kBQ2;
    const long long rw = (long long)kBQ2 + 2LL * a.r;
    a.rwp = (int)(rw < a.n ? rw : a.n);
  }
  const size_t dyn = sizeof(uint32_t) * ((size_t)a.rwp / 32 + 2 + nxc + 1);
  // the spans' block counts (the host checks that they fit the grid limits)
  const long long pairs = (long long)a.H * a.B;
  const unsigned fwd_blocks = (unsigned)(a.span_major ? a.nkc * fwd_span(a).per * pairs : a.n_gr + a.nqb * pairs);
  const int col_per = a.bp_band ? col_span<DT, true>(a).per : col_span<DT, false>(a).per;
  const unsigned col_blocks = (unsigned)(a.span_major ? a.nkc * col_per * pairs
                                                      : ((a.n_gr + 7) & ~7) + a.n_bcol + a.n_gcol);
  if (!a.no_profile) profile_mark(s, 0);
  hipLaunchKernelGGL(k_attn_fwd<DT>, dim3(fwd_blocks), dim3(kThreads), dyn, s, a);
  if (!a.no_profile) profile_mark(s, 1);
  if (col_blocks > 0) {
    if (a.bp_band)
      hipLaunchKernelGGL((k_attn_cols<DT, true>), dim3(col_blocks), dim3(kThreads), 0, s, a);
    else
      hipLaunchKernelGGL((k_attn_cols<DT, false>), dim3(col_blocks), dim3(kThreads), 0, s, a);
  }
  if (!a.no_profile) profile_mark(s, 2);
  return hipGetLastError();
}

hipError_t launch_window_attention(int dtype, const AttnArgs& a, hipStream_t s) {
  return dtype == 1 ? launch_window_t<1>(a, s) : launch_window_t<0>(a, s);
}

static ScorePartials score_partials(const float* part, int B, int n, int H, int G, const AttnGeom& g) {
  ScorePartials sp;
  sp.band = part;
  sp.gcol = sp.band + (size_t)B * H * n;
  sp.grow = sp.gcol + (size_t)B * H * g.nqr * G;
  sp.n = n;
  sp.H = H;
  sp.G = G;
  sp.ngc = g.ngc;
  sp.nqr = g.nqr;
  return sp;
}

hipError_t launch_score_from_partials(const float* partials, const int* valid_len, const int* gpos, int B, int n,
                                      int H, int G, const AttnGeom& g, float* scores, hipStream_t s) {
  dim3 grid((n + kScoreKeys - 1) / kScoreKeys, B);
  const ScorePartials sp = score_partials(partials, B, n, H, G, g);
  const int* gp = G > 0 ? gpos : nullptr;
  if (g.ngc == 0)
    hipLaunchKernelGGL(k_score_from_partials<0>, grid, dim3(kScoreKeys * kScoreGroups), 0, s, sp, valid_len, gp,
                       scores);
  else if (g.ngc == 1)
    hipLaunchKernelGGL(k_score_from_partials<1>, grid, dim3(kScoreKeys * kScoreGroups), 0, s, sp, valid_len, gp,
                       scores);
  else if (g.ngc == 2)
    hipLaunchKernelGGL(k_score_from_partials<2>, grid, dim3(kScoreKeys * kScoreGroups), 0, s, sp, valid_len, gp,
                       scores);
  else
    hipLaunchKernelGGL(k_score_from_partials<-1>, grid, dim3(kScoreKeys * kScoreGroups), 0, s, sp, valid_len, gp,
                       scores);
  return hipGetLastError();
}

size_t band_parts_floats(int B, int H, int n, int window, int G) {
  const AttnGeom g = attn_geom(n, window, G);
  // the 16-byte variant's span (segments of 256 keys) covers the other's
  return (size_t)B * H * ((n + kBandRows - 1) / kBandRows) * band_segments(g.rb, 4) * 256;
}

hipError_t launch_score_from_band(const float* bp, const int* valid_len, const int* gpos, int B, int n, int H, int G,
                                  const AttnGeom& g, float* partials, float* parts, float* scores, hipStream_t s) {
  ScorePartials sp = score_partials(partials, B, n, H, G, g);
  ScorePartialsOut po{partials, const_cast<float*>(sp.gcol), const_cast<float*>(sp.grow)};
  // 16-byte loads need every row's first entry for a lane's first key
  // (2r * i + key + r, plus the head's offset b * H * n * (2r + 1)) on a
  // 4-float boundary
  const bool vec4 = g.rb % 4 == 0 && n % 4 == 0 && reinterpret_cast<uintptr_t>(bp) % 16 == 0;
  const int vec = vec4 ? 4 : 1, nseg = band_segments(g.rb, vec);
  const int threads = 64 * (nseg < 4 ? nseg : 4);
  const long long blocks = (long long)B * H * ((n + kBandRows - 1) / kBandRows) + (G > 0 ? (long long)B * H * g.nqr : 0);
  if (vec4)
    hipLaunchKernelGGL(k_band_rows<4>, dim3((unsigned)blocks), dim3(threads), 0, s, bp, valid_len, B, n, H, G, g,
                       nseg, parts, po);
  else
    hipLaunchKernelGGL(k_band_rows<1>, dim3((unsigned)blocks), dim3(threads), 0, s, bp, valid_len, B, n, H, G, g,
                       nseg, parts, po);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_band_keys, dim3((unsigned)((n + 255) / 256), (unsigned)(B * H)), dim3(256), 0, s, bp,
                     valid_len, B, n, H, G, g, nseg, 64 * vec, parts, po);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_score_from_partials(partials, valid_len, gpos, B, n, H, G, g, scores, s);
}

}  // namespace sc
