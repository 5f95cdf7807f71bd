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
  SC_DEV void store(T* lds) const {
#pragma unroll
    for (int i = 0; i < kCpt; ++i) {
      const int c = threadIdx.x + kThreads * i, row = c / kCpr, part = c % kCpr;
      *reinterpret_cast<uint4*>(lds + row * P + part * kEpc) = r[i];
    }
  }
};

// ------------------------------------------------------------ pass 1 tile ---
// One 64-key tile for the 16 queries of a wave.  s[st][i] is the logit of
// (key 16*st + 4g + i, query lr).  ok(st, i) masks keys (kMasked only).
// The running max m_use is in scaled log2 units; softmax_scale >= 0, so the
// tile max is taken on the raw logits and scaled once.
template <int DT, bool kMasked, typename OkFn>
SC_DEV void softmax_tile(const typename Tr<DT>::Frag (&qf)[Tr<DT>::kChunks], const typename Tr<DT>::T* sK,
                         const typename Tr<DT>::T* sV, float c2, int lr, int g, float& m_use, float& l_run,
                         f32x4 (&o)[4], OkFn ok) {
  using TR = Tr<DT>;
  constexpr int P = TR::kPitch;
  f32x4 s[4];
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    typename TR::Frag kf[TR::kChunks];
    TR::load_frags(sK + (16 * st + lr) * P, g, kf);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < TR::kChunks; ++c) acc = TR::mma(kf[c], qf[c], acc);
    s[st] = acc;
  }
  bool valid[4][4];
  float tmax = -INFINITY;
#pragma unroll
  for (int st = 0; st < 4; ++st)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      valid[st][i] = !kMasked || ok(st, i);
      tmax = fmaxf(tmax, valid[st][i] ? s[st][i] : -INFINITY);
    }
  tmax = group_max(tmax) * c2;
  if (tmax > m_use + kTau) {
    const float f = fast_exp2(m_use - tmax);
    l_run *= f;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) o[dt] *= f;
    m_use = tmax;
  }
  float p[4][4];
#pragma unroll
  for (int st = 0; st < 4; ++st)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float e = fast_exp2(fmaf(s[st][i], c2, -m_use));
      p[st][i] = valid[st][i] ? e : 0.f;
      l_run += p[st][i];
    }
  if constexpr (DT == 1) {
    // keys of lane group g in MFMA order: 32kc + 4g + (0..3), then 32kc + 16 + 4g + (0..3)
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      bf16x8 pb;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pb[i] = (__bf16)p[2 * kc][i];
        pb[4 + i] = (__bf16)p[2 * kc + 1][i];
      }
      const typename TR::T* v0 = sV + (32 * kc + 4 * g + (lr >> 2)) * P + 4 * (lr & 3);
      const typename TR::T* v1 = v0 + 16 * P;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const i16x4 a0 = lds_read_tr16(v0 + 16 * dt);
        const i16x4 a1 = lds_read_tr16(v1 + 16 * dt);
        const i16x8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
        o[dt] = TR::mma(__builtin_bit_cast(bf16x8, a), pb, o[dt]);
      }
    }
  } else {
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) o[dt] = TR::mma(sV[(16 * st + 4 * g + i) * P + 16 * dt + lr], p[st][i], o[dt]);
  }
}

// ------------------------------------------------------------ pass 2 tile ---
// Column sums of exact probabilities for the 16 keys of sub-tile `w` of the
// staged tile over the 64 queries of the block.  Result register (qst, i) of
// the MFMA is (query 16*qst + 4g + i, key lr).  ok(qst, i) masks pairs;
// emit(qst, i, p) sees every probability (used for the band layout).
template <int DT, bool kMasked, typename OkFn, typename EmitFn>
SC_DEV float score_tile(const typename Tr<DT>::Frag (&qf)[4][Tr<DT>::kChunks], const float (&l2)[4][4],
                        const typename Tr<DT>::T* sK, int w, float c2, int lr, int g, OkFn ok, EmitFn emit) {
  using TR = Tr<DT>;
  typename TR::Frag kf[TR::kChunks];
  TR::load_frags(sK + (16 * w + lr) * TR::kPitch, g, kf);
  float cs = 0.f;
#pragma unroll
  for (int qst = 0; qst < 4; ++qst) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < TR::kChunks; ++c) acc = TR::mma(qf[qst][c], kf[c], acc);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float p = fast_exp2(fmaf(acc[i], c2, -l2[qst][i]));
      if (kMasked && !ok(qst, i)) p = 0.f;
      emit(qst, i, p);
      cs += p;
    }
  }
  return group_sum(cs);
}

struct NoEmit {
  SC_DEV void operator()(int, int, float) const {}
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

// Slot of global key `key` of sequence row gp[0..G) (ascending), or -1.
SC_DEV int find_slot(const int* gp, int G, int key) {
  int lo = 0, hi = G - 1;
  while (lo <= hi) {
    const int mid = (lo + hi) >> 1;
    const int p = gp[mid];
    if (p == key) return mid;
    if (p >= 0 && p < key) lo = mid + 1;
    else hi = mid - 1;
  }
  return -1;
}

// ------------------------------------------------------- window kernels -----
// Geometry of one window block (sequence b, head h, queries q0 .. q0+63) and
// its LDS tables: the global-token bitmask over the key range [kt0, kt1) and
// the list of 64-slot chunks that hold global keys outside that range.
struct WinBlock {
  int qb, bh, h, b, L, q0, kt0, kt1, nkt, nwords, nxc, ntile;
};

SC_DEV WinBlock win_block(const AttnArgs& a) {
  WinBlock wb;
  const int lin = xcd_remap(blockIdx.x, a.nqb * a.H * a.B);
  wb.qb = lin % a.nqb;
  wb.bh = lin / a.nqb;
  wb.h = wb.bh % a.H;
  wb.b = wb.bh / a.H;
  wb.L = clampi(a.valid_len[wb.b], 0, a.n);
  wb.q0 = wb.qb * kBQ;
  wb.kt0 = max(0, wb.q0 - a.r);
  wb.kt1 = min(wb.L, wb.q0 + kBQ + a.r);
  wb.nkt = (wb.kt1 - wb.kt0 + kBK - 1) / kBK;
  wb.nwords = (wb.kt1 - wb.kt0 + 31) >> 5;
  wb.nxc = (a.gpos && a.G > 0) ? (a.G + kBK - 1) / kBK : 0;
  wb.ntile = wb.nkt;
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
  for (int i = tid; i < wb.nwords; i += kThreads) sBits[i] = 0u;
  for (int i = tid; i < wb.nxc; i += kThreads) sXList[i] = 0;
  __syncthreads();
  for (int j = tid; j < (gp ? a.G : 0); j += kThreads) {
    const int p = gp[j];
    if (p >= wb.kt0 && p < wb.kt1)
      atomicOr(&sBits[(p - wb.kt0) >> 5], 1u << ((p - wb.kt0) & 31));
    else if (p >= 0 && p < wb.L)
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

// Tile loader shared by both passes: band tiles are contiguous key ranges,
// global-slot tiles gather the rows of global keys outside the band.
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
      if (Vg) stv.load_range(Vg, a.ld_in, k0, wb.kt1);
    } else {
      const int c = sXList[t - wb.nkt];
      stk.load_rows(Kg, a.ld_in, [&](int row) { return slot_row(c, row); });
      if (Vg) stv.load_rows(Vg, a.ld_in, [&](int row) { return slot_row(c, row); });
      if (threadIdx.x < kBK) pos_reg = slot_row(c, threadIdx.x);
    }
  }
  SC_DEV void store(int t, T* sK, T* sV, int* sPos) const {
    stk.store(sK);
    if (sV) stv.store(sV);
    if (t >= wb.nkt && threadIdx.x < kBK) sPos[threadIdx.x] = pos_reg;
  }
};

// Pass 1: O, LSE (and the log2 LSE handed to pass 2) for the non-global
// queries of the block; zero rows for padding queries.
template <int DT>
__global__ __launch_bounds__(kThreads) SC_OCC(3) void k_window_attn(AttnArgs a) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  using Frag = typename TR::Frag;
  constexpr int P = TR::kPitch;
  __shared__ __attribute__((aligned(16))) T sQ[kBQ * P];
  __shared__ __attribute__((aligned(16))) T sK[2][kBK * P];
  __shared__ __attribute__((aligned(16))) T sV[2][kBK * P];
  __shared__ int sPos[2][kBK];
  __shared__ int sNx;
  extern __shared__ uint32_t sDyn[];  // [global bitmask over the band range][active global-slot chunks]

  const WinBlock wb = win_block(a);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, lr = lane & 15;
  const int n = a.n, r = a.r, L = wb.L, q0 = wb.q0, kt0 = wb.kt0, kt1 = wb.kt1, nkt = wb.nkt;
  const T* Qg = static_cast<const T*>(a.q) + wb.b * a.bs_in + wb.h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + wb.b * a.bs_in + wb.h * kHeadDim;
  const T* Vg = static_cast<const T*>(a.v) + wb.b * a.bs_in + wb.h * kHeadDim;
  T* Og = static_cast<T*>(a.out) + wb.b * a.bs_out + wb.h * kHeadDim;
  float* lseg = a.lse ? a.lse + (long long)wb.bh * n : nullptr;
  float* l2g = a.win_lse2 ? a.win_lse2 + (long long)wb.bh * n : nullptr;

  if (q0 >= L) {  // padding block: zero output rows
    constexpr int kEpc = 16 / sizeof(T), kCpr = kHeadDim / kEpc;
    for (int c = tid; c < kBQ * kCpr; c += kThreads) {
      const int q = q0 + c / kCpr;
      if (q < n) zero16(Og + (long long)q * a.ld_out + (c % kCpr) * kEpc);
    }
    if (lseg)
      for (int i = tid; i < kBQ; i += kThreads)
        if (q0 + i < n) lseg[q0 + i] = -INFINITY;
    return;
  }
  uint32_t* sBits = sDyn;
  int* sXList = reinterpret_cast<int*>(sDyn + a.rwp / 32 + 2);
  {  // padding query rows are staged as zeros: their (unused) logits stay finite
    Stage<DT> sq;
    sq.load_range(Qg + (long long)q0 * a.ld_in, a.ld_in, 0, L - q0);
    sq.store(sQ);
  }
  const int ntile = win_tables(a, wb, sBits, sXList, &sNx);
  auto gbit = [&](int k) -> bool {
    const int o = k - kt0;
    return (sBits[o >> 5] >> (o & 31)) & 1u;
  };
  WinLoader<DT> ld{a, wb, wb.nxc ? a.gpos + (long long)wb.b * a.G : nullptr, sXList};

  Frag qf[TR::kChunks];
  TR::load_frags(sQ + (16 * w + lr) * P, g, qf);
  const int qa = q0 + 16 * w;
  const int qrow = qa + lr;
  float m_use = kNegBig, l_run = 0.f;
  f32x4 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // band tiles: double-buffered, the next tile's loads overlap this tile's math
  ld.load(0, Kg, Vg);
  ld.store(0, sK[0], sV[0], sPos[0]);
  __syncthreads();
  for (int t = 0; t < nkt; ++t) {
    const int buf = t & 1;
    if (t + 1 < nkt) ld.load(t + 1, Kg, Vg);
    const int k0 = kt0 + t * kBK;
    const bool near = k0 <= qa + 15 + r && k0 + kBK - 1 >= qa - r;
    if (near || tile_gmask(sBits, t, wb.nwords) != 0ull) {
      const bool interior = k0 + kBK <= kt1 && k0 >= qa + 15 - r && k0 + kBK - 1 <= qa + r;
      if (interior) {
        softmax_tile<DT, false>(qf, sK[buf], sV[buf], a.c2, lr, g, m_use, l_run, o, [](int, int) { return true; });
      } else {
        // key index inside the tile: 16*st + 4g + i; allowed when it lies in
        // [lo, hi] (window and sequence end) or is a global key of the band.
        // Branch-free: the tile's global keys come as one 64-bit mask (bits
        // beyond kt1 are never set).
        const int lo = qrow - r - k0, hi = min(qrow + r, kt1 - 1) - k0;
        const unsigned long long gm = tile_gmask(sBits, t, wb.nwords) >> (4 * g);
        softmax_tile<DT, true>(qf, sK[buf], sV[buf], a.c2, lr, g, m_use, l_run, o, [&](int s4, int i) {
          const int kk = 16 * s4 + 4 * g + i;
          return ((kk >= lo) & (kk <= hi)) | (bool)((gm >> (16 * s4 + i)) & 1ull);
        });
      }
    }
    if (t + 1 < nkt) ld.store(t + 1, sK[buf ^ 1], sV[buf ^ 1], sPos[buf ^ 1]);
    __syncthreads();
  }
  // global keys outside the band (few tiles; not pipelined)
  for (int t = nkt; t < ntile; ++t) {
    ld.load(t, Kg, Vg);
    ld.store(t, sK[0], sV[0], sPos[0]);
    __syncthreads();
    const int* sp = sPos[0];
    softmax_tile<DT, true>(qf, sK[0], sV[0], a.c2, lr, g, m_use, l_run, o,
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
  // excluded rows (global or padding) get +inf: their pass-2 probabilities are 0
  if (g == 0 && l2g && qrow < n) l2g[qrow] = qvalid ? lse2 : INFINITY;
}

// Pass 2: exact probabilities of the block's non-global queries, summed per
// key into the band and global-key partials (and written to the paper's band
// layout when requested).  Wave w owns key sub-tile w of each staged tile.
template <int DT, bool kBandProbs>
__global__ __launch_bounds__(kThreads) SC_OCC(kBandProbs ? 2 : 4) void k_window_score(AttnArgs a) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  using Frag = typename TR::Frag;
  constexpr int P = TR::kPitch;
  __shared__ __attribute__((aligned(16))) T sQ[kBQ * P];
  __shared__ __attribute__((aligned(16))) T sK[2][kBK * P];
  __shared__ int sPos[2][kBK];
  __shared__ int sNx;
  extern __shared__ uint32_t sDyn[];

  const WinBlock wb = win_block(a);
  if (wb.q0 >= wb.L) return;  // the score reduction never reads padding blocks
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, lr = lane & 15;
  const int n = a.n, r = a.r, G = a.G, L = wb.L, q0 = wb.q0, kt0 = wb.kt0, kt1 = wb.kt1, nkt = wb.nkt;
  const T* Qg = static_cast<const T*>(a.q) + wb.b * a.bs_in + wb.h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + wb.b * a.bs_in + wb.h * kHeadDim;
  const float* l2g = a.win_lse2 + (long long)wb.bh * n;
  const int* gp = wb.nxc ? a.gpos + (long long)wb.b * G : nullptr;
  uint32_t* sBits = sDyn;
  int* sXList = reinterpret_cast<int*>(sDyn + a.rwp / 32 + 2);
  {
    Stage<DT> sq;
    sq.load_range(Qg + (long long)q0 * a.ld_in, a.ld_in, 0, L - q0);
    sq.store(sQ);
  }
  const int ntile = win_tables(a, wb, sBits, sXList, &sNx);
  auto gbit = [&](int k) -> bool {
    const int o = k - kt0;
    return (sBits[o >> 5] >> (o & 31)) & 1u;
  };
  WinLoader<DT> ld{a, wb, gp, sXList};
  ld.load(0, Kg, nullptr);
  ld.store(0, sK[0], nullptr, sPos[0]);
  // the block's log2-LSE go through LDS: values a loop consumes must not come
  // from outstanding global loads (those would be waited for in every tile)
  __shared__ float sL2[kBQ];
  if (tid < kBQ) sL2[tid] = q0 + tid < L ? l2g[q0 + tid] : INFINITY;

  Frag qf2[4][TR::kChunks];
  float l2[4][4];
  float* pb = a.part_band ? a.part_band + ((long long)wb.bh * a.nqb + wb.qb) * a.rwp : nullptr;
  float* pe = a.part_band ? a.part_extra + ((long long)wb.bh * a.nqb + wb.qb) * G : nullptr;
  float* bpb = kBandProbs ? a.bp_band + (long long)wb.bh * n * a.bw : nullptr;
  float* bpc = kBandProbs ? a.bp_gcol + (long long)wb.bh * n * G : nullptr;
  // global-key partials of slots never visited stay zero (written before the
  // first barrier of the loop below, overwritten after it)
  if (pe)
    for (int j = tid; j < G; j += kThreads) pe[j] = 0.f;
  __syncthreads();
#pragma unroll
  for (int qst = 0; qst < 4; ++qst) {
    TR::load_frags(sQ + (16 * qst + lr) * P, g, qf2[qst]);
#pragma unroll
    for (int i = 0; i < 4; ++i) l2[qst][i] = sL2[16 * qst + 4 * g + i];
  }

  for (int t = 0; t < nkt; ++t) {
    const int buf = t & 1;
    if (t + 1 < nkt) ld.load(t + 1, Kg, nullptr);
    const int k0 = kt0 + t * kBK;
    const int key = k0 + 16 * w + lr;
    const bool kin = key < kt1;
    const bool kglob = kin && gbit(key);
    // query index inside the block: 16*qst + 4g + i; allowed within
    // [key - r - q0, key + r - q0] or when the key is global
    const int lo = key - r - q0, hi = key + r - q0;
    auto ok = [&](int qst, int i) {
      const int qq = 16 * qst + 4 * g + i;
      return kin & (kglob | ((qq >= lo) & (qq <= hi)));
    };
    float cs;
    if constexpr (kBandProbs) {
      const int kslot = kglob ? find_slot(gp, G, key) : -1;
      cs = score_tile<DT, true>(qf2, l2, sK[buf], w, a.c2, lr, g, ok, [&](int qst, int i, float p) {
        const int q = q0 + 16 * qst + 4 * g + i;
        if (!(q < L) || !kin || p == 0.f) return;
        if (kglob) {
          if (kslot >= 0) bpc[(long long)q * G + kslot] = p;
        } else if (abs(q - key) <= a.rb) {
          bpb[(long long)q * a.bw + (key - q + a.rb)] = p;
        }
      });
    } else {
      const bool interior = k0 + kBK <= kt1 && k0 >= q0 + kBQ - 1 - r && k0 + kBK - 1 <= q0 + r;
      cs = interior ? score_tile<DT, false>(qf2, l2, sK[buf], w, a.c2, lr, g, ok, NoEmit{})
                    : score_tile<DT, true>(qf2, l2, sK[buf], w, a.c2, lr, g, ok, NoEmit{});
    }
    if (pb && g == 0 && kin) pb[key - kt0] = cs;
    if (t + 1 < nkt) ld.store(t + 1, sK[buf ^ 1], nullptr, sPos[buf ^ 1]);
    __syncthreads();
  }
  // global keys outside the band
  for (int t = nkt; t < ntile; ++t) {
    ld.load(t, Kg, nullptr);
    ld.store(t, sK[0], nullptr, sPos[0]);
    __syncthreads();
    const int slot = kBK * sXList[t - nkt] + 16 * w + lr;
    const bool kvalid = sPos[0][16 * w + lr] >= 0;
    auto ok = [&](int, int) { return kvalid; };
    float cs;
    if constexpr (kBandProbs) {
      cs = score_tile<DT, true>(qf2, l2, sK[0], w, a.c2, lr, g, ok, [&](int qst, int i, float p) {
        const int q = q0 + 16 * qst + 4 * g + i;
        if (kvalid && q < L && p != 0.f) bpc[(long long)q * G + slot] = p;
      });
    } else {
      cs = score_tile<DT, true>(qf2, l2, sK[0], w, a.c2, lr, g, ok, NoEmit{});
    }
    if (pe && g == 0 && slot < G) pe[slot] = cs;
    __syncthreads();
  }
}

// -------------------------------------------------- global-row kernels -----
// Global query rows attend to every valid key: a dense strip, split over key
// ranges of kGlobalKeySpan.  Block = 64 global slots x one key range.
struct GrBlock {
  int kc, gc, h, b, bh;
};
SC_DEV GrBlock gr_block(const AttnArgs& a) {
  GrBlock r;
  int lin = blockIdx.x;
  r.kc = lin % a.nkc;
  lin /= a.nkc;
  r.gc = lin % a.ngc;
  lin /= a.ngc;
  r.h = lin % a.H;
  r.b = lin / a.H;
  r.bh = r.b * a.H + r.h;
  return r;
}

template <int DT>
__global__ __launch_bounds__(kThreads) void k_global_rows_fwd(AttnArgs a) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  constexpr int P = TR::kPitch;
  __shared__ __attribute__((aligned(16))) T sQ[kBQ * P];
  __shared__ __attribute__((aligned(16))) T sK[2][kBK * P];
  __shared__ __attribute__((aligned(16))) T sV[2][kBK * P];
  __shared__ int sPos[kGlobalChunk];
  const GrBlock blk = gr_block(a);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, lr = lane & 15;
  const int L = clampi(a.valid_len[blk.b], 0, a.n);
  const int kbeg = blk.kc * kGlobalKeySpan;
  if (kbeg >= L) return;
  const int kend = min(L, kbeg + kGlobalKeySpan);
  const int* gp = a.gpos + (long long)blk.b * a.G;
  int valid = 0;
  if (tid < kGlobalChunk) {
    const int j = kGlobalChunk * blk.gc + tid;
    const int p = j < a.G ? gp[j] : -1;
    valid = p >= 0 && p < L;
    sPos[tid] = valid ? p : -1;
  }
  if (!__syncthreads_or(valid)) return;
  const T* Qg = static_cast<const T*>(a.q) + blk.b * a.bs_in + blk.h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + blk.b * a.bs_in + blk.h * kHeadDim;
  const T* Vg = static_cast<const T*>(a.v) + blk.b * a.bs_in + blk.h * kHeadDim;
  const int ntile = (kend - kbeg + kBK - 1) / kBK;
  Stage<DT> stk, stv;
  {
    Stage<DT> sq;
    sq.load_rows(Qg, a.ld_in, [&](int row) { return sPos[row]; });
    sq.store(sQ);
  }
  stk.load_range(Kg, a.ld_in, kbeg, kend);
  stv.load_range(Vg, a.ld_in, kbeg, kend);
  stk.store(sK[0]);
  stv.store(sV[0]);
  __syncthreads();
  typename TR::Frag qf[TR::kChunks];
  TR::load_frags(sQ + (16 * w + lr) * P, g, qf);
  float m_use = kNegBig, l_run = 0.f;
  f32x4 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int t = 0; t < ntile; ++t) {
    const int buf = t & 1, k0 = kbeg + t * kBK;
    if (t + 1 < ntile) {
      stk.load_range(Kg, a.ld_in, k0 + kBK, kend);
      stv.load_range(Vg, a.ld_in, k0 + kBK, kend);
    }
    if (k0 + kBK <= kend) {
      softmax_tile<DT, false>(qf, sK[buf], sV[buf], a.c2, lr, g, m_use, l_run, o, [](int, int) { return true; });
    } else {
      const int hi = kend - 1 - k0;
      softmax_tile<DT, true>(qf, sK[buf], sV[buf], a.c2, lr, g, m_use, l_run, o,
                             [&](int s4, int i) { return 16 * s4 + 4 * g + i <= hi; });
    }
    if (t + 1 < ntile) {
      stk.store(sK[buf ^ 1]);
      stv.store(sV[buf ^ 1]);
    }
    __syncthreads();
  }
  const float l_row = group_sum(l_run);
  const int slot = kGlobalChunk * blk.gc + 16 * w + lr;
  const long long idx = ((long long)blk.bh * a.nkc + blk.kc) * a.Gp + slot;
  if (g == 0) {
    a.gr_ml[2 * idx] = m_use;
    a.gr_ml[2 * idx + 1] = l_row;
  }
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) *reinterpret_cast<f32x4*>(a.gr_o + idx * kHeadDim + 16 * dt + 4 * g) = o[dt];
}

// One wave per (sequence, head, global slot): merge the key-range partials.
template <int DT>
__global__ __launch_bounds__(kThreads) void k_global_rows_merge(AttnArgs a) {
  using T = typename Tr<DT>::T;
  const long long wid = (long long)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (wid >= (long long)a.B * a.H * a.Gp) return;
  const int slot = (int)(wid % a.Gp);
  const int bh = (int)(wid / a.Gp), b = bh / a.H, h = bh % a.H;
  const int L = clampi(a.valid_len[b], 0, a.n);
  const int p = slot < a.G ? a.gpos[(long long)b * a.G + slot] : -1;
  if (!(p >= 0 && p < L)) {
    if (lane == 0) a.gr_lse2[wid] = INFINITY;
    return;
  }
  const int nk = (L + kGlobalKeySpan - 1) / kGlobalKeySpan;
  float m = kNegBig;
  for (int kc = 0; kc < nk; ++kc) m = fmaxf(m, a.gr_ml[2 * (((long long)bh * a.nkc + kc) * a.Gp + slot)]);
  float l = 0.f, acc = 0.f;
  for (int kc = 0; kc < nk; ++kc) {
    const long long idx = ((long long)bh * a.nkc + kc) * a.Gp + slot;
    const float f = fast_exp2(a.gr_ml[2 * idx] - m);
    l += a.gr_ml[2 * idx + 1] * f;
    acc += a.gr_o[idx * kHeadDim + lane] * f;
  }
  const float lse2 = m + fast_log2(l);
  T* Og = static_cast<T*>(a.out) + b * a.bs_out + (long long)p * a.ld_out + h * kHeadDim;
  Og[lane] = (T)(acc / l);
  if (lane == 0) {
    if (a.lse) a.lse[(long long)bh * a.n + p] = lse2 * kLn2;
    a.gr_lse2[wid] = lse2;
  }
}

// Column sums over the global query rows of one slot chunk, per key.
template <int DT>
__global__ __launch_bounds__(kThreads) void k_global_rows_score(AttnArgs a) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  constexpr int P = TR::kPitch;
  __shared__ __attribute__((aligned(16))) T sQ[kBQ * P];
  __shared__ __attribute__((aligned(16))) T sK[2][kBK * P];
  __shared__ int sPos[kGlobalChunk];
  const GrBlock blk = gr_block(a);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, lr = lane & 15;
  const int L = clampi(a.valid_len[blk.b], 0, a.n);
  const int kbeg = blk.kc * kGlobalKeySpan;
  if (kbeg >= L) return;
  const int kend = min(L, kbeg + kGlobalKeySpan);
  const int* gp = a.gpos + (long long)blk.b * a.G;
  float* pg = a.part_grow ? a.part_grow + ((long long)blk.bh * a.ngc + blk.gc) * a.n : nullptr;
  float* bpr = a.bp_grow ? a.bp_grow + (long long)blk.bh * a.G * a.n : nullptr;
  int valid = 0;
  if (tid < kGlobalChunk) {
    const int j = kGlobalChunk * blk.gc + tid;
    const int p = j < a.G ? gp[j] : -1;
    valid = p >= 0 && p < L;
    sPos[tid] = valid ? p : -1;
  }
  if (!__syncthreads_or(valid)) {
    if (pg)
      for (int k = kbeg + tid; k < kend; k += kThreads) pg[k] = 0.f;
    return;
  }
  const T* Qg = static_cast<const T*>(a.q) + blk.b * a.bs_in + blk.h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + blk.b * a.bs_in + blk.h * kHeadDim;
  const int ntile = (kend - kbeg + kBK - 1) / kBK;
  Stage<DT> stk;
  {
    Stage<DT> sq;
    sq.load_rows(Qg, a.ld_in, [&](int row) { return sPos[row]; });
    sq.store(sQ);
  }
  stk.load_range(Kg, a.ld_in, kbeg, kend);
  stk.store(sK[0]);
  __syncthreads();
  typename TR::Frag qf[4][TR::kChunks];
  float l2[4][4];
#pragma unroll
  for (int qst = 0; qst < 4; ++qst) {
    TR::load_frags(sQ + (16 * qst + lr) * P, g, qf[qst]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      l2[qst][i] = a.gr_lse2[(long long)blk.bh * a.Gp + kGlobalChunk * blk.gc + 16 * qst + 4 * g + i];
  }
  for (int t = 0; t < ntile; ++t) {
    const int buf = t & 1, k0 = kbeg + t * kBK;
    if (t + 1 < ntile) stk.load_range(Kg, a.ld_in, k0 + kBK, kend);
    const int key = k0 + 16 * w + lr;
    const bool kin = key < kend;
    auto ok = [&](int, int) { return kin; };
    float cs;
    if (bpr) {
      cs = score_tile<DT, true>(qf, l2, sK[buf], w, a.c2, lr, g, ok, [&](int qst, int i, float p) {
        const int slot = kGlobalChunk * blk.gc + 16 * qst + 4 * g + i;
        if (kin && slot < a.G && p != 0.f) bpr[(long long)slot * a.n + key] = p;
      });
    } else {
      cs = score_tile<DT, true>(qf, l2, sK[buf], w, a.c2, lr, g, ok, NoEmit{});
    }
    if (pg && g == 0 && kin) pg[key] = cs;
    if (t + 1 < ntile) stk.store(sK[buf ^ 1]);
    __syncthreads();
  }
}

// ------------------------------------------------------ score reduction ----
// scores[b, k] = (sum over heads of: the band partials of every query block
// whose band holds k, the global-key partials if k is global, and the
// global-row sums) / (H * L).  Workgroup = 64 keys of one sequence; wave w
// sums heads w, w + nw, ...; the nw wave sums are then added in wave order.
// Fixed order everywhere; no atomics.
constexpr int kScoreKeys = 64;
constexpr int kScoreMaxWaves = 16;

__global__ __launch_bounds__(64 * kScoreMaxWaves) void k_score_from_partials(const float* part, const int* valid_len,
                                                                             const int* gpos, int B, int n, int H,
                                                                             int G, AttnGeom geo, float* scores) {
  __shared__ int smap[kScoreKeys];
  __shared__ float red[kScoreMaxWaves][kScoreKeys];
  const int b = blockIdx.y, kb = blockIdx.x * kScoreKeys, tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6, nw = blockDim.x >> 6;
  const int k = kb + lane;
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
    const float* band = part;
    const float* extra = band + (size_t)B * H * geo.nqb * geo.rwp;
    const float* grow = extra + (size_t)B * H * geo.nqb * G;
    const int r = geo.r;
    const int nqbv = (L + kBQ - 1) / kBQ;
    // blocks whose key range [max(0, qb*64 - r), qb*64 + 64 + r) holds k
    const int qlo = k - r - (kBQ - 1) <= 0 ? 0 : (k - r) / kBQ;
    const int qhi = min(nqbv - 1, (k + r) / kBQ);
    const int slot = smap[lane];
    for (int h = w; h < H; h += nw) {
      const long long bh = (long long)b * H + h;
      const float* pb = band + bh * geo.nqb * geo.rwp;
      for (int qb = qlo; qb <= qhi; ++qb) acc += pb[(long long)qb * geo.rwp + (k - max(0, qb * kBQ - r))];
      if (slot >= 0) {
        const float* pe = extra + bh * geo.nqb * G + slot;
        for (int qb = 0; qb < nqbv; ++qb) acc += pe[(long long)qb * G];
      }
      for (int gc = 0; gc < geo.ngc; ++gc) acc += grow[(bh * geo.ngc + gc) * n + k];
    }
  }
  red[w][lane] = acc;
  __syncthreads();
  if (w == 0 && k < n) {
    float tot = 0.f;
    for (int i = 0; i < nw; ++i) tot += red[i][lane];
    scores[(long long)b * n + k] = k < L ? tot / ((float)H * (float)L) : 0.f;
  }
}

// Paper layout: the score of key k is its band sub-diagonal (entries (i, j)
// with i - r + j = k), its global column and its entries of the global rows.
__global__ __launch_bounds__(256) void k_score_from_band(const float* bp, const int* valid_len, const int* gpos,
                                                          int B, int n, int H, int G, AttnGeom geo, float* scores) {
  __shared__ int smap[256];
  const int b = blockIdx.y, kb = blockIdx.x * 256, tid = threadIdx.x, k = kb + tid;
  const int L = clampi(valid_len[b], 0, n);
  smap[tid] = -1;
  __syncthreads();
  if (gpos)
    for (int j = tid; j < G; j += 256) {
      const int p = gpos[(long long)b * G + j];
      if (p >= kb && p < kb + 256 && p < L) smap[p - kb] = j;
    }
  __syncthreads();
  if (k >= n) return;
  if (k >= L) {
    scores[(long long)b * n + k] = 0.f;
    return;
  }
  const float* band = bp;
  const float* gcol = band + (size_t)B * H * n * geo.bw;
  const float* grow = gcol + (size_t)B * H * n * G;
  const int rb = geo.rb, slot = smap[tid];
  float acc = 0.f;
  for (int h = 0; h < H; ++h) {
    const long long bh = (long long)b * H + h;
    // walk the rows that can reach this block's keys; for a fixed row the
    // threads read consecutive band entries (coalesced)
    const int i_end = min(L, kb + 256 + rb);
    for (int i = max(0, kb - rb); i < i_end; ++i) {
      const int j = k - i + rb;
      if (j >= 0 && j < geo.bw) acc += band[(bh * n + i) * geo.bw + j];
    }
    if (slot >= 0)
      for (int i = 0; i < L; ++i) acc += gcol[(bh * n + i) * G + slot];
    for (int s = 0; s < G; ++s) acc += grow[(bh * G + s) * n + k];
  }
  scores[(long long)b * n + k] = acc / ((float)H * (float)L);
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
  g.rb = window / 2 < n - 1 ? window / 2 : n - 1;
  g.bw = 2 * g.rb + 1;
  return g;
}

size_t partials_floats(int B, int H, int n, const AttnGeom& g, int G) {
  return (size_t)B * H * ((size_t)g.nqb * (g.rwp + G) + (size_t)g.ngc * n);
}

size_t band_probs_floats(int B, int H, int n, const AttnGeom& g, int G) {
  return (size_t)B * H * n * ((size_t)g.bw + 2 * (size_t)G);
}

// ------------------------------------------------- benchmark kernel timing
namespace {
constexpr int kMaxProfiled = 4096;
bool g_prof_on = false;
int g_prof_count = 0;
hipEvent_t g_prof_ev[2 * kMaxProfiled];
bool g_prof_created[2 * kMaxProfiled] = {};

void profile_begin(hipStream_t s) {
  if (!g_prof_on || g_prof_count >= kMaxProfiled) return;
  const int i = 2 * g_prof_count;
  for (int j = i; j < i + 2; ++j)
    if (!g_prof_created[j]) g_prof_created[j] = hipEventCreate(&g_prof_ev[j]) == hipSuccess;
  if (g_prof_created[i]) (void)hipEventRecord(g_prof_ev[i], s);
}

void profile_end(hipStream_t s) {
  if (!g_prof_on || g_prof_count >= kMaxProfiled) return;
  const int i = 2 * g_prof_count + 1;
  if (g_prof_created[i]) (void)hipEventRecord(g_prof_ev[i], s);
  ++g_prof_count;
}
}  // namespace

int profile_set(int enable) {
  g_prof_on = enable != 0;
  if (g_prof_on) g_prof_count = 0;
  return 0;
}

int profile_read(double* total_ms, long long* launches) {
  double tot = 0.0;
  for (int i = 0; i < g_prof_count; ++i) {
    if (!g_prof_created[2 * i] || !g_prof_created[2 * i + 1]) return -1;
    if (hipEventSynchronize(g_prof_ev[2 * i + 1]) != hipSuccess) return -1;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, g_prof_ev[2 * i], g_prof_ev[2 * i + 1]) != hipSuccess) return -1;
    tot += ms;
  }
  *total_ms = tot;
  *launches = g_prof_count;
  g_prof_count = 0;
  return 0;
}

template <int DT>
static hipError_t launch_window_t(const AttnArgs& a, hipStream_t s) {
  if (a.G > 0 && a.gpos) {
    const unsigned grid = (unsigned)(a.nkc * a.ngc * a.H * a.B);
    hipLaunchKernelGGL(k_global_rows_fwd<DT>, dim3(grid), dim3(kThreads), 0, s, a);
    const long long waves = (long long)a.B * a.H * a.Gp;
    hipLaunchKernelGGL(k_global_rows_merge<DT>, dim3((unsigned)((waves + 3) / 4)), dim3(kThreads), 0, s, a);
  }
  const int nxc = a.G > 0 && a.gpos ? (a.G + kBK - 1) / kBK : 0;
  const size_t dyn = sizeof(uint32_t) * ((size_t)a.rwp / 32 + 2 + nxc + 1);
  const unsigned blocks = (unsigned)(a.nqb * a.H * a.B);
  profile_begin(s);
  hipLaunchKernelGGL(k_window_attn<DT>, dim3(blocks), dim3(kThreads), dyn, s, a);
  if (a.bp_band)
    hipLaunchKernelGGL((k_window_score<DT, true>), dim3(blocks), dim3(kThreads), dyn, s, a);
  else if (a.part_band)
    hipLaunchKernelGGL((k_window_score<DT, false>), dim3(blocks), dim3(kThreads), dyn, s, a);
  profile_end(s);
  if (a.G > 0 && a.gpos && (a.part_grow || a.bp_grow)) {
    const unsigned grid = (unsigned)(a.nkc * a.ngc * a.H * a.B);
    hipLaunchKernelGGL(k_global_rows_score<DT>, dim3(grid), dim3(kThreads), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_window_attention(int dtype, const AttnArgs& a, hipStream_t s) {
  return dtype == 1 ? launch_window_t<1>(a, s) : launch_window_t<0>(a, s);
}

hipError_t launch_score_from_partials(const float* partials, const int* valid_len, const int* gpos, int B, int n,
                                      int H, int G, const AttnGeom& g, float* scores, hipStream_t s) {
  dim3 grid((n + kScoreKeys - 1) / kScoreKeys, B);
  const int nw = H < kScoreMaxWaves ? H : kScoreMaxWaves;
  hipLaunchKernelGGL(k_score_from_partials, grid, dim3(64 * nw), 0, s, partials, valid_len, G > 0 ? gpos : nullptr, B,
                     n, H, G, g, scores);
  return hipGetLastError();
}

hipError_t launch_score_from_band(const float* bp, const int* valid_len, const int* gpos, int B, int n, int H, int G,
                                  const AttnGeom& g, float* scores, hipStream_t s) {
  dim3 grid((n + 255) / 256, B);
  hipLaunchKernelGGL(k_score_from_band, grid, dim3(256), 0, s, bp, valid_len, G > 0 ? gpos : nullptr, B, n, H, G, g,
                     scores);
  return hipGetLastError();
}

}  // namespace sc
