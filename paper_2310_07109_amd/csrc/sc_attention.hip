// Sliding-window + global-token sparse attention with exact importance-score
// partials, for gfx950 (SparseCoder, arXiv 2310.07109: Sec. 4.2.1 window,
// Sec. 3.1 global tokens, Sec. 5.5 score extraction).
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
//           and S^T = K.Q^T is computed on MFMA so that a lane holds one query
//           and 4 keys of each 16-key sub-tile.  Online softmax in the log2
//           domain with a lazily raised running max (rescale only when a tile
//           max exceeds it by 8), P rounded to the storage type, O^T += V^T.P^T
//           on MFMA.  Ends with O, and LSE for the exact second pass.
//   pass 2  (only when score partials are requested) the same tiles again; each
//           wave owns one 16-key sub-tile for all 64 queries, S = Q.K^T puts a
//           key in each lane and 4 queries per register, P = exp2(S*c - LSE2)
//           is exact, and the column sums are reduced inside the lane, then
//           across the 4 lane groups with shuffles.  One float per (block,
//           key) goes to HBM; no atomics, fixed summation order.
#include "sc_device.h"
#include "sc_internal.h"

namespace sc {
namespace {

constexpr int kThreads = 256;
constexpr int kBQ = kQueryBlock;
constexpr int kBK = kKeyTile;
constexpr float kTau = 8.0f;       // lazy-rescale slack in log2 units
constexpr float kNegBig = -1e30f;  // running-max sentinel (finite: avoids inf - inf)

// --------------------------------------------------------------- staging ----
// Tiles of 64 rows x 64 head dims move HBM -> registers -> LDS in two steps so
// that the loads of tile t+1 are in flight while tile t is computed.  Each
// thread moves kCpt 16-byte chunks of K (and of V).  rowfn(row) gives the
// source token of a tile row, or -1 for a zero row.
template <int DT>
struct Stage {
  using T = typename Tr<DT>::T;
  static constexpr int kEpc = 16 / sizeof(T);              // elements per chunk
  static constexpr int kCpr = kHeadDim / kEpc;             // chunks per row
  static constexpr int kCpt = 64 * kCpr / kThreads;        // chunks per thread
  static constexpr int P = Tr<DT>::kPitch;
  uint4 kr[kCpt];
  uint4 vr[kCpt];

  template <typename RowFn>
  SC_DEV void load_k(const T* g, long long ld, RowFn rowfn) {
#pragma unroll
    for (int i = 0; i < kCpt; ++i) {
      const int c = threadIdx.x + kThreads * i, row = c / kCpr, part = c % kCpr;
      const int src = rowfn(row);
      kr[i] = src >= 0 ? *reinterpret_cast<const uint4*>(g + (long long)src * ld + part * kEpc)
                       : make_uint4(0, 0, 0, 0);
    }
  }
  // V: f32 like K; bf16 as two consecutive rows x one chunk per thread (for
  // the transposed LDS layout).
  template <typename RowFn>
  SC_DEV void load_v(const T* g, long long ld, RowFn rowfn) {
    if constexpr (DT == 0) {
#pragma unroll
      for (int i = 0; i < kCpt; ++i) {
        const int c = threadIdx.x + kThreads * i, row = c / kCpr, part = c % kCpr;
        const int src = rowfn(row);
        vr[i] = src >= 0 ? *reinterpret_cast<const uint4*>(g + (long long)src * ld + part * kEpc)
                         : make_uint4(0, 0, 0, 0);
      }
    } else {
      const int part = threadIdx.x & 7, k0 = 2 * (threadIdx.x >> 3);
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int src = rowfn(k0 + i);
        vr[i] = src >= 0 ? *reinterpret_cast<const uint4*>(g + (long long)src * ld + 8 * part)
                         : make_uint4(0, 0, 0, 0);
      }
    }
  }
  SC_DEV void store_k(T* lds) const {
#pragma unroll
    for (int i = 0; i < kCpt; ++i) {
      const int c = threadIdx.x + kThreads * i, row = c / kCpr, part = c % kCpr;
      *reinterpret_cast<uint4*>(lds + row * P + part * kEpc) = kr[i];
    }
  }
  // bf16 V goes to LDS transposed, [dim][key position]: within each 32-key
  // half, keys 4q..4q+3 and 16+4q..16+4q+3 become 8 adjacent entries, the order
  // in which one lane group holds P for the P.V MFMA, so that one 16-byte LDS
  // read feeds the MFMA.
  SC_DEV void store_v(T* lds) const {
    if constexpr (DT == 0) {
#pragma unroll
      for (int i = 0; i < kCpt; ++i) {
        const int c = threadIdx.x + kThreads * i, row = c / kCpr, part = c % kCpr;
        *reinterpret_cast<uint4*>(lds + row * P + part * kEpc) = vr[i];
      }
    } else {
      const int part = threadIdx.x & 7, k0 = 2 * (threadIdx.x >> 3);
      const int half = k0 >> 5, t = k0 & 31;
      const int pos = 32 * half + (t < 16 ? 8 * (t >> 2) + (t & 3) : 8 * ((t - 16) >> 2) + 4 + (t & 3));
      const uint32_t av[4] = {vr[0].x, vr[0].y, vr[0].z, vr[0].w};
      const uint32_t bv[4] = {vr[1].x, vr[1].y, vr[1].z, vr[1].w};
      uint32_t* base = reinterpret_cast<uint32_t*>(lds);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t lo = (av[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
        const uint32_t hi = (bv[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
        base[((8 * part + j) * P + pos) >> 1] = lo | (hi << 16);  // pos even: k0 + 1 lands at pos + 1
      }
    }
  }
};

// Direct (unpipelined) copy of 64 rows into LDS, for the query tile.
template <int DT, typename RowFn>
SC_DEV void stage_rows(typename Tr<DT>::T* lds, const typename Tr<DT>::T* g, long long ld, RowFn rowfn) {
  Stage<DT> st;
  st.load_k(g, ld, rowfn);
  st.store_k(lds);
}

// ------------------------------------------------------------ pass 1 tile ---
// One 64-key tile for the 16 queries of a wave.  s holds S^T sub-tiles:
// s[st][i] is (key 16*st + 4g + i, query lr).  ok(st, i) masks keys.
template <int DT, bool kMasked, typename OkFn>
SC_DEV void softmax_tile(const typename Tr<DT>::Frag (&qf)[Tr<DT>::kChunks], const typename Tr<DT>::T* sK,
                         const typename Tr<DT>::T* sV, float c2, int lr, int g, float& m_use, float& l_run,
                         f32x4 (&o)[4], OkFn ok) {
  using TR = Tr<DT>;
  f32x4 s[4];
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    typename TR::Frag kf[TR::kChunks];
    TR::load_frags(sK + (16 * st + lr) * TR::kPitch, g, kf);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < TR::kChunks; ++c) acc = TR::mma(kf[c], qf[c], acc);
    s[st] = acc;
  }
  float tmax = -INFINITY;
#pragma unroll
  for (int st = 0; st < 4; ++st)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float x = s[st][i] * c2;
      if (kMasked && !ok(st, i)) x = -INFINITY;
      s[st][i] = x;
      tmax = fmaxf(tmax, x);
    }
  tmax = group_max(tmax);
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
      p[st][i] = fast_exp2(s[st][i] - m_use);
      l_run += p[st][i];
    }
  if constexpr (DT == 1) {
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      bf16x8 pb;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pb[i] = (__bf16)p[2 * kc][i];
        pb[4 + i] = (__bf16)p[2 * kc + 1][i];
      }
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const bf16x8 va = *reinterpret_cast<const bf16x8*>(sV + (16 * dt + lr) * TR::kPitch + 32 * kc + 8 * g);
        o[dt] = TR::mma(va, pb, o[dt]);
      }
    }
  } else {
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) o[dt] = TR::mma(sV[(16 * st + 4 * g + i) * TR::kPitch + 16 * dt + lr], p[st][i], o[dt]);
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

// ------------------------------------------------------- window kernel ------
template <int DT>
__global__ __launch_bounds__(kThreads) void k_window_attn(AttnArgs a) {
  using TR = Tr<DT>;
  using T = typename TR::T;
  using Frag = typename TR::Frag;
  constexpr int P = TR::kPitch;
  __shared__ __attribute__((aligned(16))) T sQ[kBQ * P];
  __shared__ __attribute__((aligned(16))) T sK[2][kBK * P];
  __shared__ __attribute__((aligned(16))) T sV[2][kBK * P];
  __shared__ float sL2[kBQ];
  __shared__ int sPos[2][kBK];
  extern __shared__ uint32_t sDyn[];  // [global bitmask over the band range][active global-slot chunks]

  const int total = a.nqb * a.H * a.B;
  const int lin = xcd_remap(blockIdx.x, total);
  const int qb = lin % a.nqb, bh = lin / a.nqb, h = bh % a.H, b = bh / a.H;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, lr = lane & 15;
  const int n = a.n, r = a.r, G = a.G;
  const int L = clampi(a.valid_len[b], 0, n);
  const int q0 = qb * kBQ;
  const T* Qg = static_cast<const T*>(a.q) + b * a.bs_in + h * kHeadDim;
  const T* Kg = static_cast<const T*>(a.k) + b * a.bs_in + h * kHeadDim;
  const T* Vg = static_cast<const T*>(a.v) + b * a.bs_in + h * kHeadDim;
  T* Og = static_cast<T*>(a.out) + b * a.bs_out + h * kHeadDim;
  float* lseg = a.lse ? a.lse + (long long)bh * n : nullptr;
  const int* gp = (a.gpos && G > 0) ? a.gpos + (long long)b * G : nullptr;

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

  const int kt0 = max(0, q0 - r);
  const int kt1 = min(L, q0 + kBQ + r);
  const int nkt = (kt1 - kt0 + kBK - 1) / kBK;
  const int nwords = (kt1 - kt0 + 31) >> 5;
  const int nxc = gp ? (G + kBK - 1) / kBK : 0;
  uint32_t* sBits = sDyn;                  // nwords
  int* sXList = reinterpret_cast<int*>(sDyn + a.rwp / 32 + 2);  // nxc + 1 entries
  __shared__ int sNx;

  for (int i = tid; i < nwords; i += kThreads) sBits[i] = 0u;
  for (int i = tid; i < nxc; i += kThreads) sXList[i] = 0;
  if (tid == 0) sNx = 0;
  __syncthreads();
  // global keys inside the band range -> bitmask; outside -> mark their chunk
  for (int j = tid; j < (gp ? G : 0); j += kThreads) {
    const int p = gp[j];
    if (p >= kt0 && p < kt1)
      atomicOr(&sBits[(p - kt0) >> 5], 1u << ((p - kt0) & 31));
    else if (p >= 0 && p < L)
      sXList[j / kBK] = 1;
  }
  // padding query rows are staged as zeros: their (unused) logits stay finite
  stage_rows<DT>(sQ, Qg, a.ld_in, [&](int row) { const int q = q0 + row; return q < L ? q : -1; });
  __syncthreads();
  if (tid == 0) {  // compact the list of chunks holding global keys outside the band
    int m = 0;
    for (int c = 0; c < nxc; ++c)
      if (sXList[c]) sXList[m++] = c;
    sNx = m;
  }
  __syncthreads();
  const int ntile = nkt + sNx;
  auto gbit = [&](int k) -> bool {
    const int o = k - kt0;
    return (sBits[o >> 5] >> (o & 31)) & 1u;
  };
  // source token of row `row` of tile t: band tiles first, then global-slot tiles
  auto rowf = [&](int t, int row) -> int {
    if (t < nkt) {
      const int k = kt0 + t * kBK + row;
      return k < kt1 ? k : -1;
    }
    const int j = kBK * sXList[t - nkt] + row;
    const int p = j < G ? gp[j] : -1;
    return (p >= 0 && p < L && (p < kt0 || p >= kt1)) ? p : -1;
  };

  // ---- pass 1: softmax + P.V for this wave's 16 queries
  Frag qf[TR::kChunks];
  TR::load_frags(sQ + (16 * w + lr) * P, g, qf);
  const int qa = q0 + 16 * w;
  const int qrow = qa + lr;
  float m_use = kNegBig, l_run = 0.f;
  f32x4 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  Stage<DT> st;
  int pos_reg = -1;
  auto load = [&](int t, bool with_v) {
    st.load_k(Kg, a.ld_in, [&](int row) { return rowf(t, row); });
    if (with_v) st.load_v(Vg, a.ld_in, [&](int row) { return rowf(t, row); });
    if (tid < kBK) pos_reg = rowf(t, tid);
  };
  auto store = [&](int buf, bool with_v) {
    st.store_k(sK[buf]);
    if (with_v) st.store_v(sV[buf]);
    if (tid < kBK) sPos[buf][tid] = pos_reg;
  };

  load(0, true);
  store(0, true);
  __syncthreads();
  for (int t = 0; t < ntile; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntile) load(t + 1, true);
    if (t < nkt) {
      const int k0 = kt0 + t * kBK;
      const uint32_t gw = sBits[2 * t] | (2 * t + 1 < nwords ? sBits[2 * t + 1] : 0u);
      const bool near = k0 <= qa + 15 + r && k0 + kBK - 1 >= qa - r;
      if (near || gw != 0u) {
        const bool interior = k0 + kBK <= kt1 && k0 >= qa + 15 - r && k0 + kBK - 1 <= qa + r;
        if (interior) {
          softmax_tile<DT, false>(qf, sK[buf], sV[buf], a.c2, lr, g, m_use, l_run, o, [](int, int) { return true; });
        } else {
          softmax_tile<DT, true>(qf, sK[buf], sV[buf], a.c2, lr, g, m_use, l_run, o, [&](int s4, int i) {
            const int k = k0 + 16 * s4 + 4 * g + i;
            return k < kt1 && (abs(qrow - k) <= r || gbit(k));
          });
        }
      }
    } else {
      const int* sp = sPos[buf];
      softmax_tile<DT, true>(qf, sK[buf], sV[buf], a.c2, lr, g, m_use, l_run, o,
                             [&](int s4, int i) { return sp[16 * s4 + 4 * g + i] >= 0; });
    }
    if (t + 1 < ntile) store(buf ^ 1, true);
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
    for (int dt = 0; dt < 4; ++dt) store_row4<DT>(Og + (long long)qrow * a.ld_out + 16 * dt + 4 * g, f32x4{0.f, 0.f, 0.f, 0.f});
    if (g == 0 && lseg) lseg[qrow] = -INFINITY;
  }
  if (g == 0) sL2[16 * w + lr] = qvalid ? lse2 : INFINITY;
  if (!a.part_band && !a.bp_band) return;  // uniform across the block

  // ---- pass 2: exact probabilities, column sums per key
  load(0, false);
  store(0, false);
  __syncthreads();
  Frag qf2[4][TR::kChunks];
  float l2[4][4];
#pragma unroll
  for (int qst = 0; qst < 4; ++qst) {
    TR::load_frags(sQ + (16 * qst + lr) * P, g, qf2[qst]);
#pragma unroll
    for (int i = 0; i < 4; ++i) l2[qst][i] = sL2[16 * qst + 4 * g + i];
  }
  float* pb = a.part_band ? a.part_band + ((long long)bh * a.nqb + qb) * a.rwp : nullptr;
  float* pe = a.part_band ? a.part_extra + ((long long)bh * a.nqb + qb) * G : nullptr;
  float* bpb = a.bp_band ? a.bp_band + (long long)bh * n * a.bw : nullptr;
  float* bpc = a.bp_band ? a.bp_gcol + (long long)bh * n * G : nullptr;
  // global-key partials of slots never visited stay zero
  if (pe)
    for (int j = tid; j < G; j += kThreads) pe[j] = 0.f;

  for (int t = 0; t < ntile; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntile) load(t + 1, false);
    float cs;
    if (t < nkt) {
      const int k0 = kt0 + t * kBK;
      const int key = k0 + 16 * w + lr;
      auto ok = [&](int qst, int i) {
        const int q = q0 + 16 * qst + 4 * g + i;
        return key < kt1 && (abs(q - key) <= r || gbit(key));
      };
      if (bpb) {
        const bool kglob = key < kt1 && gbit(key);
        const int kslot = kglob ? find_slot(gp, G, key) : -1;
        cs = score_tile<DT, true>(qf2, l2, sK[buf], w, a.c2, lr, g, ok, [&](int qst, int i, float p) {
          const int q = q0 + 16 * qst + 4 * g + i;
          if (!(q < L) || key >= kt1 || p == 0.f) return;
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
      if (pb && g == 0 && key < kt1) pb[key - kt0] = cs;
    } else {
      const int slot = kBK * sXList[t - nkt] + 16 * w + lr;
      const bool kvalid = sPos[buf][16 * w + lr] >= 0;
      auto ok = [&](int, int) { return kvalid; };
      if (bpc) {
        cs = score_tile<DT, true>(qf2, l2, sK[buf], w, a.c2, lr, g, ok, [&](int qst, int i, float p) {
          const int q = q0 + 16 * qst + 4 * g + i;
          if (kvalid && q < L && p != 0.f) bpc[(long long)q * G + slot] = p;
        });
      } else {
        cs = score_tile<DT, true>(qf2, l2, sK[buf], w, a.c2, lr, g, ok, NoEmit{});
      }
      if (pe && g == 0 && slot < G) pe[slot] = cs;
    }
    if (t + 1 < ntile) store(buf ^ 1, false);
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
  auto rowf = [&](int t, int row) { const int k = kbeg + t * kBK + row; return k < kend ? k : -1; };
  Stage<DT> st;
  auto load = [&](int t) {
    st.load_k(Kg, a.ld_in, [&](int row) { return rowf(t, row); });
    st.load_v(Vg, a.ld_in, [&](int row) { return rowf(t, row); });
  };
  stage_rows<DT>(sQ, Qg, a.ld_in, [&](int row) { return sPos[row]; });
  load(0);
  st.store_k(sK[0]);
  st.store_v(sV[0]);
  __syncthreads();
  typename TR::Frag qf[TR::kChunks];
  TR::load_frags(sQ + (16 * w + lr) * P, g, qf);
  float m_use = kNegBig, l_run = 0.f;
  f32x4 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int t = 0; t < ntile; ++t) {
    const int buf = t & 1, k0 = kbeg + t * kBK;
    if (t + 1 < ntile) load(t + 1);
    if (k0 + kBK <= kend)
      softmax_tile<DT, false>(qf, sK[buf], sV[buf], a.c2, lr, g, m_use, l_run, o, [](int, int) { return true; });
    else
      softmax_tile<DT, true>(qf, sK[buf], sV[buf], a.c2, lr, g, m_use, l_run, o,
                             [&](int s4, int i) { return k0 + 16 * s4 + 4 * g + i < kend; });
    if (t + 1 < ntile) {
      st.store_k(sK[buf ^ 1]);
      st.store_v(sV[buf ^ 1]);
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
  Stage<DT> st;
  auto load = [&](int t) {
    st.load_k(Kg, a.ld_in, [&](int row) { const int k = kbeg + t * kBK + row; return k < kend ? k : -1; });
  };
  stage_rows<DT>(sQ, Qg, a.ld_in, [&](int row) { return sPos[row]; });
  load(0);
  st.store_k(sK[0]);
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
    const int buf = t & 1;
    if (t + 1 < ntile) load(t + 1);
    const int key = kbeg + t * kBK + 16 * w + lr;
    auto ok = [&](int, int) { return key < kend; };
    float cs;
    if (bpr) {
      cs = score_tile<DT, true>(qf, l2, sK[buf], w, a.c2, lr, g, ok, [&](int qst, int i, float p) {
        const int slot = kGlobalChunk * blk.gc + 16 * qst + 4 * g + i;
        if (key < kend && slot < a.G && p != 0.f) bpr[(long long)slot * a.n + key] = p;
      });
    } else {
      cs = score_tile<DT, true>(qf, l2, sK[buf], w, a.c2, lr, g, ok, NoEmit{});
    }
    if (pg && g == 0 && key < kend) pg[key] = cs;
    if (t + 1 < ntile) st.store_k(sK[buf ^ 1]);
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

size_t attn_workspace_bytes(int B, int H, const AttnGeom& g) {
  if (g.Gp == 0) return 0;
  const size_t per = (size_t)B * H * g.Gp;
  return sizeof(float) * (per * g.nkc * (2 + kHeadDim) + per);
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
  profile_begin(s);
  hipLaunchKernelGGL(k_window_attn<DT>, dim3((unsigned)(a.nqb * a.H * a.B)), dim3(kThreads), dyn, s, a);
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
