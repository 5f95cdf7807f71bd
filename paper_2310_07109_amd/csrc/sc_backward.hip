// LTP soft pruning on gfx950: the training form of the pruning (SparseCoder,
// arXiv 2310.07109, Sec. 4.2.2 step 1: the model and the per-layer
// thresholds are trained through a soft mask before the mask is binarised)
// and its backward through the sparse attention and the importance scores.
//
// Forward (k_soft_mask, one wave per token):
//   m_k = sigmoid((s_k - theta) / T) for valid tokens that are not kept
//   global tokens, 1 for those, 0 for padding;  y[k] = m_k * out[k].
//
// Backward, given dL/dy and optionally dL/dm (e.g. from a regulariser):
//   k_soft_rows     one wave per token: dO = bf16(m * dy); dm = sum dy * out
//                   (+ dL/dm); ds = dm m (1 - m) / T (0 for kept global
//                   tokens and padding); g = ds / (H L); D = dO . out per head;
//                   ds summed per 4 tokens for the threshold's gradient.
//   k_bwd_rows<0>   D_q += sum_j P[q][j] g_j (the score's share of the row
//                   term of the softmax backward).
//   k_bwd_dfin      D of the global query rows from their span partials.
//   k_bwd_rows<1>   dQ_q = alpha sum_j dS[q][j] K_j, with
//                   dS = P (dO_q . V_j + g_j - D_q) and P = exp2(S c2 - LSE2)
//                   recomputed from the forward's LSE.
//   k_bwd_cols      dK_j = alpha sum_q dS[q][j] Q_q, dV_j = sum_q P[q][j] dO_q.
//   k_bwd_finish    the global rows' dQ and the global keys' dK, dV from their
//                   span partials; dtheta = -sum ds.
// Row-side work (D, dQ) is done per 64-query block over the block's band key
// tiles plus tiles of gathered global keys, and per (64 global query rows,
// 512-key span) for the global rows.  Column-side work (dK, dV) is done per
// 64-key block over its band query tiles plus tiles of gathered global query
// rows, and per (64 global keys, 512-query span) for the global keys.  Each
// allowed pair is counted once on each side: (q, k) with k global lives in the
// global-key tiles and the global-column blocks, q global in the global-row
// blocks and the global-query tiles, the rest in the band.  Every sum has a
// fixed order; no atomics.
//
// MFMA layouts are the forward's: S^T = K Q^T puts a query in each lane and
// 4 keys per register (row side), S = Q K^T a key in each lane and 4 queries
// per register (column side); the second product of each side reads its
// row-major LDS tile with transposed reads, rows in MFMA k order.
#include <type_traits>

#include "sc_device.h"
#include "sc_internal.h"

namespace sc {
namespace {

using TRb = Tr<1>;

SC_DEV float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Whether token k of the sequence is a used global slot (G small: one pass of
// the wave over the slots).
SC_DEV bool wave_is_global(const int* gp, int G, int k) {
  bool hit = false;
  for (int j = threadIdx.x & 63; j < G; j += 64) hit |= gp[j] == k;
  return __builtin_amdgcn_ballot_w64(hit) != 0ull;
}

// ------------------------------------------------------------ forward mask --
__global__ __launch_bounds__(256) void k_soft_mask(SoftArgs a) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const long long t = (long long)blockIdx.x * 4 + w;
  if (t >= (long long)a.B * a.n) return;
  const int b = (int)(t / a.n), k = (int)(t % a.n);
  const int L = clampi(a.valid_len[b], 0, a.n);
  const long long ld = (long long)a.H * kHeadDim;
  float m = 0.f;
  if (k < L) {
    const bool g = a.keep_global && a.gpos && wave_is_global(a.gpos + (long long)b * a.G, a.G, k);
    m = g ? 1.f : 1.f / (1.f + __expf(-(a.scores[t] - a.theta) * a.inv_t));
  }
  if (lane == 0) a.mask_out[t] = m;
  const __bf16* o = a.o + t * ld;
  __bf16* y = a.y + t * ld;
  if (k >= L) {  // padding: y = 0 without reading out
    for (int u = lane; u < a.H * 8; u += 64) *reinterpret_cast<uint4*>(y + 8 * u) = make_uint4(0, 0, 0, 0);
    return;
  }
  for (int base = 0; base < a.H * 8; base += 128) {  // two passes' loads in flight
    bf16x8 x[2];
#pragma unroll
    for (int ps = 0; ps < 2; ++ps) x[ps] = *reinterpret_cast<const bf16x8*>(o + 8 * min(base + 64 * ps + lane, a.H * 8 - 1));
#pragma unroll
    for (int ps = 0; ps < 2; ++ps) {
      const int u = base + 64 * ps + lane;
      if (u < a.H * 8) {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[ps][e] = (__bf16)(m * (float)x[ps][e]);
        *reinterpret_cast<bf16x8*>(y + 8 * u) = x[ps];
      }
    }
  }
}

// ------------------------------------------------------------- row terms --
// One wave per token; returns the token's score gradient ds (0 for padding).
SC_DEV float soft_row(const SoftArgs& a, long long t, int lane) {
  const int b = (int)(t / a.n), k = (int)(t % a.n), H = a.H;
  const int L = clampi(a.valid_len[b], 0, a.n);
  const long long ld = (long long)H * kHeadDim;
  const __bf16* dy = a.dy + t * ld;
  const __bf16* o = a.o + t * ld;
  __bf16* dO = a.dO + t * ld;
  float* Dq = a.Dq + (long long)b * H * a.n + k;  // head h at Dq[h * n]
  if (k >= L) {
    for (int u = lane; u < H * 8; u += 64) *reinterpret_cast<uint4*>(dO + 8 * u) = make_uint4(0, 0, 0, 0);
    for (int h = lane; h < H; h += 64) Dq[(long long)h * a.n] = 0.f;
    if (lane == 0) a.gk[t] = 0.f;
    return 0.f;
  }
  const float m = a.mask[t];
  float dm = 0.f;
  // 16-byte units: unit u holds dims 8(u % 8) .. of head u / 8; in each pass
  // of the wave, lanes 8j .. 8j + 7 hold the whole of one head.  Two passes'
  // loads are issued before any of them is used.
  for (int base = 0; base < H * 8; base += 128) {
    bf16x8 yv[2], ov[2];
#pragma unroll
    for (int ps = 0; ps < 2; ++ps) {
      const int u = min(base + 64 * ps + lane, H * 8 - 1);  // clamped: loads stay in the row
      yv[ps] = *reinterpret_cast<const bf16x8*>(dy + 8 * u);
      ov[ps] = *reinterpret_cast<const bf16x8*>(o + 8 * u);
    }
#pragma unroll
    for (int ps = 0; ps < 2; ++ps) {
      const int u = base + 64 * ps + lane;
      float hd = 0.f;
      if (u < H * 8) {
        bf16x8 dv;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float yf = (float)yv[ps][e], of = (float)ov[ps][e];
          dm = fmaf(yf, of, dm);
          dv[e] = (__bf16)(m * yf);
          hd = fmaf((float)dv[e], of, hd);
        }
        *reinterpret_cast<bf16x8*>(dO + 8 * u) = dv;
      }
      hd += __shfl_xor(hd, 1, 64);
      hd += __shfl_xor(hd, 2, 64);
      hd += __shfl_xor(hd, 4, 64);
      if ((lane & 7) == 0 && u < H * 8) Dq[(long long)(u >> 3) * a.n] = hd;
    }
  }
  dm = wave_sum(dm);
  if (a.dmask) dm += a.dmask[t];
  const bool g = a.keep_global && a.gpos && wave_is_global(a.gpos + (long long)b * a.G, a.G, k);
  const float ds = g ? 0.f : dm * m * (1.f - m) * a.inv_t;
  if (lane == 0) a.gk[t] = ds / ((float)H * (float)L);
  return ds;
}

// Workgroup = 4 tokens; their ds are added in wave order into dsv[workgroup]
// (the threshold's gradient sums these partials).
__global__ __launch_bounds__(256) void k_soft_rows(SoftArgs a) {
  __shared__ float red[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const long long t = (long long)blockIdx.x * 4 + w;
  const float ds = t < (long long)a.B * a.n ? soft_row(a, t, lane) : 0.f;
  if (lane == 0) red[w] = ds;
  __syncthreads();
  if (threadIdx.x == 0) a.dsv[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

// ---------------------------------------------------------- tile helpers --
// acc[dt] += A^T B where A is a 64-row bf16 tile (rows in MFMA k order:
// lane (g, lr) supplies dims 16 dt + 4 (lr & 3) .. of rows 32 kc + 4g + lr / 4
// and 32 kc + 16 + 4g + lr / 4) and B the packed bf16 operand of chunk kc.
SC_DEV void mma_tr(const __bf16* tile, const bf16x8 (&pb)[2], f32x4 (&acc)[4]) {
  const int ln = threadIdx.x & 63, lr = ln & 15, g = ln >> 4;
#pragma unroll
  for (int kc = 0; kc < 2; ++kc) {
    const int vr = 32 * kc + 4 * g + (lr >> 2), bsel = (lr >> 1) & 1, e = 4 * (lr & 1);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const i16x4 a0 = lds_read_tr16(tile + TRb::off(vr, 2 * dt + bsel) + e);
      const i16x4 a1 = lds_read_tr16(tile + TRb::off(vr + 16, 2 * dt + bsel) + e);
      const bf16x8 af = __builtin_bit_cast(bf16x8, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
      acc[dt] = TRb::mma(af, pb[kc], acc[dt]);
    }
  }
}

// s[st] = init[st] + A_st B^T for the four 16-row sub-tiles of an LDS tile A
// (rows 16 st + lr) and a register operand B of the wave's 16 rows.
SC_DEV void mma_rows(const __bf16* tile, const bf16x8 (&bf)[2], f32x4 (&s)[4], int lr, int g,
                     const f32x4 (&init)[4]) {
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    bf16x8 af[2];
    TRb::load_frags(tile, 16 * st + lr, g, af);
    f32x4 c = init[st];
    c = TRb::mma(af[0], bf[0], c);
    c = TRb::mma(af[1], bf[1], c);
    s[st] = c;
  }
}
SC_DEV void mma_rows(const __bf16* tile, const bf16x8 (&bf)[2], f32x4 (&s)[4], int lr, int g) {
  const f32x4 z[4] = {};
  mma_rows(tile, bf, s, lr, g, z);
}

// The global-token bitmask of a sequence in LDS (band blocks).
SC_DEV void build_bits(uint32_t* bits, const int* gp, int G, int L, int n) {
  const int nw = (n + 31) >> 5;
  for (int i = threadIdx.x; i < nw; i += blockDim.x) bits[i] = 0u;
  __syncthreads();
  if (gp)
    for (int j = threadIdx.x; j < G; j += blockDim.x) {
      const int p = gp[j];
      if (p >= 0 && p < L) atomicOr(&bits[p >> 5], 1u << (p & 31));
    }
  __syncthreads();
}

SC_DEV bool bit_of(const uint32_t* bits, int t) { return (bits[t >> 5] >> (t & 31)) & 1u; }

SC_DEV void store4_bf16(__bf16* p, f32x4 v, float scale) {
  bf16x4 x;
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = (__bf16)(v[i] * scale);
  *reinterpret_cast<bf16x4*>(p) = x;
}

// ------------------------------------------------------------- row side --
// kMode 0: D += P g;  kMode 1: dQ.  kGRows: global-row blocks (64 gathered
// global queries x one 512-key span) instead of band blocks (64 queries).
// LDS of the row side (K and V tiles, double-buffered, and their metadata)
// and of the column side (Q and dO tiles); one launch may hold both kinds.
struct RowSmemK {  // the D pass reads K only
  __bf16 sK[2][64 * 64];
  float sBias[2][64];  // 0 for a key counted in this tile, -inf otherwise
  float sG[2][64];
};
struct RowSmem {
  __bf16 sK[2][64 * 64];
  float sBias[2][64];
  float sG[2][64];
  __bf16 sV[2][64 * 64];
};
struct ColSmem {
  __bf16 sQ[2][64 * 64];
  __bf16 sO[2][64 * 64];  // dO rows
  float sL2[2][64];       // LSE2 of a query counted in this tile, +inf otherwise
  float sD[2][64];
};
union BwdSmem {
  RowSmem row;
  ColSmem col;
};

template <int kMode, bool kGRows, typename Smem>
SC_DEV void bwd_rows(const SoftArgs& a, int blk, Smem& sm, uint32_t* sBits) {
  auto& sK = sm.sK;
  auto& sBias = sm.sBias;
  auto& sG = sm.sG;
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6), lr = lane & 15,
            g = lane >> 4;
  const int H = a.H, n = a.n, G = a.G, r = a.r;
  int bh, q0 = 0, span = 0, gc = 0;
  if constexpr (!kGRows) {  // a (sequence, head)'s query blocks in order on one XCD
    const int nqb = (n + 63) / 64;
    int qb;
    xcd_pair_map(blk, nqb, a.B * H, bh, qb);
    q0 = 64 * qb;
  } else {
    span = blk % a.nsp;
    blk /= a.nsp;
    const int ngc = a.Gp / 64;
    gc = blk % ngc;
    bh = blk / ngc;
  }
  const int b = bh / H, h = bh % H;
  const int L = clampi(a.valid_len[b], 0, n);
  const int* gp = a.gpos ? a.gpos + (long long)b * G : nullptr;
  const long long ld = (long long)H * kHeadDim;
  const unsigned ldb = (unsigned)(2 * ld);
  const long long seq = (long long)b * n * ld + (long long)h * kHeadDim;
  if constexpr (!kGRows) {
    if (q0 >= L) {
      if (kMode == 1)  // padding queries: zero gradient rows
        for (int i = tid; i < 64 * 8; i += 256) {
          const int q = q0 + i / 8;
          if (q < n) *reinterpret_cast<uint4*>(a.dq + seq + q * ld + 8 * (i % 8)) = make_uint4(0, 0, 0, 0);
        }
      return;
    }
    build_bits(sBits, gp, G, L, n);
  } else {
    if (span * kBwdSpan >= L) return;
  }
  // this lane's query
  int q, slot = 0;
  bool qok;
  if constexpr (!kGRows) {
    q = q0 + 16 * w + lr;
    qok = q < L && !bit_of(sBits, q);
  } else {
    slot = 64 * gc + 16 * w + lr;
    q = (gp && slot < G) ? gp[slot] : -1;
    qok = q >= 0 && q < L;
  }
  const int qs = qok ? q : 0;
  bf16x8 qf[2], df[2];
  qf[0] = *reinterpret_cast<const bf16x8*>(a.q + seq + qs * ld + 8 * g);
  qf[1] = *reinterpret_cast<const bf16x8*>(a.q + seq + qs * ld + 32 + 8 * g);
  if constexpr (kMode == 1) {
    df[0] = *reinterpret_cast<const bf16x8*>(a.dO + seq + qs * ld + 8 * g);
    df[1] = *reinterpret_cast<const bf16x8*>(a.dO + seq + qs * ld + 32 + 8 * g);
  }
  const long long dqi = (long long)bh * n + qs;
  const float lse2 = qok ? a.lse[dqi] * kLog2e : 0.f;
  const float Dv = (kMode == 1 && qok) ? a.Dq[dqi] : 0.f;
  const float c2 = a.c2;
  // key tiles: the band, then the gathered global keys (band blocks); or the span
  int kt0, kt1, ngt = 0;
  if constexpr (!kGRows) {
    kt0 = max(0, q0 - r);
    kt1 = min(L, q0 + 64 + r);
    ngt = gp ? (G + 63) / 64 : 0;
  } else {
    kt0 = span * kBwdSpan;
    kt1 = min(L, kt0 + kBwdSpan);
  }
  const int nband = (kt1 - kt0 + 63) / 64, nt = nband + ngt;
  // key of tile row R of tile tt, or -1 where no pair of this block's side is
  // counted in that tile; dma_row: a valid row to load in its place
  auto key_of = [&](int tt, int R) {
    if (tt < nband) {
      const int key = kt0 + 64 * tt + R;
      return (key < kt1 && (kGRows || !bit_of(sBits, key))) ? key : -1;
    }
    const int sl = 64 * (tt - nband) + R;
    const int key = sl < G ? gp[sl] : -1;
    return (key >= 0 && key < L) ? key : -1;
  };
  auto issue = [&](int tt, int buf) {
    const int lane2 = opaque_lane();
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int R0 = 16 * w + 8 * j, R = R0 + (lane2 >> 3);
      int row;
      if (tt < nband) {
        row = min(kt0 + 64 * tt + R, L - 1);
      } else {
        const int sl = 64 * (tt - nband) + R;
        row = sl < G ? gp[sl] : 0;
        row = (row >= 0 && row < L) ? row : 0;
      }
      const unsigned u = (lane2 & 7) ^ (lane2 >> 3), voff = (unsigned)row * ldb + 16u * u;
      lds_dma16(a.k + seq, voff, lds_addr(&sK[buf][R0 * TRb::kPitch]));
      if constexpr (kMode == 1) lds_dma16(a.v + seq, voff, lds_addr(&sm.sV[buf][R0 * TRb::kPitch]));
    }
  };
  float pg = 0.f;
  f32x4 acc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // one tile; kEdge: the band condition is checked per pair (edge tiles of a
  // band block), else every counted key of the tile is in the band of every
  // query of the block.  Lanes of queries not counted here compute values
  // that are never stored.
  auto tile = [&](auto edge_c, int t, int cur) {
    constexpr bool kEdge = decltype(edge_c)::value;
    const int kbase = kt0 + 64 * t;
    f32x4 s[4];
    mma_rows(sK[cur], qf, s, lr, g);
    float p[4][4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const f32x4 bias = *reinterpret_cast<const f32x4*>(&sBias[cur][16 * st + 4 * g]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float x = fmaf(s[st][i], c2, -lse2) + bias[i];
        if constexpr (kEdge) x = (unsigned)(kbase + 16 * st + 4 * g + i - q + r) <= (unsigned)(2 * r) ? x : -INFINITY;
        p[st][i] = fast_exp2(x);
      }
    }
    if constexpr (kMode == 0) {
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        const f32x4 gg = *reinterpret_cast<const f32x4*>(&sG[cur][16 * st + 4 * g]);
#pragma unroll
        for (int i = 0; i < 4; ++i) pg = fmaf(p[st][i], gg[i], pg);
      }
    } else {
      // dP^T + g: the MFMA accumulates onto the keys' score gradients
      f32x4 gg[4], dp[4];
#pragma unroll
      for (int st = 0; st < 4; ++st) gg[st] = *reinterpret_cast<const f32x4*>(&sG[cur][16 * st + 4 * g]);
      mma_rows(sm.sV[cur], df, dp, lr, g, gg);
      bf16x8 pb[2];
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int i = 0; i < 4; ++i) pb[st >> 1][4 * (st & 1) + i] = (__bf16)(p[st][i] * (dp[st][i] - Dv));
      mma_tr(sK[cur], pb, acc);
    }
  };
  if (nt > 0) {
    issue(0, 0);
    if (tid < 64) {
      const int key = key_of(0, tid);
      sBias[0][tid] = key >= 0 ? 0.f : -INFINITY;
      sG[0][tid] = key >= 0 ? a.gk[(long long)b * n + key] : 0.f;
    }
  }
  for (int t = 0; t < nt; ++t) {
    const int cur = t & 1;
    wait_dma();
    __syncthreads();  // tile t and its metadata are in LDS; buffers of tile t - 1 are free
    const bool more = t + 1 < nt;
    if (more) issue(t + 1, cur ^ 1);
    float nbias = 0.f, ng = 0.f;
    if (tid < 64 && more) {
      const int nkey = key_of(t + 1, tid);
      nbias = nkey >= 0 ? 0.f : -INFINITY;
      ng = nkey >= 0 ? a.gk[(long long)b * n + nkey] : 0.f;
    }
    const int kbase = kt0 + 64 * t;
    const bool edge = !kGRows && t < nband && !(kbase >= q0 + 63 - r && kbase + 63 <= q0 + r);
    if (edge)
      tile(std::true_type{}, t, cur);
    else
      tile(std::false_type{}, t, cur);
    if (tid < 64 && more) {  // the metadata buffer of tile t + 1 was last read by tile t - 1
      sBias[cur ^ 1][tid] = nbias;
      sG[cur ^ 1][tid] = ng;
    }
  }
  if constexpr (kMode == 0) {
    const float tot = group_sum(pg);
    if (g == 0 && qok) {
      if constexpr (!kGRows)
        a.Dq[dqi] += tot;
      else
        a.gpg[((long long)bh * a.nsp + span) * a.Gp + slot] = tot;
    }
  } else {
    if constexpr (!kGRows) {
      __bf16* dst = a.dq + seq + q * ld;
      if (qok) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) store4_bf16(dst + 16 * dt + 4 * g, acc[dt], a.alpha);
      } else if (q >= L && q < n) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) *reinterpret_cast<uint2*>(dst + 16 * dt + 4 * g) = make_uint2(0, 0);
      }
    } else if (qok) {
      float* dst = a.gdq + (((long long)bh * a.nsp + span) * a.Gp + slot) * kHeadDim;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        f32x4 v = acc[dt];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] *= a.alpha;
        *reinterpret_cast<f32x4*>(dst + 16 * dt + 4 * g) = v;
      }
    }
  }
}

// D of the global query rows: + their span partials, in span order.
__global__ __launch_bounds__(64) void k_bwd_dfin(SoftArgs a) {
  const int bh = blockIdx.x, b = bh / a.H, n = a.n;
  const int L = clampi(a.valid_len[b], 0, n);
  const int nspv = (L + kBwdSpan - 1) / kBwdSpan;
  for (int j = threadIdx.x; j < a.G; j += 64) {
    const int q = a.gpos[(long long)b * a.G + j];
    if (q < 0 || q >= L) continue;
    float tot = a.Dq[(long long)bh * n + q];
    for (int sp = 0; sp < nspv; ++sp) tot += a.gpg[((long long)bh * a.nsp + sp) * a.Gp + j];
    a.Dq[(long long)bh * n + q] = tot;
  }
}

// ---------------------------------------------------------- column side --
// dK, dV.  kGCols: global-column blocks (64 gathered global keys x one
// 512-query span) instead of band blocks (64 keys).
template <bool kGCols>
SC_DEV void bwd_cols(const SoftArgs& a, int blk, ColSmem& sm, uint32_t* sBits) {
  auto& sQ = sm.sQ;
  auto& sO = sm.sO;
  auto& sL2 = sm.sL2;
  auto& sD = sm.sD;
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6), lr = lane & 15,
            g = lane >> 4;
  const int H = a.H, n = a.n, G = a.G, r = a.r;
  int bh, k0 = 0, span = 0, gc = 0;
  if constexpr (!kGCols) {  // a (sequence, head)'s key blocks in order on one XCD
    const int nkb = (n + 63) / 64;
    int kb;
    xcd_pair_map(blk, nkb, a.B * H, bh, kb);
    k0 = 64 * kb;
  } else {
    span = blk % a.nsp;
    blk /= a.nsp;
    const int ngc = a.Gp / 64;
    gc = blk % ngc;
    bh = blk / ngc;
  }
  const int b = bh / H, h = bh % H;
  const int L = clampi(a.valid_len[b], 0, n);
  const int* gp = a.gpos ? a.gpos + (long long)b * G : nullptr;
  const long long ld = (long long)H * kHeadDim;
  const unsigned ldb = (unsigned)(2 * ld);
  const long long seq = (long long)b * n * ld + (long long)h * kHeadDim;
  if constexpr (!kGCols) {
    if (k0 >= L) {  // padding keys: zero gradient rows
      for (int i = tid; i < 64 * 8; i += 256) {
        const int k = k0 + i / 8;
        if (k < n) {
          *reinterpret_cast<uint4*>(a.dk + seq + k * ld + 8 * (i % 8)) = make_uint4(0, 0, 0, 0);
          *reinterpret_cast<uint4*>(a.dv + seq + k * ld + 8 * (i % 8)) = make_uint4(0, 0, 0, 0);
        }
      }
      return;
    }
    build_bits(sBits, gp, G, L, n);
  } else {
    if (span * kBwdSpan >= L) return;
  }
  int k, slot = 0;
  bool kok;
  if constexpr (!kGCols) {
    k = k0 + 16 * w + lr;
    kok = k < L && !bit_of(sBits, k);
  } else {
    slot = 64 * gc + 16 * w + lr;
    k = (gp && slot < G) ? gp[slot] : -1;
    kok = k >= 0 && k < L;
  }
  const int ks = kok ? k : 0;
  bf16x8 kf[2], vf[2];
  kf[0] = *reinterpret_cast<const bf16x8*>(a.k + seq + ks * ld + 8 * g);
  kf[1] = *reinterpret_cast<const bf16x8*>(a.k + seq + ks * ld + 32 + 8 * g);
  vf[0] = *reinterpret_cast<const bf16x8*>(a.v + seq + ks * ld + 8 * g);
  vf[1] = *reinterpret_cast<const bf16x8*>(a.v + seq + ks * ld + 32 + 8 * g);
  const float gkv = kok ? a.gk[(long long)b * n + k] : 0.f;
  const float c2 = a.c2;
  int qt0, qt1, ngt = 0;
  if constexpr (!kGCols) {
    qt0 = max(0, k0 - r);
    qt1 = min(L, k0 + 64 + r);
    ngt = gp ? (G + 63) / 64 : 0;
  } else {
    qt0 = span * kBwdSpan;
    qt1 = min(L, qt0 + kBwdSpan);
  }
  const int nband = (qt1 - qt0 + 63) / 64, nt = nband + ngt;
  auto query_of = [&](int tt, int R) {
    if (tt < nband) {
      const int qq = qt0 + 64 * tt + R;
      return (qq < qt1 && (kGCols || !bit_of(sBits, qq))) ? qq : -1;
    }
    const int sl = 64 * (tt - nband) + R;
    const int qq = sl < G ? gp[sl] : -1;
    return (qq >= 0 && qq < L) ? qq : -1;
  };
  auto issue = [&](int tt, int buf) {
    const int lane2 = opaque_lane();
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int R0 = 16 * w + 8 * j, R = R0 + (lane2 >> 3);
      int row;
      if (tt < nband) {
        row = min(qt0 + 64 * tt + R, L - 1);
      } else {
        const int sl = 64 * (tt - nband) + R;
        row = sl < G ? gp[sl] : 0;
        row = (row >= 0 && row < L) ? row : 0;
      }
      const unsigned u = (lane2 & 7) ^ (lane2 >> 3), voff = (unsigned)row * ldb + 16u * u;
      lds_dma16(a.q + seq, voff, lds_addr(&sQ[buf][R0 * TRb::kPitch]));
      lds_dma16(a.dO + seq, voff, lds_addr(&sO[buf][R0 * TRb::kPitch]));
    }
  };
  f32x4 accK[4], accV[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
    accK[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    accV[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // one tile; kEdge: the band condition is checked per pair.  Lanes of keys
  // not counted here compute values that are never stored.
  auto tile = [&](auto edge_c, int t, int cur) {
    constexpr bool kEdge = decltype(edge_c)::value;
    const int qbase = qt0 + 64 * t;
    f32x4 s[4], dp[4];
    const f32x4 gk4[4] = {f32x4{gkv, gkv, gkv, gkv}, f32x4{gkv, gkv, gkv, gkv}, f32x4{gkv, gkv, gkv, gkv},
                          f32x4{gkv, gkv, gkv, gkv}};
    mma_rows(sQ[cur], kf, s, lr, g);
    mma_rows(sO[cur], vf, dp, lr, g, gk4);  // dP + g of the lane's key
    bf16x8 pP[2], pS[2];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const f32x4 l2 = *reinterpret_cast<const f32x4*>(&sL2[cur][16 * st + 4 * g]);
      const f32x4 dd = *reinterpret_cast<const f32x4*>(&sD[cur][16 * st + 4 * g]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float x = fmaf(s[st][i], c2, -l2[i]);
        if constexpr (kEdge) x = (unsigned)(qbase + 16 * st + 4 * g + i - k + r) <= (unsigned)(2 * r) ? x : -INFINITY;
        const float p = fast_exp2(x);
        pP[st >> 1][4 * (st & 1) + i] = (__bf16)p;
        pS[st >> 1][4 * (st & 1) + i] = (__bf16)(p * (dp[st][i] - dd[i]));
      }
    }
    mma_tr(sO[cur], pP, accV);
    mma_tr(sQ[cur], pS, accK);
  };
  if (nt > 0) {
    issue(0, 0);
    if (tid < 64) {
      const int qq = query_of(0, tid);
      sL2[0][tid] = qq >= 0 ? a.lse[(long long)bh * n + qq] * kLog2e : INFINITY;
      sD[0][tid] = qq >= 0 ? a.Dq[(long long)bh * n + qq] : 0.f;
    }
  }
  for (int t = 0; t < nt; ++t) {
    const int cur = t & 1;
    wait_dma();
    __syncthreads();  // tile t and its metadata are in LDS; buffers of tile t - 1 are free
    const bool more = t + 1 < nt;
    if (more) issue(t + 1, cur ^ 1);
    float nl2 = INFINITY, nd = 0.f;
    if (tid < 64 && more) {
      const int nq = query_of(t + 1, tid);
      if (nq >= 0) {
        nl2 = a.lse[(long long)bh * n + nq] * kLog2e;
        nd = a.Dq[(long long)bh * n + nq];
      }
    }
    const int qbase = qt0 + 64 * t;
    const bool edge = !kGCols && t < nband && !(qbase >= k0 + 63 - r && qbase + 63 <= k0 + r);
    if (edge)
      tile(std::true_type{}, t, cur);
    else
      tile(std::false_type{}, t, cur);
    if (tid < 64 && more) {  // the metadata buffer of tile t + 1 was last read by tile t - 1
      sL2[cur ^ 1][tid] = nl2;
      sD[cur ^ 1][tid] = nd;
    }
  }
  if constexpr (!kGCols) {
    if (kok) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        store4_bf16(a.dk + seq + k * ld + 16 * dt + 4 * g, accK[dt], a.alpha);
        store4_bf16(a.dv + seq + k * ld + 16 * dt + 4 * g, accV[dt], 1.f);
      }
    } else if (k >= L && k < n) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        *reinterpret_cast<uint2*>(a.dk + seq + k * ld + 16 * dt + 4 * g) = make_uint2(0, 0);
        *reinterpret_cast<uint2*>(a.dv + seq + k * ld + 16 * dt + 4 * g) = make_uint2(0, 0);
      }
    }
  } else if (kok) {
    const long long o = (((long long)bh * a.nsp + span) * a.Gp + slot) * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      f32x4 v = accK[dt];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] *= a.alpha;
      *reinterpret_cast<f32x4*>(a.gdk + o + 16 * dt + 4 * g) = v;
      *reinterpret_cast<f32x4*>(a.gdv + o + 16 * dt + 4 * g) = accV[dt];
    }
  }
}

// Block ranges of the two main launches, each starting at a multiple of 8 so
// that the band blocks' XCD mapping holds: the global-span blocks first (few,
// long), then the band blocks.
struct BwdGrid {
  int gr, gc, band;  // padded block counts of global-row, global-column and band segments
};

// D pass: [global rows][band rows].
__global__ __launch_bounds__(256) void k_bwd_dpass(SoftArgs a, BwdGrid gd) {
  __shared__ __align__(16) RowSmemK sm;
  extern __shared__ uint32_t sBits[];
  const int blk = blockIdx.x;
  if (blk < gd.gr) {
    if (blk < a.B * a.H * (a.Gp / 64) * a.nsp) bwd_rows<0, true>(a, blk, sm, sBits);
    return;
  }
  bwd_rows<0, false>(a, blk - gd.gr, sm, sBits);
}

// Gradients: [global columns][global rows][band rows (dQ)][band columns (dK, dV)].
__global__ __launch_bounds__(256) void k_bwd_grad(SoftArgs a, BwdGrid gd) {
  __shared__ __align__(16) BwdSmem sm;
  extern __shared__ uint32_t sBits[];
  const int nglob = a.B * a.H * (a.Gp / 64) * a.nsp;
  int blk = blockIdx.x;
  if (blk < gd.gc) {
    if (blk < nglob) bwd_cols<true>(a, blk, sm.col, sBits);
    return;
  }
  blk -= gd.gc;
  if (blk < gd.gr) {
    if (blk < nglob) bwd_rows<1, true>(a, blk, sm.row, sBits);
    return;
  }
  blk -= gd.gr;
  if (blk < gd.band) {
    if (blk < a.B * a.H * ((a.n + 63) / 64)) bwd_rows<1, false>(a, blk, sm.row, sBits);
    return;
  }
  bwd_cols<false>(a, blk - gd.band, sm.col, sBits);
}

// Global rows' dQ and global keys' dK, dV: sums of the span partials in span
// order, one thread per (sequence, head, slot, dim) with all its loads in
// flight (blocks 0 .. nfin - 1); dtheta = -sum ds in a fixed order (the last
// block).
constexpr int kFinSpans = 16;  // spans summed with every load issued first (longer sequences loop)

__global__ __launch_bounds__(256) void k_bwd_finish(SoftArgs a, int nfin) {
  __shared__ float red[256];
  const int tid = threadIdx.x, n = a.n, H = a.H;
  if ((int)blockIdx.x == nfin) {
    // thread t adds the 4-float groups t, t + 256, ... with eight groups in
    // flight, then the scalar tail; the threads' sums meet in a fixed tree
    const long long tot = ((long long)a.B * n + 3) / 4, nv = tot / 4;  // one partial per 4 tokens
    const f32x4* v4 = reinterpret_cast<const f32x4*>(a.dsv);
    float part[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (long long base = tid; base < nv; base += 256 * 8) {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const long long i = base + 256LL * u;
        if (i < nv) {
          const f32x4 x = v4[i];
          part[u] += (x[0] + x[1]) + (x[2] + x[3]);
        }
      }
    }
    float acc = ((part[0] + part[1]) + (part[2] + part[3])) + ((part[4] + part[5]) + (part[6] + part[7]));
    for (long long i = 4 * nv + tid; i < tot; i += 256) acc += a.dsv[i];
    red[tid] = acc;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
      if (tid < off) red[tid] += red[tid + off];
      __syncthreads();
    }
    if (tid == 0) *a.dtheta = -red[0];
    return;
  }
  const long long e = (long long)blockIdx.x * 256 + tid;  // (bh, slot, dim)
  const int c = (int)(e % kHeadDim), j = (int)((e / kHeadDim) % a.G), bh = (int)(e / ((long long)kHeadDim * a.G));
  if (bh >= a.B * H) return;
  const int b = bh / H, h = bh % H;
  const int L = clampi(a.valid_len[b], 0, n);
  const int p = a.gpos[(long long)b * a.G + j];
  if (p < 0 || p >= L) return;
  const int nspv = (L + kBwdSpan - 1) / kBwdSpan;
  const long long o0 = ((long long)bh * a.nsp * a.Gp + j) * kHeadDim + c, so = (long long)a.Gp * kHeadDim;
  float sq = 0.f, sk = 0.f, sv = 0.f;
  for (int base = 0; base < nspv; base += kFinSpans) {
    float xq[kFinSpans], xk[kFinSpans], xv[kFinSpans];
#pragma unroll
    for (int u = 0; u < kFinSpans; ++u) {
      const bool in = base + u < nspv;
      const long long o = o0 + (long long)(in ? base + u : 0) * so;
      xq[u] = in ? a.gdq[o] : 0.f;
      xk[u] = in ? a.gdk[o] : 0.f;
      xv[u] = in ? a.gdv[o] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kFinSpans; ++u) {
      if (base + u < nspv) {
        sq += xq[u];
        sk += xk[u];
        sv += xv[u];
      }
    }
  }
  const long long ld = (long long)H * kHeadDim;
  const long long at = (long long)b * n * ld + (long long)p * ld + (long long)h * kHeadDim + c;
  a.dq[at] = (__bf16)sq;
  a.dk[at] = (__bf16)sk;
  a.dv[at] = (__bf16)sv;
}

}  // namespace

hipError_t launch_soft_mask(const SoftArgs& a, hipStream_t s) {
  const long long rows = (long long)a.B * a.n;
  hipLaunchKernelGGL(k_soft_mask, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_soft_backward(const SoftArgs& a, hipStream_t s) {
  const long long rows = (long long)a.B * a.n;
  const int bh = a.B * a.H, nb = (a.n + 63) / 64;
  const size_t bits = sizeof(uint32_t) * (((size_t)a.n + 31) / 32);
  const int nglob = bh * (a.Gp / 64) * a.nsp;  // 0 without global tokens
  BwdGrid gd;
  gd.gr = (nglob + 7) & ~7;
  gd.gc = gd.gr;
  gd.band = ((bh * nb) + 7) & ~7;
  hipLaunchKernelGGL(k_soft_rows, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_bwd_dpass, dim3((unsigned)(gd.gr + bh * nb)), dim3(256), bits, s, a, gd);
  if (a.G > 0) hipLaunchKernelGGL(k_bwd_dfin, dim3((unsigned)bh), dim3(64), 0, s, a);
  hipLaunchKernelGGL(k_bwd_grad, dim3((unsigned)(gd.gc + gd.gr + gd.band + bh * nb)), dim3(256), bits, s, a, gd);
  const long long nel = (a.G > 0 && a.gpos) ? (long long)bh * a.G * kHeadDim : 0;
  const int nfin = (int)((nel + 255) / 256);
  hipLaunchKernelGGL(k_bwd_finish, dim3((unsigned)(nfin + 1)), dim3(256), 0, s, a, nfin);
  return hipGetLastError();
}

}  // namespace sc
