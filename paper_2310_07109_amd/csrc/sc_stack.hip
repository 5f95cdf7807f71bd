// Projections and normalisation of the attention-only encoder stack
// (SparseCoder, arXiv 2310.07109, Sec. 4.2 / Fig. 5: the encoder layer around
// the sparse attention; RoBERTa shapes).
//
// k_gemm_bf16   Y[rows, N] = X[rows, K] . W[K, N], bf16 operands, fp32
//               accumulation on v_mfma_f32_16x16x32_bf16.  Workgroup tile
//               128 x 128, 4 waves of 64 x 64, K step 32.  W is row-major
//               [K, N] (as stored by the caller), so its tile is transposed
//               while it is written to LDS to give each lane 8 consecutive k.
//               Rows of sequence b at or beyond len[b] are skipped: the GEMM
//               runs on the surviving tokens only.  Epilogue: bf16 store,
//               fp32 store, or GELU (exact form, x * Phi(x)) then bf16 store
//               for the first feed-forward product.
// k_gemm_v2     the same product when K % 32 == 0 and N % 128 == 0 (the
//               encoder's shapes): 128 x 128 workgroup tile, K stages of 32
//               brought into LDS by gfx950's direct global->LDS loads, three
//               stage buffers with two stages in flight (48 KB, so three
//               workgroups share a CU).  X rows are stored as 64-byte rows
//               whose 16-byte units are XOR-swizzled by bits 2-3 of the row
//               and read as 16-byte A fragments; W stays row-major ([k][n], 256-byte rows,
//               units swizzled by twice the row's low 3 bits) and the B
//               fragments (8 consecutive k of one column) come from transposing
//               LDS reads (ds_read_b64_tr_b16).  Those reads hand each lane the
//               rows 4g..4g+3 and 16+4g..16+4g+3 of a 32-row chunk, so W's rows
//               are loaded into that order and the lane receives k = 8g..8g+7.
//               All N tiles of one M tile run on one XCD (X is fetched once);
//               M tile t of sequence b goes to XCD (t + b) mod 8, so that the
//               first tiles of the sequences (often the only live ones after
//               pruning) spread over the XCDs.
//               Split reduction for small float32 products: when the
//               surviving rows fill few tiles (after pruning, often one per
//               sequence), S blocks per output tile each take K / S of the
//               reduction and write float32 partial sums into slabs; the
//               residual LayerNorm adds the slabs in the fixed order
//               s = 0 .. S-1.  Both kernels derive S from the lengths, so the
//               host needs no synchronisation.
// k_residual_ln y = bf16(LayerNorm(x + t)), one wavefront per row, fp32
//               statistics (biased variance), gamma = 1, beta = 0.
#include <algorithm>

#include "sc_device.h"
#include "sc_internal.h"

namespace sc {
namespace {

constexpr int kBM = 128, kBN = 128, kBKg = 32;
constexpr int kGPitch = kBKg + 8;  // 80-byte rows: 16 consecutive rows hit distinct banks

SC_DEV float gelu_exact(float v) { return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f)); }

__global__ __launch_bounds__(256) void k_gemm_bf16(const __bf16* __restrict__ X, const __bf16* __restrict__ W,
                                                   void* __restrict__ Y, int mode, int n, int K, int N,
                                                   const int* __restrict__ len) {
  __shared__ __attribute__((aligned(16))) __bf16 sX[kBM * kGPitch];
  __shared__ __attribute__((aligned(16))) __bf16 sW[kBN * kGPitch];  // transposed: [col][k]
  const int b = blockIdx.z;
  const int m0 = blockIdx.y * kBM, n0 = blockIdx.x * kBN;
  const int rows = len ? clampi(len[b], 0, n) : n;
  if (m0 >= rows) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, lr = lane & 15;
  const int wm = (w >> 1) * 64, wn = (w & 1) * 64;
  const __bf16* Xb = X + (long long)b * n * K;
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < K; k0 += kBKg) {
    __syncthreads();
    // X tile: 128 rows x 4 chunks of 8
#pragma unroll
    for (int c = tid; c < kBM * 4; c += 256) {
      const int row = c >> 2, part = c & 3;
      const int m = m0 + row;
      __bf16* d = sX + row * kGPitch + 8 * part;
      if (m < rows && k0 + 8 * part < K)
        copy16(d, Xb + (long long)m * K + k0 + 8 * part);
      else
        zero16(d);
    }
    // W tile: 32 k-rows x 128 cols, two k-rows per thread, transposed
    {
      const int kp = tid >> 4, part = tid & 15;
      const int kk = k0 + 2 * kp, col = n0 + 8 * part;
      uint4 a = make_uint4(0, 0, 0, 0), c = make_uint4(0, 0, 0, 0);
      if (col < N) {
        if (kk < K) a = *reinterpret_cast<const uint4*>(W + (long long)kk * N + col);
        if (kk + 1 < K) c = *reinterpret_cast<const uint4*>(W + (long long)(kk + 1) * N + col);
      }
      const uint32_t av[4] = {a.x, a.y, a.z, a.w}, cv[4] = {c.x, c.y, c.z, c.w};
      uint32_t* base = reinterpret_cast<uint32_t*>(sW);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t lo = (av[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
        const uint32_t hi = (cv[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
        base[((8 * part + j) * kGPitch + 2 * kp) >> 1] = lo | (hi << 16);
      }
    }
    __syncthreads();
    bf16x8 af[4], bfr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const bf16x8*>(sX + (wm + 16 * i + lr) * kGPitch + 8 * g);
#pragma unroll
    for (int j = 0; j < 4; ++j) bfr[j] = *reinterpret_cast<const bf16x8*>(sW + (wn + 16 * j + lr) * kGPitch + 8 * g);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
  }
  // result (row wm + 16i + 4g + e, col wn + 16j + lr)
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = m0 + wm + 16 * i + 4 * g + e;
      if (m >= rows) continue;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int col = n0 + wn + 16 * j + lr;
        if (col >= N) continue;
        const long long off = ((long long)b * n + m) * N + col;
        if (mode == kGemmF32)
          static_cast<float*>(Y)[off] = acc[i][j][e];
        else if (mode == kGemmGeluBf16)
          static_cast<__bf16*>(Y)[off] = (__bf16)gelu_exact(acc[i][j][e]);
        else
          static_cast<__bf16*>(Y)[off] = (__bf16)acc[i][j][e];
      }
    }
}

// k per stage of k_gemm_v2 and stage buffers (kNBuf - 1 stages in flight).
// 32 x 3 (48 KB of LDS, three workgroups per CU) measured faster than 64 x 2
// (64 KB, two per CU), 32 x 4 (two per CU, three stages in flight) and
// 64 x 3 (one per CU): workgroups per CU matter more than prefetch depth.
constexpr int kGK = 32;
constexpr int kNBuf = 3;
constexpr int kXUnits = kGK / 8;     // 16-byte units per X row
constexpr int kDmaPerStage = kGK / 8;  // direct loads per thread and stage (X and W)

struct GemmSmem {
  __attribute__((aligned(16))) __bf16 x[kNBuf][kBM * kGK];  // [row][k], 2 kGK-byte rows
  __attribute__((aligned(16))) __bf16 w[kNBuf][kGK * kBN];  // [k][n], 256-byte rows
};

// X rows of 8 units (64 k) swizzle by the row's low 3 bits; rows of 4 units
// (32 k) by bits 2-3, so that 16 consecutive rows read at one unit hit 16
// distinct 16-byte bank groups
SC_DEV int gx_off(int row, int unit) {
  return row * kGK + 8 * (unit ^ (kXUnits == 8 ? (row & 7) : ((row >> 2) & 3)));
}
// s_waitcnt vmcnt(n) alone (expcnt and lgkmcnt at their no-wait maxima)
template <int N>
SC_DEV void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
SC_DEV int gw_off(int row, int unit) { return row * kBN + 8 * (unit ^ (2 * (row & 7))); }
// W row held by LDS row r of a stage: within each 32-row chunk, LDS row
// 4g + t holds k = 8g + t and LDS row 16 + 4g + t holds k = 8g + 4 + t.
SC_DEV int gw_krow(int r) { return (r & ~31) + 8 * ((r & 15) >> 2) + 4 * ((r >> 4) & 1) + (r & 3); }

// Split of the reduction (see the header): tiles = 128-row tiles of the
// surviving rows (per sequence), S = number of K ranges.  S doubles while
// the partial sums stay within kGemmSplitRows rows, the launch within
// kSplitBlocks workgroups, and every range keeps at least 3 stages.  One
// wave computes it with lane b reading len[b] (B <= kSplitMaxB, else no
// split); excl = live tiles of the sequences before the lane's, incl = excl
// plus the lane's own.
constexpr int kSplitMaxB = 64, kSplitMax = 8, kSplitBlocks = 1024;
struct SplitPlan {
  int tiles, S;
};
SC_DEV SplitPlan split_plan(const int* len, int B, int n, int Nt, int nk, int& excl, int& incl) {
  const int lane = threadIdx.x & 63;
  const bool ok = len && B <= kSplitMaxB;
  const int c = ok && lane < B ? (clampi(len[lane], 0, n) + kBM - 1) / kBM : 0;
  incl = c;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(incl, d, 64);
    if (lane >= d) incl += y;
  }
  excl = incl - c;
  SplitPlan p{__builtin_amdgcn_readlane(incl, 63), 1};
  if (!ok) return p;
  while (2 * p.S <= kSplitMax && p.tiles * 2 * p.S * kBM <= kGemmSplitRows &&
         p.tiles * Nt * 2 * p.S <= kSplitBlocks && nk % (2 * p.S) == 0 && nk / (2 * p.S) >= 3)
    p.S *= 2;
  return p;
}

SC_DEV void gemm_store(void* Y, int mode, long long off, float v) {
  if (mode == kGemmF32)
    static_cast<float*>(Y)[off] = v;
  else if (mode == kGemmGeluBf16)
    static_cast<__bf16*>(Y)[off] = (__bf16)gelu_exact(v);
  else
    static_cast<__bf16*>(Y)[off] = (__bf16)v;
}

// part: float32 slabs of the split reduction (NULL: no split; mode must be
// kGemmF32 otherwise).
__global__ __launch_bounds__(256) void k_gemm_v2(const __bf16* __restrict__ X, const __bf16* __restrict__ W,
                                                 void* __restrict__ Y, int mode, int B, int n, int K, int N,
                                                 const int* __restrict__ len, float* __restrict__ part) {
  __shared__ GemmSmem sm;
  const int Nt = N / kBN, Mt = (n + kBM - 1) / kBM, nk = K / kGK;
  int excl = 0, incl = 0;
  const SplitPlan sp = part ? split_plan(len, B, n, Nt, nk, excl, incl) : SplitPlan{0, 1};
  int b = -1, t = 0, nt = 0, ks = 0, tile = 0;
  if (sp.S > 1) {
    // block i: K range i % S of output tile (i / S) % Nt of the (i / S / Nt)-th live M tile
    int item = blockIdx.x;
    if (item >= sp.tiles * Nt * sp.S) return;
    ks = item % sp.S;
    item /= sp.S;
    nt = item % Nt;
    tile = item / Nt;
    const unsigned long long owner = __ballot(incl > tile);  // lanes of the sequence holding the tile and after
    b = __builtin_ctzll(owner);
    t = tile - __shfl(excl, b, 64);
  } else {
    // block i runs on XCD i % 8 and takes the (i / 8 / Nt)-th M tile of that
    // XCD (tiles t = (x - b) mod 8, +8, ... of sequences b = 0, 1, ...) with
    // N tile (i / 8) % Nt
    const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3;
    const int jm = j / Nt;
    nt = j % Nt;
    for (int bb = 0, acc = 0; bb < B; ++bb) {
      const int t0 = (xcd - bb) & 7;
      const int cnt = t0 < Mt ? (Mt - t0 + 7) / 8 : 0;
      if (jm < acc + cnt) {
        b = bb;
        t = t0 + 8 * (jm - acc);
        break;
      }
      acc += cnt;
    }
  }
  if (b < 0) return;
  const int m0 = t * kBM, n0 = nt * kBN;
  const int rows = len ? clampi(len[b], 0, n) : n;
  if (m0 >= rows) return;
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6), g = lane >> 4,
            lr = lane & 15;
  const int wm = (w >> 1) * 64, wn = (w & 1) * 64;
  const __bf16* Xb = X + (long long)b * n * K;
  const unsigned xrow_b = 2u * (unsigned)K, wrow_b = 2u * (unsigned)N;  // byte offsets fit in 32 bits (host)
  auto issue = [&](int k0, int bf) {
    const int ln = opaque_lane();
    constexpr int kXRows = 64 / kXUnits;  // X rows per load (1 KB)
#pragma unroll
    for (int t = 0; t < 32 / kXRows; ++t) {  // X: wave w fills rows 32w .. 32w+31
      const int R0 = 32 * w + kXRows * t, R = R0 + ln / kXUnits;
      const int u = (ln % kXUnits) ^ (kXUnits == 8 ? (R & 7) : ((R >> 2) & 3));
      const int gr = min(m0 + R, rows - 1);
      lds_dma16(Xb, (unsigned)gr * xrow_b + 2u * (unsigned)(k0 + 8 * u), lds_addr(sm.x[bf] + R0 * kGK));
    }
#pragma unroll
    for (int t = 0; t < kGK / 16; ++t) {  // W: wave w fills rows kGK/4 w .., 4 rows per load
      const int R0 = (kGK / 4) * w + 4 * t, R = R0 + (ln >> 4);
      const int u = (ln & 15) ^ (2 * (R & 7));
      lds_dma16(W, (unsigned)(k0 + gw_krow(R)) * wrow_b + 2u * (unsigned)(n0 + 8 * u), lds_addr(sm.w[bf] + R0 * kBN));
    }
  };
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) acc[i][jn] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int per = nk / sp.S, s0 = ks * per, s1 = s0 + per;  // this block's stages
  // stages s0 .. s0 + kNBuf - 2 in flight; stage s + kNBuf - 1 is issued into
  // the buffer read in stage s - 1 once the barrier of stage s has passed
#pragma unroll
  for (int p = 0; p < kNBuf - 1; ++p)
    if (s0 + p < s1) issue((s0 + p) * kGK, p);
  for (int s = s0; s < s1; ++s) {
    const int later = min(s1 - 1 - s, kNBuf - 2);  // stages issued after s, still in flight
    if constexpr (kNBuf >= 4) {
      if (later >= 2) wait_vm<2 * kDmaPerStage>();
      else if (later == 1) wait_vm<kDmaPerStage>();
      else wait_vm<0>();
    } else if constexpr (kNBuf == 3) {
      if (later >= 1) wait_vm<kDmaPerStage>();
      else wait_vm<0>();
    } else {
      wait_vm<0>();
    }
    __syncthreads();
    if (s + kNBuf - 1 < s1) issue((s + kNBuf - 1) * kGK, (s - s0 + kNBuf - 1) % kNBuf);
    const int bf = (s - s0) % kNBuf;
    const __bf16* sx = sm.x[bf];
    const __bf16* sw = sm.w[bf];
#pragma unroll
    for (int kc = 0; kc < kGK / 32; ++kc) {
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const bf16x8*>(sx + gx_off(wm + 16 * i + lr, 4 * kc + g));
      const int vr = 32 * kc + 4 * g + (lr >> 2), bsel = (lr >> 1) & 1, e = 4 * (lr & 1);
#pragma unroll
      for (int jn = 0; jn < 4; ++jn) {
        const int U = 2 * ((wn >> 4) + jn) + bsel;
        const i16x4 a0 = lds_read_tr16(sw + gw_off(vr, U) + e);
        const i16x4 a1 = lds_read_tr16(sw + gw_off(vr + 16, U) + e);
        bfr[jn] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int jn = 0; jn < 4; ++jn)
          acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[jn], acc[i][jn], 0, 0, 0);
    }
  }
  // result (row wm + 16i + 4g + e, col wn + 16jn + lr); split: partial ks of
  // element (128 tile + m - m0, col) at part[(128 (ks tiles + tile) + m - m0) N + col]
  if (sp.S > 1) {
    float* slab = part + ((long long)(ks * sp.tiles + tile) * kBM - m0) * N;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + wm + 16 * i + 4 * g + e;
        if (m >= rows) continue;
#pragma unroll
        for (int jn = 0; jn < 4; ++jn) slab[(long long)m * N + n0 + wn + 16 * jn + lr] = acc[i][jn][e];
      }
    return;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = m0 + wm + 16 * i + 4 * g + e;
      if (m >= rows) continue;
#pragma unroll
      for (int jn = 0; jn < 4; ++jn)
        gemm_store(Y, mode, ((long long)b * n + m) * N + n0 + wn + 16 * jn + lr, acc[i][jn][e]);
    }
}

// v[4u + q] = x[c + q] + t[c + q] for the columns c = 4 lane + 256 u .. +3
// (D a multiple of 64), t being the sum of S partial sums that lie `stride`
// floats apart, added in the order s = 0 .. S-1; 16-byte loads of t.
template <int S, int kPer>
SC_DEV void ln_load(float (&v)[kPer], const __bf16* xp, const float* tp, long long stride, int D, int lane) {
#pragma unroll
  for (int u = 0; u < kPer / 4; ++u) {
    const int c = 4 * lane + 256 * u;
    if (c < D) {
      float4 a = *reinterpret_cast<const float4*>(tp + c);
#pragma unroll
      for (int k = 1; k < S; ++k) {
        const float4 e = *reinterpret_cast<const float4*>(tp + k * stride + c);
        a.x += e.x;
        a.y += e.y;
        a.z += e.z;
        a.w += e.w;
      }
      const bf16x4 xv = *reinterpret_cast<const bf16x4*>(xp + c);
      v[4 * u] = a.x + (float)xv[0];
      v[4 * u + 1] = a.y + (float)xv[1];
      v[4 * u + 2] = a.z + (float)xv[2];
      v[4 * u + 3] = a.w + (float)xv[3];
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) v[4 * u + q] = 0.f;
    }
  }
}

// part, K: the partial sums and reduction length of the product that wrote
// t, when it may have split its reduction (t itself is then unused).
// kMaxPer = elements per lane (D <= 64 kMaxPer).  Occupancy bound: 6 waves
// per SIMD at 16 elements per lane (80 VGPRs, which the unsplit rows need
// for latency hiding; the split path's wide loads are then issued in a few
// rounds), 4 at 32.
template <int kMaxPer>
__global__ __launch_bounds__(256, kMaxPer <= 16 ? 6 : 4) void k_residual_ln(const __bf16* __restrict__ xr, const float* __restrict__ t,
                                                     __bf16* __restrict__ y, int B, int n, int D, float eps,
                                                     const int* __restrict__ len, const float* __restrict__ part,
                                                     int K) {
  const long long row = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= (long long)B * n) return;
  const int b = (int)(row / n), j = (int)(row % n);
  if (j >= clampi(len[b], 0, n)) return;
  const __bf16* xp = xr + row * D;
  __bf16* yp = y + row * D;
  float v[kMaxPer];
  // loaded as written by an unsplit product before the plan is known (replaced after a split)
  ln_load<1, kMaxPer>(v, xp, t + row * D, 0, D, lane);
  int excl = 0, incl = 0;
  const SplitPlan sp = part ? split_plan(len, B, n, D / kBN, K / kGK, excl, incl) : SplitPlan{0, 1};
  if (sp.S > 1) {  // the row's place: its tile among the live tiles, then its row in the tile
    const int tile = j / kBM + __shfl(excl, b, 64);
    const float* tp = part + ((long long)tile * kBM + j % kBM) * D;
    const long long stride = (long long)sp.tiles * kBM * D;  // between the partial sums
    if (sp.S == 2)
      ln_load<2, kMaxPer>(v, xp, tp, stride, D, lane);
    else if (sp.S == 4)
      ln_load<4, kMaxPer>(v, xp, tp, stride, D, lane);
    else
      ln_load<8, kMaxPer>(v, xp, tp, stride, D, lane);
  }
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) s += v[u];
  for (int m = 1; m < 64; m <<= 1) s += __shfl_xor(s, m, 64);
  const float mean = s / (float)D;
  float q = 0.f;
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int c = 4 * lane + 256 * (u / 4);
    const float dv = c < D ? v[u] - mean : 0.f;
    q += dv * dv;
  }
  for (int m = 1; m < 64; m <<= 1) q += __shfl_xor(q, m, 64);
  const float inv = 1.0f / sqrtf(q / (float)D + eps);
#pragma unroll
  for (int u = 0; u < kMaxPer / 4; ++u) {
    const int c = 4 * lane + 256 * u;
    if (c < D) {
      bf16x4 o;
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) o[q4] = (__bf16)((v[4 * u + q4] - mean) * inv);
      *reinterpret_cast<bf16x4*>(yp + c) = o;
    }
  }
}

}  // namespace

namespace {
bool gemm_v2_ok(int n, int K, int N) {
  return K % kGK == 0 && N % kBN == 0 && K > 0 && N > 0 && (long long)n * K * 2 < (1LL << 32) &&
         (long long)K * N * 2 < (1LL << 32);
}
}  // namespace

hipError_t launch_gemm_bf16(const void* x, const void* w, void* y, int mode, int B, int n, int K, int N,
                            const int* len, float* part, hipStream_t s) {
  if (gemm_v2_ok(n, K, N)) {
    // per XCD at most B * ceil(Mt / 8) M tiles; a split launch needs at most kSplitBlocks
    const long long per_xcd = (long long)B * (((n + kBM - 1) / kBM + 7) / 8);
    long long blocks = 8 * (long long)(N / kBN) * per_xcd;
    if (part && mode == kGemmF32 && len) blocks = std::max<long long>(blocks, kSplitBlocks);
    else part = nullptr;
    hipLaunchKernelGGL(k_gemm_v2, dim3((unsigned)blocks), dim3(256), 0, s, static_cast<const __bf16*>(x),
                       static_cast<const __bf16*>(w), y, mode, B, n, K, N, len, part);
    return hipGetLastError();
  }
  dim3 grid((N + kBN - 1) / kBN, (n + kBM - 1) / kBM, B);
  hipLaunchKernelGGL(k_gemm_bf16, grid, dim3(256), 0, s, static_cast<const __bf16*>(x),
                     static_cast<const __bf16*>(w), y, mode, n, K, N, len);
  return hipGetLastError();
}

hipError_t launch_residual_layernorm(const void* x_res, const float* t, void* y, int B, int n, int D, float eps,
                                     const int* len, const float* part, int K, hipStream_t s) {
  const long long rows = (long long)B * n;
  if (!gemm_v2_ok(n, K, D)) part = nullptr;  // the product took the path without a split
  auto* kern = D <= 1024 ? k_residual_ln<16> : k_residual_ln<32>;  // D <= 2048 (checked by the caller)
  hipLaunchKernelGGL(kern, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, static_cast<const __bf16*>(x_res), t,
                     static_cast<__bf16*>(y), B, n, D, eps, len, part, K);
  return hipGetLastError();
}

}  // namespace sc
