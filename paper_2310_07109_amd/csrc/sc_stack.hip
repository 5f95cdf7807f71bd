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
//               fp32 store, or GELU (x * Phi(x), erf by Abramowitz & Stegun 7.1.26) then bf16 store
//               for the first feed-forward product.
// k_gemm_v3     the same product when K % 32 == 0 and N % 128 == 0 (the
//               encoder's shapes), on packed rows: the surviving rows of all
//               sequences are numbered in order on the device (prefix sum of
//               the lengths) and cut into shared tiles, so that the product
//               runs on ceil(R / BM) tiles of the R surviving rows instead of
//               one partly empty tile per sequence.  Tiles of 256 x 128 rows x
//               columns once R >= 8192 (4 waves of 128 x 64, two stage
//               buffers), else 128 x 128 (4 waves of 64 x 64, three buffers):
//               48 KB either way, three workgroups per CU.  K stages of 32
//               arrive by gfx950's direct global->LDS loads.  X rows are stored
//               as 64-byte rows whose 16-byte units are XOR-swizzled by bits 2-3
//               of the row and read as 16-byte A fragments; W stays row-major
//               ([k][n], 256-byte rows, units swizzled by twice the row's low
//               3 bits) and the B fragments (8 consecutive k of one column) come
//               from transposing LDS reads (ds_read_b64_tr_b16).  Those reads
//               hand each lane the rows 4g..4g+3 and 16+4g..16+4g+3 of a 32-row
//               chunk, so W's rows are loaded into that order and the lane
//               receives k = 8g..8g+7.  Items (tile, N tile, K range) go to the
//               XCDs in contiguous ranges.
//               Split reduction for small float32 products: when the packed
//               rows fill few tiles (after pruning), S blocks per output tile
//               each take K / S of the reduction and write float32 partial
//               sums into slabs; the residual LayerNorm adds the slabs in the
//               fixed order s = 0 .. S-1.  Both kernels derive the packing and
//               S from the lengths, so the host needs no synchronisation.
// k_residual_ln y = bf16(LayerNorm(x + t)), one wavefront per packed row, fp32
//               statistics (biased variance), gamma = 1, beta = 0.
#include <algorithm>

#include "sc_device.h"
#include "sc_internal.h"

namespace sc {
namespace {

constexpr int kBM = 128, kBN = 128, kBKg = 32;
constexpr int kGPitch = kBKg + 8;  // 80-byte rows: 16 consecutive rows hit distinct banks

// GELU, x Phi(x) = x (1 + erf(x / sqrt 2)) / 2, with erfc(z) for z = |x| / sqrt 2
// from Abramowitz & Stegun, Handbook of Mathematical Functions, eq. 7.1.26
// (erfc(z) = (a1 t + ... + a5 t^5) exp(-z^2), t = 1 / (1 + p z), absolute
// error <= 1.5e-7): for x >= 0 the result is x (1 - erfc / 2), for x < 0
// x erfc / 2.  Evaluated in float32 it stays within 6e-7 of the exact GELU
// (1.7e-4 relative where |GELU| >= 1e-3), far inside the bf16 rounding of the
// stored activation; one reciprocal, one exponential and five FMAs instead
// of the library erff.
SC_DEV float gelu_exact(float v) {
  const float z = fabsf(v) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, z, 1.0f));
  const float poly =
      t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f), -0.284496736f), 0.254829592f);
  const float ec = poly * fast_exp2(-z * z * kLog2e);
  return v >= 0.f ? v * fmaf(-0.5f, ec, 1.0f) : 0.5f * v * ec;
}

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

// ---------------------------------------------------------------------------
// Packed rows.  The surviving rows of all sequences are numbered in sequence
// order (packed row p of sequence b is its row p - pre[b], pre = exclusive
// prefix sum of the lengths), so that the products run on ceil(R / BM) tiles
// of R = sum of the lengths rows instead of one partly empty tile per
// sequence and 128 rows.  Every workgroup derives the numbering from the
// lengths itself: the host never learns them.

// Wave 0 writes pre[0 .. B] (pre[B] = R); lengths clamped to [0, n], all n
// without lengths.
SC_DEV void pack_prefix(int* pre, const int* len, int B, int n) {
  if (threadIdx.x >= 64) return;
  const int lane = threadIdx.x;
  int carry = 0;
  for (int c = 0; c < B; c += 64) {
    const int b = c + lane;
    const int v = b < B ? (len ? clampi(len[b], 0, n) : n) : 0;
    int incl = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int y = __shfl_up(incl, d, 64);
      if (lane >= d) incl += y;
    }
    if (b < B) pre[b] = carry + incl - v;
    carry += __shfl(incl, 63, 64);
  }
  if (lane == 0) pre[B] = carry;
}

// The sequence holding packed row p < pre[B]: the largest b with pre[b] <= p
// (empty sequences share their start with the next one).
SC_DEV int pack_seq(const int* pre, int B, int p) {
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pre[mid] <= p) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Tiles of the packed product.  R rows in tiles of bm rows: 256 once the
// rows fill at least kBigRows (the taller tile's lower traffic per flop
// pays); 64 when the 64-row tiles of an unsplit product still fit one round
// of kOneRound workgroups (few rows: more, smaller tiles keep more CUs busy,
// and each CU pulls (64 + 128) / (128 + 128) of the bytes); 128 otherwise.
// Split reduction (float32 outputs with slabs only, 128-row tiles): S
// blocks per output tile each take K / S of the reduction; S doubles while
// the partial sums stay within kGemmSplitRows rows, the launch within
// kSplitBlocks workgroups and every range keeps at least 3 stages.  The
// product and the residual LayerNorm that adds its slabs compute the same
// plan from the same lengths.
constexpr int kBigRows = 8192, kOneRound = 256, kSplitMax = 8, kSplitBlocks = 1024;
struct GemmPlan {
  int bm, T, S;
};
SC_DEV GemmPlan gemm_plan(int R, int Nt, int nk, bool split) {
  GemmPlan p;
  p.S = 1;
  if (R >= kBigRows) {
    p.bm = 256;
    p.T = (R + 255) / 256;
    return p;
  }
  if (!split && (R + 63) / 64 * Nt <= kOneRound) {
    p.bm = 64;
    p.T = (R + 63) / 64;
    return p;
  }
  p.bm = 128;
  p.T = (R + 127) / 128;
  if (split)
    while (2 * p.S <= kSplitMax && p.T * 2 * p.S * 128 <= kGemmSplitRows && p.T * Nt * 2 * p.S <= kSplitBlocks &&
           nk % (2 * p.S) == 0 && nk / (2 * p.S) >= 3)
      p.S *= 2;
  return p;
}

// k per stage; W tile 32 x 128 per stage.
constexpr int kGK = 32;
constexpr int kXUnits = kGK / 8;  // 16-byte units per X row
constexpr int kStageBytes = 49152;  // stage buffers: 4 x (64 + 128), 3 x (128 + 128) or 2 x (256 + 128) x 32 bf16

// X rows of 4 units (32 k) swizzle by bits 2-3 of the row, so that 16
// consecutive rows read at one unit hit 16 distinct 16-byte bank groups
SC_DEV int gx_off(int row, int unit) { return row * kGK + 8 * (unit ^ ((row >> 2) & 3)); }
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

template <int kMode>
SC_DEV void gemm_store(void* Y, long long off, float v) {
  if constexpr (kMode == kGemmF32)
    static_cast<float*>(Y)[off] = v;
  else if constexpr (kMode == kGemmGeluBf16)
    static_cast<__bf16*>(Y)[off] = (__bf16)gelu_exact(v);
  else
    static_cast<__bf16*>(Y)[off] = (__bf16)v;
}

// One output tile of BM x 128 (4 waves of BM/2 x 64, BM = 64, 128, 256) over this block's
// stages s0 .. s1-1, kNBuf stage buffers with kNBuf - 1 stages in flight;
// grow[r] = global row of tile row r (-1: past the packed rows).  slab: the
// split's partial sums of this tile (row r at slab + r N), else NULL.
template <int BM, int kNBuf, int kMode>
SC_DEV void gemm_tile(const __bf16* __restrict__ X, const __bf16* __restrict__ W, void* __restrict__ Y,
                      char* stage, const int* grow, int K, int N, int n0, int s0, int s1, float* slab) {
  constexpr int FI = BM / 32;        // 16-row fragments per wave (wave tile BM/2 x 64)
  constexpr int XL = BM / 64;        // X loads per wave and stage (16 rows each)
  constexpr int kDmaPerStage = XL + 2;
  constexpr int kXBytes = BM * kGK * 2, kWBytes = kGK * kBN * 2;
  static_assert(kNBuf * (kXBytes + kWBytes) <= kStageBytes, "stage buffers");
  __bf16* sxb = reinterpret_cast<__bf16*>(stage);
  __bf16* swb = reinterpret_cast<__bf16*>(stage + kNBuf * kXBytes);
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6), g = lane >> 4,
            lr = lane & 15;
  const int wm = (w >> 1) * (BM / 2), wn = (w & 1) * 64;
  const unsigned xrow_b = 2u * (unsigned)K, wrow_b = 2u * (unsigned)N;  // byte offsets fit in 32 bits (host)
  // this lane's X rows (global, rows past the packed ones re-read the tile's first row)
  unsigned xoff[XL];
#pragma unroll
  for (int t = 0; t < XL; ++t) {
    const int R = (BM / 4) * w + 16 * t + lane / kXUnits;
    const int gr = grow[R];
    xoff[t] = (unsigned)(gr >= 0 ? gr : grow[0]) * xrow_b;
  }
  auto issue = [&](int k0, int bf) {
    const int ln = opaque_lane();
#pragma unroll
    for (int t = 0; t < XL; ++t) {  // X: wave w fills rows BM/4 w .. , 16 rows per load
      const int R0 = (BM / 4) * w + 16 * t, R = R0 + ln / kXUnits;
      const int u = (ln % kXUnits) ^ ((R >> 2) & 3);
      lds_dma16(X, xoff[t] + 2u * (unsigned)(k0 + 8 * u), lds_addr(sxb + (bf * BM + R0) * kGK));
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {  // W: wave w fills rows 8w .., 4 rows per load
      const int R0 = 8 * w + 4 * t, R = R0 + (ln >> 4);
      const int u = (ln & 15) ^ (2 * (R & 7));
      lds_dma16(W, (unsigned)(k0 + gw_krow(R)) * wrow_b + 2u * (unsigned)(n0 + 8 * u),
                lds_addr(swb + (bf * kGK + R0) * kBN));
    }
  };
  f32x4 acc[FI][4];
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) acc[i][jn] = f32x4{0.f, 0.f, 0.f, 0.f};
  // stages s0 .. s0 + kNBuf - 2 in flight; stage s + kNBuf - 1 is issued into
  // the buffer read in stage s - 1 once the barrier of stage s has passed
#pragma unroll
  for (int p = 0; p < kNBuf - 1; ++p)
    if (s0 + p < s1) issue((s0 + p) * kGK, p);
  for (int s = s0; s < s1; ++s) {
    const int later = min(s1 - 1 - s, kNBuf - 2);  // stages issued after s, still in flight
    if constexpr (kNBuf == 4) {
      if (later >= 2) wait_vm<2 * kDmaPerStage>();
      else if (later == 1) wait_vm<kDmaPerStage>();
      else wait_vm<0>();
    } else if constexpr (kNBuf == 3) {
      if (later >= 1) wait_vm<kDmaPerStage>();
      else wait_vm<0>();
    } else {
      static_assert(kNBuf == 2, "two to four stage buffers");
      wait_vm<0>();
    }
    __syncthreads();
    if (s + kNBuf - 1 < s1) issue((s + kNBuf - 1) * kGK, (s - s0 + kNBuf - 1) % kNBuf);
    const int bf = (s - s0) % kNBuf;
    const __bf16* sx = sxb + bf * BM * kGK;
    const __bf16* sw = swb + bf * kGK * kBN;
    bf16x8 af[FI], bfr[4];
#pragma unroll
    for (int i = 0; i < FI; ++i) af[i] = *reinterpret_cast<const bf16x8*>(sx + gx_off(wm + 16 * i + lr, g));
    const int vr = 4 * g + (lr >> 2), bsel = (lr >> 1) & 1, e = 4 * (lr & 1);
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) {
      const int U = 2 * ((wn >> 4) + jn) + bsel;
      const i16x4 a0 = lds_read_tr16(sw + gw_off(vr, U) + e);
      const i16x4 a1 = lds_read_tr16(sw + gw_off(vr + 16, U) + e);
      bfr[jn] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
    }
#pragma unroll
    for (int i = 0; i < FI; ++i)
#pragma unroll
      for (int jn = 0; jn < 4; ++jn)
        acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[jn], acc[i][jn], 0, 0, 0);
  }
  // result (tile row wm + 16i + 4g + e, col wn + 16jn + lr)
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = wm + 16 * i + 4 * g + e;
      const int gr = grow[r];
      if (gr < 0) continue;
      const int col = n0 + wn + lr;
      if (slab) {
#pragma unroll
        for (int jn = 0; jn < 4; ++jn) slab[(long long)r * N + col + 16 * jn] = acc[i][jn][e];
      } else {
#pragma unroll
        for (int jn = 0; jn < 4; ++jn) gemm_store<kMode>(Y, (long long)gr * N + col + 16 * jn, acc[i][jn][e]);
      }
    }
}

// Y[row, N] = X[row, K] . W[K, N] over the surviving rows of the B
// sequences (row j of sequence b at b n + j, j < len[b]).  part: float32
// slabs of a split reduction (kGemmF32 only), NULL for none.  Items (packed
// tile t, N tile, K range ks), ks fastest, are dealt to the XCDs in
// contiguous ranges (workgroup i runs on XCD i % 8): an XCD keeps its tiles'
// X rows in its L2 and sweeps the N tiles.
// At most 168 VGPRs: three waves per SIMD, which the three workgroups per
// CU that the stage buffers allow need.
template <int kMode>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void k_gemm_v3(const __bf16* __restrict__ X, const __bf16* __restrict__ W,
                                                 void* __restrict__ Y, int B, int n, int K, int N,
                                                 const int* __restrict__ len, float* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) char stage[kStageBytes];
  __shared__ int grow[256];
  int* pre = reinterpret_cast<int*>(stage);  // until the first stage lands
  pack_prefix(pre, len, B, n);
  __syncthreads();
  const int R = pre[B], Nt = N / kBN, nk = K / kGK;
  const GemmPlan pl = gemm_plan(R, Nt, nk, kMode == kGemmF32 && part != nullptr);
  const long long items = (long long)pl.T * Nt * pl.S;
  const int x = blockIdx.x & 7;
  const long long item = items * x / 8 + (blockIdx.x >> 3);
  if (item >= items * (x + 1) / 8) return;
  const int ks = (int)(item % pl.S), nt = (int)(item / pl.S % Nt), t = (int)(item / pl.S / Nt);
  const int m0 = t * pl.bm;
  if ((int)threadIdx.x < pl.bm) {
    const int p = m0 + threadIdx.x;
    int gr = -1;
    if (p < R) {
      const int b = pack_seq(pre, B, p);
      gr = b * n + (p - pre[b]);
    }
    grow[threadIdx.x] = gr;
  }
  __syncthreads();  // the prefix table is dead from here: the stages overwrite it
  const int per = nk / pl.S, s0 = ks * per, s1 = s0 + per;
  float* slab = pl.S > 1 ? part + ((long long)ks * pl.T * 128 + m0) * N : nullptr;
  if (pl.bm == 256)
    gemm_tile<256, 2, kMode>(X, W, Y, stage, grow, K, N, nt * kBN, s0, s1, nullptr);
  else if (pl.bm == 128)
    gemm_tile<128, 3, kMode>(X, W, Y, stage, grow, K, N, nt * kBN, s0, s1, slab);
  else
    gemm_tile<64, 4, kMode>(X, W, Y, stage, grow, K, N, nt * kBN, s0, s1, nullptr);
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

// One row of the residual LayerNorm: y = bf16(LayerNorm(x + t)) at global
// row `row`, packed index p (where a split product left its partial sums).
template <int kMaxPer>
SC_DEV void ln_row(const __bf16* __restrict__ xr, const float* __restrict__ t, __bf16* __restrict__ y, int D,
                   float eps, const float* __restrict__ part, const GemmPlan& pl, long long row, int p, int lane) {
  const __bf16* xp = xr + row * D;
  __bf16* yp = y + row * D;
  float v[kMaxPer];
  if (pl.S == 1) {
    ln_load<1, kMaxPer>(v, xp, t + row * D, 0, D, lane);
  } else {  // the row's partial sums sit at its packed index in each slab
    const float* tp = part + (long long)p * D;
    const long long stride = (long long)pl.T * 128 * D;
    if (pl.S == 2)
      ln_load<2, kMaxPer>(v, xp, tp, stride, D, lane);
    else if (pl.S == 4)
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
    if (256 * u < D && c < D) {
      bf16x4 o;
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) o[q4] = (__bf16)((v[4 * u + q4] - mean) * inv);
      *reinterpret_cast<bf16x4*>(yp + c) = o;
    }
  }
}

// part, K: the slabs and reduction length of the product that wrote t, when
// it may have split its reduction (t itself is then unused).  One wavefront
// per packed row, rows dealt round-robin over the launch's waves.  kMaxPer =
// elements per lane (D <= 64 kMaxPer).  pre: dynamic LDS of B + 1 ints.
template <int kMaxPer>
__global__ __launch_bounds__(256) void k_residual_ln(const __bf16* __restrict__ xr, const float* __restrict__ t,
                                                     __bf16* __restrict__ y, int B, int n, int D, float eps,
                                                     const int* __restrict__ len, const float* __restrict__ part,
                                                     int K) {
  extern __shared__ int pre[];
  pack_prefix(pre, len, B, n);
  __syncthreads();
  const int R = pre[B];
  const int lane = threadIdx.x & 63;
  const GemmPlan pl = gemm_plan(R, D / kBN, K / kGK, part != nullptr);
  for (int p = blockIdx.x * 4 + (threadIdx.x >> 6); p < R; p += gridDim.x * 4) {
    const int b = pack_seq(pre, B, p);
    ln_row<kMaxPer>(xr, t, y, D, eps, part, pl, (long long)b * n + (p - pre[b]), p, lane);
  }
}

}  // namespace

namespace {
// Shapes of the packed product: K and N whole stages and tiles, 32-bit byte
// offsets over all B n rows of X and over W, the prefix table in the stage
// buffers.
bool gemm_v3_ok(int B, int n, int K, int N) {
  return K % kGK == 0 && N % kBN == 0 && K > 0 && N > 0 && B <= kPackMaxB &&
         (long long)B * n * K * 2 < (1LL << 32) && (long long)K * N * 2 < (1LL << 32);
}
}  // namespace

hipError_t launch_gemm_bf16(const void* x, const void* w, void* y, int mode, int B, int n, int K, int N,
                            const int* len, float* part, hipStream_t s) {
  if (gemm_v3_ok(B, n, K, N)) {
    // items: at most ceil(B n / 128) 128-row tiles x N tiles, kSplitBlocks for
    // a split, kOneRound for 64-row tiles
    const long long tiles = ((long long)B * n + 127) / 128 * (N / kBN);
    if (!(part && mode == kGemmF32)) part = nullptr;
    const long long items = std::max<long long>(tiles, part ? kSplitBlocks : kOneRound);
    const dim3 grid((unsigned)(8 * ((items + 7) / 8))), block(256);
    const __bf16* xb = static_cast<const __bf16*>(x);
    const __bf16* wb = static_cast<const __bf16*>(w);
    if (mode == kGemmF32)
      hipLaunchKernelGGL(k_gemm_v3<kGemmF32>, grid, block, 0, s, xb, wb, y, B, n, K, N, len, part);
    else if (mode == kGemmGeluBf16)
      hipLaunchKernelGGL(k_gemm_v3<kGemmGeluBf16>, grid, block, 0, s, xb, wb, y, B, n, K, N, len, nullptr);
    else
      hipLaunchKernelGGL(k_gemm_v3<kGemmBf16>, grid, block, 0, s, xb, wb, y, B, n, K, N, len, nullptr);
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
  if (!gemm_v3_ok(B, n, K, D)) part = nullptr;  // the product took the path without a split
  auto* kern = D <= 1024 ? k_residual_ln<16> : k_residual_ln<32>;  // D <= 2048 (checked by the caller)
  // one wave per row, at most 1024 workgroups (later rows loop; with the
  // grid sized by the lengths' upper bound n, a pruned layer's few rows would
  // otherwise come with thousands of workgroups that only build the prefix
  // table: 7.5 -> 6.3 us in the stack's late layers)
  const long long blocks = std::min<long long>((rows + 3) / 4, 1024);
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), sizeof(int) * (B + 1), s,
                     static_cast<const __bf16*>(x_res), t, static_cast<__bf16*>(y), B, n, D, eps, len, part, K);
  return hipGetLastError();
}

}  // namespace sc
