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
// k_residual_ln y = bf16(LayerNorm(x + t)), one wavefront per row, fp32
//               statistics (biased variance), gamma = 1, beta = 0.
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

__global__ __launch_bounds__(256) void k_residual_ln(const __bf16* __restrict__ xr, const float* __restrict__ t,
                                                     __bf16* __restrict__ y, int B, int n, int D, float eps,
                                                     const int* __restrict__ len) {
  const long long row = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= (long long)B * n) return;
  const int b = (int)(row / n), j = (int)(row % n);
  if (j >= clampi(len[b], 0, n)) return;
  const __bf16* xp = xr + row * D;
  const float* tp = t + row * D;
  __bf16* yp = y + row * D;
  constexpr int kMaxPer = 32;  // D <= 2048
  float v[kMaxPer];
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int c = lane + 64 * u;
    v[u] = c < D ? (float)xp[c] + tp[c] : 0.f;
    s += v[u];
  }
  for (int m = 1; m < 64; m <<= 1) s += __shfl_xor(s, m, 64);
  const float mean = s / (float)D;
  float q = 0.f;
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int c = lane + 64 * u;
    const float dv = c < D ? v[u] - mean : 0.f;
    q += dv * dv;
  }
  for (int m = 1; m < 64; m <<= 1) q += __shfl_xor(q, m, 64);
  const float inv = 1.0f / sqrtf(q / (float)D + eps);
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int c = lane + 64 * u;
    if (c < D) yp[c] = (__bf16)((v[u] - mean) * inv);
  }
}

__global__ void k_record_len(const int* len, int* dst, int B) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < B) dst[i] = len[i];
}

}  // namespace

hipError_t launch_gemm_bf16(const void* x, const void* w, void* y, int mode, int B, int n, int K, int N,
                            const int* len, hipStream_t s) {
  dim3 grid((N + kBN - 1) / kBN, (n + kBM - 1) / kBM, B);
  hipLaunchKernelGGL(k_gemm_bf16, grid, dim3(256), 0, s, static_cast<const __bf16*>(x),
                     static_cast<const __bf16*>(w), y, mode, n, K, N, len);
  return hipGetLastError();
}

hipError_t launch_residual_layernorm(const void* x_res, const float* t, void* y, int B, int n, int D, float eps,
                                     const int* len, hipStream_t s) {
  const long long rows = (long long)B * n;
  hipLaunchKernelGGL(k_residual_ln, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s,
                     static_cast<const __bf16*>(x_res), t, static_cast<__bf16*>(y), B, n, D, eps, len);
  return hipGetLastError();
}

hipError_t launch_record_len(const int* len, int* dst, int B, hipStream_t s) {
  hipLaunchKernelGGL(k_record_len, dim3((B + 255) / 256), dim3(256), 0, s, len, dst, B);
  return hipGetLastError();
}

}  // namespace sc
