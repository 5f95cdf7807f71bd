// LDS read throughput per CU for the two read forms of the window
// attention's tile loop: 16-byte fragment reads (ds_read_b128: the K and Q
// MFMA operands) and 8-byte transposing reads (ds_read_b64_tr_b16: the V
// operand).  A measurement aid for the bottleneck analysis (bench.py
// --probe-lds), built into libsc_probe.so: not part of the hot path or of
// libsc.so's interface.
//
// kBlocksPerCu workgroups of 4 waves per CU (the attention's residency), each
// holding 32 KB of LDS; every wave issues groups of 8 independent reads and
// waits for them, so the time is the LDS's delivery rate.  Addresses stay
// inside the workgroup's 32 KB (the highest group starts at byte 24560).
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr int kLdsBytes = 32768, kThreads = 256;

template <int kOp>
__global__ __launch_bounds__(kThreads) void k_lds_rate(unsigned* out, int iters) {
  __shared__ __attribute__((aligned(16))) unsigned lds[kLdsBytes / 4];
  const int tid = threadIdx.x, lane = tid & 63;
  for (int i = tid; i < kLdsBytes / 4; i += kThreads) lds[i] = (unsigned)i * 2654435761u;
  __syncthreads();
  const unsigned base = (unsigned)(uintptr_t)(const __attribute__((address_space(3))) void*)lds;
  // group start: 16-byte aligned, at most 0x5FF0, so that 8 reads spaced 1 KB
  // (b128) or 512 B (tr_b64) apart end below 32 KB
  unsigned off = (unsigned)(lane * 16 + (tid >> 6) * 4096) & 0x5FF0u;
  unsigned acc = 0;
  for (int it = 0; it < iters; ++it) {
    const unsigned a = base + off;
    if constexpr (kOp == 0) {
      uint4 v0, v1, v2, v3, v4, v5, v6, v7;
      asm volatile(
          "ds_read_b128 %0, %8\n\tds_read_b128 %1, %8 offset:1024\n\tds_read_b128 %2, %8 offset:2048\n\t"
          "ds_read_b128 %3, %8 offset:3072\n\tds_read_b128 %4, %8 offset:4096\n\tds_read_b128 %5, %8 offset:5120\n\t"
          "ds_read_b128 %6, %8 offset:6144\n\tds_read_b128 %7, %8 offset:7168\n\ts_waitcnt lgkmcnt(0)"
          : "=v"(v0), "=v"(v1), "=v"(v2), "=v"(v3), "=v"(v4), "=v"(v5), "=v"(v6), "=v"(v7)
          : "v"(a)
          : "memory");
      acc ^= v0.x ^ v1.y ^ v2.z ^ v3.w ^ v4.x ^ v5.y ^ v6.z ^ v7.w;
    } else {
      uint2 v0, v1, v2, v3, v4, v5, v6, v7;
      asm volatile(
          "ds_read_b64_tr_b16 %0, %8\n\tds_read_b64_tr_b16 %1, %8 offset:512\n\tds_read_b64_tr_b16 %2, %8 offset:1024\n\t"
          "ds_read_b64_tr_b16 %3, %8 offset:1536\n\tds_read_b64_tr_b16 %4, %8 offset:2048\n\t"
          "ds_read_b64_tr_b16 %5, %8 offset:2560\n\tds_read_b64_tr_b16 %6, %8 offset:3072\n\t"
          "ds_read_b64_tr_b16 %7, %8 offset:3584\n\ts_waitcnt lgkmcnt(0)"
          : "=v"(v0), "=v"(v1), "=v"(v2), "=v"(v3), "=v"(v4), "=v"(v5), "=v"(v6), "=v"(v7)
          : "v"(a)
          : "memory");
      acc ^= v0.x ^ v1.y ^ v2.x ^ v3.y ^ v4.x ^ v5.y ^ v6.x ^ v7.y;
    }
    off = (off + 8192u) & 0x5FF0u;
  }
  if (acc == 0x9e3779b9u) out[0] = acc;  // keeps the reads alive; practically never true
}

}  // namespace

// op 0: ds_read_b128, 1: ds_read_b64_tr_b16.  Runs `blocks` workgroups of 256
// threads, `iters` groups of 8 reads per thread; *ms = kernel time
// (hipEvents, after one untimed launch), *bytes = bytes delivered to the
// waves.
extern "C" int sc_probe_lds_rate(int op, int blocks, int iters, double* ms, double* bytes) {
  unsigned* out = nullptr;
  if (hipMalloc(&out, sizeof(unsigned)) != hipSuccess) return -1;
  auto launch = [&]() {
    if (op == 0)
      hipLaunchKernelGGL(k_lds_rate<0>, dim3(blocks), dim3(kThreads), 0, 0, out, iters);
    else
      hipLaunchKernelGGL(k_lds_rate<1>, dim3(blocks), dim3(kThreads), 0, 0, out, iters);
  };
  hipEvent_t e0, e1;
  hipEventCreate(&e0);
  hipEventCreate(&e1);
  launch();
  hipEventRecord(e0, 0);
  launch();
  hipEventRecord(e1, 0);
  hipEventSynchronize(e1);
  float t = 0.f;
  hipEventElapsedTime(&t, e0, e1);
  hipEventDestroy(e0);
  hipEventDestroy(e1);
  hipFree(out);
  *ms = t;
  *bytes = (double)blocks * kThreads * iters * 8 * (op == 0 ? 16 : 8);
  return (int)hipGetLastError();
}
