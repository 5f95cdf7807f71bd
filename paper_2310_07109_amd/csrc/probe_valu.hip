// Issue rate of the two VALU forms the window attention's cost model counts
// (v_fma_f32 and v_exp_f32 on gfx950).  A measurement aid for the roofline
// figures (bench.py --probe-valu), built into its own library: not part of
// the hot path or of libsc.so's interface.
//
// Every wave runs kChains independent dependency chains of one instruction
// kind, unrolled, at 8 waves per SIMD, so the time per instruction is the
// SIMD's issue rate rather than the instruction's latency.  The exp chain
// computes x = exp2(-|x|) (the negation and absolute value are free operand
// modifiers), which stays in (0, 1].
#include <hip/hip_runtime.h>

namespace {

constexpr int kChains = 8, kUnroll = 4, kThreads = 256;

template <int kOp>
__global__ __launch_bounds__(kThreads) void k_valu_rate(float* out, int iters, float a, float b) {
  float x[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) x[c] = (float)(threadIdx.x + c) * 1e-3f;
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
#pragma unroll
      for (int c = 0; c < kChains; ++c) {
        if constexpr (kOp == 0)
          x[c] = fmaf(x[c], a, b);
        else
          x[c] = __builtin_amdgcn_exp2f(-fabsf(x[c]));
      }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c) s += x[c];
  if (s == 1.2345678f) out[threadIdx.x] = s;  // keeps the chains alive; never true in practice
}

}  // namespace

// op 0: v_fma_f32, 1: v_exp_f32.  Runs `blocks` workgroups of 256 threads,
// `iters` x 32 instructions per thread; *ms = kernel time (hipEvents, after
// one untimed launch), *wave_instr = wave64 instructions executed.
extern "C" int sc_probe_valu_rate(int op, int blocks, int iters, double* ms, double* wave_instr) {
  float* out = nullptr;
  if (hipMalloc(&out, sizeof(float) * kThreads) != hipSuccess) return -1;
  auto launch = [&]() {
    if (op == 0)
      hipLaunchKernelGGL(k_valu_rate<0>, dim3(blocks), dim3(kThreads), 0, 0, out, iters, 0.999f, 1e-4f);
    else
      hipLaunchKernelGGL(k_valu_rate<1>, dim3(blocks), dim3(kThreads), 0, 0, out, iters, 0.f, 0.f);
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
  *wave_instr = (double)blocks * (kThreads / 64) * iters * kUnroll * kChains;
  return (int)hipGetLastError();
}
