// Device-side building blocks of the gfx950 kernels: vector types, MFMA
// fragment traits for the two storage types, cross-lane helpers.
//
// Lane conventions (wave64, v_mfma_f32_16x16x* family): lane l has row/column
// index lr = l % 16 and lane group g = l / 16.  A 16x16 fp32 result tile puts
// element (4g + i, lr) in lane l, register i.  Both operands of one MFMA are
// loaded with the same per-lane pattern along the contraction dimension, so the
// products pair up whatever order the hardware uses inside a lane group.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define SC_DEV __device__ __forceinline__

namespace sc {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kHeadDim = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

SC_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// IEEE 754-2019 maximum (NaN-propagating): compiles to v_maximum3_f32 without
// the NaN-quieting copies that fmaxf needs on MFMA results in IEEE mode.
SC_DEV float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }
SC_DEV float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// Cross-row exchanges on the VALU (gfx950 v_permlane16/32_swap).  With both
// operands equal to v, permlane16_swap returns (rows 0,0,2,2 ; rows 1,1,3,3)
// of v and permlane32_swap returns (low half twice ; high half twice), so the
// sum of the two results is the all-reduce over lanes l and l^16 (resp. l^32),
// computed in the same order in every lane.
SC_DEV float xor16_sum(float v) {
  const unsigned u = __builtin_bit_cast(unsigned, v);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __builtin_bit_cast(float, (unsigned)r[0]) + __builtin_bit_cast(float, (unsigned)r[1]);
}
SC_DEV float xor32_sum(float v) {
  const unsigned u = __builtin_bit_cast(unsigned, v);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_bit_cast(float, (unsigned)r[0]) + __builtin_bit_cast(float, (unsigned)r[1]);
}
SC_DEV float xor16_max(float v) {
  const unsigned u = __builtin_bit_cast(unsigned, v);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return vmax(__builtin_bit_cast(float, (unsigned)r[0]), __builtin_bit_cast(float, (unsigned)r[1]));
}
SC_DEV float xor32_max(float v) {
  const unsigned u = __builtin_bit_cast(unsigned, v);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return vmax(__builtin_bit_cast(float, (unsigned)r[0]), __builtin_bit_cast(float, (unsigned)r[1]));
}

// Sum / max over the four lane groups (lanes lr, lr+16, lr+32, lr+48); every
// lane gets the same result, combined in the same order.
SC_DEV float group_sum(float v) { return xor32_sum(xor16_sum(v)); }
SC_DEV float group_max(float v) { return xor32_max(xor16_max(v)); }

typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((ext_vector_type(8))) short i16x8;

// gfx950 LDS transpose read (ds_read_tr16_b64): every lane supplies the
// address of 4 consecutive 16-bit elements; within each group of 16 lanes,
// lane j receives element j % 4 of the blocks read by lanes j/4, 4 + j/4,
// 8 + j/4 and 12 + j/4 (in that order).
SC_DEV i16x4 lds_read_tr16(const void* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(const_cast<void*>(p)));
}

// The lane id, opaque to the compiler: values derived from it are
// recomputed where they are used instead of being hoisted out of the tile
// loops and held in registers across them.
SC_DEV int opaque_lane() {
  int lane;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane));
  return lane;
}

// One direct load: lane i's 16 bytes at base + voff land at LDS byte address
// lds + 16 i (gfx950 global_load_lds_dwordx4, destination base in m0).  Inline
// assembly on purpose: the compiler cannot tell these writes from later LDS
// reads of the other tile buffer and would wait for them before every read;
// here they are completed explicitly by wait_dma() before the barrier that
// publishes the tile.
SC_DEV unsigned lds_addr(const void* p) {
  return (unsigned)(size_t)(const __attribute__((address_space(3))) void*)p;
}
SC_DEV void lds_dma16(const void* base, unsigned voff, unsigned lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(base), "s"(lds)
               : "memory", "m0");
}
SC_DEV void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2): workgroup i runs on XCD i % 8.  For a grid of `pairs` x `inner`
// blocks (a (sequence, head) pair and its query or key blocks), block i is
// mapped to (pair, idx) so that the inner blocks of a pair run on one XCD in
// order (neighbours share K/V tiles in that L2) and the pairs are dealt
// round-robin over the XCDs, which spreads sequences of different length
// evenly.  When pairs is not a multiple of 8 the last pairs % 8 pairs keep
// the plain order.  The caller's block index must start at a multiple of 8.
SC_DEV void xcd_pair_map(int i, int inner, int pairs, int& pair, int& idx) {
  const int full = pairs & ~7;
  if (i < full * inner) {
    const int x = i & 7, j = i >> 3;
    pair = 8 * (j / inner) + x;
    idx = j % inner;
  } else {
    const int rest = i - full * inner;
    pair = full + rest / inner;
    idx = rest % inner;
  }
}

// The same dealing of pairs to XCDs for work split into nspan spans of `per`
// blocks per pair, but span-major: an XCD runs span 0 of all its pairs, then
// span 1 of all of them, and so on, with a pair's blocks of one span in order.
// Work at the start of the sequences (all there is once pruning has shortened
// them) is dispatched first, and the blocks that only find a span beyond
// their sequence's length come last.  Block i -> (pair, span c, block o of
// the span).  The last pairs % 8 pairs follow, span-major among themselves.
SC_DEV void xcd_span_map(int i, int nspan, int per, int pairs, int& pair, int& c, int& o) {
  const int full = pairs & ~7;
  if (i < full * nspan * per) {
    const int x = i & 7, j = i >> 3, row = (full >> 3) * per;  // blocks per span on one XCD
    c = j / row;
    const int r = j - c * row;
    pair = 8 * (r / per) + x;
    o = r % per;
  } else {
    const int rest = i - full * nspan * per, row = (pairs - full) * per;
    c = rest / row;
    const int r = rest - c * row;
    pair = full + r / per;
    o = r % per;
  }
}

template <int DT>
struct Tr;

// LDS tiles hold rows of 64 head dims in 16-byte units.  off(row, unit) is
// the element offset of a unit in a key / query tile (read as MFMA fragments,
// one 16-byte unit per lane); voff(row, unit) the same in a value tile (read
// with the 8-byte transposed reads).  Each storage type picks layouts that are
// free of LDS bank conflicts for those reads.

// bfloat16: one MFMA v_mfma_f32_16x16x32_bf16 covers 32 of the 64 head dims;
// a lane holds 8 consecutive dims (16 bytes) of its row.  Rows are unpadded
// (128 B) with the unit index XOR-swizzled by the row's low 3 bits, for key,
// query and value tiles alike: the 16-byte fragment reads (lane -> row lr,
// unit g) and the transposed 8-byte reads of value tiles then touch distinct
// LDS banks (measured on gfx950: as fast as linear reads, where a padded
// 144-byte pitch made the fragment reads 1.7x slower), and whole rows stay
// 128-byte runs that the direct global->LDS loads can fill.
template <>
struct Tr<1> {
  using T = __bf16;
  using Frag = bf16x8;
  static constexpr int kChunks = 2;
  static constexpr int kPitch = 64;  // elements per row
  static constexpr int kPitchV = 64;
  SC_DEV static int off(int row, int unit) { return row * kPitch + 8 * (unit ^ (row & 7)); }
  SC_DEV static int voff(int row, int unit) { return off(row, unit); }
  SC_DEV static f32x4 mma(Frag a, Frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  SC_DEV static void load_frags(const T* tile, int row, int g, Frag (&f)[kChunks]) {
    f[0] = *reinterpret_cast<const bf16x8*>(tile + off(row, g));
    f[1] = *reinterpret_cast<const bf16x8*>(tile + off(row, 4 + g));
  }
};

// float32: v_mfma_f32_16x16x4_f32 covers 4 dims per instruction, one per lane
// group.  Chunk c = 4m + i gives lane group g the dim 16m + 4g + i, so one
// 16-byte LDS read fills four chunks.  All rows are padded to 272 bytes.
template <>
struct Tr<0> {
  using T = float;
  using Frag = float;
  static constexpr int kChunks = 16;
  static constexpr int kPitch = 68;
  static constexpr int kPitchV = 68;
  SC_DEV static int off(int row, int unit) { return row * kPitch + 4 * unit; }
  SC_DEV static int voff(int row, int unit) { return row * kPitchV + 4 * unit; }
  SC_DEV static f32x4 mma(Frag a, Frag b, f32x4 c) { return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0); }
  SC_DEV static void load_frags(const T* tile, int row, int g, Frag (&f)[kChunks]) {
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      f32x4 v = *reinterpret_cast<const f32x4*>(tile + off(row, 4 * m + g));
      f[4 * m + 0] = v[0];
      f[4 * m + 1] = v[1];
      f[4 * m + 2] = v[2];
      f[4 * m + 3] = v[3];
    }
  }
};

// 16-byte global <-> LDS copies of whole rows of 64 head dims.
template <typename T>
SC_DEV void copy16(T* dst, const T* src) {
  *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(src);
}
template <typename T>
SC_DEV void zero16(T* dst) {
  *reinterpret_cast<uint4*>(dst) = make_uint4(0, 0, 0, 0);
}

SC_DEV int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

}  // namespace sc
