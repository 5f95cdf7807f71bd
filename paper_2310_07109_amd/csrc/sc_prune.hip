// Binarised mask and hard pruning (SparseCoder, arXiv 2310.07109, Sec. 4.2.2
// steps 2-3): keep a token iff its score is strictly above the layer
// threshold (or it is a global token and those are kept), then compact the
// survivors, in order, into a shorter sequence.
//
// k_prune_scan   one workgroup of 1024 threads per sequence walks the tokens
//                1024 at a time: a wavefront ballot + mbcnt gives each kept
//                token its rank inside its wave, an LDS scan of the 16 wave
//                totals gives the wave offsets, and a running carry links the
//                chunks.  Exact and deterministic (integer work only).
//                Top-k rule (an alternative to the threshold, in the family
//                of SpAtten's cascade token pruning cited in Sec. 3.3): each
//                sequence keeps its ceil(keep_ratio * C) highest-scored
//                candidates (C = valid tokens, less the global ones when those
//                are kept anyway); equal scores go to the lower index.  The
//                K-th largest score is found exactly by a radix select on the
//                order-preserving 32-bit image of the float (four 8-bit digits,
//                an LDS histogram and a 256-bin suffix scan per digit); tied
//                scores are ranked in index order by the same block scan.  Up
//                to 8192 tokens a thread owns 8 consecutive tokens, keeps
//                their keys in registers through the digit passes, and two
//                block-wide scans (ties, then kept tokens) rank the sequence.
// k_gather_rows  one wavefront per output row copies the kept input row with
//                16-byte lanes (coalesced), for up to four tensors at once.
// k_prune_compact the threshold rule and the compaction in one launch, for
//                16-byte aligned rows: workgroup (c, b) owns tokens
//                [64c, 64c + 64) of sequence b.  It counts the kept tokens
//                before its chunk itself (every score before it, read from
//                L2), ranks its own tokens with a ballot, writes their
//                survivor slots and copies their rows; the last chunk's
//                workgroup, whose count spans the whole sequence, writes the
//                new length and the -1 tails.  No workgroup waits on another.
#include <algorithm>

#include "sc_device.h"
#include "sc_internal.h"

namespace sc {
namespace {

constexpr int kScanThreads = 1024;
constexpr int kScanWaves = kScanThreads / 64;
constexpr int kTopkE = 8;  // tokens per thread held in registers by the top-k path


// Exclusive rank of this lane among the lanes of its wave whose flag is set,
// and the wave's total.
SC_DEV int wave_rank(bool flag, int& total) {
  const unsigned long long m = __ballot(flag);
  total = __popcll(m);
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Block-wide exclusive scan of one flag per thread; returns this thread's
// offset and writes the block total to `total`.  Contains barriers.
SC_DEV int block_rank(bool flag, int* s_wave, int& total) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int wt;
  const int r = wave_rank(flag, wt);
  if (lane == 0) s_wave[w] = wt;
  __syncthreads();
  if (w == 0) {
    const int v = lane < kScanWaves ? s_wave[lane] : 0;
    int incl = v;
#pragma unroll
    for (int off = 1; off < kScanWaves; off <<= 1) {
      const int u = __shfl_up(incl, off, 64);
      if (lane >= off) incl += u;
    }
    if (lane < kScanWaves) s_wave[kScanWaves + lane] = incl - v;
    if (lane == kScanWaves - 1) s_wave[2 * kScanWaves] = incl;
  }
  __syncthreads();
  total = s_wave[2 * kScanWaves];
  const int off = s_wave[kScanWaves + w] + r;
  __syncthreads();  // s_wave is reused by the next call
  return off;
}

// Block-wide exclusive sum of one count per thread; returns this thread's
// offset and writes the block total to `total`.  Contains barriers.
SC_DEV int block_excl_sum(int v, int* s_wave, int& total) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int u = __shfl_up(incl, off, 64);
    if (lane >= off) incl += u;
  }
  if (lane == 63) s_wave[w] = incl;
  __syncthreads();
  if (w == 0) {
    const int x = lane < kScanWaves ? s_wave[lane] : 0;
    int winc = x;
#pragma unroll
    for (int off = 1; off < kScanWaves; off <<= 1) {
      const int u = __shfl_up(winc, off, 64);
      if (lane >= off) winc += u;
    }
    if (lane < kScanWaves) s_wave[kScanWaves + lane] = winc - x;
    if (lane == kScanWaves - 1) s_wave[2 * kScanWaves] = winc;
  }
  __syncthreads();
  total = s_wave[2 * kScanWaves];
  const int off = s_wave[kScanWaves + w] + incl - v;
  __syncthreads();  // s_wave is reused by the next call
  return off;
}

// Order-preserving image of a float score (ascending keys = ascending
// values; -0 maps to +0 so that equal scores have equal keys).
SC_DEV uint32_t score_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inclusive prefix sum over threads 0..255 of v (threads 256+ pass 0 and get
// a meaningless result).  Contains barriers; all threads must call it.
SC_DEV int scan256(int v, int* s_tmp) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int u = __shfl_up(incl, off, 64);
    if (lane >= off) incl += u;
  }
  if (lane == 63 && w < 4) s_tmp[w] = incl;
  __syncthreads();
  int add = 0;
  for (int j = 0; j < w && j < 4; ++j) add += s_tmp[j];
  __syncthreads();  // s_tmp is reused by the next call
  return incl + add;
}

__global__ __launch_bounds__(kScanThreads) void k_prune_scan(PruneArgs p) {
  __shared__ int s_wave[2 * kScanWaves + 1];
  __shared__ int s_hist[256];
  __shared__ int s_sel[2];
  __shared__ int s_tmp[4];
  extern __shared__ uint32_t s_gbits[];  // global-token bitmask over [0, n)
  const int b = blockIdx.x, tid = threadIdx.x, n = p.n;
  const int L = clampi(p.valid_len[b], 0, n);
  const int nwords = (n + 31) >> 5;
  const int* gp = (p.gpos && p.G > 0) ? p.gpos + (long long)b * p.G : nullptr;
  for (int i = tid; i < nwords; i += kScanThreads) s_gbits[i] = 0u;
  __syncthreads();
  if (gp)
    for (int j = tid; j < p.G; j += kScanThreads) {
      const int q = gp[j];
      if (q >= 0 && q < L) atomicOr(&s_gbits[q >> 5], 1u << (q & 31));
    }
  __syncthreads();
  const float* s = p.scores + (long long)b * n;
  auto is_glob = [&](int k) { return (bool)((s_gbits[k >> 5] >> (k & 31)) & 1u); };
  // top-k: candidates, their count C, K = ceil(keep_ratio * C), the K-th
  // largest key T and the number `want` of candidates with key T to keep.
  // Key 0 marks a non-candidate (no float maps to it but a negative NaN).
  auto cand_key = [&](int k) -> uint32_t {
    return (k < L && !(p.keep_global && is_glob(k))) ? score_key(s[k]) : 0u;
  };
  uint32_t T = 0u;
  int want = 0;
  bool none = true;  // no candidate is kept by rank
  // top-k over at most kTopkE * kScanThreads tokens: thread t owns the E
  // consecutive tokens [t E, t E + E) and keeps their keys in registers for
  // the count, the four digit passes and the ranking
  const bool own = p.topk && n <= kTopkE * kScanThreads;
  const int E = (n + kScanThreads - 1) / kScanThreads, k0 = tid * E;
  uint32_t okey[kTopkE];
  unsigned ogk = 0u;  // bit e: token k0 + e is kept as a global token
  if (own) {
#pragma unroll
    for (int e = 0; e < kTopkE; ++e) {
      const int k = k0 + e;
      ogk |= (unsigned)(e < E && k < L && p.keep_global && is_glob(k)) << e;
      okey[e] = e < E ? cand_key(k) : 0u;
    }
  }
  if (p.topk) {
    if (tid == 0) s_sel[0] = 0;
    __syncthreads();
    int cnt = 0;
    if (own) {
#pragma unroll
      for (int e = 0; e < kTopkE; ++e) cnt += okey[e] != 0u;
    } else {
      for (int k = tid; k < L; k += kScanThreads) cnt += cand_key(k) != 0u;
    }
    // candidate count: per-wave sums, one LDS atomic per wave
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off, 64);
    if ((tid & 63) == 0) atomicAdd(&s_sel[0], cnt);
    __syncthreads();
    const int C = s_sel[0];
    __syncthreads();
    const double prod = (double)p.keep_ratio * (double)C;
    const int K = prod <= 0.0 ? 0 : (prod >= (double)C ? C : (int)ceil(prod));
    none = K == 0;
    want = K;
    for (int shift = 24; shift >= 0 && !none; shift -= 8) {
      if (tid < 256) s_hist[tid] = 0;
      __syncthreads();
      const uint32_t hmask = shift == 24 ? 0u : ~0u << (shift + 8);
      if (own) {
#pragma unroll
        for (int e = 0; e < kTopkE; ++e) {
          const uint32_t key = okey[e];
          if (key != 0u && (key & hmask) == (T & hmask)) atomicAdd(&s_hist[(key >> shift) & 255u], 1);
        }
      } else {
        for (int k = tid; k < L; k += kScanThreads) {
          const uint32_t key = cand_key(k);
          if (key != 0u && (key & hmask) == (T & hmask)) atomicAdd(&s_hist[(key >> shift) & 255u], 1);
        }
      }
      __syncthreads();
      // bins from the top: the digit whose bin holds the want-th largest key
      const int c = tid < 256 ? s_hist[255 - tid] : 0;
      const int incl = scan256(c, s_tmp);
      if (tid < 256 && incl >= want && incl - c < want) {
        s_sel[0] = 255 - tid;
        s_sel[1] = want - (incl - c);
      }
      __syncthreads();
      T |= (uint32_t)s_sel[0] << shift;
      want = s_sel[1];
      __syncthreads();  // s_sel is rewritten by the next digit
    }
  }
  int* kidx = p.keep_idx + (long long)b * n;
  int* nidx = p.new_index + (long long)b * n;
  const int* oin = p.orig_in ? p.orig_in + (long long)b * n : nullptr;
  int* oout = p.orig_out ? p.orig_out + (long long)b * n : nullptr;
  int carry = 0, tie_carry = 0;
  if (own) {
    // ties before a token, in token order, then the kept tokens before it:
    // two block scans for the whole sequence
    int nt = 0;
#pragma unroll
    for (int e = 0; e < kTopkE; ++e) nt += !none && okey[e] != 0u && okey[e] == T;
    int ties;
    int tr = block_excl_sum(nt, s_wave, ties);
    unsigned keepm = 0u;
    int nk = 0;
#pragma unroll
    for (int e = 0; e < kTopkE; ++e) {
      const uint32_t key = okey[e];
      const bool cand = key != 0u && !none;
      const bool tie = cand && key == T;
      const bool kp = ((ogk >> e) & 1u) || (cand && (key > T || (tie && tr < want)));
      tr += tie;
      keepm |= (unsigned)kp << e;
      nk += kp;
    }
    int pos = block_excl_sum(nk, s_wave, carry);
#pragma unroll
    for (int e = 0; e < kTopkE; ++e) {
      const int k = k0 + e;
      if (e < E && k < n) {
        if ((keepm >> e) & 1u) {
          kidx[pos] = k;
          if (oout) oout[pos] = oin ? oin[k] : k;
          nidx[k] = pos++;
        } else {
          nidx[k] = -1;
        }
      }
    }
  }
  for (int base = 0; base < n && !own; base += kScanThreads) {
    const int k = base + tid;
    bool keep = false;
    if (!p.topk) {
      if (k < L) keep = s[k] > p.threshold || (p.keep_global && is_glob(k));
    } else {
      const bool gkeep = k < L && p.keep_global && is_glob(k);
      const uint32_t key = cand_key(k);
      const bool cand = key != 0u && !none;
      const bool tie = cand && key == T;
      int ties;
      const int tr = tie_carry + block_rank(tie, s_wave, ties);
      tie_carry += ties;
      keep = gkeep || (cand && (key > T || (tie && tr < want)));
    }
    int total;
    const int pos = carry + block_rank(keep, s_wave, total);
    if (keep) {
      kidx[pos] = k;
      if (oout) oout[pos] = oin ? oin[k] : k;
    }
    if (k < n) nidx[k] = keep ? pos : -1;
    carry += total;
  }
  if (tid == 0) {
    p.new_len[b] = carry;
    if (p.len_copy) p.len_copy[b] = carry;
  }
  for (int j = carry + tid; j < n; j += kScanThreads) {
    kidx[j] = -1;
    if (oout) oout[j] = -1;
  }
  if (!p.new_gpos || p.G == 0) return;
  __syncthreads();  // new_index written by this block is visible to it
  int gcarry = 0;
  int* ngp = p.new_gpos + (long long)b * p.G;
  for (int base = 0; base < p.G; base += kScanThreads) {
    const int j = base + tid;
    int q = -1;
    if (j < p.G) {
      const int pos = gp[j];
      if (pos >= 0 && pos < L) q = nidx[pos];
    }
    int total;
    const int at = gcarry + block_rank(q >= 0, s_wave, total);
    if (q >= 0) ngp[at] = q;
    gcarry += total;
  }
  for (int j = gcarry + tid; j < p.G; j += kScanThreads) ngp[j] = -1;
}

constexpr int kChunk = 64;   // tokens per workgroup of k_prune_compact
constexpr int kPcThreads = 256;

// Threshold rule: keep(k) = k < L and (score > threshold or (keep_global and
// k global)), compared in float32 as in k_prune_scan.
__global__ __launch_bounds__(kPcThreads) void k_prune_compact(PruneArgs p, GatherArgs g) {
  extern __shared__ uint32_t s_gbits[];  // global-token bitmask over [0, c1)
  __shared__ int s_red[2][kPcThreads / 64];
  __shared__ int s_k[kChunk], s_pos[kChunk];
  __shared__ int s_nk, s_gchunk;
  constexpr int kPre = 16;  // scores per thread loaded before the length and the bitmap are known
  const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6, n = p.n;
  const int c0 = blockIdx.x * kChunk, c1 = min(c0 + kChunk, n);
  const bool last = c1 == n;
  const float* s = p.scores + (long long)b * n;
  // issued together: the length, this thread's global slot, the first
  // kPre * 256 scores before the chunk (clamped into it) and the chunk's own
  // score (wave 0)
  const int Lraw = p.valid_len[b];
  const int* gp = (p.gpos && p.G > 0) ? p.gpos + (long long)b * p.G : nullptr;
  const int q0 = gp && tid < p.G ? gp[tid] : -1;
  float v[kPre];
#pragma unroll
  for (int i = 0; i < kPre; ++i) v[i] = c0 > 0 ? s[min(tid + kPcThreads * i, c0 - 1)] : 0.f;
  const float own = s[min(c0 + lane, c1 - 1)];
  const int L = clampi(Lraw, 0, n);
  const int nwords = (c1 + 31) >> 5;
  for (int i = tid; i < nwords; i += kPcThreads) s_gbits[i] = 0u;
  __syncthreads();
  if (q0 >= 0 && q0 < L && q0 < c1) atomicOr(&s_gbits[q0 >> 5], 1u << (q0 & 31));
  for (int j = tid + kPcThreads; gp && j < p.G; j += kPcThreads) {
    const int q = gp[j];
    if (q >= 0 && q < L && q < c1) atomicOr(&s_gbits[q >> 5], 1u << (q & 31));
  }
  __syncthreads();
  // bitmask reads clamped into [0, c1) and the rule in bitwise form: no
  // branch separates the reads, so they are waited for together
  auto glob = [&](int k) { return ((s_gbits[min(k, c1 - 1) >> 5] >> (k & 31)) & 1u) != 0u; };
  const bool kg = p.keep_global != 0;
  const float thr = p.threshold;
  // kept tokens, and kept global tokens, before the chunk
  int cnt = 0, gcnt = 0;
  const int lim = min(c0, L);
#pragma unroll
  for (int i = 0; i < kPre; ++i) {
    const int k = tid + kPcThreads * i;
    const bool gl = glob(k);
    const bool kp = (k < lim) & ((v[i] > thr) | (kg & gl));
    cnt += kp;
    gcnt += kp & gl;
  }
  for (int base = kPre * kPcThreads; base < lim; base += 8 * kPcThreads) {  // longer sequences
    float u[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) u[i] = s[min(base + tid + kPcThreads * i, lim - 1)];  // clamped, past lim discarded
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int k = base + tid + kPcThreads * i;
      const bool gl = glob(k);
      const bool kp = (k < lim) & ((u[i] > thr) | (kg & gl));
      cnt += kp;
      gcnt += kp & gl;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    cnt += __shfl_xor(cnt, off, 64);
    gcnt += __shfl_xor(gcnt, off, 64);
  }
  if (lane == 0) {
    s_red[0][w] = cnt;
    s_red[1][w] = gcnt;
  }
  __syncthreads();
  int before = 0, gbefore = 0;
#pragma unroll
  for (int i = 0; i < kPcThreads / 64; ++i) {
    before += s_red[0][i];
    gbefore += s_red[1][i];
  }
  int* kidx = p.keep_idx + (long long)b * n;
  const int* oin = p.orig_in ? p.orig_in + (long long)b * n : nullptr;
  int* oout = p.orig_out ? p.orig_out + (long long)b * n : nullptr;
  int* ngp = (p.new_gpos && gp) ? p.new_gpos + (long long)b * p.G : nullptr;
  if (w == 0) {  // the chunk's own tokens, one per lane
    const int k = c0 + lane;
    const bool gl = glob(k);
    const bool kp = (k < c1) & (k < L) & ((own > thr) | (kg & gl));
    const bool gk = kp & gl;
    int tot, gtot;
    const int r = wave_rank(kp, tot);
    const int gr = wave_rank(gk, gtot);
    if (kp) {
      const int pos = before + r;
      kidx[pos] = k;
      if (oout) oout[pos] = oin ? oin[k] : k;
      s_k[r] = k;
      s_pos[r] = pos;
      // surviving global tokens keep their ascending order
      if (gk && ngp) ngp[gbefore + gr] = pos;
    }
    if (lane == 0) {
      s_nk = tot;
      s_gchunk = gtot;
    }
  }
  __syncthreads();
  const int nk = s_nk;
  if (last) {  // this workgroup's count spans the sequence
    const int total = before + nk;
    if (tid == 0) {
      p.new_len[b] = total;
      if (p.len_copy) p.len_copy[b] = total;
    }
    for (int j = total + tid; j < n; j += kPcThreads) {
      kidx[j] = -1;
      if (oout) oout[j] = -1;
    }
    if (ngp)
      for (int j = gbefore + s_gchunk + tid; j < p.G; j += kPcThreads) ngp[j] = -1;
  }
  // rows of the kept tokens: wave w copies rows w, w + 4, ..., four rows at a
  // time, each lane two 16-byte units per row and round.  Rows and units past
  // the end are clamped to the last valid ones for both the load and the
  // store (a second, identical write), so that no branch separates the eight
  // loads or the eight stores.
  for (int t = 0; t < g.nt; ++t) {
    const long long rb = g.row_bytes[t];
    const int nu = (int)(rb >> 4);
    const char* src = g.src[t] + (long long)b * n * rb;
    char* dst = g.dst[t] + (long long)b * n * rb;
    for (int i0 = w; i0 < nk; i0 += 16)
      for (int u0 = 0; u0 < nu; u0 += 128) {
        const int r0 = min(i0, nk - 1), r1 = min(i0 + 4, nk - 1), r2 = min(i0 + 8, nk - 1),
                  r3 = min(i0 + 12, nk - 1);
        const long long ua = 16LL * min(u0 + lane, nu - 1), ub = 16LL * min(u0 + lane + 64, nu - 1);
        const char *s0 = src + s_k[r0] * rb, *s1 = src + s_k[r1] * rb, *s2 = src + s_k[r2] * rb,
                   *s3 = src + s_k[r3] * rb;
        const uint4 v0a = *reinterpret_cast<const uint4*>(s0 + ua), v0b = *reinterpret_cast<const uint4*>(s0 + ub);
        const uint4 v1a = *reinterpret_cast<const uint4*>(s1 + ua), v1b = *reinterpret_cast<const uint4*>(s1 + ub);
        const uint4 v2a = *reinterpret_cast<const uint4*>(s2 + ua), v2b = *reinterpret_cast<const uint4*>(s2 + ub);
        const uint4 v3a = *reinterpret_cast<const uint4*>(s3 + ua), v3b = *reinterpret_cast<const uint4*>(s3 + ub);
        char *d0 = dst + s_pos[r0] * rb, *d1 = dst + s_pos[r1] * rb, *d2 = dst + s_pos[r2] * rb,
             *d3 = dst + s_pos[r3] * rb;
        *reinterpret_cast<uint4*>(d0 + ua) = v0a;
        *reinterpret_cast<uint4*>(d0 + ub) = v0b;
        *reinterpret_cast<uint4*>(d1 + ua) = v1a;
        *reinterpret_cast<uint4*>(d1 + ub) = v1b;
        *reinterpret_cast<uint4*>(d2 + ua) = v2a;
        *reinterpret_cast<uint4*>(d2 + ub) = v2b;
        *reinterpret_cast<uint4*>(d3 + ua) = v3a;
        *reinterpret_cast<uint4*>(d3 + ub) = v3b;
      }
  }
}

// One wavefront per (sequence, output row); blockIdx.z selects the tensor.
__global__ __launch_bounds__(256) void k_gather_rows(GatherArgs a) {
  const int t = blockIdx.z, b = blockIdx.y;
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (j >= a.n || j >= a.new_len[b]) return;
  const int k = a.keep_idx[(long long)b * a.n + j];
  if (k < 0 || k >= a.n) return;
  const long long rb = a.row_bytes[t];
  const char* src = a.src[t] + ((long long)b * a.n + k) * rb;
  char* dst = a.dst[t] + ((long long)b * a.n + j) * rb;
  if (((rb | (long long)(uintptr_t)a.src[t] | (long long)(uintptr_t)a.dst[t]) & 15) == 0) {
    for (long long o = 16LL * lane; o < rb; o += 16 * 64)
      *reinterpret_cast<uint4*>(dst + o) = *reinterpret_cast<const uint4*>(src + o);
  } else if (((rb | (long long)(uintptr_t)a.src[t] | (long long)(uintptr_t)a.dst[t]) & 3) == 0) {
    for (long long o = 4LL * lane; o < rb; o += 4 * 64)
      *reinterpret_cast<uint32_t*>(dst + o) = *reinterpret_cast<const uint32_t*>(src + o);
  } else {
    for (long long o = lane; o < rb; o += 64) dst[o] = src[o];
  }
}

// Zero fill, 16 bytes per thread and store where the buffer allows it.
__global__ void k_fill_zero(uint32_t* p, long long words) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if ((reinterpret_cast<uintptr_t>(p) & 15) == 0) {
    const long long quads = words >> 2;
    if (i < quads) reinterpret_cast<uint4*>(p)[i] = make_uint4(0u, 0u, 0u, 0u);
    if (i < (words & 3)) p[4 * quads + i] = 0u;
  } else if (i < words) {
    p[i] = 0u;
  }
}

// Device-resident preconditions of one sequence's descriptor arrays (one
// wave per sequence): 0 <= valid_len[b] <= n; global slots hold ascending,
// distinct positions below valid_len[b], then only unused (-1) slots.  The
// violations found are OR-ed into *err as SC_VALID_* bits.
__global__ __launch_bounds__(64) void k_validate_desc(const int* valid_len, const int* gpos, int n, int G,
                                                      int* err) {
  const int b = blockIdx.x, lane = threadIdx.x;
  const int L = valid_len[b];
  int bits = 0;
  if (lane == 0 && (L < 0 || L > n)) bits |= kValidLen;
  if (gpos) {
    const int* gp = gpos + (long long)b * G;
    for (int j = lane; j < G; j += 64) {
      const int p = gp[j], prev = j > 0 ? gp[j - 1] : -2;
      if (p < -1 || p >= L) bits |= kValidPosRange;
      if (p >= 0 && prev == -1) bits |= kValidPosUnusedFirst;
      if (p >= 0 && prev >= 0 && prev >= p) bits |= kValidPosOrder;
    }
  }
  // one atomic per kind of violation and wave (vector memory atomics)
  for (int bit = 1; bit <= kValidPosUnusedFirst; bit <<= 1)
    if (__ballot((bits & bit) != 0) != 0ull && lane == 0) atomicOr(err, bit);
}

__global__ void k_copy_i32(const int* src, int* dst, long long count) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) dst[i] = src[i];
}

__global__ void k_iota_orig(const int* valid_len, int* orig, int B, int n) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long long)B * n) return;
  const int b = (int)(i / n), j = (int)(i % n);
  orig[i] = j < clampi(valid_len[b], 0, n) ? j : -1;
}

}  // namespace

hipError_t launch_prune(const PruneArgs& p, hipStream_t s) {
  const size_t dyn = sizeof(uint32_t) * (((size_t)p.n + 31) / 32 + 1);
  hipLaunchKernelGGL(k_prune_scan, dim3(p.B), dim3(kScanThreads), dyn, s, p);
  return hipGetLastError();
}

hipError_t launch_prune_gather(const PruneArgs& p, const GatherArgs& g, hipStream_t s) {
  bool aligned = !p.topk;
  for (int t = 0; t < g.nt; ++t)
    aligned = aligned && ((g.row_bytes[t] | (long long)(uintptr_t)g.src[t] | (long long)(uintptr_t)g.dst[t]) & 15) == 0;
  if (!aligned) {
    hipError_t e = launch_prune(p, s);
    return e != hipSuccess ? e : launch_gather(g, s);
  }
  const size_t dyn = sizeof(uint32_t) * (((size_t)p.n + 31) / 32 + 1);
  hipLaunchKernelGGL(k_prune_compact, dim3((p.n + kChunk - 1) / kChunk, p.B), dim3(kPcThreads), dyn, s, p, g);
  return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs& g, hipStream_t s) {
  if (g.nt == 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather_rows, dim3((g.n + 3) / 4, g.B, g.nt), dim3(256), 0, s, g);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
  const long long words = (long long)(bytes / 4);
  if (words <= 0) return hipSuccess;
  const long long threads = (reinterpret_cast<uintptr_t>(p) & 15) == 0 ? std::max(words >> 2, 3LL) : words;
  hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, static_cast<uint32_t*>(p),
                     words);
  return hipGetLastError();
}

hipError_t launch_validate_desc(const int* valid_len, const int* gpos, int B, int n, int G, int* err, hipStream_t s) {
  const hipError_t e = launch_fill_zero(err, sizeof(int), s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_validate_desc, dim3((unsigned)B), dim3(64), 0, s, valid_len, gpos, n, G, err);
  return hipGetLastError();
}

hipError_t launch_copy_i32(const int* src, int* dst, long long count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy_i32, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, src, dst, count);
  return hipGetLastError();
}

hipError_t launch_iota_orig(const int* valid_len, int* orig, int B, int n, hipStream_t s) {
  const long long count = (long long)B * n;
  hipLaunchKernelGGL(k_iota_orig, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, valid_len, orig, B, n);
  return hipGetLastError();
}

}  // namespace sc
