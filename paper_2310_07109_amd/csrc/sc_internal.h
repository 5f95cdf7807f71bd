// Internal launch interface between the C ABI (sc_api.hip) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sc {

constexpr int kQueryBlock = 64;    // queries per window-attention workgroup
constexpr int kKeyTile = 64;       // keys per LDS tile
constexpr int kGlobalChunk = 32;   // global slots per workgroup of the global-row / global-column blocks
constexpr int kGlobalKeySpan = 512;  // keys per split of the global-row kernels

// Geometry + pointers of one attention launch sequence.  Element strides let
// the same kernels read q/k/v out of a fused [tokens, 3*D] projection.
struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  void* out;
  float* lse;             // [B, H, n] or null
  const int* valid_len;   // [B]
  const int* gpos;        // [B, G] or null
  long long ld_in, bs_in;   // elements between tokens / sequences of q, k, v
  long long ld_out, bs_out; // same for out
  int B, n, H, G, r;      // r = half window, clamped to [0, n]
  int causal;             // 1: keys after the query are never attended
  int skip_pad_out;       // 1: output rows of padding-only query blocks are left unwritten
  int no_profile;         // 1: never record benchmark events for this call
  int span_major;         // 1: dispatch the attention blocks span-major (xcd_span_map), for
                          //    sequences much shorter than n; 0: pair by pair (xcd_pair_map)
                          //    unless n is at most 4096 (the launch then takes the span order)
  float c2;               // softmax scale * log2(e)
  // score partials (null: skip the exact-probability column sums)
  float* part_band;       // [B, H, n]      band column sums of non-global keys
  float* part_extra;      // [B, H, nqr, G] global-key columns per 512-query range
  float* part_grow;       // [B, H, ngc, n] column sums over the global rows
  int nqb, rwp, ngc, nkc, Gp, nkb, nqr;
  int n_gr, n_bcol, n_gcol;  // block counts of the global-row, band-column and global-column parts
  // global-row split partials (workspace)
  float* gr_ml;           // [B, H, nkc, Gp, 2]
  float* gr_o;            // [B, H, nkc, Gp, 64]
  float* gr_lse2;         // [B, H, Gp]
  float* win_lse2;        // [B, H, n] log2-LSE of the window rows (+inf: excluded)
  // paper band layout (null unless requested)
  float* bp_band;         // [B, H, n, bw]
  float* bp_gcol;         // [B, H, n, G]
  float* bp_grow;         // [B, H, G, n]
  int bw, rb;             // bw = 2 * rb + 1
};

struct AttnGeom {
  int nqb, rwp, ngc, Gp, nkc, r, bw, rb, nkb, nqr;
};

AttnGeom attn_geom(int n, int window, int G);
size_t partials_floats(int B, int H, int n, const AttnGeom& g, int G);
size_t band_probs_floats(int B, int H, int n, const AttnGeom& g, int G);

hipError_t launch_window_attention(int dtype, const AttnArgs& a, hipStream_t s);
// benchmark timing of the window-attention kernel (events on the launch stream)
int profile_set(int enable);
int profile_read(double* fwd_ms, double* cols_ms, long long cap, long long* calls);
hipError_t launch_score_from_partials(const float* partials, const int* valid_len, const int* gpos, int B, int n,
                                      int H, int G, const AttnGeom& g, float* scores, hipStream_t s);
// per-row-block partial sums of the band layout, a part of sc_ltp_score's
// workspace in the band mode
size_t band_parts_floats(int B, int H, int n, int window, int G);
hipError_t launch_score_from_band(const float* bp, const int* valid_len, const int* gpos, int B, int n, int H, int G,
                                  const AttnGeom& g, float* partials, float* parts, float* scores, hipStream_t s);

struct PruneArgs {
  const float* scores;     // [B, n]
  const int* valid_len;    // [B]
  const int* gpos;         // [B, G] or null
  int B, n, G;
  float threshold;
  int keep_global;
  int topk;                // 0: threshold rule; 1: keep the ceil(keep_ratio * C) best candidates per sequence
  float keep_ratio;
  int* keep_idx;           // [B, n]
  int* new_len;            // [B]
  int* new_gpos;           // [B, G] or null
  const int* orig_in;      // [B, n] or null
  int* orig_out;           // [B, n] or null
  int* new_index;          // workspace [B, n]
  int* len_copy;           // [B] or null: a second copy of new_len (e.g. a per-layer record)
};
hipError_t launch_prune(const PruneArgs& p, hipStream_t s);

// LTP soft pruning, training form: forward mask and the backward of
// y = mask * attention(q, k, v) through the attention and the scores.  All
// token tensors are contiguous [B, n, H, 64] bf16.
constexpr int kBwdSpan = 512;  // keys (queries) per global-row (global-column) block of the backward

struct SoftArgs {
  const __bf16 *q, *k, *v, *o, *dy;
  const float* lse;     // [B, H, n] natural log (forward output)
  const float* mask;    // [B, n]
  const float* dmask;   // [B, n] or null
  const float* scores;  // [B, n] (forward mask only)
  __bf16* y;            // [B, n, H, 64] (forward mask only)
  float* mask_out;      // [B, n] (forward mask only)
  __bf16 *dq, *dk, *dv;
  float* dtheta;        // one float
  const int* valid_len;
  const int* gpos;      // [B, G] or null
  int B, n, H, G, r;
  int keep_global;
  float alpha, c2;      // softmax scale, and scale * log2(e)
  float theta, inv_t;   // threshold (forward) and 1 / temperature
  int nsp, Gp;          // spans of kBwdSpan tokens; G padded to a multiple of 64
  // workspace
  __bf16* dO;           // [B, n, H, 64]  mask * dy
  float* Dq;            // [B, H, n]      sum_j P dL/dP of each query row
  float* gk;            // [B, n]         score gradient of each key over H * L
  float* dsv;           // [B n / 4]      score gradients summed per 4 tokens (for the threshold's)
  float* gpg;           // [B, H, nsp, Gp]      global rows: sum_j P g per key span
  float* gdq;           // [B, H, nsp, Gp, 64]  global rows: dQ per key span
  float* gdk;           // [B, H, nsp, Gp, 64]  global keys: dK per query span
  float* gdv;           // [B, H, nsp, Gp, 64]  global keys: dV per query span
};
hipError_t launch_soft_mask(const SoftArgs& a, hipStream_t s);
hipError_t launch_soft_backward(const SoftArgs& a, hipStream_t s);

struct GatherArgs {
  int B, n, nt;
  const char* src[4];
  char* dst[4];
  long long row_bytes[4];
  const int* keep_idx;
  const int* new_len;
};
hipError_t launch_gather(const GatherArgs& g, hipStream_t s);
// The prune of p followed by the gather of g (keep_idx and new_len of g are
// p's): one launch for the threshold rule on 16-byte aligned rows, else the
// two above.
hipError_t launch_prune_gather(const PruneArgs& p, const GatherArgs& g, hipStream_t s);

// Stack pieces.
// y[rows, N] = x[rows, K] . W[K, N] (bf16 in, fp32 accumulate), rows of
// sequence b limited to len[b] (others untouched); output bf16 or fp32.
// GEMM epilogues: bf16 store, fp32 store, GELU then bf16 store.  The
// surviving rows of all sequences are packed into shared row tiles on the
// device (B <= kPackMaxB).
// part (float32, kGemmSplitRows * N, or NULL): with kGemmF32, a product
// whose packed rows fill few tiles splits its reduction into slabs there
// instead of writing y; the residual LayerNorm given the same part,
// lengths and K adds them.
constexpr int kGemmBf16 = 0, kGemmF32 = 1, kGemmGeluBf16 = 2;
constexpr int kGemmSplitRows = 128 * 128;
constexpr int kPackMaxB = 8192;
hipError_t launch_gemm_bf16(const void* x, const void* w, void* y, int mode, int B, int n, int K, int N,
                            const int* len, float* part, hipStream_t s);
// y = bf16(LayerNorm(x_res + t)) per row, rows of sequence b < len[b]; t or,
// when part is not NULL, the slabs of the product of reduction length K that
// wrote it.  B <= kPackMaxB.
hipError_t launch_residual_layernorm(const void* x_res, const float* t, void* y, int B, int n, int D, float eps,
                                     const int* len, const float* part, int K, hipStream_t s);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);
// Bits of the device-side descriptor check (the same values as SC_VALID_* in
// sc.h): a length outside [0, n]; a global position below -1 or not below
// its sequence's length; used positions not strictly ascending; a used slot
// after an unused one.
constexpr int kValidLen = 1, kValidPosRange = 2, kValidPosOrder = 4, kValidPosUnusedFirst = 8;
// *err = 0, then the bits of the violations found in valid_len [B] and
// gpos [B, G] (NULL when G == 0).
hipError_t launch_validate_desc(const int* valid_len, const int* gpos, int B, int n, int G, int* err, hipStream_t s);
hipError_t launch_copy_i32(const int* src, int* dst, long long count, hipStream_t s);
hipError_t launch_iota_orig(const int* valid_len, int* orig, int B, int n, hipStream_t s);

}  // namespace sc
