// C ABI of the library (declared in include/sc.h): argument validation on the
// host, workspace carving, and launch sequencing on the caller's stream.
// Nothing here allocates device memory or synchronises.
#include <algorithm>
#include <cfloat>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "../../include/sc.h"
#include "sc_internal.h"

namespace {

using sc::AttnArgs;
using sc::AttnGeom;

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

size_t elem_size(int dtype) { return dtype == SC_BF16 ? 2 : 4; }

sc_status check_desc(const sc_attn_desc* d) {
  if (!d) return SC_EINVAL;
  if (d->B < 1 || d->n < 1 || d->H < 1 || d->window < 0 || d->G < 0 || d->G > d->n) return SC_EINVAL;
  if (!d->valid_len) return SC_EINVAL;
  if (d->G > 0 && !d->global_pos) return SC_EINVAL;
  if (!std::isfinite(d->softmax_scale) || d->softmax_scale < 0.f) return SC_EINVAL;
  if (d->dtype != SC_F32 && d->dtype != SC_BF16) return SC_EINVAL;
  if (d->causal != 0 && d->causal != 1) return SC_EINVAL;
  if (d->d != 64) return SC_EUNSUPPORTED;
  if (d->causal && d->dtype != SC_BF16) return SC_EUNSUPPORTED;
  // grid sizes must fit the launch limits: 64-row blocks, and the attention
  // launches' per-span work (at most 8 window or band-column blocks and two
  // blocks per 32 global slots in every key span)
  const long long nspan = (d->n + sc::kGlobalKeySpan - 1) / sc::kGlobalKeySpan;
  const long long ngc = (d->G + sc::kGlobalChunk - 1) / sc::kGlobalChunk;
  const long long blocks = std::max((long long)((d->n + 63) / 64), nspan * (8 + 2 * ngc)) * d->H * d->B;
  if (blocks + 8 >= (1LL << 31)) return SC_EUNSUPPORTED;  // + padding of a block count to a multiple of 8
  if ((long long)d->B * d->n >= (1LL << 31)) return SC_EUNSUPPORTED;
  // tile loads address one sequence's rows with 32-bit byte offsets
  if ((long long)d->n * d->H * d->d * (long long)elem_size(d->dtype) >= (1LL << 32)) return SC_EUNSUPPORTED;
  return SC_OK;
}

size_t tensor_bytes(const sc_attn_desc* d) { return (size_t)d->B * d->n * d->H * d->d * elem_size(d->dtype); }

// Carves 256-byte aligned pieces out of the caller's workspace.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* p) : base(static_cast<char*>(p)) {}
  template <typename T>
  T* take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

AttnArgs make_attn_args(const sc_attn_desc* d, const AttnGeom& geo) {
  AttnArgs a;
  std::memset(&a, 0, sizeof(a));
  a.valid_len = d->valid_len;
  a.gpos = d->G > 0 ? d->global_pos : nullptr;
  a.ld_in = (long long)d->H * d->d;
  a.bs_in = a.ld_in * d->n;
  a.ld_out = a.ld_in;
  a.bs_out = a.bs_in;
  a.B = d->B;
  a.n = d->n;
  a.H = d->H;
  a.G = d->G;
  a.r = geo.r;
  a.causal = d->causal;
  // Scale in log2 units.  The kernels need c2 > 0 (disallowed logits are set
  // to -inf and exp2(-inf * c2) must be 0); a zero scale becomes the smallest
  // normal float, which yields the same fp32 probabilities for logits below
  // 2^26 in magnitude (every scaled logit then rounds away next to 1 in exp2).
  a.c2 = std::max(d->softmax_scale * 1.4426950408889634f, FLT_MIN);
  a.nqb = geo.nqb;
  a.rwp = geo.rwp;
  a.ngc = geo.ngc;
  a.nkc = geo.nkc;
  a.Gp = geo.Gp;
  a.bw = geo.bw;
  a.rb = geo.rb;
  a.nkb = geo.nkb;
  a.nqr = geo.nqr;
  return a;
}

void carve_attn_ws(AttnArgs& a, Carver& c) {
  a.win_lse2 = c.take<float>((size_t)a.B * a.H * a.n);
  if (a.Gp == 0) return;
  const size_t per = (size_t)a.B * a.H * a.Gp;
  a.gr_ml = c.take<float>(per * a.nkc * 2);
  a.gr_o = c.take<float>(per * a.nkc * 64);
  a.gr_lse2 = c.take<float>(per);
}

void set_partials(AttnArgs& a, float* sp) {
  a.part_band = sp;
  a.part_extra = sp ? sp + (size_t)a.B * a.H * a.n : nullptr;
  a.part_grow = sp ? a.part_extra + (size_t)a.B * a.H * a.nqr * a.G : nullptr;
}

size_t attn_ws_size(const sc_attn_desc* d) {
  const AttnGeom geo = sc::attn_geom(d->n, d->window, d->G);
  AttnArgs a = make_attn_args(d, geo);
  Carver c(nullptr);
  carve_attn_ws(a, c);
  return c.off;
}

}  // namespace

#ifdef SC_DEBUG
// Debug build: the device word of the descriptor check.
static __device__ int32_t g_debug_err;
#endif

namespace {
#ifdef SC_DEBUG
// Debug build: before an entry point enqueues anything, its descriptor's
// device-resident arrays are checked and the stream drained; then the entry
// point's own work is waited for and a failed launch or execution reported.
sc_status debug_pre(const sc_attn_desc* d, void* stream) {
  if (check_desc(d) != SC_OK) return SC_OK;  // the entry point reports it
  int32_t* err = nullptr;
  if (hipGetSymbolAddress(reinterpret_cast<void**>(&err), HIP_SYMBOL(g_debug_err)) != hipSuccess || !err)
    return SC_EHIP;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (sc::launch_validate_desc(d->valid_len, d->G > 0 ? d->global_pos : nullptr, d->B, d->n, d->G, err, s) !=
      hipSuccess)
    return SC_EHIP;
  int32_t bits = 0;
  if (hipMemcpyAsync(&bits, err, sizeof(bits), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return SC_EHIP;
  return bits != 0 ? SC_EINVAL : SC_OK;
}

sc_status debug_post(sc_status st, void* stream) {
  if (st != SC_OK) return st;
  if (hipStreamSynchronize(static_cast<hipStream_t>(stream)) != hipSuccess || hipGetLastError() != hipSuccess)
    return SC_EHIP;
  return SC_OK;
}
#endif
}  // namespace

#ifdef SC_DEBUG
#define SC_DEBUG_CALL(d, stream, call)          \
  do {                                          \
    const sc_status pre_ = debug_pre(d, stream); \
    if (pre_ != SC_OK) return pre_;             \
    return debug_post(call, stream);            \
  } while (0)
#else
#define SC_DEBUG_CALL(d, stream, call) return call
#endif

extern "C" {

const char* sc_status_str(sc_status s) {
  switch (s) {
    case SC_OK: return "ok";
    case SC_EINVAL: return "invalid argument";
    case SC_EUNSUPPORTED: return "unsupported argument";
    case SC_EWORKSPACE: return "workspace missing or too small";
    case SC_EHIP: return "HIP runtime error";
    case SC_ENOSCRATCH: return "problem needs more workspace than the no-allocation entry point's static buffer holds";
    default: return "unknown status";
  }
}

size_t sc_score_partials_size(const sc_attn_desc* d) {
  if (check_desc(d) != SC_OK) return 0;
  const AttnGeom geo = sc::attn_geom(d->n, d->window, d->G);
  return sizeof(float) * sc::partials_floats(d->B, d->H, d->n, geo, d->G);
}

size_t sc_band_probs_size(const sc_attn_desc* d) {
  if (check_desc(d) != SC_OK) return 0;
  const AttnGeom geo = sc::attn_geom(d->n, d->window, d->G);
  return sizeof(float) * sc::band_probs_floats(d->B, d->H, d->n, geo, d->G);
}

size_t sc_window_attention_workspace_size(const sc_attn_desc* d) {
  if (check_desc(d) != SC_OK) return 0;
  return attn_ws_size(d);
}

}  // extern "C"

namespace {

sc_status window_attention(const sc_attn_desc* d, const void* q, const void* k, const void* v, void* out, float* lse,
                           float* score_partials, float* band_probs, void* workspace, size_t ws_bytes, void* stream,
                           bool no_profile) {
  sc_status st = check_desc(d);
  if (st != SC_OK) return st;
  if (!q || !k || !v || !out) return SC_EINVAL;
  if (d->causal && band_probs) return SC_EUNSUPPORTED;
  const size_t tb = tensor_bytes(d);
  if (overlaps(out, tb, q, tb) || overlaps(out, tb, k, tb) || overlaps(out, tb, v, tb)) return SC_EINVAL;
  const size_t lse_b = sizeof(float) * d->B * d->H * d->n;
  if (lse && (overlaps(lse, lse_b, out, tb) || overlaps(lse, lse_b, q, tb) || overlaps(lse, lse_b, k, tb) ||
              overlaps(lse, lse_b, v, tb)))
    return SC_EINVAL;
  const size_t need = attn_ws_size(d);
  if (!workspace || ws_bytes < need) return SC_EWORKSPACE;
  const size_t sp_b = sc_score_partials_size(d), bp_b = sc_band_probs_size(d);
  if (score_partials && (overlaps(score_partials, sp_b, out, tb) || overlaps(score_partials, sp_b, workspace, need)))
    return SC_EINVAL;
  if (band_probs && (overlaps(band_probs, bp_b, out, tb) || overlaps(band_probs, bp_b, score_partials, sp_b) ||
                     overlaps(band_probs, bp_b, workspace, need)))
    return SC_EINVAL;
  const AttnGeom geo = sc::attn_geom(d->n, d->window, d->G);
  AttnArgs a = make_attn_args(d, geo);
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.lse = lse;
  a.no_profile = no_profile ? 1 : 0;
  Carver c(workspace);
  carve_attn_ws(a, c);
  set_partials(a, score_partials);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (band_probs) {
    a.bp_band = band_probs;
    a.bp_gcol = band_probs + (size_t)d->B * d->H * d->n * geo.bw;
    a.bp_grow = a.bp_gcol + (size_t)d->B * d->H * d->n * d->G;
    if (sc::launch_fill_zero(band_probs, bp_b, s) != hipSuccess) return SC_EHIP;
  }
  return sc::launch_window_attention(d->dtype, a, s) == hipSuccess ? SC_OK : SC_EHIP;
}

}  // namespace

// ------------------------------------------- no-allocation window attention
// Workspace of sc_window_attention_noalloc: a fixed device array that every
// GPU the library runs on holds until the process ends.  In host code its name
// is only a stand-in for the symbol; the device address comes from
// hipGetSymbolAddress, once per device (with that device current), and only
// that address is handed to the kernels.
static __device__ __align__(256) unsigned char scratch[SC_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Device address of `scratch` on the current device (which the caller's
// stream must belong to).
sc_status scratch_address(void* stream, void** addr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return SC_EHIP;
  if (dev >= kMaxDevices) return SC_EUNSUPPORTED;
  hipDevice_t sdev = -1;
  if (hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev) != hipSuccess) return SC_EHIP;
  if (sdev != dev) return SC_EINVAL;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SC_EHIP;
    g_scratch_dev[dev] = p;
  }
  *addr = g_scratch_dev[dev];
  return SC_OK;
}
}  // namespace

extern "C" {

static sc_status sc_window_attention_impl(const sc_attn_desc* d, const void* q, const void* k, const void* v, void* out,
                                          float* lse, float* score_partials, float* band_probs, void* workspace,
                                          size_t ws_bytes, void* stream) {
  return window_attention(d, q, k, v, out, lse, score_partials, band_probs, workspace, ws_bytes, stream, false);
}

sc_status sc_window_attention(const sc_attn_desc* d, const void* q, const void* k, const void* v, void* out, float* lse,
                              float* score_partials, float* band_probs, void* workspace, size_t ws_bytes,
                              void* stream) {
  SC_DEBUG_CALL(d, stream,
                sc_window_attention_impl(d, q, k, v, out, lse, score_partials, band_probs, workspace, ws_bytes,
                                         stream));
}

static sc_status sc_window_attention_noalloc_impl(const sc_attn_desc* d, const void* q, const void* k, const void* v,
                                                  void* out, float* lse, float* score_partials, float* band_probs,
                                                  void* stream) {
  sc_status st = check_desc(d);
  if (st != SC_OK) return st;
  if (attn_ws_size(d) > (size_t)SC_NOALLOC_SCRATCH_BYTES) return SC_ENOSCRATCH;
  void* ws = nullptr;
  st = scratch_address(stream, &ws);
  if (st != SC_OK) return st;
  return window_attention(d, q, k, v, out, lse, score_partials, band_probs, ws, (size_t)SC_NOALLOC_SCRATCH_BYTES,
                          stream, true);
}

sc_status sc_window_attention_noalloc(const sc_attn_desc* d, const void* q, const void* k, const void* v, void* out,
                                      float* lse, float* score_partials, float* band_probs, void* stream) {
  SC_DEBUG_CALL(d, stream,
                sc_window_attention_noalloc_impl(d, q, k, v, out, lse, score_partials, band_probs, stream));
}

size_t sc_ltp_score_workspace_size(const sc_attn_desc* d, int32_t mode) {
  // the band layout is first reduced to per-row-block partial sums, then to
  // the partials of the fused path
  if (mode != SC_SCORE_FROM_BAND_PROBS || check_desc(d) != SC_OK) return 0;
  return sc_score_partials_size(d) + sizeof(float) * sc::band_parts_floats(d->B, d->H, d->n, d->window, d->G);
}

static sc_status sc_ltp_score_impl(const sc_attn_desc* d, int32_t mode, const float* src, float* scores,
                                   void* workspace, size_t ws_bytes, void* stream) {
  sc_status st = check_desc(d);
  if (st != SC_OK) return st;
  if (!src || !scores) return SC_EINVAL;
  if (mode != SC_SCORE_FROM_PARTIALS && mode != SC_SCORE_FROM_BAND_PROBS) return SC_EINVAL;
  const size_t src_b = mode == SC_SCORE_FROM_PARTIALS ? sc_score_partials_size(d) : sc_band_probs_size(d);
  const size_t sc_b = sizeof(float) * d->B * d->n;
  if (overlaps(src, src_b, scores, sc_b)) return SC_EINVAL;
  const size_t need = sc_ltp_score_workspace_size(d, mode);
  if (need > 0) {
    if (!workspace || ws_bytes < need) return SC_EWORKSPACE;
    if (overlaps(workspace, need, src, src_b) || overlaps(workspace, need, scores, sc_b)) return SC_EINVAL;
  }
  const AttnGeom geo = sc::attn_geom(d->n, d->window, d->G);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = mode == SC_SCORE_FROM_PARTIALS
                     ? sc::launch_score_from_partials(src, d->valid_len, d->global_pos, d->B, d->n, d->H, d->G, geo,
                                                      scores, s)
                     : sc::launch_score_from_band(src, d->valid_len, d->global_pos, d->B, d->n, d->H, d->G, geo,
                                                  static_cast<float*>(workspace),
                                                  static_cast<float*>(workspace) + sc_score_partials_size(d) / 4,
                                                  scores, s);
  return e == hipSuccess ? SC_OK : SC_EHIP;
}

sc_status sc_ltp_score(const sc_attn_desc* d, int32_t mode, const float* src, float* scores, void* workspace,
                       size_t ws_bytes, void* stream) {
  SC_DEBUG_CALL(d, stream,
                sc_ltp_score_impl(d, mode, src, scores, workspace, ws_bytes, stream));
}

size_t sc_ltp_prune_compact_workspace_size(const sc_attn_desc* d) {
  if (check_desc(d) != SC_OK) return 0;
  return sizeof(int32_t) * (size_t)d->B * d->n;
}

namespace {

// Threshold (topk = 0) or top-k (topk = 1) selection, then the gather.
sc_status prune_compact(const sc_attn_desc* d, const float* scores, float threshold, int topk, float keep_ratio,
                        int32_t keep_global, int32_t n_tensors, const void* const* src, void* const* dst,
                        const int64_t* row_bytes, int32_t* keep_idx, int32_t* new_len, int32_t* new_global_pos,
                        const int32_t* orig_idx_in, int32_t* orig_idx_out, void* workspace, size_t ws_bytes,
                        void* stream) {
  sc_status st = check_desc(d);
  if (st != SC_OK) return st;
  if (!scores || !keep_idx || !new_len) return SC_EINVAL;
  if (n_tensors < 0 || n_tensors > 4) return SC_EINVAL;
  if (n_tensors > 0 && (!src || !dst || !row_bytes)) return SC_EINVAL;
  const size_t need = sc_ltp_prune_compact_workspace_size(d);
  if (!workspace || ws_bytes < need) return SC_EWORKSPACE;
  const size_t bn = (size_t)d->B * d->n;
  const size_t i32b = sizeof(int32_t) * bn;
  sc::GatherArgs ga;
  std::memset(&ga, 0, sizeof(ga));
  ga.B = d->B;
  ga.n = d->n;
  ga.nt = n_tensors;
  for (int t = 0; t < n_tensors; ++t) {
    if (!src[t] || !dst[t] || row_bytes[t] <= 0) return SC_EINVAL;
    const size_t tb = bn * (size_t)row_bytes[t];
    if (overlaps(src[t], tb, dst[t], tb)) return SC_EINVAL;
    if (overlaps(dst[t], tb, keep_idx, i32b) || overlaps(dst[t], tb, workspace, need)) return SC_EINVAL;
    ga.src[t] = static_cast<const char*>(src[t]);
    ga.dst[t] = static_cast<char*>(dst[t]);
    ga.row_bytes[t] = row_bytes[t];
  }
  if (orig_idx_in && orig_idx_out && overlaps(orig_idx_in, i32b, orig_idx_out, i32b)) return SC_EINVAL;
  if (overlaps(keep_idx, i32b, workspace, need) || overlaps(keep_idx, i32b, scores, sizeof(float) * bn))
    return SC_EINVAL;
  sc::PruneArgs p;
  p.scores = scores;
  p.valid_len = d->valid_len;
  p.gpos = d->G > 0 ? d->global_pos : nullptr;
  p.B = d->B;
  p.n = d->n;
  p.G = d->G;
  p.threshold = threshold;
  p.keep_global = keep_global ? 1 : 0;
  p.topk = topk;
  p.keep_ratio = keep_ratio;
  p.keep_idx = keep_idx;
  p.new_len = new_len;
  p.new_gpos = new_global_pos;
  p.orig_in = orig_idx_in;
  p.orig_out = orig_idx_out;
  p.new_index = static_cast<int*>(workspace);
  p.len_copy = nullptr;
  hipStream_t s = static_cast<hipStream_t>(stream);
  ga.keep_idx = keep_idx;
  ga.new_len = new_len;
  return sc::launch_prune_gather(p, ga, s) == hipSuccess ? SC_OK : SC_EHIP;
}

}  // namespace

static sc_status sc_ltp_prune_compact_impl(const sc_attn_desc* d, const float* scores, float threshold,
                                           int32_t keep_global, int32_t n_tensors, const void* const* src,
                                           void* const* dst, const int64_t* row_bytes, int32_t* keep_idx,
                                           int32_t* new_len, int32_t* new_global_pos, const int32_t* orig_idx_in,
                                           int32_t* orig_idx_out, void* workspace, size_t ws_bytes, void* stream) {
  return prune_compact(d, scores, threshold, 0, 0.f, keep_global, n_tensors, src, dst, row_bytes, keep_idx, new_len,
                       new_global_pos, orig_idx_in, orig_idx_out, workspace, ws_bytes, stream);
}

sc_status sc_ltp_prune_compact(const sc_attn_desc* d, const float* scores, float threshold, int32_t keep_global,
                               int32_t n_tensors, const void* const* src, void* const* dst, const int64_t* row_bytes,
                               int32_t* keep_idx, int32_t* new_len, int32_t* new_global_pos, const int32_t* orig_idx_in,
                               int32_t* orig_idx_out, void* workspace, size_t ws_bytes, void* stream) {
  SC_DEBUG_CALL(d, stream,
                sc_ltp_prune_compact_impl(d, scores, threshold, keep_global, n_tensors, src, dst, row_bytes,
                                          keep_idx, new_len, new_global_pos, orig_idx_in, orig_idx_out, workspace,
                                          ws_bytes, stream));
}

static sc_status sc_topk_prune_compact_impl(const sc_attn_desc* d, const float* scores, float keep_ratio,
                                            int32_t keep_global, int32_t n_tensors, const void* const* src,
                                            void* const* dst, const int64_t* row_bytes, int32_t* keep_idx,
                                            int32_t* new_len, int32_t* new_global_pos, const int32_t* orig_idx_in,
                                            int32_t* orig_idx_out, void* workspace, size_t ws_bytes, void* stream) {
  if (!(keep_ratio >= 0.f && keep_ratio <= 1.f)) return SC_EINVAL;  // also rejects NaN
  return prune_compact(d, scores, 0.f, 1, keep_ratio, keep_global, n_tensors, src, dst, row_bytes, keep_idx, new_len,
                       new_global_pos, orig_idx_in, orig_idx_out, workspace, ws_bytes, stream);
}

sc_status sc_topk_prune_compact(const sc_attn_desc* d, const float* scores, float keep_ratio, int32_t keep_global,
                                int32_t n_tensors, const void* const* src, void* const* dst, const int64_t* row_bytes,
                                int32_t* keep_idx, int32_t* new_len, int32_t* new_global_pos,
                                const int32_t* orig_idx_in, int32_t* orig_idx_out, void* workspace, size_t ws_bytes,
                                void* stream) {
  SC_DEBUG_CALL(d, stream,
                sc_topk_prune_compact_impl(d, scores, keep_ratio, keep_global, n_tensors, src, dst, row_bytes,
                                           keep_idx, new_len, new_global_pos, orig_idx_in, orig_idx_out, workspace,
                                           ws_bytes, stream));
}

// ------------------------------------------------------------ soft pruning --
namespace {

bool soft_desc_ok(const sc_attn_desc* d, sc_status* st) {
  *st = check_desc(d);
  if (*st != SC_OK) return false;
  if (d->dtype != SC_BF16 || d->causal) {
    *st = SC_EUNSUPPORTED;
    return false;
  }
  return true;
}

// Workspace pieces of the backward (pointers null when base is null).
size_t carve_soft(const sc_attn_desc* d, void* base, sc::SoftArgs* a) {
  Carver c(base);
  const size_t bn = (size_t)d->B * d->n, bhn = bn * d->H;
  const int nsp = (d->n + sc::kBwdSpan - 1) / sc::kBwdSpan, Gp = ((d->G + 63) / 64) * 64;
  const size_t part = (size_t)d->B * d->H * nsp * Gp;
  a->dO = c.take<__bf16>(bhn * 64);
  a->Dq = c.take<float>(bhn);
  a->gk = c.take<float>(bn);
  a->dsv = c.take<float>((bn + 3) / 4);
  a->gpg = c.take<float>(part > 0 ? part : 1);
  a->gdq = c.take<float>(part > 0 ? part * 64 : 1);
  a->gdk = c.take<float>(part > 0 ? part * 64 : 1);
  a->gdv = c.take<float>(part > 0 ? part * 64 : 1);
  a->nsp = nsp;
  a->Gp = Gp;
  return c.off;
}

sc::SoftArgs soft_args(const sc_attn_desc* d) {
  sc::SoftArgs a;
  std::memset(&a, 0, sizeof(a));
  a.B = d->B;
  a.n = d->n;
  a.H = d->H;
  a.G = d->G;
  a.r = d->window / 2 < d->n ? d->window / 2 : d->n;
  a.valid_len = d->valid_len;
  a.gpos = d->G > 0 ? d->global_pos : nullptr;
  a.alpha = d->softmax_scale;
  a.c2 = d->softmax_scale * 1.4426950408889634f;
  return a;
}

}  // namespace

static sc_status sc_ltp_soft_mask_impl(const sc_attn_desc* d, const float* scores, float theta, float temperature,
                                       int32_t keep_global, const void* out, float* mask, void* y, void* stream) {
  sc_status st;
  if (!soft_desc_ok(d, &st)) return st;
  if (!scores || !out || !mask || !y) return SC_EINVAL;
  if (!std::isfinite(theta) || !(temperature > 0.f) || !std::isfinite(temperature)) return SC_EINVAL;
  const size_t tb = tensor_bytes(d), sb = sizeof(float) * (size_t)d->B * d->n;
  if (overlaps(y, tb, out, tb) || overlaps(y, tb, scores, sb) || overlaps(y, tb, mask, sb) ||
      overlaps(mask, sb, scores, sb) || overlaps(mask, sb, out, tb))
    return SC_EINVAL;
  sc::SoftArgs a = soft_args(d);
  a.scores = scores;
  a.o = static_cast<const __bf16*>(out);
  a.mask_out = mask;
  a.y = static_cast<__bf16*>(y);
  a.theta = theta;
  a.inv_t = 1.f / temperature;
  a.keep_global = keep_global ? 1 : 0;
  return sc::launch_soft_mask(a, static_cast<hipStream_t>(stream)) == hipSuccess ? SC_OK : SC_EHIP;
}

sc_status sc_ltp_soft_mask(const sc_attn_desc* d, const float* scores, float theta, float temperature,
                           int32_t keep_global, const void* out, float* mask, void* y, void* stream) {
  SC_DEBUG_CALL(d, stream,
                sc_ltp_soft_mask_impl(d, scores, theta, temperature, keep_global, out, mask, y, stream));
}

size_t sc_ltp_soft_backward_workspace_size(const sc_attn_desc* d) {
  sc_status st;
  if (!soft_desc_ok(d, &st)) return 0;
  sc::SoftArgs a;
  return carve_soft(d, nullptr, &a);
}

static sc_status sc_ltp_soft_backward_impl(const sc_attn_desc* d, const void* q, const void* k, const void* v,
                                           const void* out, const float* lse, const float* mask, float temperature,
                                           int32_t keep_global, const void* dy, const float* dmask, void* dq, void* dk,
                                           void* dv, float* dtheta, void* workspace, size_t ws_bytes, void* stream) {
  sc_status st;
  if (!soft_desc_ok(d, &st)) return st;
  if (!q || !k || !v || !out || !lse || !mask || !dy || !dq || !dk || !dv || !dtheta) return SC_EINVAL;
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return SC_EINVAL;
  const size_t need = sc_ltp_soft_backward_workspace_size(d);
  if (!workspace || ws_bytes < need) return SC_EWORKSPACE;
  const size_t tb = tensor_bytes(d), sb = sizeof(float) * (size_t)d->B * d->n;
  const size_t lb = sizeof(float) * (size_t)d->B * d->H * d->n;
  const void* ins[] = {q, k, v, out, dy};
  const void* outs[] = {dq, dk, dv};
  for (const void* o : outs) {
    for (const void* i : ins)
      if (overlaps(o, tb, i, tb)) return SC_EINVAL;
    if (overlaps(o, tb, lse, lb) || overlaps(o, tb, mask, sb) || overlaps(o, tb, workspace, need) ||
        overlaps(o, tb, dtheta, sizeof(float)) || (dmask && overlaps(o, tb, dmask, sb)))
      return SC_EINVAL;
  }
  if (overlaps(dq, tb, dk, tb) || overlaps(dq, tb, dv, tb) || overlaps(dk, tb, dv, tb)) return SC_EINVAL;
  for (const void* i : ins)
    if (overlaps(workspace, need, i, tb)) return SC_EINVAL;
  if (overlaps(workspace, need, lse, lb) || overlaps(workspace, need, mask, sb) ||
      overlaps(workspace, need, dtheta, sizeof(float)) || (dmask && overlaps(workspace, need, dmask, sb)))
    return SC_EINVAL;
  sc::SoftArgs a = soft_args(d);
  carve_soft(d, workspace, &a);
  a.q = static_cast<const __bf16*>(q);
  a.k = static_cast<const __bf16*>(k);
  a.v = static_cast<const __bf16*>(v);
  a.o = static_cast<const __bf16*>(out);
  a.dy = static_cast<const __bf16*>(dy);
  a.lse = lse;
  a.mask = mask;
  a.dmask = dmask;
  a.dq = static_cast<__bf16*>(dq);
  a.dk = static_cast<__bf16*>(dk);
  a.dv = static_cast<__bf16*>(dv);
  a.dtheta = dtheta;
  a.inv_t = 1.f / temperature;
  a.keep_global = keep_global ? 1 : 0;
  return sc::launch_soft_backward(a, static_cast<hipStream_t>(stream)) == hipSuccess ? SC_OK : SC_EHIP;
}

sc_status sc_ltp_soft_backward(const sc_attn_desc* d, const void* q, const void* k, const void* v, const void* out,
                               const float* lse, const float* mask, float temperature, int32_t keep_global,
                               const void* dy, const float* dmask, void* dq, void* dk, void* dv, float* dtheta,
                               void* workspace, size_t ws_bytes, void* stream) {
  SC_DEBUG_CALL(d, stream,
                sc_ltp_soft_backward_impl(d, q, k, v, out, lse, mask, temperature, keep_global, dy, dmask, dq, dk,
                                          dv, dtheta, workspace, ws_bytes, stream));
}

// ------------------------------------------------------------------ stack --
namespace {

struct StackWs {
  __bf16 *qkv, *o, *oc, *xc, *xa, *xb;
  __bf16 *x1, *h;  // feed-forward block: attention sub-layer output, hidden activations
  float *t, *scores, *partials;
  float* split;  // slabs of the split reductions of the output and second feed-forward products
  int *len_a, *len_b, *gp_a, *gp_b, *orig_a, *orig_b, *keep_idx, *new_index;
  AttnArgs attn;
};

// Workspace of the stack; F = feed-forward width (0: attention-only layers).
size_t carve_stack(const sc_attn_desc* d, int F, void* base, StackWs* ws) {
  const AttnGeom geo = sc::attn_geom(d->n, d->window, d->G);
  const size_t D = (size_t)d->H * d->d, bn = (size_t)d->B * d->n, G = (size_t)d->G;
  Carver c(base);
  StackWs w;
  w.qkv = c.take<__bf16>(bn * 3 * D);
  w.o = c.take<__bf16>(bn * D);
  w.oc = c.take<__bf16>(bn * D);
  w.xc = c.take<__bf16>(bn * D);
  w.xa = c.take<__bf16>(bn * D);
  w.xb = c.take<__bf16>(bn * D);
  w.x1 = F > 0 ? c.take<__bf16>(bn * D) : nullptr;
  w.h = F > 0 ? c.take<__bf16>(bn * (size_t)F) : nullptr;
  w.t = c.take<float>(bn * D);
  w.split = c.take<float>((size_t)sc::kGemmSplitRows * D);
  w.scores = c.take<float>(bn);
  w.partials = c.take<float>(sc::partials_floats(d->B, d->H, d->n, geo, d->G));
  w.len_a = c.take<int>(d->B);
  w.len_b = c.take<int>(d->B);
  w.gp_a = c.take<int>(G > 0 ? d->B * G : 1);
  w.gp_b = c.take<int>(G > 0 ? d->B * G : 1);
  w.orig_a = c.take<int>(bn);
  w.orig_b = c.take<int>(bn);
  w.keep_idx = c.take<int>(bn);
  w.new_index = c.take<int>(bn);
  // the attention workspace and the partials do not depend on the window
  w.attn = make_attn_args(d, geo);
  carve_attn_ws(w.attn, c);
  if (ws) *ws = w;
  return c.off;
}

// The window-dependent geometry of the attention arguments.
void set_window(AttnArgs& a, int n, int window, int G) {
  const AttnGeom geo = sc::attn_geom(n, window, G);
  a.r = geo.r;
  a.nqb = geo.nqb;
  a.rwp = geo.rwp;
  a.rb = geo.rb;
  a.bw = geo.bw;
  a.nkb = geo.nkb;
}

// Layers of the stack: windows (host, NULL = desc->window for every layer);
// W1 / W2 NULL = attention-only layers, else feed-forward width F.
sc_status run_stack(const sc_attn_desc* d, int32_t n_layers, const int32_t* windows, const void* x_in,
                    const void* const* Wqkv, const void* const* Wo, const void* const* W1, const void* const* W2,
                    int32_t F, const float* thresholds, int32_t keep_global, float ln_eps, void* x_out,
                    int32_t* final_len, int32_t* orig_idx, int32_t* kept_per_layer, void* workspace, size_t ws_bytes,
                    void* stream) {
  sc_status st = check_desc(d);
  if (st != SC_OK) return st;
  if (d->dtype != SC_BF16 || d->causal) return SC_EUNSUPPORTED;
  if ((long long)d->H * d->d > 2048) return SC_EUNSUPPORTED;
  if ((long long)d->n * 3 * d->H * d->d * 2 >= (1LL << 32)) return SC_EUNSUPPORTED;  // fused q|k|v rows
  if (d->B > sc::kPackMaxB) return SC_EUNSUPPORTED;  // row packing of the products and LayerNorms
  if (n_layers < 1 || !x_in || !Wqkv || !Wo || !thresholds || !x_out || !final_len) return SC_EINVAL;
  if (!(ln_eps > 0.f) || !std::isfinite(ln_eps)) return SC_EINVAL;
  const bool ffn = W1 != nullptr;
  if (ffn && (!W2 || F <= 0 || F % 8 != 0)) return SC_EINVAL;
  for (int l = 0; l < n_layers; ++l) {
    if (!Wqkv[l] || !Wo[l]) return SC_EINVAL;
    if (ffn && (!W1[l] || !W2[l])) return SC_EINVAL;
    if (windows && windows[l] < 0) return SC_EINVAL;
  }
  const size_t need = carve_stack(d, ffn ? F : 0, nullptr, nullptr);
  if (!workspace || ws_bytes < need) return SC_EWORKSPACE;
  const size_t D = (size_t)d->H * d->d, bn = (size_t)d->B * d->n, xb = bn * D * 2;
  if (overlaps(x_out, xb, x_in, xb) || overlaps(x_out, xb, workspace, need) || overlaps(x_in, xb, workspace, need))
    return SC_EINVAL;
  StackWs w;
  carve_stack(d, ffn ? F : 0, workspace, &w);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int B = d->B, n = d->n, H = d->H, G = d->G, Di = (int)D;
  bool ok = true;
  auto chk = [&](hipError_t e) { ok = ok && e == hipSuccess; };
  int *len_cur = w.len_a, *len_nxt = w.len_b, *gp_cur = w.gp_a, *gp_nxt = w.gp_b;
  int *orig_cur = w.orig_a, *orig_nxt = w.orig_b;
  chk(sc::launch_copy_i32(d->valid_len, len_cur, B, s));
  if (G > 0) chk(sc::launch_copy_i32(d->global_pos, gp_cur, (long long)B * G, s));
  chk(sc::launch_iota_orig(d->valid_len, orig_cur, B, n, s));
  const __bf16* cur = static_cast<const __bf16*>(x_in);
  for (int l = 0; l < n_layers && ok; ++l) {
    const int window = windows ? windows[l] : d->window;
    __bf16* nxt = (l == n_layers - 1) ? static_cast<__bf16*>(x_out) : ((l & 1) ? w.xb : w.xa);
    // a1: qkv projection of the surviving rows
    chk(sc::launch_gemm_bf16(cur, Wqkv[l], w.qkv, sc::kGemmBf16, B, n, Di, 3 * Di, len_cur, nullptr, s));
    // a2-a5: sparse attention reading q|k|v out of the fused projection
    AttnArgs a = w.attn;
    set_window(a, n, window, G);
    a.q = w.qkv;
    a.k = w.qkv + D;
    a.v = w.qkv + 2 * D;
    a.ld_in = 3 * (long long)D;
    a.bs_in = a.ld_in * n;
    a.out = w.o;
    a.ld_out = (long long)D;
    a.bs_out = a.ld_out * n;
    a.lse = nullptr;
    a.skip_pad_out = 1;  // O is read only at the kept rows (the gather below)
    a.span_major = l > 0 ? 1 : 0;  // pruned layers: short sequences in an n-row batch (n up to 4096: always)
    a.valid_len = len_cur;
    a.gpos = G > 0 ? gp_cur : nullptr;
    set_partials(a, w.partials);
    chk(sc::launch_window_attention(SC_BF16, a, s));
    // a6: importance scores
    const AttnGeom geo = sc::attn_geom(n, window, G);
    chk(sc::launch_score_from_partials(w.partials, len_cur, G > 0 ? gp_cur : nullptr, B, n, H, G, geo, w.scores, s));
    // a7-a8: threshold, scan, gather of O and of the residual input
    sc::PruneArgs p;
    p.scores = w.scores;
    p.valid_len = len_cur;
    p.gpos = G > 0 ? gp_cur : nullptr;
    p.B = B;
    p.n = n;
    p.G = G;
    p.threshold = thresholds[l];
    p.keep_global = keep_global ? 1 : 0;
    p.topk = 0;
    p.keep_ratio = 0.f;
    p.keep_idx = w.keep_idx;
    p.new_len = len_nxt;
    p.new_gpos = G > 0 ? gp_nxt : nullptr;
    p.orig_in = orig_cur;
    p.orig_out = orig_nxt;
    p.new_index = w.new_index;
    p.len_copy = kept_per_layer ? kept_per_layer + (size_t)l * B : nullptr;
    sc::GatherArgs ga;
    std::memset(&ga, 0, sizeof(ga));
    ga.B = B;
    ga.n = n;
    ga.nt = 2;
    ga.src[0] = reinterpret_cast<const char*>(w.o);
    ga.dst[0] = reinterpret_cast<char*>(w.oc);
    ga.src[1] = reinterpret_cast<const char*>(cur);
    ga.dst[1] = reinterpret_cast<char*>(w.xc);
    ga.row_bytes[0] = ga.row_bytes[1] = (long long)D * 2;
    ga.keep_idx = w.keep_idx;
    ga.new_len = len_nxt;
    chk(sc::launch_prune_gather(p, ga, s));
    // a9: output projection, residual, LayerNorm on the survivors
    chk(sc::launch_gemm_bf16(w.oc, Wo[l], w.t, sc::kGemmF32, B, n, Di, Di, len_nxt, w.split, s));
    if (!ffn) {
      chk(sc::launch_residual_layernorm(w.xc, w.t, nxt, B, n, Di, ln_eps, len_nxt, w.split, Di, s));
    } else {
      // feed-forward block: h = GELU(x1 . W1), then LayerNorm(x1 + h . W2)
      chk(sc::launch_residual_layernorm(w.xc, w.t, w.x1, B, n, Di, ln_eps, len_nxt, w.split, Di, s));
      chk(sc::launch_gemm_bf16(w.x1, W1[l], w.h, sc::kGemmGeluBf16, B, n, Di, F, len_nxt, nullptr, s));
      chk(sc::launch_gemm_bf16(w.h, W2[l], w.t, sc::kGemmF32, B, n, F, Di, len_nxt, w.split, s));
      chk(sc::launch_residual_layernorm(w.x1, w.t, nxt, B, n, Di, ln_eps, len_nxt, w.split, F, s));
    }
    cur = nxt;
    int* tmp;
    tmp = len_cur; len_cur = len_nxt; len_nxt = tmp;
    tmp = gp_cur; gp_cur = gp_nxt; gp_nxt = tmp;
    tmp = orig_cur; orig_cur = orig_nxt; orig_nxt = tmp;
  }
  chk(sc::launch_copy_i32(len_cur, final_len, B, s));
  if (orig_idx) chk(sc::launch_copy_i32(orig_cur, orig_idx, (long long)bn, s));
  return ok ? SC_OK : SC_EHIP;
}

}  // namespace

size_t sc_encoder_attn_stack_workspace_size(const sc_attn_desc* d, int32_t n_layers) {
  if (check_desc(d) != SC_OK || n_layers < 1) return 0;
  return carve_stack(d, 0, nullptr, nullptr);
}

static sc_status sc_encoder_attn_stack_impl(const sc_attn_desc* d, int32_t n_layers, const void* x_in,
                                            const void* const* Wqkv, const void* const* Wo, const float* thresholds,
                                            int32_t keep_global, float ln_eps, void* x_out, int32_t* final_len,
                                            int32_t* orig_idx, int32_t* kept_per_layer, void* workspace,
                                            size_t ws_bytes, void* stream) {
  return run_stack(d, n_layers, nullptr, x_in, Wqkv, Wo, nullptr, nullptr, 0, thresholds, keep_global, ln_eps, x_out,
                   final_len, orig_idx, kept_per_layer, workspace, ws_bytes, stream);
}

sc_status sc_encoder_attn_stack(const sc_attn_desc* d, int32_t n_layers, const void* x_in, const void* const* Wqkv,
                                const void* const* Wo, const float* thresholds, int32_t keep_global, float ln_eps,
                                void* x_out, int32_t* final_len, int32_t* orig_idx, int32_t* kept_per_layer,
                                void* workspace, size_t ws_bytes, void* stream) {
  SC_DEBUG_CALL(d, stream,
                sc_encoder_attn_stack_impl(d, n_layers, x_in, Wqkv, Wo, thresholds, keep_global, ln_eps, x_out,
                                           final_len, orig_idx, kept_per_layer, workspace, ws_bytes, stream));
}

size_t sc_encoder_stack_workspace_size(const sc_attn_desc* d, int32_t n_layers, int32_t ffn_dim) {
  if (check_desc(d) != SC_OK || n_layers < 1 || ffn_dim <= 0) return 0;
  return carve_stack(d, ffn_dim, nullptr, nullptr);
}

static sc_status sc_encoder_stack_impl(const sc_attn_desc* d, int32_t n_layers, const int32_t* windows,
                                       const void* x_in, const void* const* Wqkv, const void* const* Wo,
                                       const void* const* W1, const void* const* W2, int32_t ffn_dim,
                                       const float* thresholds, int32_t keep_global, float ln_eps, void* x_out,
                                       int32_t* final_len, int32_t* orig_idx, int32_t* kept_per_layer, void* workspace,
                                       size_t ws_bytes, void* stream) {
  if (!W1 || !W2) return SC_EINVAL;
  return run_stack(d, n_layers, windows, x_in, Wqkv, Wo, W1, W2, ffn_dim, thresholds, keep_global, ln_eps, x_out,
                   final_len, orig_idx, kept_per_layer, workspace, ws_bytes, stream);
}

sc_status sc_encoder_stack(const sc_attn_desc* d, int32_t n_layers, const int32_t* windows, const void* x_in,
                           const void* const* Wqkv, const void* const* Wo, const void* const* W1, const void* const* W2,
                           int32_t ffn_dim, const float* thresholds, int32_t keep_global, float ln_eps, void* x_out,
                           int32_t* final_len, int32_t* orig_idx, int32_t* kept_per_layer, void* workspace,
                           size_t ws_bytes, void* stream) {
  SC_DEBUG_CALL(d, stream,
                sc_encoder_stack_impl(d, n_layers, windows, x_in, Wqkv, Wo, W1, W2, ffn_dim, thresholds, keep_global,
                                      ln_eps, x_out, final_len, orig_idx, kept_per_layer, workspace, ws_bytes,
                                      stream));
}

sc_status sc_validate_desc(const sc_attn_desc* d, int32_t* err, void* stream) {
  const sc_status st = check_desc(d);
  if (st != SC_OK) return st;
  if (!err) return SC_EINVAL;
  return sc::launch_validate_desc(d->valid_len, d->G > 0 ? d->global_pos : nullptr, d->B, d->n, d->G, err,
                                  static_cast<hipStream_t>(stream)) == hipSuccess
             ? SC_OK
             : SC_EHIP;
}

sc_status sc_profile_window_kernel(int32_t enable) {
  sc::profile_set(enable);
  return SC_OK;
}

sc_status sc_profile_window_kernel_read(double* fwd_ms, double* cols_ms, int64_t capacity, int64_t* calls) {
  if (!calls || capacity < 0 || (capacity > 0 && (!fwd_ms || !cols_ms))) return SC_EINVAL;
  long long cnt = 0;
  if (sc::profile_read(fwd_ms, cols_ms, capacity, &cnt) != 0) return SC_EHIP;
  *calls = cnt;
  return SC_OK;
}

}  // extern "C"
