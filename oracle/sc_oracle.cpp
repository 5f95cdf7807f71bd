// SparseCoder oracle: a plain, slow, obviously correct CPU implementation of
// sliding-window + global-token sparse self-attention with learned-token-pruning
// scores, threshold masking, compaction, and the attention-only encoder stack.
//
// TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call this code:
// only the tests, the smoke check and the benchmark's CPU-baseline leg do.  It
// shares no code, header, table or helper with the HIP library.
//
// Everything is computed in double precision from the exact input values.
// Sources (SparseCoder, arXiv 2310.07109):
//   * sliding-window local attention: token i attends to its neighbours within
//     the window (Sec. 4.2.1, Fig. 4); global ("special") tokens attend to every
//     token and are attended to by every token (Sec. 3.2.1 "Global attention", Fig. 3b-c; Sec. 5.5);
//   * importance score of a token: attention probabilities accumulated down the
//     token's column after the row-wise softmax (Sec. 1, Fig. 1 caption;
//     Sec. 3.3), for sparse attention the band's sub-diagonal plus the global
//     rows and columns (Sec. 5.5); normalised here to the mean over heads and
//     valid queries;
//   * binarised mask: keep iff score > layer threshold, strictly (Sec. 4.2.2,
//     the display equation of step 2); hard pruning removes masked tokens
//     (Sec. 4.2.2 step 3) and later layers see the shorter sequence (Sec. 4.2).
//   * top-k pruning (a rank rule in place of the threshold; not the paper's
//     rule, a variant from the token-pruning families of its Sec. 3.3): the
//     ceil(keep_ratio * C) best-scored candidates per sequence are kept;
//   * soft pruning, the training form (Sec. 4.2.2 step 1): a sigmoid soft mask
//     of the score against the threshold scales the layer output, and its
//     backward gives the gradients of Q, K, V and the threshold.
// Where the paper is silent the readings are: half-width r = floor(w/2) with
// |i - j| <= r inclusive; the softmax scale is an argument; prefix padding
// (tokens >= valid length are neither queries nor keys); scores divided by
// H * valid length so that they sum to one over a sequence; kept tokens stay in
// ascending order; global tokens are kept when keep_global is set.
//
// Pins: tests/test_oracle_pins.py checks every function here against brute
// force, closed forms, library routines and invariants.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <vector>
#ifdef _OPENMP
#include <omp.h>
#endif

namespace {

int set_threads(int nthreads) {
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
  return omp_get_max_threads();
#else
  (void)nthreads;
  return 1;
#endif
}

// Round a double to the nearest bfloat16 value (8 significant bits), ties to
// even, returned as a double.  bfloat16 keeps float32's exponent range.
double round_bf16(double x) {
  if (x == 0.0 || !std::isfinite(x)) return x;
  int e;
  std::frexp(x, &e);  // |x| = f * 2^e, f in [0.5, 1)
  int ulp_exp = e - 8;
  if (ulp_exp < -133) ulp_exp = -133;  // subnormal spacing of float32
  double ulp = std::ldexp(1.0, ulp_exp);
  double q = std::nearbyint(x / ulp) * ulp;  // default rounding mode: ties to even
  const double maxbf = std::ldexp(255.0, 120);  // (2 - 2^-7) * 2^127
  if (std::fabs(q) > maxbf) return std::copysign(std::numeric_limits<double>::infinity(), x);
  return q;
}

// The attention of one (sequence, head).  Rows are tokens; row stride is `ld`
// doubles between consecutive tokens.  Writes out rows (stride ld_out), the
// per-query log-sum-exp, and adds every probability P[q][k] into colsum[k].
// causal: keys after the query are never attended (the decoder variant the
// paper's Sec. 7.2 names as future work).
void attend_one_head(int n, int d, int L, int r, const std::vector<char>& is_global, double alpha,
                     const double* q, const double* k, const double* v, long ld, double* out, long ld_out,
                     double* lse, double* colsum, bool causal) {
  std::vector<int> nbr;
  std::vector<double> s;
  nbr.reserve(n);
  s.reserve(n);
  for (int i = 0; i < n; ++i) {
    double* o = out + (long)i * ld_out;
    if (i >= L) {  // padding query: no token, no output
      for (int c = 0; c < d; ++c) o[c] = 0.0;
      lse[i] = -std::numeric_limits<double>::infinity();
      continue;
    }
    // Allowed(i, j): both valid, and inside the window or either one global;
    // causal: and j <= i.
    nbr.clear();
    const int jend = causal ? std::min(i + 1, L) : L;
    for (int j = 0; j < jend; ++j)
      if (std::abs(i - j) <= r || is_global[i] || is_global[j]) nbr.push_back(j);
    s.assign(nbr.size(), 0.0);
    double m = -std::numeric_limits<double>::infinity();
    for (size_t t = 0; t < nbr.size(); ++t) {
      const double* qi = q + (long)i * ld;
      const double* kj = k + (long)nbr[t] * ld;
      double acc = 0.0;
      for (int c = 0; c < d; ++c) acc += qi[c] * kj[c];
      s[t] = alpha * acc;
      m = std::max(m, s[t]);
    }
    double z = 0.0;
    for (size_t t = 0; t < nbr.size(); ++t) z += std::exp(s[t] - m);
    for (int c = 0; c < d; ++c) o[c] = 0.0;
    for (size_t t = 0; t < nbr.size(); ++t) {
      double p = std::exp(s[t] - m) / z;
      const double* vj = v + (long)nbr[t] * ld;
      for (int c = 0; c < d; ++c) o[c] += p * vj[c];
      colsum[nbr[t]] += p;
    }
    lse[i] = m + std::log(z);
  }
}

std::vector<char> global_flags(int n, int L, int G, const int32_t* gp) {
  std::vector<char> f(n, 0);
  for (int j = 0; j < G; ++j) {
    int p = gp[j];
    if (p >= 0 && p < L) f[p] = 1;
  }
  return f;
}

}  // namespace

extern "C" {

// Exposed so the tests can pin the rounding against a library conversion.
double orc_round_bf16(double x) { return round_bf16(x); }

// Sparse attention over a padded batch, layout [B, n, H, d] (token-major).
//   window: full width w; a query attends to keys with |i - j| <= floor(w/2).
//   global_pos: [B, G]; entries outside [0, valid_len[b]) are unused slots.
//   out [B, n, H, d]; lse [B, H, n] (-inf for padding rows); scores [B, n]:
//   s_k = (1 / (H * L)) * sum_h sum_{q < L} P_h[q][k] for k < L, 0 otherwise.
//   colsum (optional) [B, H, n]: the per-head column sums before averaging.
static int sparse_attention(int B, int n, int H, int d, int window, int G, const int32_t* global_pos,
                            const int32_t* valid_len, double alpha, const double* q, const double* k,
                            const double* v, double* out, double* lse, double* scores, double* colsum, bool causal,
                            int nthreads) {
  if (B < 0 || n < 0 || H <= 0 || d <= 0 || window < 0 || G < 0) return -1;
  set_threads(nthreads);
  const int r = window / 2;
  const long ld = (long)H * d;
  std::vector<double> cs((size_t)B * H * n, 0.0);
#pragma omp parallel for schedule(dynamic, 1)
  for (long bh = 0; bh < (long)B * H; ++bh) {
    int b = (int)(bh / H), h = (int)(bh % H);
    int L = std::min(std::max(valid_len[b], 0), n);
    std::vector<char> g = global_flags(n, L, G, global_pos + (long)b * G);
    long base = (long)b * n * ld + (long)h * d;
    attend_one_head(n, d, L, r, g, alpha, q + base, k + base, v + base, ld, out + base, ld,
                    lse + ((long)b * H + h) * n, cs.data() + ((size_t)b * H + h) * n, causal);
  }
  for (int b = 0; b < B; ++b) {
    int L = std::min(std::max(valid_len[b], 0), n);
    for (int j = 0; j < n; ++j) {
      double acc = 0.0;
      if (j < L)
        for (int h = 0; h < H; ++h) acc += cs[((size_t)b * H + h) * n + j];
      scores[(long)b * n + j] = (j < L) ? acc / ((double)H * L) : 0.0;
    }
  }
  if (colsum) std::memcpy(colsum, cs.data(), cs.size() * sizeof(double));
  return 0;
}

int orc_sparse_attention(int B, int n, int H, int d, int window, int G, const int32_t* global_pos,
                         const int32_t* valid_len, double alpha, const double* q, const double* k,
                         const double* v, double* out, double* lse, double* scores, double* colsum,
                         int nthreads) {
  return sparse_attention(B, n, H, d, window, G, global_pos, valid_len, alpha, q, k, v, out, lse, scores, colsum,
                          false, nthreads);
}

// The causal variant: as orc_sparse_attention with Allowed(i, j) also requiring
// j <= i (band, global rows and global columns alike).
int orc_sparse_attention_causal(int B, int n, int H, int d, int window, int G, const int32_t* global_pos,
                                const int32_t* valid_len, double alpha, const double* q, const double* k,
                                const double* v, double* out, double* lse, double* scores, double* colsum,
                                int nthreads) {
  return sparse_attention(B, n, H, d, window, G, global_pos, valid_len, alpha, q, k, v, out, lse, scores, colsum,
                          true, nthreads);
}

// Compaction of sequence b from its keep flags: kept tokens in ascending order
// (keep_idx, new_len), surviving global tokens renumbered (new_global_pos),
// original positions composed (orig_out).
static void compact_sequence(int b, int n, int L, int G, const int32_t* global_pos, const std::vector<char>& keep,
                             int32_t* keep_idx, int32_t* new_len, int32_t* new_global_pos, const int32_t* orig_in,
                             int32_t* orig_out) {
  std::vector<int> new_index(n, -1);
  int cnt = 0;
  for (int k = 0; k < n; ++k) {
    if (k < L && keep[k]) {
      new_index[k] = cnt;
      keep_idx[(long)b * n + cnt] = k;
      ++cnt;
    }
  }
  for (int j = cnt; j < n; ++j) keep_idx[(long)b * n + j] = -1;
  new_len[b] = cnt;
  int gc = 0;
  for (int j = 0; j < G; ++j) {
    int p = global_pos[(long)b * G + j];
    if (p >= 0 && p < L && new_index[p] >= 0) new_global_pos[(long)b * G + gc++] = new_index[p];
  }
  for (int j = gc; j < G; ++j) new_global_pos[(long)b * G + j] = -1;
  if (orig_out) {
    for (int j = 0; j < n; ++j) {
      int src = keep_idx[(long)b * n + j];
      orig_out[(long)b * n + j] = src < 0 ? -1 : (orig_in ? orig_in[(long)b * n + src] : src);
    }
  }
}

// Binarised mask and hard pruning of one layer.  The decision is taken on the
// float32 score against the float32 threshold: keep iff k < L and (s > theta
// or (keep_global and k is global)).  Kept tokens keep their relative order.
//   keep_idx [B, n]: input index of the j-th kept token, -1 for j >= new_len.
//   new_global_pos [B, G]: surviving global tokens renumbered, -1 padded.
//   orig_in (optional) [B, n] composes into orig_out [B, n] = orig_in[keep_idx]
//   (identity when orig_in is NULL), -1 beyond new_len.
int orc_ltp_prune(int B, int n, int G, const int32_t* global_pos, const int32_t* valid_len,
                  const float* scores, float threshold, int keep_global, int32_t* keep_idx, int32_t* new_len,
                  int32_t* new_global_pos, const int32_t* orig_in, int32_t* orig_out) {
  if (B < 0 || n < 0 || G < 0) return -1;
  for (int b = 0; b < B; ++b) {
    int L = std::min(std::max(valid_len[b], 0), n);
    std::vector<char> g = global_flags(n, L, G, global_pos + (long)b * G);
    std::vector<char> keep(n, 0);
    for (int k = 0; k < L; ++k) keep[k] = scores[(long)b * n + k] > threshold || (keep_global && g[k]);
    compact_sequence(b, n, L, G, global_pos, keep, keep_idx, new_len, new_global_pos, orig_in, orig_out);
  }
  return 0;
}

// Top-k pruning: the same compaction with a rank rule instead of the
// threshold (the paper's Sec. 3.3 places LTP among token-pruning methods, some
// of which keep a fixed fraction of the tokens by rank).  Per sequence the
// candidates are the valid tokens, except the global ones when keep_global is
// set (those are kept anyway); of C candidates the K = ceil(keep_ratio * C)
// (in double, clamped to [0, C]) with the largest float32 scores are kept,
// equal scores going to the lower index.
int orc_topk_prune(int B, int n, int G, const int32_t* global_pos, const int32_t* valid_len, const float* scores,
                   float keep_ratio, int keep_global, int32_t* keep_idx, int32_t* new_len, int32_t* new_global_pos,
                   const int32_t* orig_in, int32_t* orig_out) {
  if (B < 0 || n < 0 || G < 0) return -1;
  for (int b = 0; b < B; ++b) {
    int L = std::min(std::max(valid_len[b], 0), n);
    std::vector<char> g = global_flags(n, L, G, global_pos + (long)b * G);
    std::vector<char> keep(n, 0);
    std::vector<int> cand;
    for (int k = 0; k < L; ++k) {
      if (keep_global && g[k])
        keep[k] = 1;
      else
        cand.push_back(k);
    }
    const long C = (long)cand.size();
    const double prod = (double)keep_ratio * (double)C;
    const long K = prod <= 0.0 ? 0 : (prod >= (double)C ? C : (long)std::ceil(prod));
    // candidates are in index order; a stable sort by descending score keeps
    // that order among equal scores
    const float* s = scores + (long)b * n;
    std::stable_sort(cand.begin(), cand.end(), [&](int x, int y) { return s[x] > s[y]; });
    for (long i = 0; i < K; ++i) keep[cand[i]] = 1;
    compact_sequence(b, n, L, G, global_pos, keep, keep_idx, new_len, new_global_pos, orig_in, orig_out);
  }
  return 0;
}

// Row gather of a padded [B, n, row_bytes] tensor: dst row j = src row
// keep_idx[j] for j < new_len[b]; rows at or beyond new_len are left untouched.
int orc_gather_rows(int B, int n, long row_bytes, const void* src, void* dst, const int32_t* keep_idx,
                    const int32_t* new_len) {
  const char* s = static_cast<const char*>(src);
  char* t = static_cast<char*>(dst);
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < new_len[b]; ++j) {
      int k = keep_idx[(long)b * n + j];
      std::memcpy(t + ((long)b * n + j) * row_bytes, s + ((long)b * n + k) * row_bytes, row_bytes);
    }
  return 0;
}

// LayerNorm of one row (gamma = 1, beta = 0, biased variance, eps inside the
// square root), rounded to bf16.
static void layer_norm_bf16(const std::vector<double>& t, long D, double ln_eps, double* yr) {
  double mean = 0.0;
  for (long c = 0; c < D; ++c) mean += t[c];
  mean /= (double)D;
  double var = 0.0;
  for (long c = 0; c < D; ++c) var += (t[c] - mean) * (t[c] - mean);
  var /= (double)D;
  double inv = 1.0 / std::sqrt(var + ln_eps);
  for (long c = 0; c < D; ++c) yr[c] = round_bf16((t[c] - mean) * inv);
}

// GELU in its exact form, x * Phi(x) with the standard normal CDF Phi.
static double gelu(double v) { return 0.5 * v * (1.0 + std::erf(v / std::sqrt(2.0))); }

// One encoder layer (RoBERTa-shaped, post-LN, no biases; Sec. 4.2, Fig. 5):
//   qkv = bf16(x . Wqkv)            [columns q | k | v, each head-major]
//   O   = bf16(sparse attention(q, k, v))
//   s   = float32(importance scores); keep / compaction as orc_ltp_prune
//   x1  = bf16(LayerNorm(x + O . Wo)) on the kept rows
// and, with a feed-forward block (W1 non-NULL), on the kept rows
//   h   = bf16(GELU(x1 . W1))       W1 [D, F]
//   y   = bf16(LayerNorm(x1 + h . W2))   W2 [F, D]
// else y = x1.  LayerNorm: gamma = 1, beta = 0, biased variance, eps inside
// the square root.  x: [B, n, D] exact bf16 values; Wqkv: [D, 3D] and Wo:
// [D, D] row-major.  Outputs: y [B, n, D] compacted (rows >= new_len zero),
// keep_idx [B, n], new_len [B], new_global_pos [B, G], scores (optional)
// [B, n] float32.
static int encoder_layer(int B, int n, int H, int d, int window, int G, const int32_t* global_pos,
                         const int32_t* valid_len, double alpha, const double* x, const double* Wqkv,
                         const double* Wo, const double* W1, const double* W2, int F, float threshold,
                         int keep_global, double ln_eps, double* y, int32_t* keep_idx, int32_t* new_len,
                         int32_t* new_global_pos, float* scores_out, int nthreads) {
  if (B < 0 || n < 0 || H <= 0 || d <= 0 || (W1 && F <= 0)) return -1;
  set_threads(nthreads);
  const long D = (long)H * d, D3 = 3 * D;
  std::vector<double> qv((size_t)B * n * D), kv((size_t)B * n * D), vv((size_t)B * n * D);
  // a1: projection, double accumulation, bf16 storage.  Padding rows are
  // left zero: the attention never reads them.
#pragma omp parallel for schedule(dynamic, 16)
  for (long row = 0; row < (long)B * n; ++row) {
    if (row % n >= std::min(std::max(valid_len[row / n], 0), n)) {
      for (long j = 0; j < D; ++j) qv[row * D + j] = kv[row * D + j] = vv[row * D + j] = 0.0;
      continue;
    }
    const double* xr = x + row * D;
    std::vector<double> acc(D3, 0.0);
    for (long c = 0; c < D; ++c) {
      double xv = xr[c];
      const double* w = Wqkv + c * D3;
      for (long j = 0; j < D3; ++j) acc[j] += xv * w[j];
    }
    for (long j = 0; j < D; ++j) {
      qv[row * D + j] = round_bf16(acc[j]);
      kv[row * D + j] = round_bf16(acc[D + j]);
      vv[row * D + j] = round_bf16(acc[2 * D + j]);
    }
  }
  std::vector<double> o((size_t)B * n * D), lse((size_t)B * H * n), sc((size_t)B * n);
  int rc = orc_sparse_attention(B, n, H, d, window, G, global_pos, valid_len, alpha, qv.data(), kv.data(),
                                vv.data(), o.data(), lse.data(), sc.data(), nullptr, nthreads);
  if (rc) return rc;
  for (auto& e : o) e = round_bf16(e);
  std::vector<float> s32((size_t)B * n);
  for (size_t i = 0; i < s32.size(); ++i) s32[i] = (float)sc[i];
  if (scores_out) std::memcpy(scores_out, s32.data(), s32.size() * sizeof(float));
  orc_ltp_prune(B, n, G, global_pos, valid_len, s32.data(), threshold, keep_global, keep_idx, new_len,
                new_global_pos, nullptr, nullptr);
  // a9 (and the feed-forward block) on the kept rows.
#pragma omp parallel for schedule(dynamic, 4)
  for (long row = 0; row < (long)B * n; ++row) {
    int b = (int)(row / n), j = (int)(row % n);
    double* yr = y + row * D;
    if (j >= new_len[b]) {
      for (long c = 0; c < D; ++c) yr[c] = 0.0;
      continue;
    }
    long src = (long)b * n + keep_idx[row];
    std::vector<double> t(D);
    for (long c = 0; c < D; ++c) t[c] = x[src * D + c];
    for (long c = 0; c < D; ++c) {
      double ov = o[src * D + c];
      const double* w = Wo + c * D;
      for (long e = 0; e < D; ++e) t[e] += ov * w[e];
    }
    if (!W1) {
      layer_norm_bf16(t, D, ln_eps, yr);
      continue;
    }
    std::vector<double> x1(D), h(F, 0.0);
    layer_norm_bf16(t, D, ln_eps, x1.data());
    for (long c = 0; c < D; ++c) {
      const double* w = W1 + c * (long)F;
      for (long f = 0; f < F; ++f) h[f] += x1[c] * w[f];
    }
    for (long f = 0; f < F; ++f) h[f] = round_bf16(gelu(h[f]));
    for (long c = 0; c < D; ++c) t[c] = x1[c];
    for (long f = 0; f < F; ++f) {
      const double* w = W2 + f * D;
      for (long c = 0; c < D; ++c) t[c] += h[f] * w[c];
    }
    layer_norm_bf16(t, D, ln_eps, yr);
  }
  return 0;
}

// One attention-only layer (no feed-forward block): encoder_layer with W1 = NULL.
int orc_encoder_layer(int B, int n, int H, int d, int window, int G, const int32_t* global_pos,
                      const int32_t* valid_len, double alpha, const double* x, const double* Wqkv,
                      const double* Wo, float threshold, int keep_global, double ln_eps, double* y,
                      int32_t* keep_idx, int32_t* new_len, int32_t* new_global_pos, float* scores_out,
                      int nthreads) {
  return encoder_layer(B, n, H, d, window, G, global_pos, valid_len, alpha, x, Wqkv, Wo, nullptr, nullptr, 0,
                       threshold, keep_global, ln_eps, y, keep_idx, new_len, new_global_pos, scores_out, nthreads);
}

// One full layer with the feed-forward block (W1 [D, F], W2 [F, D]).
int orc_encoder_layer_ffn(int B, int n, int H, int d, int window, int G, const int32_t* global_pos,
                          const int32_t* valid_len, double alpha, const double* x, const double* Wqkv,
                          const double* Wo, const double* W1, const double* W2, int F, float threshold,
                          int keep_global, double ln_eps, double* y, int32_t* keep_idx, int32_t* new_len,
                          int32_t* new_global_pos, float* scores_out, int nthreads) {
  if (!W1 || !W2) return -1;
  return encoder_layer(B, n, H, d, window, G, global_pos, valid_len, alpha, x, Wqkv, Wo, W1, W2, F, threshold,
                       keep_global, ln_eps, y, keep_idx, new_len, new_global_pos, scores_out, nthreads);
}

// The multi-layer stack: the layer applied n_layers times, each layer on the
// previous layer's compacted output and renumbered global tokens.
//   windows [n_layers]: the window of each layer (Sec. 7.1 names the scheme
//   of small windows in lower layers and large ones in higher layers); Wqkv:
//   n_layers consecutive [D, 3D] matrices; Wo: n_layers
//   consecutive [D, D]; W1 / W2 (NULL: attention-only layers): n_layers
//   consecutive [D, F] / [F, D].  thresholds [n_layers]; y [B, n, D];
//   final_len [B]; orig_idx [B, n] (input position of each surviving row, -1
//   beyond final_len); kept_per_layer [n_layers, B] (sequence length after
//   each layer's pruning).
static int encoder_stack(int B, int n, int H, int d, const int32_t* windows, int G, const int32_t* global_pos,
                         const int32_t* valid_len, double alpha, int n_layers, const double* x, const double* Wqkv,
                         const double* Wo, const double* W1, const double* W2, int F, const float* thresholds,
                         int keep_global, double ln_eps, double* y, int32_t* final_len, int32_t* orig_idx,
                         int32_t* kept_per_layer, int nthreads) {
  const long D = (long)H * d;
  std::vector<double> cur(x, x + (size_t)B * n * D), nxt((size_t)B * n * D);
  std::vector<int32_t> len(valid_len, valid_len + B), gp(global_pos, global_pos + (size_t)B * G);
  std::vector<int32_t> orig((size_t)B * n), orig2((size_t)B * n), kidx((size_t)B * n), nl(B), ngp((size_t)B * G);
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < n; ++j) orig[(size_t)b * n + j] = j < len[b] ? j : -1;
  for (int l = 0; l < n_layers; ++l) {
    int rc = encoder_layer(B, n, H, d, windows[l], G, gp.data(), len.data(), alpha, cur.data(),
                           Wqkv + (size_t)l * D * 3 * D, Wo + (size_t)l * D * D,
                           W1 ? W1 + (size_t)l * D * F : nullptr, W2 ? W2 + (size_t)l * F * D : nullptr, F,
                           thresholds[l], keep_global, ln_eps, nxt.data(), kidx.data(), nl.data(), ngp.data(),
                           nullptr, nthreads);
    if (rc) return rc;
    for (int b = 0; b < B; ++b)
      for (int j = 0; j < n; ++j) {
        int s = kidx[(size_t)b * n + j];
        orig2[(size_t)b * n + j] = s < 0 ? -1 : orig[(size_t)b * n + s];
      }
    orig.swap(orig2);
    cur.swap(nxt);
    len = nl;
    gp = ngp;
    for (int b = 0; b < B; ++b) kept_per_layer[(size_t)l * B + b] = len[b];
  }
  std::memcpy(y, cur.data(), cur.size() * sizeof(double));
  std::memcpy(final_len, len.data(), (size_t)B * sizeof(int32_t));
  std::memcpy(orig_idx, orig.data(), orig.size() * sizeof(int32_t));
  return 0;
}

// Attention-only stack with one window for every layer.
int orc_encoder_stack(int B, int n, int H, int d, int window, int G, const int32_t* global_pos,
                      const int32_t* valid_len, double alpha, int n_layers, const double* x, const double* Wqkv,
                      const double* Wo, const float* thresholds, int keep_global, double ln_eps, double* y,
                      int32_t* final_len, int32_t* orig_idx, int32_t* kept_per_layer, int nthreads) {
  std::vector<int32_t> windows(n_layers > 0 ? n_layers : 1, window);
  return encoder_stack(B, n, H, d, windows.data(), G, global_pos, valid_len, alpha, n_layers, x, Wqkv, Wo, nullptr,
                       nullptr, 0, thresholds, keep_global, ln_eps, y, final_len, orig_idx, kept_per_layer, nthreads);
}

// Full stack: per-layer windows and the feed-forward block in every layer.
int orc_encoder_stack_ffn(int B, int n, int H, int d, const int32_t* windows, int G, const int32_t* global_pos,
                          const int32_t* valid_len, double alpha, int n_layers, const double* x, const double* Wqkv,
                          const double* Wo, const double* W1, const double* W2, int F, const float* thresholds,
                          int keep_global, double ln_eps, double* y, int32_t* final_len, int32_t* orig_idx,
                          int32_t* kept_per_layer, int nthreads) {
  if (!windows || !W1 || !W2) return -1;
  return encoder_stack(B, n, H, d, windows, G, global_pos, valid_len, alpha, n_layers, x, Wqkv, Wo, W1, W2, F,
                       thresholds, keep_global, ln_eps, y, final_len, orig_idx, kept_per_layer, nthreads);
}

// ---------------------------------------------------------------------------
// LTP soft pruning, the training form of the pruning (Sec. 4.2.2 step 1: the
// model and the per-layer thresholds are trained through a soft mask before
// the mask is binarised).  The paper states the mask only in words; the form
// here is the one of the Learned Token Pruning method it adopts (a reading):
//   m_k = sigmoid((s_k - theta) / T)  for valid tokens that are not kept
//                                     global tokens,
//   m_k = 1 for valid global tokens when keep_global is set, 0 for padding,
//   y[k] = m_k * out[k]               (every head and dimension of the row),
// with s the importance score of orc_sparse_attention and T a temperature.
// The backward takes the gradient of a loss with respect to y (dy) and,
// optionally, an extra gradient with respect to the mask (dmask, e.g. from a
// regulariser on the kept fraction), and applies the chain rule in the order
// of the forward: through y = m * out to m and out; through the sigmoid to s
// and theta; through s = (column sums of P) / (H * L) and through out = P V to
// P; through the row softmax to the logits; through S = alpha Q K^T to Q, K.

static double sigmoid(double x) { return 1.0 / (1.0 + std::exp(-x)); }

// Neighbours and probabilities of valid query i of one (sequence, head), as
// attend_one_head defines them (bidirectional).
static void row_probs(int d, int L, int r, const std::vector<char>& is_global, double alpha, const double* q,
                      const double* k, long ld, int i, std::vector<int>& nbr, std::vector<double>& p) {
  nbr.clear();
  for (int j = 0; j < L; ++j)
    if (std::abs(i - j) <= r || is_global[i] || is_global[j]) nbr.push_back(j);
  p.assign(nbr.size(), 0.0);
  double m = -std::numeric_limits<double>::infinity();
  for (size_t t = 0; t < nbr.size(); ++t) {
    double acc = 0.0;
    for (int c = 0; c < d; ++c) acc += q[(long)i * ld + c] * k[(long)nbr[t] * ld + c];
    p[t] = alpha * acc;
    m = std::max(m, p[t]);
  }
  double z = 0.0;
  for (size_t t = 0; t < nbr.size(); ++t) z += std::exp(p[t] - m);
  for (size_t t = 0; t < nbr.size(); ++t) p[t] = std::exp(p[t] - m) / z;
}

// Soft mask of every token from the scores.
static void soft_mask(int B, int n, int G, const int32_t* global_pos, const int32_t* valid_len, const double* scores,
                      double theta, double T, int keep_global, double* mask) {
  for (int b = 0; b < B; ++b) {
    int L = std::min(std::max(valid_len[b], 0), n);
    std::vector<char> g = global_flags(n, L, G, global_pos + (long)b * G);
    for (int k = 0; k < n; ++k) {
      double m = 0.0;
      if (k < L) m = (keep_global && g[k]) ? 1.0 : sigmoid((scores[(long)b * n + k] - theta) / T);
      mask[(long)b * n + k] = m;
    }
  }
}

// Forward: out, lse and scores as orc_sparse_attention, then mask [B, n] and
// y [B, n, H, d] = mask * out.
int orc_soft_prune_forward(int B, int n, int H, int d, int window, int G, const int32_t* global_pos,
                           const int32_t* valid_len, double alpha, const double* q, const double* k, const double* v,
                           double theta, double T, int keep_global, double* out, double* lse, double* scores,
                           double* mask, double* y, int nthreads) {
  if (!(T > 0.0)) return -1;
  int rc = sparse_attention(B, n, H, d, window, G, global_pos, valid_len, alpha, q, k, v, out, lse, scores, nullptr,
                            false, nthreads);
  if (rc) return rc;
  soft_mask(B, n, G, global_pos, valid_len, scores, theta, T, keep_global, mask);
  const long D = (long)H * d;
  for (long t = 0; t < (long)B * n; ++t)
    for (long c = 0; c < D; ++c) y[t * D + c] = mask[t] * out[t * D + c];
  return 0;
}

// Backward of orc_soft_prune_forward for the loss gradient dy [B, n, H, d]
// (with respect to y) and dmask [B, n] (with respect to the mask, or NULL).
// Writes dq, dk, dv [B, n, H, d] and dtheta (a scalar).
// Optional error scales (each may be NULL): mq, mk, mv [B, n, H, d] and
// mtheta hold the same chain evaluated on magnitudes (every factor replaced by
// its absolute value, every difference by a sum), so that a perturbation of
// relative size u in every rounded factor moves each gradient element by at
// most about u times its scale (the running error bound of a sum of products).
int orc_soft_prune_backward(int B, int n, int H, int d, int window, int G, const int32_t* global_pos,
                            const int32_t* valid_len, double alpha, const double* q, const double* k, const double* v,
                            double theta, double T, int keep_global, const double* dy, const double* dmask,
                            double* dq, double* dk, double* dv, double* dtheta, double* mq, double* mk, double* mv,
                            double* mtheta, int nthreads) {
  if (B < 0 || n < 0 || H <= 0 || d <= 0 || window < 0 || G < 0 || !(T > 0.0)) return -1;
  const long D = (long)H * d;
  const size_t bnD = (size_t)B * n * D;
  std::vector<double> out(bnD), lse((size_t)B * H * n), scores((size_t)B * n), mask((size_t)B * n);
  int rc = sparse_attention(B, n, H, d, window, G, global_pos, valid_len, alpha, q, k, v, out.data(), lse.data(),
                            scores.data(), nullptr, false, nthreads);
  if (rc) return rc;
  soft_mask(B, n, G, global_pos, valid_len, scores.data(), theta, T, keep_global, mask.data());
  // y = m * out: dL/dm_k = sum over the row of dy * out (+ dmask), dL/dout = m * dy.
  // m = sigmoid(z), z = (s - theta) / T: dL/ds = dL/dm * m (1 - m) / T and
  // dL/dtheta = - sum of the same over the masked tokens.
  std::vector<double> gs((size_t)B * n, 0.0), dout(bnD, 0.0), gsm((size_t)B * n, 0.0);
  double dth = 0.0, dthm = 0.0;
  for (int b = 0; b < B; ++b) {
    int L = std::min(std::max(valid_len[b], 0), n);
    std::vector<char> g = global_flags(n, L, G, global_pos + (long)b * G);
    for (int kk = 0; kk < L; ++kk) {
      const long t = (long)b * n + kk;
      double dm = dmask ? dmask[t] : 0.0;
      double dmm = std::fabs(dm);
      for (long c = 0; c < D; ++c) {
        dm += dy[t * D + c] * out[t * D + c];
        dmm += std::fabs(dy[t * D + c] * out[t * D + c]);
        dout[t * D + c] = mask[t] * dy[t * D + c];
      }
      if (keep_global && g[kk]) continue;  // a constant mask of 1
      const double ds = dm * mask[t] * (1.0 - mask[t]) / T;
      const double dsm = dmm * mask[t] * (1.0 - mask[t]) / T;
      // s_k = (1 / (H L)) sum_h sum_q P_h[q][k]: each P_h[q][k] receives ds / (H L)
      gs[t] = ds / ((double)H * L);
      gsm[t] = dsm / ((double)H * L);
      dth -= ds;
      dthm += dsm;
    }
  }
  *dtheta = dth;
  if (mtheta) *mtheta = dthm;
  std::fill(dq, dq + bnD, 0.0);
  std::fill(dk, dk + bnD, 0.0);
  std::fill(dv, dv + bnD, 0.0);
  const bool scales = mq && mk && mv;
  if (scales) {
    std::fill(mq, mq + bnD, 0.0);
    std::fill(mk, mk + bnD, 0.0);
    std::fill(mv, mv + bnD, 0.0);
  }
  set_threads(nthreads);
  const int r = window / 2;
#pragma omp parallel for schedule(dynamic, 1)
  for (long bh = 0; bh < (long)B * H; ++bh) {
    int b = (int)(bh / H), h = (int)(bh % H);
    int L = std::min(std::max(valid_len[b], 0), n);
    std::vector<char> g = global_flags(n, L, G, global_pos + (long)b * G);
    const long base = (long)b * n * D + (long)h * d;
    const double *qh = q + base, *kh = k + base, *vh = v + base, *doh = dout.data() + base;
    double *dqh = dq + base, *dkh = dk + base, *dvh = dv + base;
    std::vector<int> nbr;
    std::vector<double> p, dp, dpm;
    for (int i = 0; i < L; ++i) {
      row_probs(d, L, r, g, alpha, qh, kh, D, i, nbr, p);
      // out_i = sum_j P[i][j] v_j and the score term: dL/dP[i][j] = dout_i . v_j + gs_j
      dp.assign(nbr.size(), 0.0);
      dpm.assign(nbr.size(), 0.0);
      double rowdot = 0.0, rowdotm = 0.0;  // sum_j P[i][j] dL/dP[i][j]
      for (size_t t = 0; t < nbr.size(); ++t) {
        const int j = nbr[t];
        double acc = 0.0, accm = 0.0;
        for (int c = 0; c < d; ++c) {
          acc += doh[(long)i * D + c] * vh[(long)j * D + c];
          accm += std::fabs(doh[(long)i * D + c] * vh[(long)j * D + c]);
        }
        dp[t] = acc + gs[(long)b * n + j];
        dpm[t] = accm + gsm[(long)b * n + j];
        rowdot += p[t] * dp[t];
        rowdotm += p[t] * dpm[t];
      }
      for (size_t t = 0; t < nbr.size(); ++t) {
        const int j = nbr[t];
        // row softmax: dL/dS[i][j] = P[i][j] (dL/dP[i][j] - sum_l P[i][l] dL/dP[i][l]); S = alpha q_i . k_j
        const double dsij = p[t] * (dp[t] - rowdot);
        for (int c = 0; c < d; ++c) {
          dqh[(long)i * D + c] += alpha * dsij * kh[(long)j * D + c];
          dkh[(long)j * D + c] += alpha * dsij * qh[(long)i * D + c];
          dvh[(long)j * D + c] += p[t] * doh[(long)i * D + c];
        }
        if (scales) {
          const double dsm = p[t] * (dpm[t] + rowdotm);
          double *mqh = mq + base, *mkh = mk + base, *mvh = mv + base;
          for (int c = 0; c < d; ++c) {
            mqh[(long)i * D + c] += alpha * dsm * std::fabs(kh[(long)j * D + c]);
            mkh[(long)j * D + c] += alpha * dsm * std::fabs(qh[(long)i * D + c]);
            mvh[(long)j * D + c] += p[t] * std::fabs(doh[(long)i * D + c]);
          }
        }
      }
    }
  }
  return 0;
}

}  // extern "C"
