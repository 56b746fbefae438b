// Host-side iteration latency model and dynamic-chunk selection (no HIP).
//
// The scheduler of Section 3.1 picks, every iteration, the largest prefill
// chunk whose batch still meets the next-token deadlines of the decodes in it
// (dynamic chunking, Section 3.3), using a lightweight latency predictor
// trained offline (Section 3.6). The predictor here is linear in five
// roofline features of the batch (see include/hb.h), fitted by non-negative
// least squares to hb_profile cells.
#include <cmath>
#include <cstring>
#include <limits>
#include <vector>

#include "hb.h"
#include "hb_plan.h"

namespace hb {
namespace {

constexpr int NF = HB_LAT_FEATURES;

bool check_cfg(const hb_layer_config* c) {
  return c && c->n_q_heads > 0 && c->n_kv_heads > 0 && c->head_dim > 0;
}

// Features of one batch given as (chunk_len, context_len) pairs; summed in
// request order. A request with chunk_len 0 is absent (a decode-only batch).
void features_of(const hb_layer_config& c, const int32_t* chunk, const int32_t* ctx, int n, int stride, double* f) {
  const double kv_bytes_per_token = 2.0 * c.n_kv_heads * c.head_dim * 2.0;
  const double attn_flops_per_pair = 4.0 * c.n_q_heads * c.head_dim;
  double T = 0, kv = 0, ctx_pairs = 0, new_pairs = 0;
  for (int i = 0; i < n; ++i) {
    const double ch = chunk[i * stride], x = ctx[i * stride];
    if (ch == 0) continue;  // a request with no new tokens reads nothing
    T += ch;
    kv += x + ch;
    ctx_pairs += ch * x;
    new_pairs += ch * (ch + 1) / 2;
  }
  f[0] = 1.0;
  f[1] = T / 1e3;
  f[2] = kv * kv_bytes_per_token / 1e9;
  f[3] = ctx_pairs * attn_flops_per_pair / 1e12;
  f[4] = new_pairs * attn_flops_per_pair / 1e12;
}

double dot(const double* a, const double* b) {
  double s = 0;
  for (int i = 0; i < NF; ++i) s += a[i] * b[i];
  return s;
}

// Least squares on the columns in `mask`: columns scaled to unit maximum,
// Householder QR, back substitution. Returns false when a column is zero or
// the columns are (numerically) dependent.
bool solve_subset(const std::vector<double>& A, const std::vector<double>& y, int rows, unsigned mask, double* coef) {
  int cols[NF], k = 0;
  for (int j = 0; j < NF; ++j)
    if (mask & (1u << j)) cols[k++] = j;
  if (rows < k) return false;
  std::vector<double> B((size_t)rows * k), b(y.begin(), y.begin() + rows);
  double scale[NF];
  for (int a = 0; a < k; ++a) {
    double mx = 0;
    for (int r = 0; r < rows; ++r) mx = std::fmax(mx, std::fabs(A[(size_t)r * NF + cols[a]]));
    if (mx == 0) return false;
    scale[a] = 1.0 / mx;
    for (int r = 0; r < rows; ++r) B[(size_t)r * k + a] = A[(size_t)r * NF + cols[a]] * scale[a];
  }
  double diag[NF];
  for (int a = 0; a < k; ++a) {
    double norm = 0;
    for (int r = a; r < rows; ++r) norm += B[(size_t)r * k + a] * B[(size_t)r * k + a];
    norm = std::sqrt(norm);
    if (!(norm > 1e-12)) return false;
    const double alpha = B[(size_t)a * k + a] > 0 ? -norm : norm;
    // v = x - alpha e_1, stored in place of column a (rows a..)
    B[(size_t)a * k + a] -= alpha;
    double vv = 0;
    for (int r = a; r < rows; ++r) vv += B[(size_t)r * k + a] * B[(size_t)r * k + a];
    for (int c = a + 1; c < k; ++c) {
      double dv = 0;
      for (int r = a; r < rows; ++r) dv += B[(size_t)r * k + a] * B[(size_t)r * k + c];
      const double f = 2 * dv / vv;
      for (int r = a; r < rows; ++r) B[(size_t)r * k + c] -= f * B[(size_t)r * k + a];
    }
    double dv = 0;
    for (int r = a; r < rows; ++r) dv += B[(size_t)r * k + a] * b[r];
    const double f = 2 * dv / vv;
    for (int r = a; r < rows; ++r) b[r] -= f * B[(size_t)r * k + a];
    diag[a] = alpha;
  }
  double x[NF];
  for (int a = k - 1; a >= 0; --a) {
    double sum = b[a];
    for (int c = a + 1; c < k; ++c) sum -= B[(size_t)a * k + c] * x[c];
    x[a] = sum / diag[a];
  }
  for (int j = 0; j < NF; ++j) coef[j] = 0;
  for (int a = 0; a < k; ++a) coef[cols[a]] = x[a] * scale[a];
  return true;
}

}  // namespace
}  // namespace hb

using namespace hb;

extern "C" hb_status hb_latency_features(const hb_layer_config* cfg, const hb_request* requests,
                                         int32_t n_requests, double* features) {
  if (!check_cfg(cfg) || !features || n_requests < 0 || (n_requests > 0 && !requests))
    return fail(HB_ERR_INVALID, "hb_latency_features: null pointer or bad size");
  for (int i = 0; i < n_requests; ++i)
    if (requests[i].chunk_len < 0 || requests[i].context_len < 0)
      return fail(HB_ERR_INVALID, "hb_latency_features: request %d has a negative length", i);
  const int stride = sizeof(hb_request) / sizeof(int32_t);
  static_assert(sizeof(hb_request) % sizeof(int32_t) == 0, "hb_request is whole int32 words");
  features_of(*cfg, n_requests ? &requests[0].chunk_len : nullptr, n_requests ? &requests[0].context_len : nullptr,
              n_requests, stride, features);
  return HB_OK;
}

extern "C" hb_status hb_fit_latency_model(const hb_layer_config* cfg, const int32_t* chunk_sizes, int32_t n_chunk,
                                          const hb_decode_mix* mixes, int32_t n_mix, const hb_profile_cell* cells,
                                          hb_latency_model* out) {
  if (!check_cfg(cfg) || !chunk_sizes || !mixes || !cells || !out || n_chunk <= 0 || n_mix <= 0)
    return fail(HB_ERR_INVALID, "hb_fit_latency_model: null pointer or empty profile");
  const int rows = n_chunk * n_mix;
  if (rows < NF) return fail(HB_ERR_INVALID, "hb_fit_latency_model: %d cells for %d features", rows, NF);
  // rows of the weighted system: features / measured, target 1 (relative error)
  std::vector<double> A((size_t)rows * NF), y(rows, 1.0), raw((size_t)rows * NF);
  std::vector<int32_t> chunk, ctx;
  for (int m = 0; m < n_mix; ++m) {
    const hb_decode_mix& mx = mixes[m];
    if (mx.n_decode < 0 || (mx.n_decode > 0 && !mx.decode_contexts) || mx.chunk_context < 0)
      return fail(HB_ERR_INVALID, "hb_fit_latency_model: mix %d malformed", m);
    for (int c = 0; c < n_chunk; ++c) {
      const int r = m * n_chunk + c;
      const double t = cells[r].median_ms;
      if (!(t > 0) || !std::isfinite(t)) return fail(HB_ERR_INVALID, "hb_fit_latency_model: cell %d median %g", r, t);
      if (chunk_sizes[c] < 0) return fail(HB_ERR_INVALID, "hb_fit_latency_model: negative chunk size");
      chunk.assign(1, chunk_sizes[c]);
      ctx.assign(1, mx.chunk_context);
      for (int i = 0; i < mx.n_decode; ++i) {
        if (mx.decode_contexts[i] < 0) return fail(HB_ERR_INVALID, "hb_fit_latency_model: negative context");
        chunk.push_back(1);
        ctx.push_back(mx.decode_contexts[i]);
      }
      features_of(*cfg, chunk.data(), ctx.data(), (int)chunk.size(), 1, &raw[(size_t)r * NF]);
      for (int j = 0; j < NF; ++j) A[(size_t)r * NF + j] = raw[(size_t)r * NF + j] / t;
    }
  }
  // non-negative least squares: the optimum is the unconstrained solution on
  // its own support, so the best non-negative subset solution is it
  double best[NF] = {}, best_res = std::numeric_limits<double>::infinity();
  for (unsigned mask = 1; mask < (1u << NF); ++mask) {
    double coef[NF];
    if (!solve_subset(A, y, rows, mask, coef)) continue;
    bool ok = true;
    for (int j = 0; j < NF; ++j) ok = ok && coef[j] >= 0;
    if (!ok) continue;
    double res = 0;
    for (int r = 0; r < rows; ++r) {
      const double e = dot(&A[(size_t)r * NF], coef) - 1.0;
      res += e * e;
    }
    if (res < best_res) {
      best_res = res;
      std::memcpy(best, coef, sizeof(best));
    }
  }
  if (!std::isfinite(best_res)) return fail(HB_ERR_INVALID, "hb_fit_latency_model: no non-negative fit");
  std::memcpy(out->coef, best, sizeof(best));
  out->fit_rel_rms = std::sqrt(best_res / rows);
  // largest under-prediction: measured / predicted - 1 over the cells
  double under = 0;
  for (int r = 0; r < rows; ++r) {
    const double pred = dot(&raw[(size_t)r * NF], best);
    if (pred > 0) under = std::fmax(under, cells[r].median_ms / pred - 1.0);
  }
  out->fit_max_under = under;
  out->n_cells = rows;
  return HB_OK;
}

extern "C" hb_status hb_predict_latency(const hb_latency_model* model, const hb_layer_config* cfg,
                                        const hb_request* requests, int32_t n_requests, double* ms) {
  if (!model || !ms) return fail(HB_ERR_INVALID, "hb_predict_latency: null pointer");
  double f[NF];
  const hb_status st = hb_latency_features(cfg, requests, n_requests, f);
  if (st != HB_OK) return st;
  *ms = dot(model->coef, f);
  return HB_OK;
}

extern "C" hb_status hb_select_chunk(const hb_latency_model* model, const hb_layer_config* cfg,
                                     const int32_t* decode_contexts, const double* decode_deadlines_ms,
                                     int32_t n_decode, double now_ms, int32_t chunk_context, int32_t max_chunk,
                                     int32_t granularity, double margin, int32_t* chunk, double* predicted_ms) {
  if (!model || !check_cfg(cfg) || !chunk || !predicted_ms || n_decode < 0 ||
      (n_decode > 0 && (!decode_contexts || !decode_deadlines_ms)))
    return fail(HB_ERR_INVALID, "hb_select_chunk: null pointer or bad size");
  if (chunk_context < 0 || max_chunk < 0 || granularity < 1 || std::isnan(now_ms) || !(margin >= 0))
    return fail(HB_ERR_INVALID, "hb_select_chunk: chunk_context %d, max_chunk %d, granularity %d, margin %g",
                chunk_context, max_chunk, granularity, margin);
  const double scale = 1.0 + margin;
  double slack = std::numeric_limits<double>::infinity();
  for (int i = 0; i < n_decode; ++i) {
    if (decode_contexts[i] < 0 || std::isnan(decode_deadlines_ms[i]))
      return fail(HB_ERR_INVALID, "hb_select_chunk: decode %d has a negative context or NaN deadline", i);
    slack = std::fmin(slack, decode_deadlines_ms[i] - now_ms);
  }
  // the batch: the chunk (row 0, chunk_len 0 for a decode-only batch), then the decodes
  std::vector<int32_t> ch(n_decode + 1, 1), cx(n_decode + 1);
  cx[0] = chunk_context;
  for (int i = 0; i < n_decode; ++i) cx[i + 1] = decode_contexts[i];
  auto predict = [&](int c) {
    ch[0] = c;
    double f[NF];
    features_of(*cfg, ch.data(), cx.data(), n_decode + 1, 1, f);
    return dot(model->coef, f);
  };
  // the prediction is non-decreasing in c (non-negative coefficients of
  // features that grow with c), so scan down from the largest candidate
  int best = 0;
  double best_ms = predict(0);
  const int top = max_chunk / granularity * granularity;
  if (max_chunk > 0) {
    const double full = predict(max_chunk);
    if (full * scale <= slack) {
      best = max_chunk;
      best_ms = full;
    } else {
      for (int c = (top == max_chunk ? top - granularity : top); c >= granularity; c -= granularity) {
        const double t = predict(c);
        if (t * scale <= slack) {
          best = c;
          best_ms = t;
          break;
        }
      }
    }
  }
  *chunk = best;
  *predicted_ms = best_ms;
  return HB_OK;
}
