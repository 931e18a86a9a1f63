// C ABI of the KVpop future-attention target library: argument validation, error
// reporting and dispatch to the gfx950 kernels. The semantics of every entry point
// are specified in include/kvpop.h.
#include "kvpop.h"

#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdlib>
#include <cstdint>
#include <string>

#include "kvpop_internal.h"

namespace {

thread_local std::string g_err_text;

struct Sizes {
  int64_t q_elems, k_elems, row_elems;  // Q, K and [B, Hq, T] element counts
};

bool mul_ok(int64_t a, int64_t b, int64_t* r) {
  if (a != 0 && b > INT64_MAX / a) return false;
  *r = a * b;
  return true;
}

int check_dims(const kvpop_dims* d, Sizes* sz) {
  if (!d) return KVPOP_EINVAL;
  if (d->batch < 1 || d->n_q_heads < 1 || d->n_kv_heads < 1 || d->seq_len < 1 || d->head_dim < 1)
    return KVPOP_EINVAL;
  if (d->n_q_heads % d->n_kv_heads != 0) return KVPOP_EINVAL;
  if (!std::isfinite(d->scale) || !(d->scale > 0.f)) return KVPOP_EINVAL;
  if (d->head_dim != 64 && d->head_dim != 128) return KVPOP_EUNSUPPORTED;
  if (d->seq_len > KVPOP_MAX_SEQ_LEN) return KVPOP_EUNSUPPORTED;
  int64_t bh, bkh, t;
  if (!mul_ok(d->batch, d->n_q_heads, &bh) || !mul_ok(bh, d->seq_len, &sz->row_elems) ||
      !mul_ok(sz->row_elems, d->head_dim, &sz->q_elems) || !mul_ok(d->batch, d->n_kv_heads, &bkh) ||
      !mul_ok(bkh, d->seq_len, &t) || !mul_ok(t, d->head_dim, &sz->k_elems) ||
      sz->q_elems > INT64_MAX / 4)
    return KVPOP_EINVAL;
  // Grid sizes stay below 2^31 workgroups: at most B * Hq * ceil(T / 32) of them.
  if (sz->row_elems / 32 + bh > INT32_MAX) return KVPOP_EUNSUPPORTED;
  return KVPOP_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool overlap(const void* a, int64_t abytes, const void* b, int64_t bbytes) {
  if (!a || !b) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return a0 < b0 + (uintptr_t)bbytes && b0 < a0 + (uintptr_t)abytes;
}

int check_band(int32_t window, int32_t horizon) {
  if (window < 0) return KVPOP_EINVAL;
  if (horizon >= 0 && horizon < window) return KVPOP_EINVAL;
  return KVPOP_OK;
}

int hip_status(int e) {
  if (e == 0) return KVPOP_OK;
  g_err_text = std::string("HIP error: ") + hipGetErrorString(static_cast<hipError_t>(e));
  return KVPOP_EHIP;
}

// Test hook for the KVPOP_EHIP path: with the environment variable
// KVPOP_TEST_FORCE_EHIP set to a nonzero hipError_t code, every entry point fails
// after validation as if its first launch had returned that code, and launches
// nothing. Unset (the normal case) it costs one getenv per call.
int forced_hip_error() {
  const char* e = std::getenv("KVPOP_TEST_FORCE_EHIP");
  return e ? std::atoi(e) : 0;
}

// Runs the launches of one entry point (a callable returning 0 or the hipError_t
// of the launch that failed) and maps the result to a status.
template <class F>
int launch(F&& f) {
  const int forced = forced_hip_error();
  if (forced != 0) return hip_status(forced);
  return hip_status(f());
}

kvpop::Launch make_launch(const kvpop_dims* d, const void* q, const void* k, const float* bias, void* stream) {
  kvpop::Launch L{};
  L.q = static_cast<const uint16_t*>(q);
  L.k = static_cast<const uint16_t*>(k);
  L.bias = bias;
  L.B = d->batch;
  L.Hq = d->n_q_heads;
  L.Hkv = d->n_kv_heads;
  L.T = d->seq_len;
  L.D = d->head_dim;
  L.scale = d->scale;
  L.stream = stream;
  return L;
}

// Validation shared by every entry point for the inputs q, k, key_bias.
int check_inputs(const kvpop_dims* d, const void* q, const void* k, const float* bias, Sizes* sz) {
  int st = check_dims(d, sz);
  if (st != KVPOP_OK) return st;
  if (!q || !k) return KVPOP_EINVAL;
  if (!aligned16(q) || !aligned16(k) || (bias && !aligned16(bias))) return KVPOP_EUNSUPPORTED;
  return KVPOP_OK;
}

// An output of `bytes` bytes must not overlap q, k, bias or `other`.
int check_output(const void* out, int64_t bytes, const Sizes& sz, const kvpop_dims* d, const void* q,
                 const void* k, const float* bias, const void* other, int64_t other_bytes) {
  if (!out) return KVPOP_EINVAL;
  if (!aligned16(out)) return KVPOP_EUNSUPPORTED;
  if (overlap(out, bytes, q, sz.q_elems * 2) || overlap(out, bytes, k, sz.k_elems * 2) ||
      overlap(out, bytes, bias, (int64_t)d->seq_len * 4) || overlap(out, bytes, other, other_bytes))
    return KVPOP_EINVAL;
  return KVPOP_OK;
}

// Validation shared by kvpop_running_topk and kvpop_running_topk_noalloc. The
// workspace (need bytes) is checked only when it is caller memory (ws != NULL).
int check_topk(const kvpop_topk_dims* d, const float* scores, const float* log_gamma, int32_t sinks, int32_t window,
               int32_t topk, int32_t* rank, int32_t* cutoff, int32_t* label, int32_t* boundary, int32_t* evict,
               const void* ws, size_t need) {
  if (!scores || !rank || !cutoff) return KVPOP_EINVAL;
  const void* ptrs[] = {scores, log_gamma, rank, cutoff, label, boundary, evict, ws};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return KVPOP_EUNSUPPORTED;
  const int64_t n = (int64_t)d->batch * d->n_heads * d->seq_len;
  if (n / d->seq_len / d->n_heads != d->batch || n * 4 > INT64_MAX / 2) return KVPOP_EINVAL;
  const int64_t b = n * 4;
  // Outputs must not overlap each other, the inputs or the workspace.
  const void* outs[] = {rank, cutoff, label, boundary, evict};
  for (int i = 0; i < 5; ++i) {
    if (!outs[i]) continue;
    if (overlap(outs[i], b, scores, b) || overlap(outs[i], b, log_gamma, (int64_t)d->n_heads * 4) ||
        overlap(outs[i], b, ws, (int64_t)need))
      return KVPOP_EINVAL;
    for (int j = i + 1; j < 5; ++j)
      if (overlap(outs[i], b, outs[j], b)) return KVPOP_EINVAL;
  }
  if (overlap(ws, (int64_t)need, scores, b) || overlap(ws, (int64_t)need, log_gamma, (int64_t)d->n_heads * 4))
    return KVPOP_EINVAL;
  return KVPOP_OK;
}

kvpop::TopkLaunch make_topk(const kvpop_topk_dims* d, const float* scores, const float* log_gamma, int32_t sinks,
                            int32_t window, int32_t topk, int32_t* rank, int32_t* cutoff, int32_t* label,
                            int32_t* boundary, int32_t* evict, void* workspace, void* stream) {
  kvpop::TopkLaunch L{};
  L.scores = scores;
  L.log_gamma = log_gamma;
  L.B = d->batch;
  L.H = d->n_heads;
  L.T = d->seq_len;
  L.sinks = sinks;
  L.window = window;
  L.topk = topk;
  L.rank = rank;
  L.cutoff = cutoff;
  L.label = label;
  L.boundary = boundary;
  L.evict = evict;
  L.workspace = workspace;
  L.stream = stream;
  return L;
}

}  // namespace

extern "C" {

int kvpop_abi_version(void) { return KVPOP_ABI_VERSION; }

const char* kvpop_strerror(int status) {
  switch (status) {
    case KVPOP_OK:
      return "success";
    case KVPOP_EINVAL:
      return "invalid argument (null pointer, bad dimension, Hq % Hkv != 0, bad scale, bad window/horizon, "
             "or overlapping buffers)";
    case KVPOP_EUNSUPPORTED:
      return "unsupported configuration (head_dim not 64/128, pointer not 16-byte aligned, or size limit)";
    case KVPOP_EHIP:
      return g_err_text.empty() ? "HIP runtime error" : g_err_text.c_str();
    case KVPOP_ETOOBIG:
      return "problem too large for the no-allocation entry point (its workspace exceeds "
             "KVPOP_NOALLOC_SCRATCH_BYTES)";
    default:
      return "unknown status code";
  }
}

int kvpop_row_lse(const kvpop_dims* dims, const void* q, const void* k, const float* key_bias, float* lse,
                  void* stream) {
  Sizes sz;
  int st = check_inputs(dims, q, k, key_bias, &sz);
  if (st != KVPOP_OK) return st;
  st = check_output(lse, sz.row_elems * 4, sz, dims, q, k, key_bias, nullptr, 0);
  if (st != KVPOP_OK) return st;
  kvpop::Launch L = make_launch(dims, q, k, key_bias, stream);
  L.out = lse;
  return launch([&] { return kvpop::launch_row_lse(L); });
}

int kvpop_future_attn_from_lse(const kvpop_dims* dims, const void* q, const void* k, const float* key_bias,
                               const float* lse, int32_t window, int32_t horizon, float* out, void* stream) {
  Sizes sz;
  int st = check_inputs(dims, q, k, key_bias, &sz);
  if (st != KVPOP_OK) return st;
  if (!lse) return KVPOP_EINVAL;
  if (!aligned16(lse)) return KVPOP_EUNSUPPORTED;
  st = check_band(window, horizon);
  if (st != KVPOP_OK) return st;
  st = check_output(out, sz.row_elems * 4, sz, dims, q, k, key_bias, lse, sz.row_elems * 4);
  if (st != KVPOP_OK) return st;
  kvpop::Launch L = make_launch(dims, q, k, key_bias, stream);
  L.lse = lse;
  L.out = out;
  L.window = window;
  L.horizon = horizon;
  return launch([&] { return kvpop::launch_future_mass(L); });
}

int kvpop_future_attn_bands(const kvpop_dims* dims, const void* q, const void* k, const float* key_bias,
                            const float* lse, int32_t n_bands, const int32_t* windows, const int32_t* horizons,
                            float* const* outs, void* stream) {
  Sizes sz;
  int st = check_inputs(dims, q, k, key_bias, &sz);
  if (st != KVPOP_OK) return st;
  if (!lse) return KVPOP_EINVAL;
  if (!aligned16(lse)) return KVPOP_EUNSUPPORTED;
  if (n_bands < 1 || n_bands > 2 || !windows || !horizons || !outs) return KVPOP_EINVAL;
  for (int i = 0; i < n_bands; ++i) {
    st = check_band(windows[i], horizons[i]);
    if (st != KVPOP_OK) return st;
    st = check_output(outs[i], sz.row_elems * 4, sz, dims, q, k, key_bias, lse, sz.row_elems * 4);
    if (st != KVPOP_OK) return st;
  }
  if (n_bands == 2 && overlap(outs[0], sz.row_elems * 4, outs[1], sz.row_elems * 4)) return KVPOP_EINVAL;
  kvpop::Launch L = make_launch(dims, q, k, key_bias, stream);
  L.lse = lse;
  L.out = outs[0];
  L.window = windows[0];
  L.horizon = horizons[0];
  if (n_bands == 2) {
    L.out1 = outs[1];
    L.window1 = windows[1];
    L.horizon1 = horizons[1];
  }
  return launch([&] { return kvpop::launch_future_mass(L); });
}

int kvpop_future_attn_scores(const kvpop_dims* dims, const void* q, const void* k, const float* key_bias,
                             const float* lse, int32_t window, int32_t horizon, int32_t agg, float eps,
                             int32_t normalize, float* out, float* scores, void* stream) {
  Sizes sz;
  int st = check_inputs(dims, q, k, key_bias, &sz);
  if (st != KVPOP_OK) return st;
  if (!lse) return KVPOP_EINVAL;
  if (!aligned16(lse)) return KVPOP_EUNSUPPORTED;
  st = check_band(window, horizon);
  if (st != KVPOP_OK) return st;
  if ((agg != KVPOP_AGG_MAX && agg != KVPOP_AGG_MEAN) || (normalize != 0 && normalize != 1) || !std::isfinite(eps) ||
      eps < 0.f)
    return KVPOP_EINVAL;
  const int64_t score_bytes = (int64_t)dims->batch * dims->n_kv_heads * dims->seq_len * 4;
  st = check_output(scores, score_bytes, sz, dims, q, k, key_bias, lse, sz.row_elems * 4);
  if (st != KVPOP_OK) return st;
  if (out) {
    st = check_output(out, sz.row_elems * 4, sz, dims, q, k, key_bias, lse, sz.row_elems * 4);
    if (st != KVPOP_OK) return st;
    if (overlap(out, sz.row_elems * 4, scores, score_bytes)) return KVPOP_EINVAL;
  }
  kvpop::Launch L = make_launch(dims, q, k, key_bias, stream);
  L.lse = lse;
  L.out = out;
  L.window = window;
  L.horizon = horizon;
  L.scores = scores;
  L.agg = agg;
  L.eps = eps;
  L.normalize = normalize;
  return launch([&] { return kvpop::launch_future_mass(L); });
}

size_t kvpop_running_topk_workspace_size(const kvpop_topk_dims* d) {
  if (!d || d->batch < 1 || d->n_heads < 1 || d->seq_len < 1 || d->seq_len > KVPOP_MAX_SEQ_LEN) return 0;
  const size_t seqs = (size_t)d->batch * (size_t)d->n_heads;
  const size_t words = kvpop::topk_workspace_words_per_seq(d->seq_len);
  if (seqs > SIZE_MAX / 4 / words) return 0;
  return seqs * words * 4;
}

int kvpop_running_topk(const kvpop_topk_dims* d, const float* scores, const float* log_gamma, int32_t sinks,
                       int32_t window, int32_t topk, int32_t* rank, int32_t* cutoff, int32_t* label,
                       int32_t* boundary, int32_t* evict, void* workspace, size_t workspace_bytes, void* stream) {
  if (!d || d->batch < 1 || d->n_heads < 1 || d->seq_len < 1) return KVPOP_EINVAL;
  if (d->seq_len > KVPOP_MAX_SEQ_LEN) return KVPOP_EUNSUPPORTED;
  if (sinks < 0 || window < 0 || topk < 1) return KVPOP_EINVAL;
  if (!scores || !rank || !cutoff || !workspace) return KVPOP_EINVAL;
  const size_t need = kvpop_running_topk_workspace_size(d);
  if (need == 0 || workspace_bytes < need) return KVPOP_EINVAL;
  const int st = check_topk(d, scores, log_gamma, sinks, window, topk, rank, cutoff, label, boundary, evict,
                            workspace, need);
  if (st != KVPOP_OK) return st;
  kvpop::TopkLaunch L = make_topk(d, scores, log_gamma, sinks, window, topk, rank, cutoff, label, boundary, evict,
                                  workspace, stream);
  return launch([&] { return kvpop::launch_running_topk(L); });
}

int kvpop_running_topk_noalloc(const kvpop_topk_dims* d, const float* scores, const float* log_gamma, int32_t sinks,
                               int32_t window, int32_t topk, int32_t* rank, int32_t* cutoff, int32_t* label,
                               int32_t* boundary, int32_t* evict, void* stream) {
  if (!d || d->batch < 1 || d->n_heads < 1 || d->seq_len < 1) return KVPOP_EINVAL;
  if (d->seq_len > KVPOP_MAX_SEQ_LEN) return KVPOP_EUNSUPPORTED;
  if (sinks < 0 || window < 0 || topk < 1) return KVPOP_EINVAL;
  const size_t need = kvpop_running_topk_workspace_size(d);
  if (need == 0) return KVPOP_EINVAL;
  if (need > (size_t)KVPOP_NOALLOC_SCRATCH_BYTES) return KVPOP_ETOOBIG;
  const int st = check_topk(d, scores, log_gamma, sinks, window, topk, rank, cutoff, label, boundary, evict,
                            nullptr, 0);
  if (st != KVPOP_OK) return st;
  return launch([&] {
    void* ws = nullptr;
    const int e = kvpop::noalloc_scratch(stream, &ws);
    if (e != 0) return e;
    kvpop::TopkLaunch L = make_topk(d, scores, log_gamma, sinks, window, topk, rank, cutoff, label, boundary,
                                    evict, ws, stream);
    return kvpop::launch_running_topk(L);
  });
}

int kvpop_sparse_attn_fwd(const kvpop_dims* dims, const void* q, const void* k, const void* v,
                          const float* key_bias, const int32_t* evict, void* o, float* lse, void* stream) {
  Sizes sz;
  int st = check_inputs(dims, q, k, key_bias, &sz);
  if (st != KVPOP_OK) return st;
  const int G = dims->n_q_heads / dims->n_kv_heads;
  if ((G & (G - 1)) != 0) return KVPOP_EUNSUPPORTED;
  if ((int64_t)dims->seq_len * dims->head_dim * 2 > INT32_MAX) return KVPOP_EUNSUPPORTED;
  if (!v || !evict) return KVPOP_EINVAL;
  if (!aligned16(v) || !aligned16(evict)) return KVPOP_EUNSUPPORTED;
  const int64_t ev_bytes = (int64_t)dims->batch * dims->n_kv_heads * dims->seq_len * 4;
  // o must not overlap q, k, key_bias, lse, v or evict; lse likewise.
  st = check_output(o, sz.q_elems * 2, sz, dims, q, k, key_bias, lse, sz.row_elems * 4);
  if (st != KVPOP_OK) return st;
  st = check_output(lse, sz.row_elems * 4, sz, dims, q, k, key_bias, o, sz.q_elems * 2);
  if (st != KVPOP_OK) return st;
  if (overlap(o, sz.q_elems * 2, v, sz.k_elems * 2) || overlap(o, sz.q_elems * 2, evict, ev_bytes) ||
      overlap(lse, sz.row_elems * 4, v, sz.k_elems * 2) || overlap(lse, sz.row_elems * 4, evict, ev_bytes))
    return KVPOP_EINVAL;
  kvpop::SparseLaunch L{};
  L.q = static_cast<const uint16_t*>(q);
  L.k = static_cast<const uint16_t*>(k);
  L.v = static_cast<const uint16_t*>(v);
  L.bias = key_bias;
  L.evict = evict;
  L.o = static_cast<uint16_t*>(o);
  L.lse = lse;
  L.B = dims->batch;
  L.Hq = dims->n_q_heads;
  L.Hkv = dims->n_kv_heads;
  L.T = dims->seq_len;
  L.D = dims->head_dim;
  L.scale = dims->scale;
  L.stream = stream;
  return launch([&] { return kvpop::launch_sparse_attn_fwd(L); });
}

int kvpop_future_attn_target(const kvpop_dims* dims, const void* q, const void* k, const float* key_bias,
                             int32_t window, int32_t horizon, float* lse_ws, float* out, void* stream) {
  Sizes sz;
  int st = check_inputs(dims, q, k, key_bias, &sz);
  if (st != KVPOP_OK) return st;
  st = check_band(window, horizon);
  if (st != KVPOP_OK) return st;
  st = check_output(lse_ws, sz.row_elems * 4, sz, dims, q, k, key_bias, out, sz.row_elems * 4);
  if (st != KVPOP_OK) return st;
  st = check_output(out, sz.row_elems * 4, sz, dims, q, k, key_bias, lse_ws, sz.row_elems * 4);
  if (st != KVPOP_OK) return st;
  kvpop::Launch L = make_launch(dims, q, k, key_bias, stream);
  return launch([&] {
    L.out = lse_ws;
    const int e = kvpop::launch_row_lse(L);
    if (e != 0) return e;
    L.lse = lse_ws;
    L.out = out;
    L.window = window;
    L.horizon = horizon;
    return kvpop::launch_future_mass(L);
  });
}

}  // extern "C"
