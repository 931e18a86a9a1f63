/*
 * kvpop.h -- C ABI of the KVpop future-attention target library (gfx950 / MI355X).
 *
 * The library computes, for every key position t and every query head, the dense
 * causal softmax probability mass that query positions at or after t place on key
 * t (KVpop, Sec. 3.1 eq. future_mass_per_group without the 1/N_t factor; App. B.1
 * eq. group_future_mass_app; App. D.1 eq. future_mass_app), without materialising
 * the T x T attention map. It works in two passes on the caller's stream:
 *
 *   pass 1  kvpop_row_lse              LSE_d = log sum_{t <= d} exp l(d, t)
 *           (App. D.1 eq. dense_lse_app; the per-query normaliser that App. D.4
 *            step 1 takes from the main attention pass)
 *   pass 2  kvpop_future_attn_from_lse out_t = sum_{d in band(t)} exp(l(d, t) - LSE_d)
 *           (App. D.1 eq. future_mass_app; App. D.4 steps 2-4 evaluate the same
 *            sum as the log-sum-exp of a transposed attention pass, App. D.2)
 *   both    kvpop_future_attn_target   pass 1 then pass 2
 *
 * with the logit (App. D.1 eq. dense_logit_app, plus an optional per-key bias)
 *
 *   l(d, t) = scale * <Q[b, qh, d, :], K[b, qh / G, t, :]> + key_bias[t],  t <= d,
 *
 * and band(t) = { d : t + window <= d <= min(T - 1, t + horizon) } (horizon < 0:
 * up to T - 1). The paper's protected window w is `window`; its finite lookahead L
 * (App. B.2) is horizon = w + L. The paper's full-future target is window = w,
 * horizon = -1; window = 0 includes the diagonal d = t.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Shapes: B = batch, Hq = query heads, Hkv = KV heads (Hq % Hkv == 0,
 *    G = Hq / Hkv), T = sequence length, D = head dim (64 or 128).
 *  - Q is bf16 [B, Hq, T, D] and K is bf16 [B, Hkv, T, D], both contiguous
 *    row-major device memory (bf16 = IEEE binary32 with the low 16 bits dropped).
 *    Query head qh reads KV head qh / G (contiguous query-head groups).
 *  - key_bias is an optional fp32 [T] device array (NULL = no bias), shared by all
 *    batch rows and heads. Values are finite or -INFINITY (key never attended: its
 *    mass is exactly 0); NaN and +INFINITY are not supported. Pass 2 factors
 *    exp(key_bias[t]) out of key t's sum when |key_bias[t]| <= 30 and otherwise
 *    adds the bias to every exponent of a guarded sweep, so any finite bias is
 *    exact to the tolerance.
 *  - lse is fp32 [B, Hq, T] holding natural-log normalisers; out is fp32
 *    [B, Hq, T] holding the linear (not log) unnormalised future mass. Keys whose
 *    band is empty (t + window > T - 1) get exactly 0.
 *  - All pointers are device pointers that the caller allocates and owns; the
 *    library allocates nothing (kvpop_running_topk_noalloc keeps a static device
 *    array, described there) and between calls keeps only a per-device cache of
 *    the compute-unit count, which sets the launch shape of small problems. Every
 *    base pointer must be 16-byte aligned. Outputs are fully overwritten (no
 *    pre-zeroing needed) and must not alias any input or each other.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream). Every
 *    call only enqueues work: it returns once the kernels are launched, and the
 *    caller must keep all buffers alive until the stream has passed them.
 *  - Arguments are validated before anything is launched; on error nothing is
 *    enqueued and no output is touched.
 *  - Thread safety: calls may be made concurrently from several host threads;
 *    the error text of KVPOP_EHIP is kept per thread.
 */
#ifndef KVPOP_H
#define KVPOP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVPOP_ABI_VERSION 3

/* Status codes returned by every entry point. */
enum {
  KVPOP_OK = 0,
  KVPOP_EINVAL = 1,       /* NULL required pointer, non-positive dimension, Hq % Hkv != 0,
                             window < 0, 0 <= horizon < window, scale not finite and > 0,
                             a bad epilogue option (agg, eps, normalize), overlapping
                             buffers, or a size whose element count overflows int64 */
  KVPOP_EUNSUPPORTED = 2, /* head_dim not in {64, 128}, a base pointer not 16-byte
                             aligned, or T above KVPOP_MAX_SEQ_LEN */
  KVPOP_EHIP = 3,         /* the HIP runtime reported an error while launching;
                             kvpop_strerror(KVPOP_EHIP) then returns its text */
  KVPOP_ETOOBIG = 4       /* kvpop_running_topk_noalloc: the problem's workspace exceeds
                             KVPOP_NOALLOC_SCRATCH_BYTES */
};

#define KVPOP_MAX_SEQ_LEN (1 << 24)

/* Problem dimensions (see the conventions above). scale is the softmax scale of
 * eq. dense_logit_app, normally 1 / sqrt(head_dim). */
typedef struct kvpop_dims {
  int32_t batch;      /* B   >= 1 */
  int32_t n_q_heads;  /* Hq  >= 1 */
  int32_t n_kv_heads; /* Hkv >= 1, Hq % Hkv == 0 */
  int32_t seq_len;    /* T   >= 1 */
  int32_t head_dim;   /* D   in {64, 128} */
  float scale;        /* > 0 and finite */
} kvpop_dims;

/* Pass 1 -- dense causal row log-normaliser (App. D.1 eq. dense_lse_app):
 *   lse[b, qh, d] = log sum_{t=0}^{d} exp(l(d, t)).
 * q: bf16 [B,Hq,T,D]; k: bf16 [B,Hkv,T,D]; key_bias: fp32 [T] or NULL;
 * lse: fp32 [B,Hq,T] output. */
int kvpop_row_lse(const kvpop_dims* dims, const void* q, const void* k, const float* key_bias,
                  float* lse, void* stream);

/* Pass 2 -- future mass from a caller-supplied normaliser (App. D.1 eq.
 * future_mass_app, App. D.2):
 *   out[b, qh, t] = sum_{d in band(t)} exp(l(d, t) - lse[b, qh, d]).
 * lse is normally the output of kvpop_row_lse on the same q, k, key_bias, which
 * makes every summand a probability (<= 1). Any other normaliser is accepted,
 * such as the sparse one of Sec. 3.2 eq. sparse_lse_main / App. D.3, which lies
 * below the dense one, so that summands of keys outside its mask exceed 1 without
 * bound. Guard: a workgroup whose fast sweep leaves a column sum above 2^64 (or
 * inf / NaN) recomputes its key block with a per-column running maximum. out is
 * then the fp32 rounding of the mass (within the relative 2e-3 bar), +INFINITY
 * where the mass exceeds the fp32 range (for example lse[d] = -INFINITY for an
 * admissible d), exactly 0 for keys biased -INFINITY. lse must not be NaN. Masses
 * below about 1e-30 lie in or near fp32's subnormal range and carry no relative
 * accuracy.
 * window >= 0; horizon < 0 (unbounded) or horizon >= window. out: fp32 [B,Hq,T]. */
int kvpop_future_attn_from_lse(const kvpop_dims* dims, const void* q, const void* k,
                               const float* key_bias, const float* lse, int32_t window,
                               int32_t horizon, float* out, void* stream);

/* Pass 2 for one or two bands of the same keys from one normaliser, in one sweep
 * (App. B.2: the target with a finite lookahead L and without one, from the same
 * LSE): for b < n_bands,
 *   outs[b][b', qh, t] = sum_{d in band_b(t)} exp(l(d, t) - lse[b', qh, d]),
 * band_b(t) = { d : t + windows[b] <= d <= min(T - 1, t + horizons[b]) }, each exactly
 * as kvpop_future_attn_from_lse computes it (same guard), up to fp32 summation
 * order. Each logit and exponential is evaluated once and added to every band that
 * holds the pair, so a band inside another costs almost nothing.
 * n_bands: 1 or 2. windows, horizons: host arrays of n_bands entries (the rules of
 * kvpop_future_attn_from_lse). outs: host array of n_bands device pointers to fp32
 * [B,Hq,T] outputs, which must not overlap each other or any input. */
int kvpop_future_attn_bands(const kvpop_dims* dims, const void* q, const void* k, const float* key_bias,
                            const float* lse, int32_t n_bands, const int32_t* windows, const int32_t* horizons,
                            float* const* outs, void* stream);

/* Both passes: kvpop_row_lse into lse_ws, then kvpop_future_attn_from_lse from it.
 * lse_ws: caller-allocated fp32 [B,Hq,T]; it holds the dense LSE on completion. */
int kvpop_future_attn_target(const kvpop_dims* dims, const void* q, const void* k,
                             const float* key_bias, int32_t window, int32_t horizon,
                             float* lse_ws, float* out, void* stream);

/* Aggregation over the G query heads of a KV head (App. B.1). */
enum {
  KVPOP_AGG_MAX = 0,  /* eq. max_group_aggregation_app: the paper's default */
  KVPOP_AGG_MEAN = 1  /* eq. mean_group_aggregation_app: probability-space mean */
};

/* Pass 2 plus the target epilogue (App. D.4 step 5; App. B.1-B.2): the per-KV-head
 * target score
 *   scores[b, h, t] = log(A_t + eps) - (normalize ? log N_t : 0),
 *   A_t = max_g out[b, h*G + g, t]  (agg = KVPOP_AGG_MAX)  or  mean_g (KVPOP_AGG_MEAN),
 *   N_t = max(1, |band(t)|)  (eq. future_count_app, clipped by the lookahead),
 * where out is the future mass of kvpop_future_attn_from_lse on the same
 * arguments. eps is added to the aggregated, unnormalised mass before the
 * logarithm, in the order of App. B (the paper leaves eps's value open; it must be
 * finite and >= 0). lse: fp32 [B,Hq,T] (as for kvpop_future_attn_from_lse).
 * out: fp32 [B,Hq,T] per-head masses, or NULL to skip writing them.
 * scores: fp32 [B,Hkv,T] output. normalize: 0 or 1. */
int kvpop_future_attn_scores(const kvpop_dims* dims, const void* q, const void* k, const float* key_bias,
                             const float* lse, int32_t window, int32_t horizon, int32_t agg, float eps,
                             int32_t normalize, float* out, float* scores, void* stream);

/* ---------------------------------------------------------------------------
 * Running top-k ranking (App. B.3, App. C; Sec. 3.1 eqs. eligible_set and
 * teacher_label). Independent of the attention passes: it works on one score per
 * (batch row, KV head, position), either the target of kvpop_future_attn_scores
 * (the teacher) or a scorer's prediction (the student's sparse mask).
 *
 * For each (b, h) sequence r[b, h, 0..T-1]:
 *   prio_t   = fl(r_t - fl(t * log_gamma[h]))      float32, decay step 1
 *              (eq. static_priority_app; log_gamma NULL means no decay)
 *   rank_t   = position of t in descending prio order, ties to the smaller t
 *              (rank 0 = highest priority)
 *   E(q)     = {t : sinks <= t <= q - window}       (eq. eligible_set)
 *   cutoff_q = the k-th smallest rank in E(q) if |E(q)| >= k, else T (every
 *              eligible token kept); the retained long-range keys of query q are
 *              the t in E(q) with rank_t <= cutoff_q (App. C.1 eq.
 *              running_topk_mask_app, App. C.2)
 *   label_q  = +1 if t_new = q - window is retained, -1 if not, 0 if E(q) is
 *              empty (eq. teacher_label)
 *   boundary_q = the retained token of E(q) with the largest rank (the teacher's
 *              cutoff token t_bnd), -1 if E(q) is empty
 *   evict_t  = the first query q >= t that no longer keeps token t under the mask
 *              of App. C.1 eq. running_topk_mask_app, T if every later query keeps
 *              it. The cutoff never increases with q (before saturation it is T;
 *              after, the k-th smallest rank of a growing set), so a dropped token
 *              never returns and that mask is exactly  t <= q < evict_t:
 *              evict_t = T for t < sinks, else
 *              min(T, max(t + window, first q with cutoff_q < rank_t)).
 * --------------------------------------------------------------------------- */
typedef struct kvpop_topk_dims {
  int32_t batch;    /* B >= 1 */
  int32_t n_heads;  /* H >= 1 (KV heads) */
  int32_t seq_len;  /* T >= 1, T <= KVPOP_MAX_SEQ_LEN */
} kvpop_topk_dims;

/* Bytes of device workspace kvpop_running_topk needs for these dimensions
 * (0 if they are invalid). */
size_t kvpop_running_topk_workspace_size(const kvpop_topk_dims* dims);

/* scores: fp32 [B,H,T]; log_gamma: fp32 [H] or NULL; sinks >= 0, window >= 0,
 * topk >= 1. Outputs int32 [B,H,T]: rank and cutoff (required), label, boundary and
 * evict (optional, NULL to skip). workspace: caller-allocated device memory of at least
 * kvpop_running_topk_workspace_size bytes, 16-byte aligned; its contents on entry
 * do not matter. All outputs are fully overwritten. */
int kvpop_running_topk(const kvpop_topk_dims* dims, const float* scores, const float* log_gamma, int32_t sinks,
                       int32_t window, int32_t topk, int32_t* rank, int32_t* cutoff, int32_t* label,
                       int32_t* boundary, int32_t* evict, void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of device scratch that kvpop_running_topk_noalloc holds per GPU (32 MiB:
 * every (B, H, T) with kvpop_running_topk_workspace_size up to this, e.g. B*H = 32
 * sequences of T = 32768 or B*H = 8 of T = 131072). */
#define KVPOP_NOALLOC_SCRATCH_BYTES (32u << 20)

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): kvpop_running_topk with
 * the same arguments and outputs but no workspace argument. Its workspace is a
 * device array of KVPOP_NOALLOC_SCRATCH_BYTES inside the library, one per GPU,
 * held from the first call on that GPU until the process ends; the call allocates
 * nothing. A problem whose kvpop_running_topk_workspace_size exceeds that is
 * rejected with KVPOP_ETOOBIG before anything is launched. All calls on one GPU
 * share its array, whose contents on entry do not matter: calls that overlap on
 * one GPU (unordered streams, or host threads without ordering) race and give
 * wrong results; calls ordered on one stream are safe. The first call on a GPU
 * looks up the array's device address (KVPOP_EHIP if that fails). */
int kvpop_running_topk_noalloc(const kvpop_topk_dims* dims, const float* scores, const float* log_gamma,
                               int32_t sinks, int32_t window, int32_t topk, int32_t* rank, int32_t* cutoff,
                               int32_t* label, int32_t* boundary, int32_t* evict, void* stream);

/* Human-readable text for a status code. For KVPOP_EHIP it is the HIP runtime's
 * message for the last failure on the calling thread. Never returns NULL; the
 * string stays valid until the next library call on the same thread. */
const char* kvpop_strerror(int status);

/* ---------------------------------------------------------------------------
 * Running top-k sparse attention forward (Sec. 3.2; App. C.1 eq.
 * running_topk_mask_app; App. C.3): the student's attention over the keys that
 * its fixed-budget mask keeps, returning the output and the sparse LSE that the
 * target pass consumes (Sec. 3.2 eq. sparse_lse_main; App. D.3).
 *
 * Key t of KV head h is kept by query q iff  t <= q < evict[b, h, t].  With evict
 * from kvpop_running_topk this is exactly the running top-k mask (sinks, protected
 * window, and the eligible tokens whose rank is within the cutoff); evict = T for
 * every key gives dense causal attention and evict[t] = t + w a sliding window.
 * For every (b, qh, q), with h = qh / G and l(q, t) = scale <q, k_t> + key_bias[t]:
 *   lse[b, qh, q]    = log sum_{kept t} exp l(q, t)        (natural log)
 *   o[b, qh, q, :]   = sum_{kept t} exp(l(q, t) - lse) v[b, h, t, :]
 * A query that keeps no key gets o = 0 and lse = -inf.
 *
 * q: bf16 [B,Hq,T,D]; k, v: bf16 [B,Hkv,T,D]; key_bias: fp32 [T] or NULL;
 * evict: int32 [B,Hkv,T]; o: bf16 [B,Hq,T,D] (output); lse: fp32 [B,Hq,T] (output).
 * The probabilities are rounded to bf16 for the product with v; the LSE uses them
 * unrounded. Requirements beyond the common ones: Hq / Hkv a power of two and
 * T * D * 2 < 2^31 (KVPOP_EUNSUPPORTED otherwise); outputs must not overlap any
 * input or each other (KVPOP_EINVAL). Device pointers, 16-byte aligned; the call
 * allocates nothing and is asynchronous on `stream`. */
int kvpop_sparse_attn_fwd(const kvpop_dims* dims, const void* q, const void* k, const void* v,
                          const float* key_bias, const int32_t* evict, void* o, float* lse, void* stream);

/* KVPOP_ABI_VERSION of the loaded library. */
int kvpop_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KVPOP_H */
