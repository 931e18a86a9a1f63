// Internal interface between the C ABI layer (kvpop_api.cpp) and the gfx950
// kernels (kvpop_kernels.hip). Not part of the public ABI.
#pragma once
#include <stdint.h>

namespace kvpop {

// Launch description shared by both passes. All sizes already validated.
struct Launch {
  const uint16_t* q;   // bf16 [B, Hq, T, D]
  const uint16_t* k;   // bf16 [B, Hkv, T, D]
  const float* bias;   // fp32 [T] or nullptr
  const float* lse;    // pass 2 input: fp32 [B, Hq, T]
  float* out;          // pass 1: lse output; pass 2: future-mass output
  int32_t B, Hq, Hkv, T, D;
  float scale;
  int32_t window;      // pass 2 only
  int32_t horizon;     // pass 2 only; < 0 = unbounded
  // Pass 2 with a second band (out1 != nullptr): its masses go to out1, from the
  // same sweep.
  float* out1;         // fp32 [B, Hq, T] or nullptr
  int32_t window1;
  int32_t horizon1;
  // Pass 2 target epilogue (scores != nullptr): per KV head and key,
  // log(agg_g out + eps) - (normalize ? log N_t : 0); agg 0 = max, 1 = mean.
  float* scores;       // fp32 [B, Hkv, T] or nullptr
  int32_t agg;
  float eps;
  int32_t normalize;
  void* stream;        // hipStream_t
};

// Running top-k ranking (kvpop_topk.hip). All sizes already validated.
struct TopkLaunch {
  const float* scores;     // fp32 [B, H, T]
  const float* log_gamma;  // fp32 [H] or nullptr (no decay)
  int32_t B, H, T;
  int32_t sinks, window, topk;
  int32_t* rank;           // [B, H, T] out
  int32_t* cutoff;         // [B, H, T] out
  int32_t* label;          // [B, H, T] out or nullptr
  int32_t* boundary;       // [B, H, T] out or nullptr
  int32_t* evict;          // [B, H, T] out or nullptr
  void* workspace;         // topk_workspace_words_per_seq(T) * B * H uint32 words
  void* stream;
};

// Running top-k sparse attention forward (kvpop_sparse_attn.hip). All sizes
// already validated; the plan fields are filled by sparse_attn_plan.
struct SparseLaunch {
  const uint16_t* q;      // bf16 [B, Hq, T, D]
  const uint16_t* k;      // bf16 [B, Hkv, T, D]
  const uint16_t* v;      // bf16 [B, Hkv, T, D]
  const float* bias;      // fp32 [T] or nullptr
  const int32_t* evict;   // int32 [B, Hkv, T]
  uint16_t* o;            // bf16 [B, Hq, T, D] out
  float* lse;             // fp32 [B, Hq, T] out
  int32_t B, Hq, Hkv, T, D;
  float scale;
  void* stream;
  // plan
  int32_t G, hpw, wq, qt, hc, nch, ntiles;
  int32_t run;            // query tiles per workgroup
  float c;                // scale * log2(e)
};
void sparse_attn_plan(SparseLaunch& L);

// Each returns 0 on success or the hipError_t of a failed launch.
int launch_row_lse(const Launch& L);
int launch_future_mass(const Launch& L);
int launch_running_topk(const TopkLaunch& L);
int launch_sparse_attn_fwd(SparseLaunch L);
size_t topk_workspace_words_per_seq(int T);
// Compute units of the device of `stream` (looked up once per device); 0 if unknown.
int stream_cus(void* stream);
// Device address of the no-allocation scratch array on the device of `stream`
// (resolved once per device); 0 or a hipError_t.
int noalloc_scratch(void* stream, void** ptr);

}  // namespace kvpop
