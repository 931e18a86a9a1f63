// gfx950 (MI355X) kernels for the KVpop future-attention target.
//
// Pass 1 (row_lse_kernel):      LSE_d = log sum_{t <= d} exp l(d, t)
//                               (KVpop App. D.1, eq. dense_lse_app)
// Pass 2 (future_mass_kernel):  m_t = sum_{d in band(t)} exp(l(d, t) - LSE_d)
//                               (KVpop App. D.1, eq. future_mass_app)
// with l(d, t) = scale * <q_d, k_t> + bias_t (eq. dense_logit_app plus an optional
// per-key bias). The paper evaluates pass 2 as the log-sum-exp of a transposed
// attention call (App. D.2); here the same column sums are accumulated directly in
// linear space, which needs no running maximum because every summand is a
// probability (<= 1) when LSE_d is the dense normaliser.
//
// Both passes recompute the logits with bf16 MFMA (v_mfma_f32_16x16x32_bf16) and
// never store the T x T matrix. The reduced index is always put on the MFMA's M
// (row) axis, so the sum for one output position stays inside one lane across a
// whole sweep (four lanes hold the rows of one column; they are combined once at
// the end): pass 1 computes tiles of K Q^T (keys on rows, queries on columns),
// pass 2 tiles of Q K^T (queries on rows, keys on columns). The operand a
// workgroup owns for its whole life (Q columns in pass 1, K columns in pass 2)
// sits in registers as the MFMA B operand; the streamed operand (the A operand)
// goes through double-buffered LDS tiles that all four waves read, so the query
// heads of one GQA group share each K tile (pass 1) and all key columns of a
// workgroup share each Q tile (pass 2).
//
// MFMA 16x16x32 lane layout (checked on gfx950): A row m = lane % 16 holds
// k = 8 (lane / 16) .. +7; B column n = lane % 16 holds the same k range; the 4
// accumulators of a lane are column n = lane % 16, rows 4 (lane / 16) + r. The
// contraction over the head dimension is order-free, so k-step s of lane l takes
// the 16-byte chunk 4 s + l / 16 of the head vector in both operands. The 16x16
// form is used rather than 32x32x16 because its MFMA chains are independent within
// a step and because the chip holds a higher clock under it (measured: 2.30 against
// 1.99 GHz at the same MFMA-busy share).
//
// Cost model. Per pair and pass the path needs 2 D MFMA flops and, on the vector
// ALU, one fma, one exp (half rate on gfx950) and one add: at D = 128 the VALU
// work equals the MFMA time at peak, so the kernels overlap the two explicitly
// (software-pipelined MFMA chains interleaved with the previous chain's
// exponentials) and keep every other VALU instruction out of the hot loop:
// tile loads go straight from global memory to LDS through buffer descriptors,
// whose range check zero-fills rows past the sequence end instead of clamping
// addresses.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>
#include <utility>


#include "kvpop_internal.h"

namespace kvpop {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// Floor of the running maximum in pass 1 (log2 units). Finite, so differences of
// two maxima never become inf - inf.
constexpr float kMaxFloor = -1.0e38f;
// A tile's partial sum above this means the reference maximum was too low.
constexpr float kOverflow = 18446744073709551616.0f;  // 2^64
// Pass 2 factors exp(bias_t) out of key t's sum only for |bias_t| <= kBiasFast
// (natural-log units); larger finite biases take the exact sweep.
constexpr float kBiasFast = 30.0f;
// Buffer descriptor word 3 for raw (untyped) gfx9 buffer access.
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// A 32-row x D bf16 tile in LDS (key rows in pass 1, query rows in pass 2) for the
// 16x16x32 layout, stored as 2 * KS4 planes of 1 KB (KS4 = D / 32 k-steps). Plane
// qs * KS4 + s holds rows 16 qs .. 16 qs + 15, chunks 4 s .. 4 s + 3, lane l's A
// operand at byte 16 l: row 16 qs + l % 16, chunk 4 s + l / 16. One contiguous,
// conflict-free 1 KB read per (16-row subtile qs, k-step), addressed by a register
// plus an immediate offset.
template <int D>
struct Tile16 {
  static constexpr int KS4 = D / 32;
  static constexpr int PLANES = 2 * KS4;
  static constexpr int ELEMS = 32 * D;
  static constexpr int PLANE = 512;  // bf16 elements per plane

  // Byte offset in a row-major [rows, D] matrix of the chunk lane l copies into its
  // plane slot for query subtile qs (the k-step adds 64 s bytes).
  static __device__ __forceinline__ int lane_voffset(int lane, int qs) {
    return (16 * qs + (lane & 15)) * D * 2 + (lane >> 4) * 16;
  }

  // Copy NP consecutive planes starting at plane p0 of the tile whose first row is
  // `rows` (`valid` <= 32 rows readable; rows >= valid read as zero) into `lds`.
  template <int NP>
  static __device__ __forceinline__ void planes_to_lds(uint16_t* lds, const uint16_t* rows, int valid, int p0,
                                                       int voff0, int voff1) {
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(rows), (short)0, valid * D * 2, kRsrcWord3);
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int p = p0 + i, qs = p / KS4, s = p - qs * KS4;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)(lds + p * PLANE), 16, qs ? voff1 : voff0, s * 64, 0,
                                               0);
    }
  }

  static __device__ __forceinline__ bf16x8 frag(const uint16_t* lds, int lane, int qs, int s) {
    return *reinterpret_cast<const bf16x8*>(lds + (qs * KS4 + s) * PLANE + lane * 8);
  }
};

// ---------------------------------------------------------------------------
// Pass 1: row log-normaliser.
//
// Workgroup = (batch b, KV head h, head chunk pc of P query heads, query block of
// BQ = 16 NW NQ / P positions). Its NW waves x NQ column subtiles of 16 (head,
// query) columns keep their Q rows in registers as the B operand of
// v_mfma_f32_16x16x32_bf16. One step streams KT = 4 key tiles of 32 rows through
// LDS (each wave copies all or half of one), shared by all P heads. A lane holds,
// per key tile, 8 key rows (2 key subtiles x 4) of each of its NQ query columns.
//
// Normalisation: every lane keeps, per query column, a reference maximum m (log2
// units) and sum = sum exp2(x - m) over its rows of each tile. Key tiles are
// visited diagonal-first: the tiles that straddle the diagonal (and any step that
// shares them) update (m, sum) exactly, as in online softmax. Every later step lies
// strictly below the diagonal and takes the exponentials against the current m with
// no per-element maximum; a lane whose running sum exceeds 2^64 after the step
// flags it, and the step is then redone exactly from the LDS tiles. Any term above
// 2^64 (a logit more than 64 log2-units above m, or inf) raises the sum past that
// bound; a sum that gets there from smaller terms only costs a redo. The result is
// the same LSE; the common path costs one fma, one exp and one add per pair.
// ---------------------------------------------------------------------------
// NW waves per workgroup: 4 (one per SIMD, two workgroups per CU), or 8 with NQ = 2
// (two per SIMD, each holding half of a 4-wave workgroup's columns; at most 128
// VGPRs, so that two such workgroups still share a CU).
template <int D, int P, bool HAS_BIAS, int NQ, int NW>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * NW, 64 * NW),
                          amdgpu_waves_per_eu(NW == 8 ? 4 : 2, NW == 8 ? 4 : 2))) void
row_lse_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const float* __restrict__ bias,
               float* __restrict__ lse, int B, int Hq, int Hkv, int T, float c, float inv_scale, int nqb, int xg,
               int zh) {
  static_assert(NQ == 2 || NQ == 4, "16-query column subtiles per wave");
  static_assert(NW == 4 || (NW == 8 && NQ == 2), "4 waves, or 8 waves of 2 subtiles");
  constexpr int KT = 4;   // 32-key tiles per step
  using TL = Tile16<D>;
  constexpr int KS4 = TL::KS4;
  constexpr int NPW = TL::PLANES * KT / NW;  // LDS planes each wave copies per step
  constexpr int SPH = NW * NQ / P;  // column subtiles per head
  static_assert(SPH >= 1, "at least one subtile per head");
  constexpr int BQ = 16 * SPH;
  constexpr int NV = 2 * 4 * NQ;        // values per lane and key tile
  constexpr int SLOTS = 2 * KS4 * NQ;   // MFMAs per key tile
  constexpr int V = NV / SLOTS;         // values per MFMA slot
  static_assert(V * SLOTS == NV, "values per slot");
  __shared__ __attribute__((aligned(16))) uint16_t sk0[KT * TL::ELEMS];
  __shared__ __attribute__((aligned(16))) uint16_t sk1[KT * TL::ELEMS];
  __shared__ __attribute__((aligned(16))) float sb0[KT * 32];
  __shared__ __attribute__((aligned(16))) float sb1[KT * 32];

  const int tid = threadIdx.x, lane = tid & 63, quad = lane >> 4, l16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index, uniform per wave
  const int G = Hq / Hkv;
  const int npc = G / P;
  const int per = B * Hkv * npc;
  // Workgroup order: heaviest (last) query block first. Workgroups are dealt to the
  // 8 XCDs round-robin (XCD = blockIdx % 8). With xg > 0 (per a multiple of 8) XCD x
  // owns the (b, KV head, head chunk) groups x, x + 8, ... and runs them xg at a
  // time, so that fewer groups share its L2; otherwise the order is query block
  // major over all groups. With zh > 0 (a grid of zh to 2 zh workgroups, zh the
  // number of CUs) every workgroup starts at once, and the dispatcher gives workgroup
  // i + zh the CU of workgroup i: the second zh take the blocks lightest first, so
  // that each CU pairs a heavy block with a light one.
  int order, rest;
  if (xg > 0) {
    const int x = (int)(blockIdx.x & 7), j = (int)(blockIdx.x >> 3);
    const int span = xg * nqb;
    const int batch = j / span, r = j - batch * span;
    order = r / xg;
    rest = x + 8 * (batch * xg + r - order * xg);
  } else if (zh > 0 && (int)blockIdx.x >= zh) {
    const int j = (int)blockIdx.x - zh;
    order = nqb - 1 - j / per;
    rest = j - (j / per) * per;
  } else {
    order = blockIdx.x / per;
    rest = blockIdx.x - order * per;
  }
  const int qb = nqb - 1 - order;  // 0 = last (heaviest) query block
  const int b = rest / (Hkv * npc);
  rest -= b * Hkv * npc;
  const int h = rest / npc;
  const int pc = rest - h * npc;
  const int i0 = qb * BQ;

  int qs[NQ], qh[NQ];
  bf16x8 qf[NQ][KS4];  // this lane's query rows (B operand), resident for the whole sweep
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    const int u = w * NQ + n;
    qs[n] = i0 + 16 * (u % SPH);
    qh[n] = h * G + pc * P + u / SPH;
    const uint16_t* row = Q + ((size_t)(b * Hq + qh[n]) * T + min(qs[n] + l16, T - 1)) * D;
#pragma unroll
    for (int s = 0; s < KS4; ++s) qf[n][s] = *reinterpret_cast<const bf16x8*>(row + (4 * s + quad) * 8);
  }

  const uint16_t* Kbh = K + (size_t)(b * Hkv + h) * T * D;
  const int kend = min(T, i0 + BQ);
  const int nkt = (kend + 31) / 32;  // key tiles 0 .. nkt - 1
  const int nfull = i0 / 32;         // tiles with every key below the block's first query
  const int ndiag = nkt - nfull;
  const int nsteps = (nkt + KT - 1) / KT;
  const int diag_steps = (ndiag + KT - 1) / KT;
  // Visiting order: diagonal tiles from the top down, then the rest from key 0 up
  // (so the workgroups of one KV head stream the same K tiles at the same time).
  auto tile_of = [&](int idx) __attribute__((always_inline)) { return idx < ndiag ? nkt - 1 - idx : idx - ndiag; };

  const int voff0 = TL::lane_voffset(lane, 0), voff1 = TL::lane_voffset(lane, 1);
  float stb = 0.f;  // raw bias of this thread's key row of the next step
  auto issue = [&](int s, uint16_t* sk) __attribute__((always_inline)) {
    // Wave w copies planes (w / KT) NPW .. of key tile w % KT of the step.
    const int wt = NW == KT ? w : w % KT;
    const int idx = s * KT + wt;
    if (idx < nkt) {
      const int t0 = tile_of(idx) * 32;
      TL::template planes_to_lds<NPW>(sk + wt * TL::ELEMS, Kbh + (size_t)t0 * D, min(32, T - t0),
                                      NW == KT ? 0 : (w / KT) * NPW, voff0, voff1);
    }
    if (HAS_BIAS && tid < KT * 32) {
      const int idx2 = s * KT + (tid >> 5);
      const int t = idx2 < nkt ? tile_of(idx2) * 32 + (tid & 31) : T;
      stb = t < T ? bias[t] : 0.f;
    }
  };
  // The arithmetic on the loaded bias stays here, after the step's compute: a use
  // of it right after the load would wait for every outstanding vector-memory
  // operation, the K tiles of the next step included.
  auto commit = [&](float* sb) __attribute__((always_inline)) {
    if (HAS_BIAS && tid < KT * 32) sb[tid] = stb * inv_scale;
  };

  float m[NQ], sum[NQ];
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    m[n] = kMaxFloor;
    sum[n] = 0.f;
  }

  // Accumulator start value of key subtile ks of tile u: 0, or bias_t / scale on
  // this lane's key rows, so that acc * c = (scale <q, k_t> + bias_t) * log2(e).
  auto acc_init = [&](const float* sb, int u, int ks) __attribute__((always_inline)) {
    if (!HAS_BIAS) return f32x4{};
    return *reinterpret_cast<const f32x4*>(&sb[u * 32 + 16 * ks + 4 * quad]);
  };

  // Exact online update of (m, sum) with the admissible entries of one tile.
  auto exact_tile = [&](const uint16_t* sk, const float* sb, int u, int t0) __attribute__((always_inline)) {
#pragma unroll
    for (int n = 0; n < NQ; ++n) {
      if (t0 > qs[n] + 15) continue;  // every key of the tile is after every query
      const bool partial = t0 + 31 > qs[n];
      f32x4 acc[2];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        acc[ks] = acc_init(sb, u, ks);
#pragma unroll
        for (int s = 0; s < KS4; ++s) acc[ks] = mfma16(TL::frag(sk + u * TL::ELEMS, lane, ks, s), qf[n][s], acc[ks]);
      }
      const int q = qs[n] + l16;
      float v[8];
      float tmax = kMaxFloor;
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        v[rr] = acc[rr >> 2][rr & 3] * c;
        if (partial && t0 + 16 * (rr >> 2) + 4 * quad + (rr & 3) > q) v[rr] = -__builtin_inff();
        tmax = fmaxf(tmax, v[rr]);
      }
      const float mn = fmaxf(m[n], tmax);
      float e = exp2_fast(v[0] - mn);
#pragma unroll
      for (int rr = 1; rr < 8; ++rr) e += exp2_fast(v[rr] - mn);
      sum[n] = sum[n] * exp2_fast(m[n] - mn) + e;
      m[n] = mn;
    }
  };
  // The exact path over every valid tile of a step.
  auto exact_step = [&](int s, const uint16_t* sk, const float* sb) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < KT; ++u) {
      const int idx = s * KT + u;
      if (idx < nkt) exact_tile(sk, sb, u, tile_of(idx) * 32);
    }
  };

  // Fast path: a software pipeline over the KT key tiles of the step with a fixed
  // issue order (scheduling barriers keep the compiler from regrouping it). Tile
  // u's unit runs 2 NQ independent MFMA chains k-step by k-step, so each A fragment
  // read from LDS feeds NQ MFMAs; the fragment register is then refilled with tile
  // u + 1's operand (used a whole unit later). Each MFMA slot also issues the VALU
  // work of tile u - 1's values, pipelined over three slots (the fma of value v, the
  // exp of value v - V and the add of value v - 2 V), query column fastest so that
  // consecutive adds go to different partial sums.
  auto fast_step = [&](const uint16_t* sk, const float* sb) __attribute__((always_inline)) {
    float nm[NQ];
#pragma unroll
    for (int n = 0; n < NQ; ++n) nm[n] = -m[n];
    bf16x8 fr[2][KS4];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int s = 0; s < KS4; ++s) fr[ks][s] = TL::frag(sk, lane, ks, s);
    f32x4 acc_prev[2][NQ];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u <= KT; ++u) {
      f32x4 acc[2][NQ];
      if (u < KT) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const f32x4 a0 = acc_init(sb, u, ks);
#pragma unroll
          for (int n = 0; n < NQ; ++n) acc[ks][n] = a0;
        }
      }
      float ts[NQ], y[NV], x[NV];
      auto add = [&](int vv) __attribute__((always_inline)) {
        const int n = vv % NQ;
        ts[n] = vv < NQ ? x[vv] : ts[n] + x[vv];  // the first terms seed the sums
      };
      int slot = 0;
#pragma unroll
      for (int s = 0; s < KS4; ++s) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
          for (int n = 0; n < NQ; ++n) {
            if (u < KT) {
              acc[ks][n] = mfma16(fr[ks][s], qf[n][s], acc[ks][n]);
              if (n == NQ - 1 && u + 1 < KT) fr[ks][s] = TL::frag(sk + (u + 1) * TL::ELEMS, lane, ks, s);
            }
            if (u > 0) {
#pragma unroll
              for (int e = 0; e < V; ++e) {
                const int vv = slot * V + e;
                const int vn = vv % NQ, rr = vv / NQ;
                y[vv] = __builtin_fmaf(acc_prev[rr >> 2][vn][rr & 3], c, nm[vn]);
                if (vv >= V) x[vv - V] = exp2_fast(y[vv - V]);
                if (vv >= 2 * V) add(vv - 2 * V);
              }
            }
            ++slot;
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      }
      if (u > 0) {
#pragma unroll
        for (int vv = NV - V; vv < NV; ++vv) x[vv] = exp2_fast(y[vv]);
#pragma unroll
        for (int vv = NV - 2 * V; vv < NV; ++vv) add(vv);
#pragma unroll
        for (int n = 0; n < NQ; ++n) sum[n] += ts[n];
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int n = 0; n < NQ; ++n) acc_prev[ks][n] = acc[ks][n];
    }
    bool ovf = false;
#pragma unroll
    for (int n = 0; n < NQ; ++n) ovf |= !(sum[n] <= kOverflow);
    return ovf;
  };

  auto step = [&](int s, const uint16_t* sk, const float* sb, uint16_t* nsk, float* nsb) __attribute__((always_inline)) {
    const bool more = s + 1 < nsteps;
    if (more) issue(s + 1, nsk);
    if (s >= diag_steps && (s + 1) * KT <= nkt) {
      float saved[NQ];
#pragma unroll
      for (int n = 0; n < NQ; ++n) saved[n] = sum[n];
      const bool ovf = fast_step(sk, sb);
      if (__builtin_amdgcn_ballot_w64(ovf) != 0) {
        // Some lane met a logit far above its reference maximum: redo exactly.
#pragma unroll
        for (int n = 0; n < NQ; ++n) sum[n] = saved[n];
        exact_step(s, sk, sb);
      }
    } else {
      exact_step(s, sk, sb);
    }
    if (more) commit(nsb);
    __syncthreads();
  };

  issue(0, sk0);
  commit(sb0);
  __syncthreads();
  for (int s = 0; s < nsteps; s += 2) {
    step(s, sk0, sb0, sk1, sb1);
    if (s + 1 < nsteps) step(s + 1, sk1, sb1, sk0, sb0);
  }

  // Merge the four lane partials of each column and write LSE (natural log).
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    float mm = m[n], sm = sum[n];
#pragma unroll
    for (int sh = 16; sh <= 32; sh *= 2) {
      const float mo = __shfl_xor(mm, sh);
      const float so = __shfl_xor(sm, sh);
      const float mx = fmaxf(mm, mo);
      sm = sm * exp2_fast(mm - mx) + so * exp2_fast(mo - mx);
      mm = mx;
    }
    const int q = qs[n] + l16;
    if (quad == 0 && q < T) lse[(size_t)(b * Hq + qh[n]) * T + q] = (mm + __log2f(sm)) * kLn2;
  }
}

// ---------------------------------------------------------------------------
// Pass 2: future mass per key.
//
// Workgroup = (batch b, KV head h, key block of BK = 4 * WK keys); wave w owns
// NSUB key subtiles of 16 (WK = 16 NSUB keys) whose K rows stay in registers as the
// B operand of v_mfma_f32_16x16x32_bf16. The workgroup sweeps the query tiles of 32
// rows that can see its keys from the last one down; one step stages the tiles of
// GC query heads of the group (two consecutive tiles when GC = 1) in LDS together
// with their LSE values, and every wave reads them all. Descending order keeps the
// key blocks of one KV head -- which all end at the last query row -- on the same
// tile at the same time, so they share it through L2.
//
// MFMA 16x16x32 lane layout (checked on gfx950): A row m = lane % 16 holds
// k = 8 (lane / 16) .. +7; B column n = lane % 16 holds the same k range; the 4
// accumulators of a lane are column n = lane % 16, rows 4 (lane / 16) + r. So k-step
// s of lane l takes the 16-byte chunk 4 s + l / 16 of the head vector in both
// operands, a 32-row query tile is two 16-row subtiles (qs), and a lane holds, per
// head and step, 8 query rows (2 qs x 4 r) of each of its NSUB keys.
//
// Per head and step a wave runs 2 NSUB independent MFMA chains of D / 32 k-steps
// (8 chains at NSUB = 4): no MFMA waits for its predecessor in the chain. Every lane
// accumulates, for its key columns, exp2(acc * c - LSE_d * log2 e) over its rows of
// each tile into a per-tile sum and then into a running column sum (a two-level sum
// keeps the fp32 error near (8 + tiles) ulp). At the end the four lane sums of each
// column are added and written: each workgroup owns its output columns, so results
// are deterministic, with no atomics. (A small grid splits the query heads of a key
// block over several workgroups; each still owns its (head, key) outputs and sums
// them in the same order.)
//
// Query rows beyond T get LSE = +inf in LDS, which zeroes their terms. A per-key
// bias is factored out of the sum, out_t = exp(bias_t) * sum_d exp(...). Query
// heads are processed GC at a time; G / GC chunks each repeat the sweep. With one
// head at a time (GC = 1) a step stages two consecutive query tiles of it, so the
// sweep takes half as many steps: on small grids the heaviest key block's chain of
// steps sets the time, and each step pays a barrier and the load latency.
//
// Guard. The fast sweep sums exp2(x) against the fixed reference 0, which is safe
// when every summand is a probability (the dense normaliser) and the factored bias
// is moderate. A caller-supplied normaliser may be smaller than the dense one (the
// sparse normaliser of App. D.3), so summands can exceed 1 without bound; a large
// bias makes the factored sum overflow or underflow. So: a workgroup whose keys
// carry a finite bias beyond +-kBiasFast runs the exact sweep from the start, and
// after a fast sweep any column sum above 2^64 (or inf / NaN) sends the whole
// workgroup through the exact sweep again. The exact sweep keeps, per column, a
// running maximum m of the summands' exponents (bias included) and the sum
// relative to it, rescaled whenever m grows, and writes exp2(m + log2 sum): the
// fp32 rounding of the mass, +inf only when the mass itself exceeds the fp32 range.
// Keys with bias -inf are never attended and get exactly 0.
//
// With EPI the kernel also finishes the target (App. D.4 step 5, App. B.1-B.2):
// it folds the G per-head masses of each key into their max or sum as the chunks
// complete, and writes log(agg + eps) - log N_t per KV head, where N_t = max(1,
// number of admissible queries). The per-head masses are then written only when
// `out` is given.
// ---------------------------------------------------------------------------

template <int D, int NSUB, int GC, bool HAS_BIAS, bool EPI, int NB>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(2, 2))) void
future_mass_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const float* __restrict__ bias,
                   const float* __restrict__ lse, float* __restrict__ out, int B, int Hq, int Hkv, int T, float c,
                   int window, int hz, float* __restrict__ scores, int agg_mean, float eps, int normalize,
                   int xgroups, int hs, int window1, int hz1, float* __restrict__ out1) {
  static_assert(NB == 1 || (NB == 2 && !EPI), "a second band only without the epilogue");
  using TL = Tile16<D>;
  constexpr int KS4 = TL::KS4;
  constexpr int WK = NSUB * 16;  // keys per wave
  constexpr int BK = 4 * WK;     // keys per workgroup
  // A step stages U = GC * TPS query tiles ("units"): TPS consecutive tiles of each
  // of GC heads. One head per step (GC = 1) takes two tiles, so that a sweep has
  // half as many steps (each step's barrier and load latency paid half as often).
  constexpr int TPS = GC == 1 ? 2 : 1;
  constexpr int U = GC * TPS;
  constexpr int PPW = U * TL::PLANES / 4;  // LDS planes each wave copies per step
  static_assert(PPW >= 1 && TL::PLANES % PPW == 0, "plane split");
  constexpr int NV = 8 * NSUB;              // values per lane, unit and step
  constexpr int SLOTS = 2 * KS4 * NSUB;     // MFMAs per unit and step
  constexpr int V = NV / SLOTS;             // values per MFMA slot
  static_assert(V * SLOTS == NV, "values per slot");
  __shared__ __attribute__((aligned(16))) uint16_t sq0[U * TL::ELEMS];
  __shared__ __attribute__((aligned(16))) uint16_t sq1[U * TL::ELEMS];
  __shared__ __attribute__((aligned(16))) float sl0[U * 32];
  __shared__ __attribute__((aligned(16))) float sl1[U * 32];

  const int tid = threadIdx.x, lane = tid & 63, quad = lane >> 4, l16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index, uniform per wave
  const int G = Hq / Hkv;
  const int nbh = B * Hkv;
  // Workgroup order. Workgroups are dealt to the 8 XCDs round-robin (XCD =
  // blockIdx % 8). With xgroups > 0 (B * Hkv a multiple of 8), XCD x owns the
  // (b, KV head) groups x, x + 8, ... and runs them xgroups at a time, each batch
  // of groups heaviest key block first: more workgroups of one group then sweep
  // the same query tiles together and share them in that XCD's L2. Otherwise the
  // order is key block major, heaviest first, over all groups.
  // A head-split launch (a small grid, no epilogue) gives each (key block, group)
  // hs workgroups, workgroup ch taking the head chunks ch, ch + hs, ...; key block
  // major, heaviest first. Every workgroup still owns its output columns.
  int kb, bh, ch = 0;
  if (hs > 1) {
    const int per = nbh * hs;
    kb = blockIdx.x / per;
    const int r = blockIdx.x - kb * per;
    bh = r / hs;
    ch = r - bh * hs;
  } else if (xgroups > 0) {
    const int nkb = (T + BK - 1) / BK;
    const int x = (int)(blockIdx.x & 7), j = (int)(blockIdx.x >> 3);
    const int span = xgroups * nkb;
    const int batch = j / span, r = j - batch * span;
    kb = r / xgroups;
    bh = x + 8 * (batch * xgroups + r - kb * xgroups);
  } else {
    kb = blockIdx.x / nbh;
    bh = blockIdx.x - kb * nbh;
  }
  const int b = bh / Hkv;
  const int h = bh - b * Hkv;
  const int j0 = kb * BK;
  const int jw = j0 + w * WK;

  // Query rows that can reach any key of the block: [j0 + window, j0 + BK - 1 + hz] within [0, T).
  // With a second band, the union of the two bands' ranges.
  const int wlo = NB == 2 ? min(window, window1) : window;
  const int hhi = NB == 2 ? max(hz, hz1) : hz;
  const long long r_lo = (long long)j0 + wlo;
  const long long r_hi = min((long long)T - 1, (long long)j0 + BK - 1 + hhi);
  int qt_hi = 0, nqt = 0;
  if (r_lo <= r_hi) {
    qt_hi = (int)(r_hi / 32);
    nqt = qt_hi - (int)(r_lo / 32) + 1;
  }
  const int nst = (nqt + TPS - 1) / TPS;  // steps; step s covers tiles qt_hi - TPS s - t, t < TPS

  // Bias of this lane's key columns: factored out (fac) by the fast sweep, added to
  // every exponent (bl2, log2 units) by the exact sweep. masked: bias -inf.
  float fac[NSUB], bl2[NSUB];
  bool masked[NSUB];
  bool big = false;
#pragma unroll
  for (int n = 0; n < NSUB; ++n) {
    fac[n] = 1.f;
    bl2[n] = 0.f;
    masked[n] = false;
    if (HAS_BIAS) {
      const int j = min(jw + 16 * n + l16, T - 1);
      const float bj = bias[j];
      masked[n] = bj == -__builtin_inff();
      bl2[n] = masked[n] ? 0.f : bj * kLog2e;
      fac[n] = masked[n] ? 0.f : exp2_fast(bl2[n]);
      big |= !masked[n] && !(__builtin_fabsf(bj) <= kBiasFast);
    }
  }

  float aggv[NSUB];  // running max or sum over query heads (EPI)
#pragma unroll
  for (int n = 0; n < NSUB; ++n) aggv[n] = 0.f;
  auto write_scores = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int n = 0; n < NSUB; ++n) {
      const int j = jw + 16 * n + l16;
      if (quad == 0 && j < T) {
        float r = __logf((agg_mean ? aggv[n] / (float)G : aggv[n]) + eps);
        if (normalize) {
          const long long cnt = min((long long)T - 1, (long long)j + hz) - ((long long)j + window) + 1;
          r -= __logf((float)max(1LL, cnt));
        }
        scores[(size_t)bh * T + j] = r;
      }
    }
  };

  if (nqt == 0) {
    // Every key of the block has an empty query range.
    if (!EPI || out) {
      for (int g = ch * GC; g < G; ++g) {
#pragma unroll
        for (int n = 0; n < NSUB; ++n) {
          const int j = jw + 16 * n + l16;
          if (quad == 0 && j < T && (hs == 1 || (g / GC) % hs == ch)) {
            out[(size_t)(b * Hq + h * G + g) * T + j] = 0.f;
            if (NB == 2) out1[(size_t)(b * Hq + h * G + g) * T + j] = 0.f;
          }
        }
      }
    }
    if (EPI) write_scores();
    return;
  }

  // Workgroup-uniform: any key of the block with a large finite bias.
  const bool all_exact = HAS_BIAS && __syncthreads_or(big);

  bf16x8 kf[NSUB][KS4];  // this lane's key rows (B operand), resident for the whole sweep
  const uint16_t* Kbh = K + (size_t)bh * T * D;
#pragma unroll
  for (int n = 0; n < NSUB; ++n) {
    const uint16_t* row = Kbh + (size_t)min(jw + 16 * n + l16, T - 1) * D;
#pragma unroll
    for (int s = 0; s < KS4; ++s) kf[n][s] = *reinterpret_cast<const bf16x8*>(row + (4 * s + quad) * 8);
  }

  const int voff0 = TL::lane_voffset(lane, 0), voff1 = TL::lane_voffset(lane, 1);
  const int pg = (w * PPW) / TL::PLANES;          // the unit (tile) this wave copies
  const int pp0 = (w * PPW) - pg * TL::PLANES;    // its first plane

  for (int gh0 = h * G + ch * GC; gh0 < (h + 1) * G; gh0 += GC * hs) {
    const size_t head0 = (size_t)(b * Hq + gh0);
    float stl = 0.f;
    // Start the loads of step s: Q tiles straight into LDS, raw LSE into a register.
    // Unit u of step s: head head0 + u / TPS, rows from (qt_hi - TPS s - u % TPS) * 32.
    // A tile below row 0 (the last step of a sweep with an odd tile count) loads
    // nothing (zero rows) and gets LSE = +inf, which zeroes its terms.
    auto issue = [&](int s, uint16_t* sq) __attribute__((always_inline)) {
      const int ti = (qt_hi - TPS * s - pg % TPS) * 32;
      TL::template planes_to_lds<PPW>(sq + pg * TL::ELEMS, Q + ((head0 + pg / TPS) * T + max(ti, 0)) * D,
                                      ti < 0 ? 0 : min(32, T - ti), pp0, voff0, voff1);
      if (tid < U * 32) {
        const int u = tid >> 5;
        const int i = (qt_hi - TPS * s - u % TPS) * 32 + (tid & 31);
        stl = i >= 0 && i < T ? lse[(head0 + u / TPS) * T + i] : __builtin_inff();
      }
    };
    auto commit = [&](float* sl) __attribute__((always_inline)) {
      if (tid < U * 32) sl[tid] = -stl * kLog2e;
    };

    float colsum[GC][NSUB];  // fast sweep: column sums; exact sweep: sums relative to mref
    float colsum1[GC][NSUB]; // fast sweep, second band
    float mref[GC][NSUB];    // exact sweep: running maximum of the exponents (log2 units)

    // -LSE_d log2 e of this lane's rows 16 qs + 4 quad + r of head g: nl[4 qs + r].
    auto read_nl = [&](const float* sl, int g, float (&nl)[8]) __attribute__((always_inline)) {
#pragma unroll
      for (int qs = 0; qs < 2; ++qs) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(&sl[g * 32 + 16 * qs + 4 * quad]);
        nl[4 * qs + 0] = v[0];
        nl[4 * qs + 1] = v[1];
        nl[4 * qs + 2] = v[2];
        nl[4 * qs + 3] = v[3];
      }
    };

    // Fully admissible step, as a software pipeline over the U units with a fixed
    // issue order (the scheduling barriers stop the compiler from regrouping it).
    // Unit g runs its 2 NSUB MFMA chains k-step by k-step, so each A fragment read
    // from LDS feeds NSUB MFMAs; right after those the fragment register is refilled
    // with unit g + 1's operand (used a whole unit later, hiding the LDS latency).
    // Each MFMA slot also issues the VALU work of unit g - 1's values, itself
    // pipelined over three slots: the fma of value v, the exp of value v - V and the
    // add of value v - 2 V, so that the three instructions after one MFMA never wait
    // for each other. Values run key-subtile fastest, so consecutive adds go to
    // different partial sums. i0: the step's first (highest) tile.
    // BANDS: bit b set = band b takes this step's sums (always 1 with one band).
    // MASKED (a band edge, one band, two key subtiles per wave): each unit's
    // accumulators start at 0 on the band's pairs and -inf elsewhere, so pairs
    // outside the band add exp2(-inf) = 0 and the step keeps the pipelined form.
    auto full_step = [&](auto bands_c, auto masked_c, int i0, const uint16_t* sq, const float* sl)
                         __attribute__((always_inline)) {
      constexpr int BANDS = decltype(bands_c)::value;
      constexpr bool MASKED = decltype(masked_c)::value;
      bf16x8 fr[2][KS4];
      float nl[2][8];
      f32x4 acc_prev[2][NSUB];
#pragma unroll
      for (int qs = 0; qs < 2; ++qs)
#pragma unroll
        for (int s = 0; s < KS4; ++s) fr[qs][s] = TL::frag(sq, lane, qs, s);
      read_nl(sl, 0, nl[0]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g <= U; ++g) {
        if (g > 0 && g < U) read_nl(sl, g, nl[g & 1]);
        f32x4 acc[2][NSUB];
#pragma unroll
        for (int qs = 0; qs < 2; ++qs)
#pragma unroll
          for (int n = 0; n < NSUB; ++n) {
            acc[qs][n] = f32x4{};
            if (MASKED && g < U) {
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const int d = i0 - 32 * (g % TPS) + 16 * qs + 4 * quad + r - (jw + 16 * n + l16);
                acc[qs][n][r] = (d >= window && d <= hz) ? 0.f : -__builtin_inff();
              }
            }
          }
        float ts[NSUB];
        float y[NV], x[NV];
        const float(&pnl)[8] = nl[(g + 1) & 1];  // unit g - 1's normalisers
        // value v of unit g - 1: key subtile v % NSUB, row slot v / NSUB = 4 qs + r
        auto val = [&](int v) __attribute__((always_inline)) {
          const int n = v % NSUB, rr = v / NSUB;
          return __builtin_fmaf(acc_prev[rr >> 2][n][rr & 3], c, pnl[rr]);
        };
        auto add = [&](int v) __attribute__((always_inline)) {
          const int n = v % NSUB;
          ts[n] = v < NSUB ? x[v] : ts[n] + x[v];  // the first terms seed the sums
        };
        int slot = 0;
#pragma unroll
        for (int s = 0; s < KS4; ++s) {
#pragma unroll
          for (int qs = 0; qs < 2; ++qs) {
#pragma unroll
            for (int n = 0; n < NSUB; ++n) {
              if (g < U) {
                acc[qs][n] = mfma16(fr[qs][s], kf[n][s], acc[qs][n]);
                if (n == NSUB - 1 && g + 1 < U) fr[qs][s] = TL::frag(sq + (g + 1) * TL::ELEMS, lane, qs, s);
              }
              if (g > 0) {
#pragma unroll
                for (int e = 0; e < V; ++e) {
                  const int v = slot * V + e;
                  y[v] = val(v);
                  if (v >= V) x[v - V] = exp2_fast(y[v - V]);
                  if (v >= 2 * V) add(v - 2 * V);
                }
              }
              ++slot;
              __builtin_amdgcn_sched_barrier(0);
            }
          }
        }
        if (g > 0) {
#pragma unroll
          for (int v = NV - V; v < NV; ++v) x[v] = exp2_fast(y[v]);
#pragma unroll
          for (int v = NV - 2 * V; v < NV; ++v) add(v);
#pragma unroll
          for (int n = 0; n < NSUB; ++n) {
            if (BANDS & 1) colsum[(g - 1) / TPS][n] += ts[n];
            if (BANDS & 2) colsum1[(g - 1) / TPS][n] += ts[n];
          }
        }
#pragma unroll
        for (int qs = 0; qs < 2; ++qs)
#pragma unroll
          for (int n = 0; n < NSUB; ++n) acc_prev[qs][n] = acc[qs][n];
      }
    };

    // Tile on a band edge. Each key subtile of the wave is classified once: outside
    // the band (skipped), inside it (summed without a mask) or across its edge (each
    // pair masked by window <= i - j <= hz). NBS: the bands taken (1 while the second
    // band lies wholly past the step, see the sweep below).
    auto edge_step = [&](auto nbs_c, const uint16_t* sq, const float* sl, int i0) __attribute__((always_inline)) {
      constexpr int NBS = decltype(nbs_c)::value;
#pragma unroll
      for (int g = 0; g < U; ++g) {
        const int iu = i0 - 32 * (g % TPS);
        bool act[NSUB], inside[NSUB], act1[NSUB], inside1[NSUB];
#pragma unroll
        for (int n = 0; n < NSUB; ++n) {
          const int dlo = iu - (jw + 16 * n + 15), dhi = iu + 31 - (jw + 16 * n);
          act[n] = !(dhi < window || dlo > hz);
          inside[n] = dlo >= window && dhi <= hz;
          act1[n] = NBS == 2 && !(dhi < window1 || dlo > hz1);
          inside1[n] = NBS == 2 && dlo >= window1 && dhi <= hz1;
        }
        float nl[8];
        read_nl(sl, g, nl);
#pragma unroll
        for (int n = 0; n < NSUB; ++n) {
          if (!act[n] && !act1[n]) continue;
          f32x4 acc[2];
#pragma unroll
          for (int qs = 0; qs < 2; ++qs) {
            acc[qs] = f32x4{};
#pragma unroll
            for (int s = 0; s < KS4; ++s) acc[qs] = mfma16(TL::frag(sq + g * TL::ELEMS, lane, qs, s), kf[n][s], acc[qs]);
          }
          float ts[2], ts1[2];
          const int base = iu + 4 * quad - (jw + 16 * n + l16);
#pragma unroll
          for (int rr = 0; rr < 8; ++rr) {
            const int d = base + 16 * (rr >> 2) + (rr & 3);
            const float e = exp2_fast(__builtin_fmaf(acc[rr >> 2][rr & 3], c, nl[rr]));
            const float xv = (inside[n] || (d >= window && d <= hz)) ? e : 0.f;
            ts[rr & 1] = rr < 2 ? xv : ts[rr & 1] + xv;  // the first terms seed the sums
            if (NBS == 2) {
              const float xv1 = (inside1[n] || (d >= window1 && d <= hz1)) ? e : 0.f;
              ts1[rr & 1] = rr < 2 ? xv1 : ts1[rr & 1] + xv1;
            }
          }
          if (act[n]) colsum[g / TPS][n] += ts[0] + ts[1];
          if (NBS == 2 && act1[n]) colsum1[g / TPS][n] += ts1[0] + ts1[1];
        }
      }
    };

    // Exact step (guarded sweep): every admissible pair's exponent x = acc * c -
    // LSE_d log2 e + bias_t log2 e, and per column an online update of (mref, colsum)
    // as in online softmax. A summand of +inf (LSE_d = -inf) makes the mass +inf.
    auto exact_step = [&](const uint16_t* sq, const float* sl, int i0, int wb, int hb) __attribute__((always_inline)) {
#pragma unroll
      for (int g = 0; g < U; ++g) {
        const int iu = i0 - 32 * (g % TPS), gh = g / TPS;
        bool act[NSUB];
#pragma unroll
        for (int n = 0; n < NSUB; ++n) {
          const int dlo = iu - (jw + 16 * n + 15), dhi = iu + 31 - (jw + 16 * n);
          act[n] = !(dhi < wb || dlo > hb);
        }
        float nl[8];
        read_nl(sl, g, nl);
#pragma unroll
        for (int n = 0; n < NSUB; ++n) {
          if (!act[n]) continue;
          f32x4 acc[2];
#pragma unroll
          for (int qs = 0; qs < 2; ++qs) {
            acc[qs] = f32x4{};
#pragma unroll
            for (int s = 0; s < KS4; ++s) acc[qs] = mfma16(TL::frag(sq + g * TL::ELEMS, lane, qs, s), kf[n][s], acc[qs]);
          }
          const int base = iu + 4 * quad - (jw + 16 * n + l16);
          float xv[8];
          float tmax = -__builtin_inff();
#pragma unroll
          for (int rr = 0; rr < 8; ++rr) {
            const int d = base + 16 * (rr >> 2) + (rr & 3);
            const float xr = __builtin_fmaf(acc[rr >> 2][rr & 3], c, nl[rr]) + bl2[n];
            xv[rr] = (d >= wb && d <= hb) ? xr : -__builtin_inff();
            tmax = fmaxf(tmax, xv[rr]);
          }
          const float mn = fmaxf(mref[gh][n], tmax);
          if (mn == __builtin_inff()) {
            mref[gh][n] = mn;
            colsum[gh][n] = 1.f;
          } else if (mn > -__builtin_inff()) {
            float e = 0.f;
#pragma unroll
            for (int rr = 0; rr < 8; ++rr) e += exp2_fast(xv[rr] - mn);
            colsum[gh][n] = colsum[gh][n] * exp2_fast(mref[gh][n] - mn) + e;
            mref[gh][n] = mn;
          }
        }
      }
    };

    auto step = [&](auto nbs_c, int s, const uint16_t* sq, const float* sl, uint16_t* nsq, float* nsl)
                    __attribute__((always_inline)) {
      constexpr int NBS = decltype(nbs_c)::value;
      const bool more = s + 1 < nst;
      if (more) issue(s + 1, nsq);
      const int i0 = (qt_hi - TPS * s) * 32;
      // Differences d = i - j over this wave's keys and the step's rows.
      const int dmin = i0 - 32 * (TPS - 1) - (jw + WK - 1);
      const int dmax = i0 + 31 - jw;
      if (NBS == 1) {
        if (dmin >= window && dmax <= hz) {
          full_step(std::integral_constant<int, 1>{}, std::false_type{}, i0, sq, sl);
        } else if (!(dmax < window || dmin > hz)) {
          if (NSUB == 2 && NB == 1) full_step(std::integral_constant<int, 1>{}, std::true_type{}, i0, sq, sl);
          else edge_step(std::integral_constant<int, 1>{}, sq, sl, i0);
        }
      } else {
        // Each band is outside this wave's pairs of the step, covers all of them,
        // or crosses them; any crossing band takes the masked path for both.
        const bool out0 = dmax < window || dmin > hz, full0 = dmin >= window && dmax <= hz;
        const bool out1 = dmax < window1 || dmin > hz1, full1 = dmin >= window1 && dmax <= hz1;
        if ((full0 || out0) && (full1 || out1)) {
          if (full0 && full1) full_step(std::integral_constant<int, 3>{}, std::false_type{}, i0, sq, sl);
          else if (full0) full_step(std::integral_constant<int, 1>{}, std::false_type{}, i0, sq, sl);
          else if (full1) full_step(std::integral_constant<int, 2>{}, std::false_type{}, i0, sq, sl);
        } else {
          edge_step(std::integral_constant<int, 2>{}, sq, sl, i0);
        }
      }
      if (more) commit(nsl);
      __syncthreads();
    };

#pragma unroll
    for (int g = 0; g < GC; ++g)
#pragma unroll
      for (int n = 0; n < NSUB; ++n) colsum[g][n] = 0.f;
    bool bad = false;
    if (!all_exact) {
      issue(0, sq0);
      commit(sl0);
      __syncthreads();
      constexpr auto one_band = std::integral_constant<int, 1>{};
      if constexpr (NB == 1) {
        for (int s = 0; s < nst; s += 2) {
          step(one_band, s, sq0, sl0, sq1, sl1);
          if (s + 1 < nst) step(one_band, s + 1, sq1, sl1, sq0, sl0);
        }
      } else {
        // Two bands. The leading steps (the highest rows) whose every row lies past
        // the second band's horizon for every key of the block take the one-band
        // code, before the second band's sums exist (with them live from the start,
        // register pressure made those steps 4% slower); the rest take both bands.
        // Step s's lowest row is (qt_hi - TPS s - TPS + 1) * 32.
        const long long x = (long long)(qt_hi - TPS + 1) * 32 - ((long long)j0 + BK - 1 + hz1) - 1;
        const int s1 = x < 0 ? 0 : (int)min((long long)nst, x / (32 * TPS) + 1);
        int s = 0;
        for (; s + 1 < s1; s += 2) {
          step(one_band, s, sq0, sl0, sq1, sl1);
          step(one_band, s + 1, sq1, sl1, sq0, sl0);
        }
        if (s < s1) step(one_band, s++, sq0, sl0, sq1, sl1);
#pragma unroll
        for (int g = 0; g < GC; ++g)
#pragma unroll
          for (int n = 0; n < NSUB; ++n) colsum1[g][n] = 0.f;
        constexpr auto two_bands = std::integral_constant<int, 2>{};
        if ((s & 1) && s < nst) {
          step(two_bands, s, sq1, sl1, sq0, sl0);
          ++s;
        }
        for (; s < nst; s += 2) {
          step(two_bands, s, sq0, sl0, sq1, sl1);
          if (s + 1 < nst) step(two_bands, s + 1, sq1, sl1, sq0, sl0);
        }
      }
      // Each of the four lane sums at most 2^62 keeps the column's sum within 2^64.
#pragma unroll
      for (int g = 0; g < GC; ++g)
#pragma unroll
        for (int n = 0; n < NSUB; ++n) {
          bad |= !masked[n] && !(colsum[g][n] <= 0.25f * kOverflow);
          if (NB == 2) bad |= !masked[n] && !(colsum1[g][n] <= 0.25f * kOverflow);
        }
    }

    // Block-wide: a large bias, or a column sum out of the safe range, takes the
    // chunk through the exact sweep.
    if (all_exact || __syncthreads_or(bad)) {
      // One exact sweep per band (over the union of the bands' query tiles).
#pragma unroll
      for (int bd = 0; bd < NB; ++bd) {
        const int wb = bd ? window1 : window, hb = bd ? hz1 : hz;
        float* ob = bd ? out1 : out;
        auto xstep = [&](int s, const uint16_t* sq, const float* sl, uint16_t* nsq, float* nsl)
                         __attribute__((always_inline)) {
          const bool more = s + 1 < nst;
          if (more) issue(s + 1, nsq);
          const int i0 = (qt_hi - TPS * s) * 32;
          const int dmin = i0 - 32 * (TPS - 1) - (jw + WK - 1);
          const int dmax = i0 + 31 - jw;
          if (!(dmax < wb || dmin > hb)) exact_step(sq, sl, i0, wb, hb);
          if (more) commit(nsl);
          __syncthreads();
        };
#pragma unroll
        for (int g = 0; g < GC; ++g)
#pragma unroll
          for (int n = 0; n < NSUB; ++n) {
            colsum[g][n] = 0.f;
            mref[g][n] = -__builtin_inff();
          }
        issue(0, sq0);
        commit(sl0);
        __syncthreads();
        for (int s = 0; s < nst; s += 2) {
          xstep(s, sq0, sl0, sq1, sl1);
          if (s + 1 < nst) xstep(s + 1, sq1, sl1, sq0, sl0);
        }
        // Merge the four lanes' (mref, sum) pairs of each column and write
        // exp2(m + log2 sum).
#pragma unroll
        for (int g = 0; g < GC; ++g) {
#pragma unroll
          for (int n = 0; n < NSUB; ++n) {
            float m = mref[g][n], sm = colsum[g][n];
#pragma unroll
            for (int sh = 16; sh <= 32; sh *= 2) {
              const float mo = __shfl_xor(m, sh);
              const float so = __shfl_xor(sm, sh);
              const float mm = fmaxf(m, mo);
              if (mm == __builtin_inff()) {
                sm = 1.f;
              } else if (mm > -__builtin_inff()) {
                sm = sm * exp2_fast(m - mm) + so * exp2_fast(mo - mm);
              }
              m = mm;
            }
            float v = 0.f;
            if (m == __builtin_inff()) v = m;
            else if (m > -__builtin_inff()) v = exp2_fast(m + __log2f(sm));
            if (masked[n]) v = 0.f;
            const int j = jw + 16 * n + l16;
            if (quad == 0 && j < T && (!EPI || ob)) ob[(head0 + g) * T + j] = v;
            if (EPI) aggv[n] = agg_mean ? aggv[n] + v : fmaxf(aggv[n], v);
          }
        }
      }
    } else {
      // Combine the four lane sums of each column and write this chunk's columns.
#pragma unroll
      for (int g = 0; g < GC; ++g) {
#pragma unroll
        for (int n = 0; n < NSUB; ++n) {
          float v = colsum[g][n] + __shfl_xor(colsum[g][n], 16);
          v += __shfl_xor(v, 32);
          if (HAS_BIAS) v = masked[n] ? 0.f : v * fac[n];
          const int j = jw + 16 * n + l16;
          if (quad == 0 && j < T && (!EPI || out)) out[(head0 + g) * T + j] = v;
          if (EPI) aggv[n] = agg_mean ? aggv[n] + v : fmaxf(aggv[n], v);
          if (NB == 2) {
            float v1 = colsum1[g][n] + __shfl_xor(colsum1[g][n], 16);
            v1 += __shfl_xor(v1, 32);
            if (HAS_BIAS) v1 = masked[n] ? 0.f : v1 * fac[n];
            if (quad == 0 && j < T) out1[(head0 + g) * T + j] = v1;
          }
        }
      }
    }
  }
  if (EPI) write_scores();
}


template <int D, int P, bool HB, int NQ, int NW>
int launch_p1_q(const Launch& L) {
  constexpr int BQ = 16 * NW * NQ / P;
  const int G = L.Hq / L.Hkv;
  const int nqb = (L.T + BQ - 1) / BQ;
  const long long per = (long long)L.B * L.Hkv * (G / P);
  const long long grid = (long long)nqb * per;
  const float c = L.scale * kLog2e;
  // One group at a time per XCD for long sequences (at least 512 query blocks, T >=
  // 32768 at P = 4): at B = 4, T = 32768 pass 1 then fetches 3.2 instead of 9.8 GB
  // from HBM per launch and holds a 2% higher clock.
  const int xg = per % 8 == 0 && nqb >= 512 ? 1 : 0;
  // A grid that the CUs hold at once (two workgroups each) pairs heavy and light
  // blocks on each CU. At B = 1, T = 4096 (512 workgroups) the heaviest CU then has
  // about 33 key steps instead of 48.
  const int ncu = stream_cus(L.stream);
  const int zh = xg == 0 && grid > ncu && grid <= 2LL * ncu && ncu % per == 0 ? ncu : 0;
  hipLaunchKernelGGL((row_lse_kernel<D, P, HB, NQ, NW>), dim3((unsigned)grid), dim3(64 * NW), 0, (hipStream_t)L.stream,
                     reinterpret_cast<const uint16_t*>(L.q), reinterpret_cast<const uint16_t*>(L.k), L.bias, L.out,
                     L.B, L.Hq, L.Hkv, L.T, c, 1.0f / L.scale, nqb, xg, zh);
  return (int)hipGetLastError();
}

// Small grids, by the number of full-height blocks (NQ = 4; P = 8 keeps that form):
//  * at most one per CU: half-height blocks (NQ = 2, 4 waves), twice the workgroups,
//    and the heaviest block, whose sweep sets the time when every workgroup starts
//    at once, has half the work (B = 1, T = 2048: 0.042 -> 0.031 ms);
//  * up to two per CU: full-height blocks as 8 waves of 2 subtiles, two waves per
//    SIMD, so that the heaviest block's MFMA and VALU work overlap even when it has
//    its CU to itself (B = 1, T = 4096: 0.087-0.092 -> 0.084 ms).
template <int D, int P, bool HB>
int launch_p1(const Launch& L) {
  const int G = L.Hq / L.Hkv;
  const long long grid4 = (long long)((L.T + 256 / P - 1) / (256 / P)) * L.B * L.Hkv * (G / P);
  if constexpr (P < 8) {
    const int ncu = stream_cus(L.stream);
    if (grid4 <= ncu) return launch_p1_q<D, P, HB, 2, 4>(L);
    if (grid4 <= 2LL * ncu) return launch_p1_q<D, P, HB, 2, 8>(L);
  }
  return launch_p1_q<D, P, HB, 4, 4>(L);
}

template <int D, int P>
int launch_p1_b(const Launch& L) {
  return L.bias ? launch_p1<D, P, true>(L) : launch_p1<D, P, false>(L);
}

template <int D>
int launch_p1_d(const Launch& L) {
  // Query heads per workgroup: the largest power of two dividing G, at most 8.
  const int G = L.Hq / L.Hkv;
  if (G % 8 == 0) return launch_p1_b<D, 8>(L);
  if (G % 4 == 0) return launch_p1_b<D, 4>(L);
  if (G % 2 == 0) return launch_p1_b<D, 2>(L);
  return launch_p1_b<D, 1>(L);
}

template <int D, int NSUB, int GC, bool HB, bool EPI, int NB>
int launch_p2(const Launch& L, int hs) {
  constexpr int BK = 4 * NSUB * 16;
  const int nkb = (L.T + BK - 1) / BK;
  const long long grid = (long long)nkb * L.B * L.Hkv;
  const float c = L.scale * kLog2e;
  int window = L.window, hz = L.horizon < 0 ? L.T : L.horizon;
  int window1 = L.window1, hz1 = NB == 2 ? (L.horizon1 < 0 ? L.T : L.horizon1) : 0;
  float *out = L.out, *out1 = L.out1;
  // Two bands: the kernel's leading one-band steps serve the band that reaches
  // further, so that band goes first (each band's sums are formed the same way in
  // either place).
  if (NB == 2 && hz1 > hz) {
    std::swap(window, window1);
    std::swap(hz, hz1);
    std::swap(out, out1);
  }
  // Groups an XCD runs at a time: one when a group has at least 128 key blocks
  // (T >= 32768: fewer groups sharing the XCD's L2 means fewer Q re-reads from HBM,
  // 30 -> 21 GB per launch at B = 4, T = 32768, and a higher clock); else half of its
  // groups when it then still has at least 4 workgroups per slot (2 per CU on its 32
  // CUs), so that the second half's heaviest blocks start early enough; otherwise
  // all of them.
  int xgroups = 0;
  const int nbh = L.B * L.Hkv;
  if (nbh % 8 == 0) {
    const int ng = nbh / 8;
    xgroups = nkb >= 128 ? 1 : (ng % 2 == 0 && (long long)ng * nkb >= 4 * 64 ? ng / 2 : ng);
  }
  hipLaunchKernelGGL((future_mass_kernel<D, NSUB, GC, HB, EPI, NB>), dim3((unsigned)(grid * hs)), dim3(256), 0,
                     (hipStream_t)L.stream, reinterpret_cast<const uint16_t*>(L.q),
                     reinterpret_cast<const uint16_t*>(L.k), L.bias, L.lse, out, L.B, L.Hq, L.Hkv, L.T, c, window, hz,
                     L.scores, L.agg, L.eps, L.normalize, hs > 1 ? 0 : xgroups, hs, window1, hz1, out1);
  return (int)hipGetLastError();
}

template <int D, int NSUB, int GC>
int launch_p2_b(const Launch& L, int hs) {
  if (L.scores)
    return L.bias ? launch_p2<D, NSUB, GC, true, true, 1>(L, 1) : launch_p2<D, NSUB, GC, false, true, 1>(L, 1);
  if (L.out1)
    return L.bias ? launch_p2<D, NSUB, GC, true, false, 2>(L, hs) : launch_p2<D, NSUB, GC, false, false, 2>(L, hs);
  return L.bias ? launch_p2<D, NSUB, GC, true, false, 1>(L, hs) : launch_p2<D, NSUB, GC, false, false, 1>(L, hs);
}

template <int D, int NSUB>
int launch_p2_gc(const Launch& L) {
  const int G = L.Hq / L.Hkv;
  constexpr int BK = 4 * NSUB * 16;
  const long long grid = (long long)((L.T + BK - 1) / BK) * L.B * L.Hkv;
  // Under 2048 workgroups (8 per CU) with a long band the heaviest key blocks set
  // the time: the query heads of each (key block, group) are then split over
  // several workgroups (not with the epilogue, which aggregates all G heads of a
  // key in one workgroup). Under 512 workgroups each takes one head, else two.
  // With a short band every block does about the same work and splitting does
  // not pay.
  const bool long_band = L.horizon < 0 || L.horizon >= L.T / 2 ||
                         (L.out1 && (L.horizon1 < 0 || L.horizon1 >= L.T / 2));
  if (!L.scores && grid < 2048 && long_band && G > 1) {
    if (grid >= 512 && G % 2 == 0) return launch_p2_b<D, NSUB, 2>(L, G / 2);
    return launch_p2_b<D, NSUB, 1>(L, G);
  }
  // Query heads per step: the largest of 4, 2, 1 that divides G.
  if (G % 4 == 0) return launch_p2_b<D, NSUB, 4>(L, 1);
  if (G % 2 == 0) return launch_p2_b<D, NSUB, 2>(L, 1);
  return launch_p2_b<D, NSUB, 1>(L, 1);
}

template <int D>
int launch_p2_d(const Launch& L) {
  // Four 16-key subtiles per wave (256 keys per workgroup) unless that leaves fewer
  // than ~2 workgroups per CU; then two (128 keys).
  // A short single band (horizon under T / 2) also takes two: its band edges are a
  // large share of the steps, and with two subtiles they keep the pipelined form.
  const long long wg2 = (long long)L.B * L.Hkv * ((L.T + 255) / 256);
  const bool short_band = L.horizon >= 0 && L.horizon < L.T / 2 && !L.out1;
  if (wg2 >= 512 && !short_band) return launch_p2_gc<D, 4>(L);
  return launch_p2_gc<D, 2>(L);
}

}  // namespace

// Compute units of the stream's device, looked up once per device.
int stream_cus(void* stream) {
  constexpr int kDevices = 64;
  static std::atomic<int> cache[kDevices];
  int dev = 0;
  if (hipStreamGetDevice((hipStream_t)stream, &dev) != hipSuccess && hipGetDevice(&dev) != hipSuccess) return 0;
  if (dev < 0 || dev >= kDevices) return 0;
  int n = cache[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 0;
    cache[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

int launch_row_lse(const Launch& L) {
  if (L.D == 64) return launch_p1_d<64>(L);
  return launch_p1_d<128>(L);
}

int launch_future_mass(const Launch& L) {
  if (L.D == 64) return launch_p2_d<64>(L);
  return launch_p2_d<128>(L);
}

}  // namespace kvpop
