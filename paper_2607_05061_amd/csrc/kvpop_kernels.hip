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
// Both passes recompute the logits with bf16 MFMA (v_mfma_f32_32x32x16_bf16) and
// never store the T x T matrix. The reduced index is always put on the MFMA's M
// (row) axis, so the sum of one output position stays inside one lane across a
// whole sweep: pass 1 computes tiles of K Q^T (keys on rows, queries on columns),
// pass 2 tiles of Q K^T (queries on rows, keys on columns). The operand that a
// workgroup owns for its whole life (Q columns in pass 1, K columns in pass 2)
// sits in registers; the streamed operand goes through a double-buffered LDS tile
// that all four waves read, so the query heads of one GQA group share each K tile
// (pass 1) and all key columns of a workgroup share each Q tile (pass 2).
//
// MFMA 32x32x16 lane layout (checked on gfx950): A row m = lane % 32 holds
// k = 8 * (lane / 32) .. +7; B column n = lane % 32 holds the same k range; the
// 16 accumulators of a lane are column n = lane % 32 and rows
// 8 * (r / 4) + 4 * (lane / 32) + r % 4. The contraction over the head dimension
// is order-free, so k-step s of a lane uses the 16-byte chunk 2 * s + lane / 32 of
// the head vector in both operands.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvpop_internal.h"

namespace kvpop {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// Floor of the running maximum in pass 1 (log2 units). Finite, so differences of
// two maxima never become inf - inf.
constexpr float kMaxFloor = -1.0e38f;
// A tile's partial sum above this means the reference maximum was too low.
constexpr float kOverflow = 18446744073709551616.0f;  // 2^64

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Row (within a 32-row tile) of accumulator r of a lane with half index hi.
__device__ __forceinline__ constexpr int acc_row(int r, int hi) { return 8 * (r >> 2) + 4 * hi + (r & 3); }

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// A 32-row x D tile of a row-major [T, D] bf16 matrix in LDS. The 16-byte chunk
// p of row r holds logical chunk p ^ (r % CPR): with 64 lanes reading one logical
// chunk from 32 consecutive rows, every 16 consecutive rows hit 16 different
// chunk slots, which spreads a ds_read_b128 over all banks.
template <int D>
struct TileIO {
  static constexpr int CPR = D / 8;             // 16-byte chunks per row
  static constexpr int PT = 32 * CPR / 256;     // chunks per thread per tile
  static_assert(PT >= 1 && (32 * CPR) % 256 == 0, "tile must split evenly over 256 threads");

  // Global -> registers: rows r0.. of `base` (a [T, D] matrix), clamped to T - 1.
  static __device__ __forceinline__ void load(u32x4 (&st)[PT], const uint16_t* __restrict__ base, int r0,
                                              int T, int tid) {
#pragma unroll
    for (int c = 0; c < PT; ++c) {
      const int id = tid + 256 * c;
      const int row = id / CPR;
      const int p = id % CPR;
      const int lc = p ^ (row & (CPR - 1));
      const int src = min(r0 + row, T - 1);
      st[c] = *reinterpret_cast<const u32x4*>(base + (size_t)src * D + lc * 8);
    }
  }
  // Registers -> LDS: chunk id lands at id * 16 bytes (linear, conflict-free).
  static __device__ __forceinline__ void store(uint16_t* lds, const u32x4 (&st)[PT], int tid) {
#pragma unroll
    for (int c = 0; c < PT; ++c) {
      const int id = tid + 256 * c;
      *reinterpret_cast<u32x4*>(lds + id * 8) = st[c];
    }
  }
  // MFMA operand for k-step s of this lane: row l32, logical chunk 2 s + hi.
  static __device__ __forceinline__ bf16x8 frag(const uint16_t* lds, int l32, int hi, int s) {
    const int p = (2 * s + hi) ^ (l32 & (CPR - 1));
    return *reinterpret_cast<const bf16x8*>(lds + (l32 * CPR + p) * 8);
  }
};

// ---------------------------------------------------------------------------
// Pass 1: row log-normaliser.
//
// Workgroup = (batch b, KV head h, head chunk pc of P query heads, query block of
// BQ = 512 / P positions). Its 4 waves x NQ = 4 column subtiles of 32 (head, query)
// columns keep their Q rows in registers (the MFMA B operand). Key tiles of 32
// rows stream through LDS as the A operand, shared by all P heads.
//
// Normalisation: every lane keeps, per column subtile, a reference maximum m
// (log2 units) and sum = sum exp2(x - m) over its 16 rows of each tile. The key
// tiles that straddle the diagonal are visited first and update (m, sum) exactly,
// as in online softmax. All later tiles lie strictly below the diagonal; for them
// the exponentials are taken against the current m without a per-element maximum,
// and only if a lane's tile sum exceeds 2^64 (a logit more than 64 log2-units
// above m, or inf) does that lane redo the tile with an exact maximum. The result
// is the same LSE; the common path costs one fma, one exp and one add per pair.
// ---------------------------------------------------------------------------
template <int D, bool HAS_BIAS>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(2, 2))) void
row_lse_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const float* __restrict__ bias,
               float* __restrict__ lse, int B, int Hq, int Hkv, int T, float c, float inv_scale, int P,
               int nqb) {
  constexpr int NQ = 4;
  constexpr int KS = D / 16;
  using IO = TileIO<D>;
  __shared__ __attribute__((aligned(16))) uint16_t sk[2][32 * D];
  __shared__ __attribute__((aligned(16))) float sb[2][32];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, hi = lane >> 5, l32 = lane & 31;
  const int G = Hq / Hkv;
  const int npc = G / P;
  const int per = B * Hkv * npc;
  const int order = blockIdx.x / per;  // 0 = last (heaviest) query block
  const int qb = nqb - 1 - order;
  int rest = blockIdx.x - order * per;
  const int b = rest / (Hkv * npc);
  rest -= b * Hkv * npc;
  const int h = rest / npc;
  const int pc = rest - h * npc;
  const int SPH = 16 / P;  // column subtiles per head in this block
  const int BQ = 32 * SPH;
  const int i0 = qb * BQ;

  int qs[NQ], qh[NQ];
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    const int u = w * NQ + n;
    qs[n] = i0 + 32 * (u % SPH);
    qh[n] = h * G + pc * P + u / SPH;
  }

  // This lane's query rows (B operand), resident for the whole sweep.
  bf16x8 qf[NQ][KS];
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    const int q = min(qs[n] + l32, T - 1);
    const uint16_t* src = Q + ((size_t)(b * Hq + qh[n]) * T + q) * D;
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[n][s] = *reinterpret_cast<const bf16x8*>(src + (2 * s + hi) * 8);
  }

  const uint16_t* Kbh = K + (size_t)(b * Hkv + h) * T * D;
  const int kend = min(T, i0 + BQ);
  const int nkt = (kend + 31) / 32;
  const int nfull = i0 / 32;  // tiles with every key below the block's first query
  const int ndiag = nkt - nfull;

  auto tile_of = [&](int s) { return s < ndiag ? nkt - 1 - s : s - ndiag; };

  u32x4 st[IO::PT];
  float stb = 0.f;
  auto fetch = [&](int s) {
    const int t0 = tile_of(s) * 32;
    IO::load(st, Kbh, t0, T, tid);
    if (HAS_BIAS && tid < 32) {
      const int t = t0 + tid;
      stb = t < T ? bias[t] * inv_scale : 0.f;
    }
  };
  auto commit = [&](int buf) {
    IO::store(sk[buf], st, tid);
    if (HAS_BIAS && tid < 32) sb[buf][tid] = stb;
  };

  float m[NQ], sum[NQ];
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    m[n] = kMaxFloor;
    sum[n] = 0.f;
  }

  fetch(0);
  commit(0);
  __syncthreads();

  for (int s = 0; s < nkt; ++s) {
    const int cur = s & 1;
    if (s + 1 < nkt) fetch(s + 1);
    const int t0 = tile_of(s) * 32;

    f32x16 acc[NQ];
    if (HAS_BIAS) {
      // Bias enters through the accumulator: C = bias_t / scale, so acc * c is
      // (scale <q, k_t> + bias_t) * log2(e).
      f32x16 ci;
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(&sb[cur][8 * g4 + 4 * hi]);
        ci[4 * g4 + 0] = v[0];
        ci[4 * g4 + 1] = v[1];
        ci[4 * g4 + 2] = v[2];
        ci[4 * g4 + 3] = v[3];
      }
#pragma unroll
      for (int n = 0; n < NQ; ++n) acc[n] = ci;
    } else {
#pragma unroll
      for (int n = 0; n < NQ; ++n) acc[n] = f32x16{};
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 a = IO::frag(sk[cur], l32, hi, ks);
#pragma unroll
      for (int n = 0; n < NQ; ++n) acc[n] = mfma32(a, qf[n][ks], acc[n]);
    }

#pragma unroll
    for (int n = 0; n < NQ; ++n) {
      if (t0 + 31 <= qs[n]) {
        // Strictly below the diagonal for every column of the subtile.
        const float nm = -m[n];
        float ts = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) ts += exp2_fast(__builtin_fmaf(acc[n][r], c, nm));
        if (!(ts <= kOverflow)) {
          float tmax = kMaxFloor;
#pragma unroll
          for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, acc[n][r] * c);
          const float mn = fmaxf(m[n], tmax);
          float e = 0.f;
#pragma unroll
          for (int r = 0; r < 16; ++r) e += exp2_fast(__builtin_fmaf(acc[n][r], c, -mn));
          sum[n] = sum[n] * exp2_fast(m[n] - mn) + e;
          m[n] = mn;
        } else {
          sum[n] += ts;
        }
      } else if (t0 <= qs[n] + 31) {
        // Straddles the diagonal: key t is admissible for query q iff t <= q.
        const int q = qs[n] + l32;
        float v[16];
        float tmax = kMaxFloor;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int t = t0 + acc_row(r, hi);
          v[r] = t <= q ? acc[n][r] * c : -__builtin_inff();
          tmax = fmaxf(tmax, v[r]);
        }
        const float mn = fmaxf(m[n], tmax);
        float e = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) e += exp2_fast(v[r] - mn);
        sum[n] = sum[n] * exp2_fast(m[n] - mn) + e;
        m[n] = mn;
      }
    }

    if (s + 1 < nkt) commit(cur ^ 1);
    __syncthreads();
  }

  // Merge the two half-wave partials of each column and write LSE (natural log).
#pragma unroll
  for (int n = 0; n < NQ; ++n) {
    const float mo = __shfl_xor(m[n], 32);
    const float so = __shfl_xor(sum[n], 32);
    const float mm = fmaxf(m[n], mo);
    const float tot = sum[n] * exp2_fast(m[n] - mm) + so * exp2_fast(mo - mm);
    const int q = qs[n] + l32;
    if (hi == 0 && q < T) lse[(size_t)(b * Hq + qh[n]) * T + q] = (mm + __log2f(tot)) * kLn2;
  }
}

// ---------------------------------------------------------------------------
// Pass 2: future mass per key.
//
// Workgroup = (batch b, KV head h, key block of BK = 4 * NK * 32 keys); wave w owns
// NK column subtiles of 32 keys whose K rows stay in registers (the MFMA B
// operand). For each query head of the group in turn, the workgroup sweeps the
// query tiles of 32 rows that can see its keys; each Q tile and its 32 LSE values
// are staged once in LDS and read by all four waves. Every lane accumulates, for
// its key column, exp2(acc * c - LSE_d * log2 e) over its 16 query rows of each
// tile into a per-tile sum and then into a running column sum (a two-level sum
// keeps the fp32 error near (16 + number of tiles) ulp). After a head's sweep the
// two half-wave sums of each column are added and written out: each workgroup owns
// its output columns, so no atomics are needed and results are deterministic.
//
// Query rows beyond T get LSE = +inf in LDS, which zeroes their terms. A per-key
// bias is factored out of the sum, out_t = exp(bias_t) * sum_d exp(...).
// ---------------------------------------------------------------------------
template <int D, int NK, bool HAS_BIAS>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(2, 2))) void
future_mass_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const float* __restrict__ bias,
                   const float* __restrict__ lse, float* __restrict__ out, int B, int Hq, int Hkv, int T, float c,
                   int window, int hz) {
  constexpr int KS = D / 16;
  constexpr int WK = NK * 32;  // keys per wave
  constexpr int BK = 4 * WK;   // keys per workgroup
  using IO = TileIO<D>;
  __shared__ __attribute__((aligned(16))) uint16_t sq[2][32 * D];
  __shared__ __attribute__((aligned(16))) float sl[2][32];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, hi = lane >> 5, l32 = lane & 31;
  const int G = Hq / Hkv;
  const int nbh = B * Hkv;
  const int kb = blockIdx.x / nbh;  // key block 0 (most query rows) first
  const int bh = blockIdx.x - kb * nbh;
  const int b = bh / Hkv;
  const int h = bh - b * Hkv;
  const int j0 = kb * BK;
  const int jw = j0 + w * WK;

  // Query rows that can reach any key of the block: [j0 + window, j0 + BK - 1 + hz] within [0, T).
  const long long r_lo = (long long)j0 + window;
  const long long r_hi = min((long long)T - 1, (long long)j0 + BK - 1 + hz);
  int qt0 = 0, nqt = 0;
  if (r_lo <= r_hi) {
    qt0 = (int)(r_lo / 32);
    nqt = (int)(r_hi / 32) - qt0 + 1;
  }

  float fac[NK];
#pragma unroll
  for (int n = 0; n < NK; ++n) {
    fac[n] = 1.f;
    if (HAS_BIAS) {
      const int j = min(jw + 32 * n + l32, T - 1);
      const float bj = bias[j];
      fac[n] = bj == -__builtin_inff() ? 0.f : exp2_fast(bj * kLog2e);
    }
  }

  if (nqt == 0) {
    // Every key of the block has an empty query range.
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int n = 0; n < NK; ++n) {
        const int j = jw + 32 * n + l32;
        if (hi == 0 && j < T) out[(size_t)(b * Hq + h * G + g) * T + j] = 0.f;
      }
    }
    return;
  }

  // This lane's key rows (B operand), resident for the whole sweep.
  bf16x8 kf[NK][KS];
  const uint16_t* Kbh = K + (size_t)bh * T * D;
#pragma unroll
  for (int n = 0; n < NK; ++n) {
    const int j = min(jw + 32 * n + l32, T - 1);
#pragma unroll
    for (int s = 0; s < KS; ++s) kf[n][s] = *reinterpret_cast<const bf16x8*>(Kbh + (size_t)j * D + (2 * s + hi) * 8);
  }

  const int nsteps = nqt * G;
  u32x4 st[IO::PT];
  float stl = 0.f;
  auto fetch = [&](int s) {
    const int g = s / nqt;
    const int i0 = (qt0 + s - g * nqt) * 32;
    const size_t head = (size_t)(b * Hq + h * G + g);
    IO::load(st, Q + head * T * D, i0, T, tid);
    if (tid < 32) {
      const int i = i0 + tid;
      stl = i < T ? -lse[head * T + i] * kLog2e : -__builtin_inff();
    }
  };
  auto commit = [&](int buf) {
    IO::store(sq[buf], st, tid);
    if (tid < 32) sl[buf][tid] = stl;
  };

  fetch(0);
  commit(0);
  __syncthreads();

  float colsum[NK];
#pragma unroll
  for (int n = 0; n < NK; ++n) colsum[n] = 0.f;
  int g = 0, qi = 0;  // head and tile index of step s

  for (int s = 0; s < nsteps; ++s) {
    const int cur = s & 1;
    if (s + 1 < nsteps) fetch(s + 1);
    const int i0 = (qt0 + qi) * 32;

    // Differences d = i - j over this wave's keys and the tile's rows.
    const int dmin = i0 - (jw + WK - 1);
    const int dmax = i0 + 31 - jw;
    const bool none = dmax < window || dmin > hz;
    if (!none) {
      f32x16 acc[NK];
#pragma unroll
      for (int n = 0; n < NK; ++n) acc[n] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 a = IO::frag(sq[cur], l32, hi, ks);
#pragma unroll
        for (int n = 0; n < NK; ++n) acc[n] = mfma32(a, kf[n][ks], acc[n]);
      }
      float nl[16];
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(&sl[cur][8 * g4 + 4 * hi]);
        nl[4 * g4 + 0] = v[0];
        nl[4 * g4 + 1] = v[1];
        nl[4 * g4 + 2] = v[2];
        nl[4 * g4 + 3] = v[3];
      }
      const bool full = dmin >= window && dmax <= hz;
      if (full) {
#pragma unroll
        for (int n = 0; n < NK; ++n) {
          float ts = 0.f;
#pragma unroll
          for (int r = 0; r < 16; ++r) ts += exp2_fast(__builtin_fmaf(acc[n][r], c, nl[r]));
          colsum[n] += ts;
        }
      } else {
#pragma unroll
        for (int n = 0; n < NK; ++n) {
          const int base = i0 + 4 * hi - (jw + 32 * n + l32);
          float ts = 0.f;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int d = base + 8 * (r >> 2) + (r & 3);
            const float e = exp2_fast(__builtin_fmaf(acc[n][r], c, nl[r]));
            ts += (d >= window && d <= hz) ? e : 0.f;
          }
          colsum[n] += ts;
        }
      }
    }

    if (s + 1 < nsteps) commit(cur ^ 1);
    __syncthreads();

    if (++qi == nqt) {
      // End of head g's sweep: combine the half-wave sums and write its columns.
#pragma unroll
      for (int n = 0; n < NK; ++n) {
        const float v = colsum[n] + __shfl_xor(colsum[n], 32);
        const int j = jw + 32 * n + l32;
        if (hi == 0 && j < T) out[(size_t)(b * Hq + h * G + g) * T + j] = HAS_BIAS ? v * fac[n] : v;
        colsum[n] = 0.f;
      }
      qi = 0;
      ++g;
    }
  }
}

template <int D, bool HB>
int launch_p1(const Launch& L, int P) {
  const int G = L.Hq / L.Hkv;
  const int BQ = 512 / P;
  const int nqb = (L.T + BQ - 1) / BQ;
  const long long grid = (long long)nqb * L.B * L.Hkv * (G / P);
  const float c = L.scale * kLog2e;
  hipLaunchKernelGGL((row_lse_kernel<D, HB>), dim3((unsigned)grid), dim3(256), 0, (hipStream_t)L.stream,
                     reinterpret_cast<const uint16_t*>(L.q), reinterpret_cast<const uint16_t*>(L.k), L.bias, L.out,
                     L.B, L.Hq, L.Hkv, L.T, c, 1.0f / L.scale, P, nqb);
  return (int)hipGetLastError();
}

template <int D, int NK, bool HB>
int launch_p2(const Launch& L) {
  constexpr int BK = 4 * NK * 32;
  const int nkb = (L.T + BK - 1) / BK;
  const long long grid = (long long)nkb * L.B * L.Hkv;
  const float c = L.scale * kLog2e;
  const int hz = L.horizon < 0 ? L.T : L.horizon;
  hipLaunchKernelGGL((future_mass_kernel<D, NK, HB>), dim3((unsigned)grid), dim3(256), 0, (hipStream_t)L.stream,
                     reinterpret_cast<const uint16_t*>(L.q), reinterpret_cast<const uint16_t*>(L.k), L.bias, L.lse,
                     L.out, L.B, L.Hq, L.Hkv, L.T, c, L.window, hz);
  return (int)hipGetLastError();
}

template <int D, int NK>
int launch_p2_nk(const Launch& L) {
  return L.bias ? launch_p2<D, NK, true>(L) : launch_p2<D, NK, false>(L);
}

template <int D>
int launch_p2_d(const Launch& L) {
  // Largest key block that still gives every CU about two workgroups.
  const long long bh = (long long)L.B * L.Hkv;
  const long long wg4 = bh * ((L.T + 511) / 512);
  const long long wg2 = bh * ((L.T + 255) / 256);
  if (wg4 >= 512) return launch_p2_nk<D, 4>(L);
  if (wg2 >= 512) return launch_p2_nk<D, 2>(L);
  return launch_p2_nk<D, 1>(L);
}

}  // namespace

int launch_row_lse(const Launch& L) {
  const int G = L.Hq / L.Hkv;
  int P = G & -G;  // largest power of two dividing G, at most 16
  if (P > 16) P = 16;
  if (L.D == 64) return L.bias ? launch_p1<64, true>(L, P) : launch_p1<64, false>(L, P);
  return L.bias ? launch_p1<128, true>(L, P) : launch_p1<128, false>(L, P);
}

int launch_future_mass(const Launch& L) {
  if (L.D == 64) return launch_p2_d<64>(L);
  return launch_p2_d<128>(L);
}

}  // namespace kvpop
