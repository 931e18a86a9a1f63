// gfx950 (MI355X) kernel for KVpop's running top-k sparse attention forward
// (Sec. 3.2, App. C.1 eq. running_topk_mask_app, App. C.3): for every query q of
// query head qh (KV head h = qh / G),
//
//   lse[q] = log sum_{t kept by q} exp l(q, t)        (Sec. 3.2 eq. sparse_lse_main)
//   o[q]   = sum_{t kept by q} exp(l(q, t) - lse[q]) v_t,
//   l(q, t) = scale <q_q, k_t> + bias_t.
//
// Token lifetimes. The running cutoff never increases with q, so a token dropped
// from the mask never returns and "t is kept by q" is t <= q < evict_t (the
// eviction query that kvpop_running_topk reports). A workgroup owning the query
// tile [q0, q1] therefore needs exactly the keys with t <= q1 and evict_t > max(t, q0)
// -- about the fixed budget s + w + k plus the tile height -- and no dense T x T
// mask or block mask: one compaction scan over evict[0 .. q1] lists them in LDS.
// Keys alive for the whole tile (t <= q0, evict_t > q1) go to list A and need no
// per-element test; keys that enter or leave inside the tile go to list P with
// (t, evict_t - t) and are tested per element as (unsigned)(q - t) < len. With the
// running top-k policy at most one token leaves per query, so list P holds fewer
// than two tile heights of keys.
//
// Compute. The gathered keys are processed in blocks of 32 like a flash-attention
// forward with the reduced index on the MFMA M axis:
//   S^T = K Q^T     v_mfma_f32_32x32x16_bf16, keys on rows, queries on columns;
//                   a lane owns one query column, so the softmax of a query stays
//                   in one lane pair (lane, lane ^ 32), combined by permlane32_swap;
//   O^T += V^T P^T  the probabilities leave the S accumulators already in the B
//                   operand layout (the key order inside a k-step is free), and
//                   V^T comes from ds_read_b64_tr_b16 over row-major V planes.
// The running maximum is lazy: it is raised (and O, l rescaled) only when a block's
// maximum exceeds it by more than 2^8, so the common block costs one fma, one exp
// and one add per element plus the bf16 packing.
//
// Workgroup = (batch b, KV head h, head chunk, query tile); 4 waves, each holding
// two (head, 32-query) columns: two heads of the same queries when G >= 2, so both
// MFMA chains of a wave share every K and V fragment read from LDS, and the same
// 32-key block serves all heads of the chunk (the GQA sharing). K and V rows are
// gathered by their positions straight from global memory into LDS
// (buffer_load ... lds, one 1 KB plane per instruction); a buffer descriptor's range
// check turns padding rows into zeros.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvpop_internal.h"

namespace kvpop {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kRsrcWord3 = 0x00020000;  // raw (untyped) buffer access
constexpr float kRescale = 8.0f;        // lazy-maximum slack of the exact variant, log2 units
constexpr float kOverflow = 64.0f;      // fast variant: largest term above the reference, log2 units
constexpr int kThreads = 256;
constexpr int kScan = 4 * kThreads;     // positions per scan step
constexpr int kCapA = 4096;             // list A capacity (entries)
constexpr int kCapP = 1536;             // list P capacity (entries)
constexpr int kPlane = 512;             // bf16 elements per 1 KB plane

__device__ __forceinline__ constexpr int acc_row(int r, int hi) { return 8 * (r >> 2) + 4 * hi + (r & 3); }

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// (x of lane l % 32, x of lane l % 32 + 32) on every lane.
__device__ __forceinline__ void pair_values(float x, float& a, float& b) {
  const int xi = __float_as_int(x);
  const auto r = __builtin_amdgcn_permlane32_swap(xi, xi, false, false);
  a = __int_as_float(r[0]);
  b = __int_as_float(r[1]);
}

// Exclusive prefix sum over the 256 threads; `total` gets the sum. `sh` holds 4 ints.
__device__ __forceinline__ int block_excl_scan(int v, int* sh, int& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[w] = x;
  __syncthreads();
  int pre = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = sh[i];
    pre += i < w ? t : 0;
    tot += t;
  }
  total = tot;
  return pre + x - v;
}

template <int D, bool HAS_BIAS>
struct Smem {
  static constexpr int KS = D / 16;  // K planes per block (k-steps over the head dim)
  static constexpr int DB = D / 32;  // 32-row blocks of the head dim
  static constexpr int VP = 2 * DB;  // V planes per block
  alignas(16) uint16_t ktile[2][KS * kPlane];
  alignas(16) uint16_t vtile[2][VP * kPlane];
  alignas(16) float btile[2][HAS_BIAS ? 64 : 4];
  alignas(16) int listA[kCapA];
  alignas(16) int posP[kCapP];  // read 16 bytes at a time
  alignas(16) int lenP[kCapP];
  alignas(16) int scan_sh[4];
};

template <int D, int HPW, bool HAS_BIAS, bool EXACT>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads), amdgpu_waves_per_eu(1, 1))) void
sparse_attn_fwd_kernel(SparseLaunch a) {
  using SM = Smem<D, HAS_BIAS>;
  constexpr int KS = SM::KS, DB = SM::DB, VP = SM::VP;
  constexpr int KPW = KS / 4, VPW = VP / 4;  // planes each wave copies per block
  static_assert(KPW >= 1 && VPW >= 1, "head dim");
  __shared__ __attribute__((aligned(16))) SM sm;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, hi = lane >> 5, col = lane & 31;
  const int T = a.T;

  // Heaviest tiles first; consecutive workgroups cover different (b, h, chunk)
  // groups of the same tile, so blockIdx % 8 (the XCD) follows the group.
  const int groups = a.B * a.Hkv * a.nch;
  const int tile = a.ntiles - 1 - (int)(blockIdx.x / groups);
  const int grp = (int)(blockIdx.x % groups);
  const int bh = grp / a.nch, chunk = grp % a.nch;
  const int b = bh / a.Hkv, h = bh % a.Hkv;
  const int q0 = tile * a.qt;
  const int q1 = min(q0 + a.qt, T) - 1;

  // This wave's two (head, 32-query) columns.
  const int hg = wave / a.wq, wq = wave % a.wq;
  int qh[2], qrow[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int head = chunk * a.hc + hg * HPW + (HPW == 2 ? c : 0);
    const int qblk = HPW == 2 ? wq : 2 * wq + c;
    qh[c] = h * a.G + head;
    qrow[c] = q0 + 32 * qblk + col;
  }

  // The exact variant only redoes tiles the fast variant flagged (NaN in lse).
  if (EXACT) {
    int flagged = 0;
#pragma unroll
    for (int c = 0; c < 2; ++c)
      if (qrow[c] < T) flagged |= __builtin_isnan(a.lse[((size_t)b * a.Hq + qh[c]) * T + qrow[c]]);
    if (!__syncthreads_or(flagged)) return;
  }

  // Q columns in registers as the B operand of S^T = K Q^T: k-step s uses the
  // 16-byte chunk 2 s + hi of the query row.
  bf16x8 qf[2][KS];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const uint16_t* row = a.q + (((size_t)b * a.Hq + qh[c]) * T + min(qrow[c], T - 1)) * D;
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[c][s] = *reinterpret_cast<const bf16x8*>(row + (2 * s + hi) * 8);
  }

  f32x16 o[2][DB];
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int d = 0; d < DB; ++d) o[c][d] = f32x16{};
  float m[2] = {-__builtin_inff(), -__builtin_inff()};
  float l[2] = {0.f, 0.f};
  bool ovf[2] = {false, false};

  const size_t kvoff = (size_t)bh * T * D;
  const int kv_bytes = T * D * 2;
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.k + kvoff), (short)0, kv_bytes, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.v + kvoff), (short)0, kv_bytes, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rb =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.bias), (short)0, HAS_BIAS ? T * 4 : 0, kRsrcWord3);
  const int32_t* ev = a.evict + (size_t)bh * T;

  // V row and column chunk this lane copies into a V plane (see compute_block for
  // the layout the transposing read expects).
  const int ks2_w = (wave * VPW) / DB;
  const int vrow = 16 * ks2_w + 8 * hi + 4 * (col >> 4) + ((lane & 7) >> 1);
  const int vcol_bytes = (16 * ((lane >> 3) & 1) + 8 * (lane & 1)) * 2;

  // Gather the 32 keys of block `blk` of `lpos` (n entries) into buffer `buf`.
  auto issue = [&](const int* lpos, int n, int blk, int buf) __attribute__((always_inline)) {
    const int e0 = blk * 32;
    const int pk = e0 + col < n ? lpos[e0 + col] : -1;
    const int pv = e0 + vrow < n ? lpos[e0 + vrow] : -1;
    const int voffK = pk >= 0 ? pk * (D * 2) + hi * 16 : kv_bytes;
    const int voffV = pv >= 0 ? pv * (D * 2) + vcol_bytes : kv_bytes;
#pragma unroll
    for (int i = 0; i < KPW; ++i) {
      const int s = wave * KPW + i;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_ptr_t)(sm.ktile[buf] + s * kPlane), 16, voffK, s * 32, 0,
                                               0);
    }
#pragma unroll
    for (int i = 0; i < VPW; ++i) {
      const int idx = wave * VPW + i;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_ptr_t)(sm.vtile[buf] + idx * kPlane), 16, voffV,
                                               (idx % DB) * 64, 0, 0);
    }
    if (HAS_BIAS && wave == 0) {
      const int voffB = pk >= 0 ? pk * 4 : T * 4;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr_t)sm.btile[buf], 4, voffB, 0, 0, 0);
    }
  };

  // One 32-key block from buffer `buf`. MASKED: per-element lifetimes from
  // (lpos, llen); otherwise only padding rows (entries >= n) are masked.
  auto compute_block = [&](const int* lpos, const int* llen, bool masked, int n, int blk,
                           int buf) __attribute__((always_inline)) {
    const int e0 = blk * 32;
    f32x16 sacc[2] = {f32x16{}, f32x16{}};
    const uint16_t* kt = sm.ktile[buf];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bf16x8 af = *reinterpret_cast<const bf16x8*>(kt + s * kPlane + lane * 8);
      sacc[0] = mfma32(af, qf[0][s], sacc[0]);
      sacc[1] = mfma32(af, qf[1][s], sacc[1]);
    }
    // With a key bias, logits in log2 units in place; without one the raw scores
    // stay (the scale is positive, so their maximum is the logits' maximum) and the
    // scale is folded into the exponential's fma.
    f32x16 (&x)[2] = sacc;
    if (HAS_BIAS) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float b2 = sm.btile[buf][acc_row(r, hi)] * kLog2e;
#pragma unroll
        for (int c = 0; c < 2; ++c) x[c][r] = __builtin_fmaf(sacc[c][r], a.c, b2);
      }
    }
    if (masked || e0 + 32 > n) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int e = e0 + 8 * g + 4 * hi;
        i32x4 pp = {0, 0, 0, 0}, ll = {0, 0, 0, 0};
        if (masked) {
          pp = *reinterpret_cast<const i32x4*>(lpos + e);
          ll = *reinterpret_cast<const i32x4*>(llen + e);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const bool valid = e + j < n;
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const bool keep = valid && (!masked || (unsigned)(qrow[c] - pp[j]) < (unsigned)ll[j]);
            x[c][4 * g + j] = keep ? x[c][4 * g + j] : -__builtin_inff();
          }
        }
      }
    }
    bf16x8 pk[2][2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      float mx = x[c][0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, x[c][r]);
      float m0, m1;
      pair_values(mx, m0, m1);
      mx = fmaxf(m0, m1);
      if (!HAS_BIAS) mx *= a.c;  // log2 units
      if (EXACT) {
        // Online maximum with lazy rescaling of the accumulators.
        if (mx > m[c] + kRescale) {
          const float f = __builtin_amdgcn_exp2f(m[c] - mx);
#pragma unroll
          for (int d = 0; d < DB; ++d) o[c][d] *= f;
          l[c] *= f;
          m[c] = mx;
        }
      } else {
        // Fixed reference: the first finite block maximum. Later terms up to 2^64
        // are exact in fp32 and bf16; beyond that the tile is flagged.
        if (m[c] == -__builtin_inff()) m[c] = mx;
        ovf[c] = ovf[c] || mx > m[c] + kOverflow;
      }
      const float mu = m[c] == -__builtin_inff() ? 0.f : m[c];
      float p[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        p[r] = HAS_BIAS ? __builtin_amdgcn_exp2f(x[c][r] - mu) : __builtin_amdgcn_exp2f(__builtin_fmaf(x[c][r], a.c, -mu));
        l[c] += p[r];
      }
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        f32x8 v8;
#pragma unroll
        for (int j = 0; j < 8; ++j) v8[j] = p[8 * k2 + j];
        pk[c][k2] = __builtin_convertvector(v8, bf16x8);
      }
    }
    // O^T += V^T P^T. Plane (k2, d) holds, at byte 512 hh + 8 l for lane
    // l = 16 g + 4 j + i4, the 4 values V[16 k2 + 8 hh + 4 (g / 2) + j][32 d + 16 (g % 2) + 4 i4 ..];
    // the transposing read then hands lane l the values of head-dim row 32 d + l % 32
    // for keys 16 k2 + 8 hh + 4 (l / 32) + 0..3, which is its A operand for the
    // contraction index 8 (l / 32) + 4 hh + j -- the same key order the S^T
    // accumulators give the B operand.
    const uint16_t* vt = sm.vtile[buf];
#pragma unroll
    for (int d = 0; d < DB; ++d) {
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const uint16_t* pl = vt + (k2 * DB + d) * kPlane;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(pl + lane * 4));
        const i16x4 up = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(pl + 256 + lane * 4));
        const i16x8 w8 = {lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
        const bf16x8 af = __builtin_bit_cast(bf16x8, w8);
        o[0][d] = mfma32(af, pk[0][k2], o[0][d]);
        o[1][d] = mfma32(af, pk[1][k2], o[1][d]);
      }
    }
  };

  // Windows of key positions [w0, w1): the compaction scan over their lifetimes
  // stops before either list could overflow, and the window's lists are then
  // processed in full. With the running top-k policy one window covers 0 .. q1.
  // (Scanning first and computing after keeps the accumulators in one place; a
  // scan interleaved with the block loop makes the compiler copy them.)
  for (int w0 = 0; w0 <= q1;) {
    int cntA = 0, cntP = 0;
    int base = w0;
    while (base <= q1 && cntA <= kCapA - kScan && cntP <= kCapP - kScan) {
      const int p0 = base + 4 * tid;
      int kind[4], len[4];
      int nf = 0, np = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int p = p0 + j;
        const int e = p <= q1 ? ev[p] : 0;
        const bool alive = p <= q1 && e > max(p, q0);  // kept by some query of the tile
        const bool full = alive && p <= q0 && e > q1;   // kept by all of them
        kind[j] = full ? 1 : (alive ? 2 : 0);
        len[j] = e - p;
        nf += full;
        np += alive && !full;
      }
      int total;
      const int ex = block_excl_scan(nf | (np << 16), sm.scan_sh, total);
      int ia = cntA + (ex & 0xFFFF), ip = cntP + (ex >> 16);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (kind[j] == 1) {
          sm.listA[ia++] = p0 + j;
        } else if (kind[j] == 2) {
          sm.posP[ip] = p0 + j;
          sm.lenP[ip++] = len[j];
        }
      }
      __syncthreads();
      cntA += total & 0xFFFF;
      cntP += total >> 16;
      base += kScan;
    }
    w0 = base;

    // Blocks of list A (no per-element test) then of list P, double-buffered:
    // block i + 1 is gathered while block i is computed.
    const int nbA = (cntA + 31) >> 5;
    const int nbt = nbA + ((cntP + 31) >> 5);
    auto source = [&](int i, const int*& lp, const int*& ll, bool& msk, int& n, int& blk)
                      __attribute__((always_inline)) {
      msk = i >= nbA;
      lp = msk ? sm.posP : sm.listA;
      ll = sm.lenP;
      n = msk ? cntP : cntA;
      blk = msk ? i - nbA : i;
    };
    if (nbt > 0) {
      {
        const int* lp;
        const int* ll;
        bool msk;
        int n, blk;
        source(0, lp, ll, msk, n, blk);
        issue(lp, n, blk, 0);
      }
      for (int i = 0; i < nbt; ++i) {
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's copies have landed
        __syncthreads();                     // all copies landed; the other buffer is free
        const int* lp;
        const int* ll;
        bool msk;
        int n, blk;
        if (i + 1 < nbt) {
          source(i + 1, lp, ll, msk, n, blk);
          issue(lp, n, blk, (i + 1) & 1);
        }
        source(i, lp, ll, msk, n, blk);
        compute_block(lp, ll, msk, n, blk, i & 1);
      }
      __syncthreads();
    }
  }

  // Epilogue: combine the two lane halves' sums, normalise, write O (bf16) and LSE.
  // A fast-variant column whose terms overflowed the fixed reference writes NaN to
  // its LSE instead; the exact variant then recomputes the whole tile.
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    float l0, l1;
    pair_values(l[c], l0, l1);
    const float lt = l0 + l1;
    const float inv = lt > 0.f ? 1.0f / lt : 0.f;
    const bool redo = !EXACT && __builtin_amdgcn_ballot_w64(ovf[c]) != 0;
    if (qrow[c] >= T) continue;
    const size_t rowi = ((size_t)b * a.Hq + qh[c]) * T + qrow[c];
    if (hi == 0)
      a.lse[rowi] = redo ? __builtin_nanf("") : lt > 0.f ? (m[c] + __builtin_amdgcn_logf(lt)) * kLn2 : -__builtin_inff();
    uint16_t* orow = a.o + rowi * D;
#pragma unroll
    for (int d = 0; d < DB; ++d) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        typedef float f32x4v __attribute__((ext_vector_type(4)));
        typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
        f32x4v v4 = {o[c][d][4 * g] * inv, o[c][d][4 * g + 1] * inv, o[c][d][4 * g + 2] * inv,
                     o[c][d][4 * g + 3] * inv};
        const bf16x4 w4 = __builtin_convertvector(v4, bf16x4);
        *reinterpret_cast<bf16x4*>(orow + 32 * d + 8 * g + 4 * hi) = w4;
      }
    }
  }
}

// The fast variant, then the exact one, which exits at once on tiles the fast one
// did not flag.
template <int D, int HPW, bool HB>
int launch_d(const SparseLaunch& L) {
  const unsigned grid = (unsigned)((long long)L.ntiles * L.B * L.Hkv * L.nch);
  hipLaunchKernelGGL((sparse_attn_fwd_kernel<D, HPW, HB, false>), dim3(grid), dim3(kThreads), 0,
                     (hipStream_t)L.stream, L);
  int e = (int)hipGetLastError();
  if (e) return e;
  hipLaunchKernelGGL((sparse_attn_fwd_kernel<D, HPW, HB, true>), dim3(grid), dim3(kThreads), 0,
                     (hipStream_t)L.stream, L);
  return (int)hipGetLastError();
}

template <int D>
int launch_hb(const SparseLaunch& L) {
  if (L.hpw == 2) return L.bias ? launch_d<D, 2, true>(L) : launch_d<D, 2, false>(L);
  return L.bias ? launch_d<D, 1, true>(L) : launch_d<D, 1, false>(L);
}

}  // namespace

void sparse_attn_plan(SparseLaunch& L) {
  L.G = L.Hq / L.Hkv;
  L.hpw = L.G >= 2 ? 2 : 1;
  const int nhp = L.G / L.hpw < 4 ? L.G / L.hpw : 4;  // head groups per workgroup
  L.wq = 4 / nhp;                                      // waves along the queries
  L.qt = 32 * (2 / L.hpw) * L.wq;
  L.hc = L.hpw * nhp;
  L.nch = L.G / L.hc;
  L.ntiles = (L.T + L.qt - 1) / L.qt;
  L.c = L.scale * kLog2e;
}

int launch_sparse_attn_fwd(SparseLaunch L) {
  sparse_attn_plan(L);
  return L.D == 128 ? launch_hb<128>(L) : launch_hb<64>(L);
}

}  // namespace kvpop
