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
// Each query keeps a fixed reference maximum (its first finite block's), so the
// accumulators are only ever touched by MFMAs; a column whose later logits exceed
// it by more than 2^64 is flagged and recomputed by an exact variant with the
// usual online rescaling.
//
// Workgroup = (batch b, KV head h, head chunk, query tile): 8 waves, two per SIMD,
// each owning one (head, 32-query) column; for G >= 2 the columns are the heads
// of a head chunk times the tile's 32-query blocks, so every 32-key block in LDS
// serves all of them (the GQA sharing). Two waves per SIMD hide each other's MFMA,
// LDS and barrier latency. K and V rows are gathered by their positions straight
// from global memory into LDS (buffer_load ... lds, one 1 KB plane per
// instruction); a buffer descriptor's range check turns padding rows into zeros.

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
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kRsrcWord3 = 0x00020000;  // raw (untyped) buffer access
constexpr float kRescale = 8.0f;        // lazy-maximum slack of the exact variant, log2 units
constexpr float kOverflowSum = 0x1p64f; // fast variant: largest block sum of terms relative to the reference
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kScan = 1024;             // positions per scan step (2 per thread)
constexpr int kCapA = 4096;             // list A capacity (entries)
constexpr int kCapP = 1536;             // list P capacity (entries)
constexpr int kPlane = 512;             // bf16 elements per 1 KB plane
constexpr int kBufs = 5;                // K/V block buffers (see the block loop)
constexpr int kChunk = 4096;            // lifetimes staged into LDS per chunk (16 KB)
constexpr int kEvBufs = 2;              // chunk buffers: the next chunk loads during the scan
constexpr int kRunMax = 16;             // most query tiles per workgroup
constexpr int kRunGrid = 4096;          // workgroups wanted before runs grow

__device__ __forceinline__ constexpr int acc_row(int r, int hi) { return 8 * (r >> 2) + 4 * hi + (r & 3); }

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// Workgroup barrier for the loops. __syncthreads() (and even an LDS-only fence)
// makes the compiler wait for every outstanding buffer load, because loads into
// LDS count as LDS writes; that would also wait for the prefetch of later blocks.
// Every wave waits for its own copies with vmcnt before arriving and has consumed
// its LDS reads of any buffer about to be refilled, so a bare s_barrier suffices;
// the memory clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void block_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Barrier after this wave's LDS writes have completed (lgkmcnt(0)), without
// waiting for outstanding buffer loads.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt at their maxima
  block_barrier();
}

// (x of lane l % 32, x of lane l % 32 + 32) on every lane.
__device__ __forceinline__ void pair_values(float x, float& a, float& b) {
  const int xi = __float_as_int(x);
  const auto r = __builtin_amdgcn_permlane32_swap(xi, xi, false, false);
  a = __int_as_float(r[0]);
  b = __int_as_float(r[1]);
}

// The transposing V reads of a block (the A operands of O^T += V^T P^T; plane
// layout at the kernel's pv). They are issued from inline asm so that the
// compiler, which cannot tell which LDS buffer a transposing read touches, does not
// wait for every outstanding buffer load (including the prefetches of later blocks)
// before them. Their registers are valid only after vfrag_wait, whose
// read-modify-write operands keep every use behind the wait.
template <int DB>
struct VFrag {
  i16x4 r[DB * 4];  // [d][k2][half]
};

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

__device__ __forceinline__ void vfrag_issue(VFrag<4>& f, uint32_t a) {
  asm volatile(
      "ds_read_b64_tr_b16 %0, %16 offset:0\n ds_read_b64_tr_b16 %1, %16 offset:512\n"
      "ds_read_b64_tr_b16 %2, %16 offset:4096\n ds_read_b64_tr_b16 %3, %16 offset:4608\n"
      "ds_read_b64_tr_b16 %4, %16 offset:1024\n ds_read_b64_tr_b16 %5, %16 offset:1536\n"
      "ds_read_b64_tr_b16 %6, %16 offset:5120\n ds_read_b64_tr_b16 %7, %16 offset:5632\n"
      "ds_read_b64_tr_b16 %8, %16 offset:2048\n ds_read_b64_tr_b16 %9, %16 offset:2560\n"
      "ds_read_b64_tr_b16 %10, %16 offset:6144\n ds_read_b64_tr_b16 %11, %16 offset:6656\n"
      "ds_read_b64_tr_b16 %12, %16 offset:3072\n ds_read_b64_tr_b16 %13, %16 offset:3584\n"
      "ds_read_b64_tr_b16 %14, %16 offset:7168\n ds_read_b64_tr_b16 %15, %16 offset:7680"
      : "=&v"(f.r[0]), "=&v"(f.r[1]), "=&v"(f.r[2]), "=&v"(f.r[3]), "=&v"(f.r[4]), "=&v"(f.r[5]), "=&v"(f.r[6]),
        "=&v"(f.r[7]), "=&v"(f.r[8]), "=&v"(f.r[9]), "=&v"(f.r[10]), "=&v"(f.r[11]), "=&v"(f.r[12]),
        "=&v"(f.r[13]), "=&v"(f.r[14]), "=&v"(f.r[15])
      : "v"(a));
}

__device__ __forceinline__ void vfrag_wait(VFrag<4>& f) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(f.r[0]), "+v"(f.r[1]), "+v"(f.r[2]), "+v"(f.r[3]), "+v"(f.r[4]), "+v"(f.r[5]), "+v"(f.r[6]),
                 "+v"(f.r[7]), "+v"(f.r[8]), "+v"(f.r[9]), "+v"(f.r[10]), "+v"(f.r[11]), "+v"(f.r[12]),
                 "+v"(f.r[13]), "+v"(f.r[14]), "+v"(f.r[15]));
}

__device__ __forceinline__ void vfrag_issue(VFrag<2>& f, uint32_t a) {
  asm volatile(
      "ds_read_b64_tr_b16 %0, %8 offset:0\n ds_read_b64_tr_b16 %1, %8 offset:512\n"
      "ds_read_b64_tr_b16 %2, %8 offset:2048\n ds_read_b64_tr_b16 %3, %8 offset:2560\n"
      "ds_read_b64_tr_b16 %4, %8 offset:1024\n ds_read_b64_tr_b16 %5, %8 offset:1536\n"
      "ds_read_b64_tr_b16 %6, %8 offset:3072\n ds_read_b64_tr_b16 %7, %8 offset:3584"
      : "=&v"(f.r[0]), "=&v"(f.r[1]), "=&v"(f.r[2]), "=&v"(f.r[3]), "=&v"(f.r[4]), "=&v"(f.r[5]), "=&v"(f.r[6]),
        "=&v"(f.r[7])
      : "v"(a));
}

__device__ __forceinline__ void vfrag_wait(VFrag<2>& f) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(f.r[0]), "+v"(f.r[1]), "+v"(f.r[2]), "+v"(f.r[3]), "+v"(f.r[4]), "+v"(f.r[5]), "+v"(f.r[6]),
                 "+v"(f.r[7]));
}

// The K fragments of a block (the A operands of S^T = K Q^T: k-step s at byte
// 1024 s + 16 lane of the K tile), read from inline asm for the same reason.
template <int KS>
struct KFrag {
  bf16x8 r[KS];
};

__device__ __forceinline__ void kfrag_issue(KFrag<8>& f, uint32_t a) {
  asm volatile(
      "ds_read_b128 %0, %8 offset:0\n ds_read_b128 %1, %8 offset:1024\n"
      "ds_read_b128 %2, %8 offset:2048\n ds_read_b128 %3, %8 offset:3072\n"
      "ds_read_b128 %4, %8 offset:4096\n ds_read_b128 %5, %8 offset:5120\n"
      "ds_read_b128 %6, %8 offset:6144\n ds_read_b128 %7, %8 offset:7168"
      : "=&v"(f.r[0]), "=&v"(f.r[1]), "=&v"(f.r[2]), "=&v"(f.r[3]), "=&v"(f.r[4]), "=&v"(f.r[5]), "=&v"(f.r[6]),
        "=&v"(f.r[7])
      : "v"(a));
}

__device__ __forceinline__ void kfrag_wait(KFrag<8>& f) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(f.r[0]), "+v"(f.r[1]), "+v"(f.r[2]), "+v"(f.r[3]), "+v"(f.r[4]), "+v"(f.r[5]), "+v"(f.r[6]),
                 "+v"(f.r[7]));
}

// Wait for the K fragments issued just before a block's V reads (8 of them for a
// 32-key block at head dim 64, 16 at 128): LDS reads complete in order, so with at
// most 15 (the counter's limit) or 8 reads outstanding the K reads have landed.
__device__ __forceinline__ void kfrag_wait_before_v(KFrag<8>& f) {
  asm volatile("s_waitcnt lgkmcnt(15)"
               : "+v"(f.r[0]), "+v"(f.r[1]), "+v"(f.r[2]), "+v"(f.r[3]), "+v"(f.r[4]), "+v"(f.r[5]), "+v"(f.r[6]),
                 "+v"(f.r[7]));
}

__device__ __forceinline__ void kfrag_wait_before_v(KFrag<4>& f) {
  asm volatile("s_waitcnt lgkmcnt(8)" : "+v"(f.r[0]), "+v"(f.r[1]), "+v"(f.r[2]), "+v"(f.r[3]));
}

__device__ __forceinline__ void kfrag_issue(KFrag<4>& f, uint32_t a) {
  asm volatile(
      "ds_read_b128 %0, %4 offset:0\n ds_read_b128 %1, %4 offset:1024\n"
      "ds_read_b128 %2, %4 offset:2048\n ds_read_b128 %3, %4 offset:3072"
      : "=&v"(f.r[0]), "=&v"(f.r[1]), "=&v"(f.r[2]), "=&v"(f.r[3])
      : "v"(a));
}

__device__ __forceinline__ void kfrag_wait(KFrag<4>& f) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(f.r[0]), "+v"(f.r[1]), "+v"(f.r[2]), "+v"(f.r[3]));
}

template <int D, bool HAS_BIAS>
struct Smem {
  static constexpr int KS = D / 16;  // K planes per block (k-steps over the head dim)
  static constexpr int DB = D / 32;  // 32-row blocks of the head dim
  static constexpr int VP = 2 * DB;  // V planes per block
  alignas(16) uint16_t ktile[kBufs][KS * kPlane];
  alignas(16) uint16_t vtile[kBufs][VP * kPlane];
  alignas(16) float btile[kBufs][HAS_BIAS ? 64 : 4];
  alignas(16) int evs[kEvBufs][kChunk];  // lifetimes of the positions being scanned
  alignas(16) int listA[kCapA];
  alignas(16) int eA[kCapA];    // lifetime ends of list A, for the next tile's lists
  alignas(16) int posP[kCapP];  // read 16 bytes at a time
  alignas(16) int lenP[kCapP];
  alignas(16) int scan_sh[2][32];
};

template <int D, int HPW, bool HAS_BIAS, bool EXACT>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads), amdgpu_waves_per_eu(2, 2))) void
sparse_attn_fwd_kernel(SparseLaunch a) {
  using SM = Smem<D, HAS_BIAS>;
  constexpr int KS = SM::KS, DB = SM::DB;
  static_assert(KS == 4 || KS == 8, "head dim 64 or 128");
  const int RUN = a.run;  // tiles per workgroup
  __shared__ __attribute__((aligned(16))) SM sm;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, hi = lane >> 5, col = lane & 31;
  const int T = a.T;

  // Workgroup order. A workgroup takes a run of RUN consecutive query tiles of one
  // (b, h, chunk) group, in ascending order; runs go heaviest first. Workgroups
  // are dealt to the 8 XCDs round-robin (XCD = blockIdx % 8): when the groups
  // divide evenly, each XCD takes its share of groups one after another, so the
  // tiles running together on an XCD share one group's keys in its L2; otherwise
  // groups interleave within each run.
  const int groups = a.B * a.Hkv * a.nch;
  const int nruns = (a.ntiles + RUN - 1) / RUN;
  int run, grp;
  if ((groups & 7) == 0) {
    const int x = (int)(blockIdx.x & 7), j = (int)(blockIdx.x >> 3);
    run = nruns - 1 - j % nruns;
    grp = x + 8 * (j / nruns);
  } else {
    run = nruns - 1 - (int)(blockIdx.x / groups);
    grp = (int)(blockIdx.x % groups);
  }
  const int bh = grp / a.nch, chunk = grp % a.nch;
  const int b = bh / a.Hkv, h = bh % a.Hkv;
  const int tile_end = min(a.ntiles, (run + 1) * RUN);

  // This wave's (head, 32-query) column: columns 2 u and 2 u + 1 are two heads of
  // the same queries when G >= 2, two query blocks of one head otherwise.
  const int u = wave >> 1, cc = wave & 1;
  const int hg = u / a.wq, wq = u % a.wq;
  const int qh = h * a.G + chunk * a.hc + hg * HPW + (HPW == 2 ? cc : 0);
  const int qcol = 32 * (HPW == 2 ? wq : 2 * wq + cc) + col;  // query offset inside a tile
  const uint16_t* qbase = a.q + ((size_t)b * a.Hq + qh) * T * D;

  const size_t kvoff = (size_t)bh * T * D;
  const int kv_bytes = T * D * 2;
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.k + kvoff), (short)0, kv_bytes, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.v + kvoff), (short)0, kv_bytes, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rb =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.bias), (short)0, HAS_BIAS ? T * 4 : 0, kRsrcWord3);
  const int32_t* ev = a.evict + (size_t)bh * T;

  // The 1 KB planes this wave copies per block: K plane `wave` (if any) and one V
  // plane (D = 128: K plane w and V plane w; D = 64: K plane w for w < 4, V plane
  // w - 4 for the others), plus the block's key biases for wave 0.
  const int kplane = wave < KS ? wave : -1;
  const int vplane = KS == 8 ? wave : (wave >= KS ? wave - KS : -1);
  const int nload = (kplane >= 0) + (vplane >= 0) + (HAS_BIAS && wave == 0);
  // V row and column chunk this lane copies into its V plane (layout at pv).
  const int vrow = 16 * (max(vplane, 0) / DB) + 8 * hi + 4 * (col >> 4) + ((lane & 7) >> 1);
  const int vcol_bytes = (16 * ((lane >> 3) & 1) + 8 * (lane & 1)) * 2;

  // State of the current tile, seen by the helpers below.
  int q0 = 0, q1 = -1, qrow = 0;
  bf16x8 qf[KS];
  f32x16 o[DB];
  float m = 0.f, l = 0.f;
  bool ovf = false;

  // Gather the 32 keys of block `blk` of `lpos` into buffer `buf`. The lists are
  // padded to whole blocks with position -1, which reads as zero rows.
  auto issue = [&](const int* lpos, int blk, int buf) __attribute__((always_inline)) {
    const int e0 = blk * 32;
    const int pk = lpos[e0 + col];
    if (kplane >= 0) {
      const int voffK = pk >= 0 ? pk * (D * 2) + hi * 16 : kv_bytes;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_ptr_t)(sm.ktile[buf] + kplane * kPlane), 16, voffK,
                                               kplane * 32, 0, 0);
    }
    if (vplane >= 0) {
      const int pv = lpos[e0 + vrow];
      const int voffV = pv >= 0 ? pv * (D * 2) + vcol_bytes : kv_bytes;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_ptr_t)(sm.vtile[buf] + vplane * kPlane), 16, voffV,
                                               (vplane % DB) * 64, 0, 0);
    }
    if (HAS_BIAS && wave == 0) {
      const int voffB = pk >= 0 ? pk * 4 : T * 4;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr_t)sm.btile[buf], 4, voffB, 0, 0, 0);
    }
  };

  // Wait until the oldest outstanding block's copies have landed, given how many
  // later blocks this wave has issued (buffer loads complete in order).
  auto wait_block = [&](int later) __attribute__((always_inline)) {
    switch (later * nload) {
      case 0: wait_vmcnt<0>(); break;
      case 1: wait_vmcnt<1>(); break;
      case 2: wait_vmcnt<2>(); break;
      case 3: wait_vmcnt<3>(); break;
      case 4: wait_vmcnt<4>(); break;
      case 5: wait_vmcnt<5>(); break;
      default: wait_vmcnt<6>(); break;
    }
  };

  // S^T = K Q^T of the block in buffer `buf`.
  auto qk = [&](int buf, f32x16& sacc) __attribute__((always_inline)) {
    sacc = f32x16{};
    const uint16_t* kt = sm.ktile[buf];
#pragma unroll
    for (int s = 0; s < KS; ++s)
      sacc = mfma32(*reinterpret_cast<const bf16x8*>(kt + s * kPlane + lane * 8), qf[s], sacc);
  };


  // Key bias and masking of block `blk` of a list (entries lpos/llen, n of them):
  // with a bias, logits in log2 units in place; without one the raw scores stay
  // (the scale is positive, so their maximum is the logits' maximum) and the scale
  // is folded into the exponential's fma.
  auto prep = [&](f32x16& x, const int* lpos, const int* llen, bool masked, int n, int blk, int buf)
                  __attribute__((always_inline)) {
    const int e0 = blk * 32;
    if (HAS_BIAS) {
#pragma unroll
      for (int r = 0; r < 16; ++r) x[r] = __builtin_fmaf(x[r], a.c, sm.btile[buf][acc_row(r, hi)] * kLog2e);
    }
    if (masked) {
      // List P: kept iff t <= q < t + len, i.e. (unsigned)(q - t) < len; padding
      // entries have len 0.
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int e = e0 + 8 * g + 4 * hi;
        const i32x4 pp = *reinterpret_cast<const i32x4*>(lpos + e);
        const i32x4 ll = *reinterpret_cast<const i32x4*>(llen + e);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          x[4 * g + j] = (unsigned)(qrow - pp[j]) < (unsigned)ll[j] ? x[4 * g + j] : -__builtin_inff();
      }
    } else if (e0 + 32 > n) {
      // The last block of list A: padding rows only.
#pragma unroll
      for (int r = 0; r < 16; ++r) x[r] = e0 + acc_row(r, hi) < n ? x[r] : -__builtin_inff();
    }
  };

  // Largest logit of a block for this lane's column (both lane halves), log2 units.
  auto block_max = [&](const f32x16& x) __attribute__((always_inline)) {
    float mx = x[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, x[r]);
    float m0, m1;
    pair_values(mx, m0, m1);
    mx = fmaxf(m0, m1);
    return HAS_BIAS ? mx : mx * a.c;  // log2 units
  };
  // The exact variant's softmax numerators of a block: online maximum with lazy
  // rescaling of the accumulators, exponentials, row sum and bf16 packing into the B
  // operand of the PV product. (The fast variant's, against a fixed reference, are
  // interleaved with the next block's QK^T product in its block loop.)
  auto softmax_exact = [&](f32x16& x, bf16x8 (&pk)[2]) __attribute__((always_inline)) {
    const float mx = block_max(x);
    if (mx > m + kRescale) {
      const float f = __builtin_amdgcn_exp2f(m - mx);
#pragma unroll
      for (int d = 0; d < DB; ++d) o[d] *= f;
      l *= f;
      m = mx;
    }
    const float mu = m == -__builtin_inff() ? 0.f : m;
    float p[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      p[r] = HAS_BIAS ? __builtin_amdgcn_exp2f(x[r] - mu) : __builtin_amdgcn_exp2f(__builtin_fmaf(x[r], a.c, -mu));
      l += p[r];
    }
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      f32x8 v8;
#pragma unroll
      for (int j = 0; j < 8; ++j) v8[j] = p[8 * k2 + j];
      pk[k2] = __builtin_convertvector(v8, bf16x8);
    }
  };

  // O^T += V^T P^T. V plane (k2, d) (1 KB at byte 1024 (k2 DB + d) of the block's
  // V tile) holds, at byte 512 hh + 8 l for lane l = 16 g + 4 j + i4, the 4 values
  // V[16 k2 + 8 hh + 4 (g / 2) + j][32 d + 16 (g % 2) + 4 i4 ..]; the transposing read
  // then hands lane l the values of head-dim row 32 d + l % 32 for keys
  // 16 k2 + 8 hh + 4 (l / 32) + 0..3, which is its A operand for the contraction
  // index 8 (l / 32) + 4 hh + j -- the same key order the S^T accumulators give the
  // B operand. Fragment (d, k2) is registers 4 d + 2 k2 (lower half) and + 1.
  auto pv = [&](const VFrag<DB>& f, const bf16x8 (&pk)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int d = 0; d < DB; ++d) {
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const i16x4 lo = f.r[4 * d + 2 * k2], up = f.r[4 * d + 2 * k2 + 1];
        const i16x8 w8 = {lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
        o[d] = mfma32(__builtin_bit_cast(bf16x8, w8), pk[k2], o[d]);
      }
    }
  };

  // Lifetimes reach LDS in chunks of kChunk positions, one chunk ahead of the scan,
  // straight from global memory (16 KB per chunk: 2 KB per wave, 2 loads).
  // Positions past the tile's last query read as 0 (never alive) through the
  // descriptor's range.
  auto stage = [&](int ch) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t re =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(ev), (short)0, (q1 + 1) * 4, kRsrcWord3);
    int* dst = sm.evs[ch & (kEvBufs - 1)];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int idx = 2 * wave + i;  // 1 KB pieces of 256 positions
      __builtin_amdgcn_raw_ptr_buffer_load_lds(re, (lds_ptr_t)(dst + idx * 256), 16, lane * 16,
                                               (ch * kChunk + idx * 256) * 4, 0, 0);
    }
  };
  int staged = 0;  // last chunk whose copies were issued
  int sstep = 0;   // LDS count exchanges so far (selects the buffer)

  // Append one candidate key per thread (t with lifetime end e; `valid` false for
  // none) to lists A and P of the current tile, in thread order after the nA / nP
  // entries already there. Returns false, leaving the lists unusable, if either
  // list would overflow.
  auto append = [&](bool valid, int t, int e, int& nA, int& nP) __attribute__((always_inline)) {
    const bool alive = valid && e > max(t, q0);  // kept by some query of the tile
    const bool full = alive && t <= q0 && e > q1;  // kept by all of them
    const uint64_t bf = __builtin_amdgcn_ballot_w64(full);
    const uint64_t bp = __builtin_amdgcn_ballot_w64(alive && !full);
    int* sh = sm.scan_sh[sstep & 1];
    if (lane == 0) {
      sh[wave] = __builtin_popcountll(bf);
      sh[16 + wave] = __builtin_popcountll(bp);
    }
    lds_sync();
    int befA = 0, befP = 0, totA = 0, totP = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const int ca = sh[w], cp = sh[16 + w];
      befA += w < wave ? ca : 0;
      befP += w < wave ? cp : 0;
      totA += ca;
      totP += cp;
    }
    // Every lane read the same counts: keep the sums in scalar registers.
    befA = __builtin_amdgcn_readfirstlane(befA);
    befP = __builtin_amdgcn_readfirstlane(befP);
    totA = __builtin_amdgcn_readfirstlane(totA);
    totP = __builtin_amdgcn_readfirstlane(totP);
    const bool fits = nA + totA <= kCapA && nP + totP <= kCapP;
    if (fits && full) {
      const int i = nA + befA + __builtin_amdgcn_mbcnt_hi((uint32_t)(bf >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bf, 0));
      sm.listA[i] = t;
      sm.eA[i] = e;
    }
    if (fits && alive && !full) {
      const int i = nP + befP + __builtin_amdgcn_mbcnt_hi((uint32_t)(bp >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bp, 0));
      sm.posP[i] = t;
      sm.lenP[i] = e - t;
    }
    nA += totA;
    nP += totP;
    ++sstep;
    return fits;
  };

  int cntA = 0, cntP = 0;  // list sizes (without padding)
  bool lists_ok = false;   // the lists hold every key of the previous tile

  // The exact variant leaves at once when the fast one flagged no tile of the run.
  if (EXACT) {
    int flagged = 0;
    for (int tile = run * RUN; tile < tile_end; ++tile) {
      const int r = tile * a.qt + qcol;
      flagged |= r < T ? __builtin_isnan(a.lse[((size_t)b * a.Hq + qh) * T + r]) : 0;
    }
    if (!__syncthreads_or(flagged)) return;
  }

  for (int tile = run * RUN; tile < tile_end; ++tile) {
    const int pq1 = q1;
    q0 = tile * a.qt;
    q1 = min(q0 + a.qt, T) - 1;
    qrow = q0 + qcol;

    // The exact variant only redoes tiles the fast variant flagged (NaN in lse); a
    // skipped tile leaves no lists for the next one.
    if (EXACT) {
      const int flagged = qrow < T ? __builtin_isnan(a.lse[((size_t)b * a.Hq + qh) * T + qrow]) : 0;
      if (!__syncthreads_or(flagged)) {
        lists_ok = false;
        continue;
      }
    }

    // Q column in registers as the B operand of S^T = K Q^T: k-step s uses the
    // 16-byte chunk 2 s + hi of the query row.
    {
      const uint16_t* row = qbase + (size_t)min(qrow, T - 1) * D;
#pragma unroll
      for (int s = 0; s < KS; ++s) qf[s] = *reinterpret_cast<const bf16x8*>(row + (2 * s + hi) * 8);
    }
#pragma unroll
    for (int d = 0; d < DB; ++d) o[d] = f32x16{};
    m = -__builtin_inff();
    l = 0.f;
    ovf = false;

    // Lists of the tile from the previous tile's (its keys still alive, reclassified,
    // plus the new positions pq1 + 1 .. q1), or from a full scan.
    bool have = false;
    if (lists_ok) {
      int pt[kCapP / kThreads], pe[kCapP / kThreads];  // list P moves to registers first
#pragma unroll
      for (int k = 0; k < kCapP / kThreads; ++k) {
        const int i = tid + k * kThreads;
        pt[k] = i < cntP ? sm.posP[i] : 0;
        pe[k] = i < cntP ? sm.posP[i] + sm.lenP[i] : 0;
      }
      int nA = 0, nP = 0;
      bool fits = true;
      // List A in place, 512 entries at a time: an entry's new index never exceeds
      // its old one, and every thread reads its entry before append's barrier.
      for (int c0 = 0; c0 < cntA; c0 += kThreads) {
        const int i = c0 + tid;
        const bool v = i < cntA;
        const int t = v ? sm.listA[i] : 0, e = v ? sm.eA[i] : 0;
        fits = append(v, t, e, nA, nP) && fits;
      }
#pragma unroll
      for (int k = 0; k < kCapP / kThreads; ++k)
        if (k * kThreads < cntP) fits = append(tid + k * kThreads < cntP, pt[k], pe[k], nA, nP) && fits;
      {
        const int p = pq1 + 1 + tid;
        const bool v = p <= q1;
        fits = append(v, p, v ? ev[p] : 0, nA, nP) && fits;
      }
      have = fits;
      cntA = nA;
      cntP = nP;
    }

    // Windows of key positions [w0, w1): the compaction scan over their lifetimes
    // stops before either list could overflow, and the window's lists are then
    // processed in full. With the running top-k policy one window covers 0 .. q1.
    // (Scanning first and computing after keeps the accumulators in one place; a
    // scan interleaved with the block loop makes the compiler copy them.)
    lists_ok = true;
    for (int w0 = 0, first = 1; w0 <= q1; first = 0) {
      if (have) {
        w0 = q1 + 1;
      } else {
        if (w0 == 0) {
          stage(0);
          staged = 0;
        }
        const int last_chunk = q1 / kChunk;
        cntA = 0;
        cntP = 0;
        int base = w0;
        while (base <= q1 && cntA <= kCapA - kScan && cntP <= kCapP - kScan) {
          if ((base & (kChunk - 1)) == 0) {
            // This chunk has landed once only the next chunk's copies (2 per wave,
            // issued after it; loads complete in order) are outstanding.
            const int c = base / kChunk;
            if (staged > c) wait_vmcnt<2>();
            else wait_vmcnt<0>();
            block_barrier();  // for every wave; chunk c - 1's buffer is free
            if (c + 1 <= last_chunk) stage(staged = c + 1);
          }
          // Thread tid looks at positions base + 512 j + tid, so each wave's ballot
          // is already in position order.
          const int* evc = sm.evs[(base / kChunk) & (kEvBufs - 1)] + (base & (kChunk - 1));
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const int p = base + 512 * j + tid;
            append(p <= q1, p, p <= q1 ? evc[512 * j + tid] : 0, cntA, cntP);
          }
          base += kScan;
        }
        lists_ok = lists_ok && first && base > q1;  // one window: the lists are complete
        w0 = base;
      }
      // Pad both lists to whole blocks: position -1 (zero rows), lifetime 0.
      if (tid < 32) {
        if (cntA + tid < ((cntA + 31) & ~31)) sm.listA[cntA + tid] = -1;
        if (cntP + tid < ((cntP + 31) & ~31)) {
          sm.posP[cntP + tid] = -1;
          sm.lenP[cntP + tid] = 0;
        }
      }
      lds_sync();  // the lists are complete and visible to every wave

      // Blocks of list A (no per-element test) then of list P.
      // The list sizes are the same in every lane (sums of counts read back from
      // LDS); taking them from lane 0 lets the block loop branch on scalars.
      cntA = __builtin_amdgcn_readfirstlane(cntA);
      cntP = __builtin_amdgcn_readfirstlane(cntP);
      const int nbA = (cntA + 31) >> 5;
      const int nbt = nbA + ((cntP + 31) >> 5);
      auto source = [&](int i, const int*& lp, bool& msk, int& n, int& blk) __attribute__((always_inline)) {
        msk = i >= nbA;
        lp = msk ? sm.posP : sm.listA;
        n = msk ? cntP : cntA;
        blk = msk ? i - nbA : i;
      };
      const int* lp;
      bool msk;
      int n, blk;
      if (EXACT && nbt > 0) {
        // Unpipelined: block i + 1 is gathered while block i is computed; buffer
        // i % kBufs is refilled at iteration i + kBufs - 1, after more barriers.
        source(0, lp, msk, n, blk);
        issue(lp, blk, 0);
        for (int i = 0; i < nbt; ++i) {
          if (i + 1 < nbt) {
            source(i + 1, lp, msk, n, blk);
            issue(lp, blk, (i + 1) % kBufs);
          }
          wait_block(i + 1 < nbt ? 1 : 0);
          block_barrier();
          source(i, lp, msk, n, blk);
          f32x16 x;
          qk(i % kBufs, x);
          prep(x, lp, sm.lenP, msk, n, blk, i % kBufs);
          bf16x8 pk[2];
          softmax_exact(x, pk);
          VFrag<DB> vf;
          vfrag_issue(vf, lds_addr(sm.vtile[i % kBufs] + lane * 4));
          vfrag_wait(vf);
          pv(vf, pk);
        }
        __syncthreads();
      } else if (nbt > 0) {
        // Software pipeline over the blocks. Iteration i computes the scores of
        // block i + 1 (MFMA) while it turns block i's scores into probabilities
        // (VALU), then multiplies block i's probabilities with its values. The
        // workgroup meets at a barrier on even iterations only: barrier i certifies
        // blocks i + 1 and i + 2 (copied since barrier i - 2), after which blocks
        // i + 3 and i + 4 are copied into the buffers of blocks i - 2 and i - 1,
        // which every wave finished with in iteration i - 1. Blocks i .. i + 4 are
        // live, one buffer each.
        for (int j = 0; j < 3 && j < nbt; ++j) {
          source(j, lp, msk, n, blk);
          issue(lp, blk, j);
        }
        wait_block(min(nbt, 3) - 1);
        block_barrier();
        // One iteration: block i's scores arrive in sc, block i + 1's leave in sn.
        // The K reads of block i + 1 go out before the V reads of block i, so the
        // QK^T product starts once they land. Its MFMAs are interleaved with block
        // i's exponentials, and the PV MFMAs (k-half major, so no two in a row
        // share an accumulator) with the packing and the row sums.
        auto iter = [&](int i, f32x16& sc, f32x16& sn, bool even) __attribute__((always_inline)) {
          if (even && i + 1 < nbt) {
            wait_vmcnt<0>();  // this wave's copies of blocks i + 1 and i + 2
            block_barrier();
#pragma unroll
            for (int j = 3; j <= 4; ++j) {
              if (i + j < nbt) {
                source(i + j, lp, msk, n, blk);
                issue(lp, blk, (i + j) % kBufs);
              }
            }
          }
          // Block i + 1's K fragments (on the last iteration a stale buffer; the
          // scores are unused) and block i's V fragments, read without the
          // compiler's waits for the copies in flight.
          KFrag<KS> kf;
          kfrag_issue(kf, lds_addr(sm.ktile[(i + 1) % kBufs] + lane * 8));
          VFrag<DB> vf;
          vfrag_issue(vf, lds_addr(sm.vtile[i % kBufs] + lane * 4));
          source(i, lp, msk, n, blk);
          prep(sc, lp, sm.lenP, msk, n, blk, i % kBufs);
          if (__builtin_amdgcn_ballot_w64(m == -__builtin_inff()) != 0) {
            // Fixed reference: the first finite block maximum, taken only until
            // every column of the wave has one.
            const float mx = block_max(sc);
            if (m == -__builtin_inff()) m = mx;
          }
          const float mu = m == -__builtin_inff() ? 0.f : m;
          kfrag_wait_before_v(kf);
          // Raised wave priority over the MFMA section: the arbiter then favours the
          // wave that is feeding the matrix core over its SIMD partner's prologue.
          __builtin_amdgcn_s_setprio(1);
          __builtin_amdgcn_sched_barrier(0);
          constexpr int EPK = 16 / KS;  // exponentials per QK^T k-step
          float p[16];
          sn = f32x16{};
#pragma unroll
          for (int st = 0; st < KS; ++st) {
            sn = mfma32(kf.r[st], qf[st], sn);
#pragma unroll
            for (int e = 0; e < EPK; ++e) {
              const int r = st * EPK + e;
              p[r] = HAS_BIAS ? __builtin_amdgcn_exp2f(sc[r] - mu)
                              : __builtin_amdgcn_exp2f(__builtin_fmaf(sc[r], a.c, -mu));
            }
            __builtin_amdgcn_sched_barrier(0);
          }
          bf16x8 pk[2];
#pragma unroll
          for (int k2 = 0; k2 < 2; ++k2) {
            f32x8 v8;
#pragma unroll
            for (int j = 0; j < 8; ++j) v8[j] = p[8 * k2 + j];
            pk[k2] = __builtin_convertvector(v8, bf16x8);
          }
          vfrag_wait(vf);
          __builtin_amdgcn_sched_barrier(0);
          float ts[2] = {p[0], p[1]};  // the first terms seed the partial sums
#pragma unroll
          for (int k2 = 0; k2 < 2; ++k2) {
#pragma unroll
            for (int d = 0; d < DB; ++d) {
              const i16x4 lo = vf.r[4 * d + 2 * k2], up = vf.r[4 * d + 2 * k2 + 1];
              const i16x8 w8 = {lo[0], lo[1], lo[2], lo[3], up[0], up[1], up[2], up[3]};
              o[d] = mfma32(__builtin_bit_cast(bf16x8, w8), pk[k2], o[d]);
#pragma unroll
              for (int e = 0; e < 8 / DB; ++e) {
                const int r = 8 * k2 + (8 / DB) * d + e;
                if (r >= 2) ts[r & 1] += p[r];
              }
              __builtin_amdgcn_sched_barrier(0);
            }
          }
          const float t = ts[0] + ts[1];
          l += t;
          // Terms up to 2^64 above the reference are exact in fp32 and bf16. A block
          // sum beyond that (or inf) means some term may exceed it: flag the column.
          ovf = ovf || !(t <= kOverflowSum);
          __builtin_amdgcn_s_setprio(0);
        };
        f32x16 sa, sb;
        qk(0, sa);
        for (int i = 0; i < nbt; i += 2) {
          iter(i, sa, sb, true);
          if (i + 1 < nbt) iter(i + 1, sb, sa, false);
        }
        __syncthreads();
      }
    }

    // Epilogue: combine the two lane halves' sums, normalise, write O (bf16) and
    // LSE. A fast-variant column whose terms overflowed the fixed reference writes
    // NaN to its LSE instead; the exact variant then recomputes the whole tile.
    float l0, l1;
    pair_values(l, l0, l1);
    const float lt = l0 + l1;
    const float inv = lt > 0.f ? 1.0f / lt : 0.f;
    const bool redo = !EXACT && __builtin_amdgcn_ballot_w64(ovf) != 0;
    if (qrow < T) {
      const size_t rowi = ((size_t)b * a.Hq + qh) * T + qrow;
      if (hi == 0)
        a.lse[rowi] = redo ? __builtin_nanf("") : lt > 0.f ? (m + __builtin_amdgcn_logf(lt)) * kLn2 : -__builtin_inff();
      uint16_t* orow = a.o + rowi * D;
#pragma unroll
      for (int d = 0; d < DB; ++d) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 v4 = {o[d][4 * g] * inv, o[d][4 * g + 1] * inv, o[d][4 * g + 2] * inv, o[d][4 * g + 3] * inv};
          *reinterpret_cast<bf16x4*>(orow + 32 * d + 8 * g + 4 * hi) = __builtin_convertvector(v4, bf16x4);
        }
      }
    }
  }
}

// The fast variant, then the exact one, which skips at once every tile the fast one
// did not flag. Both give each workgroup a run of L.run tiles.
template <int D, int HPW, bool HB>
int launch_d(const SparseLaunch& L) {
  const unsigned groups = (unsigned)(L.B * L.Hkv * L.nch);
  const unsigned grid = (unsigned)((L.ntiles + L.run - 1) / L.run) * groups;
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

// Workgroup geometry: 8 (head, 32-query) columns. With G >= 2 a wave pair holds two
// heads of the same 32 queries; the workgroup covers hc = hpw * nhp heads and a
// query tile of qt = 32 * (2 / hpw) * wq positions.
void sparse_attn_plan(SparseLaunch& L) {
  L.G = L.Hq / L.Hkv;
  L.hpw = L.G >= 2 ? 2 : 1;
  const int nhp = L.G / L.hpw < 4 ? L.G / L.hpw : 4;  // head groups per workgroup
  L.wq = 4 / nhp;                                      // wave pairs along the queries
  L.qt = 32 * (2 / L.hpw) * L.wq;
  L.hc = L.hpw * nhp;
  L.nch = L.G / L.hc;
  L.ntiles = (L.T + L.qt - 1) / L.qt;
  // Runs of consecutive tiles share their key lists, but each run is one workgroup.
  // The first tile of a run scans the lifetimes of its whole prefix (about T / 2048
  // scan steps on average), so runs of at least T / 8192 tiles keep the scans a few
  // percent of the work; beyond that, runs are shortened until the launch has about
  // kRunGrid workgroups (16 per CU). Shorter runs also keep the workgroups that run
  // together on an XCD on nearby tiles of one group, whose kept keys mostly
  // coincide: at B = 4, T = 32768 runs of 4 tiles gather 5.0 GB per call past L2
  // against 16.4 GB with runs of 16, and are 1.5-3.5% faster (two boxes); at B = 1,
  // T = 131072 runs of 16 are 3% faster than runs of 4.
  const long long tiles = (long long)L.ntiles * L.B * L.Hkv * L.nch;
  const long long by_grid = tiles / kRunGrid, by_scan = (L.T + 8191) / 8192;
  const long long r = by_grid > by_scan ? by_grid : by_scan;
  L.run = r < 1 ? 1 : (r > kRunMax ? kRunMax : (int)r);
  L.c = L.scale * kLog2e;
}

int launch_sparse_attn_fwd(SparseLaunch L) {
  sparse_attn_plan(L);
  return L.D == 128 ? launch_hb<128>(L) : launch_hb<64>(L);
}

}  // namespace kvpop
