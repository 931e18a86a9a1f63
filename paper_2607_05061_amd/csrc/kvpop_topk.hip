// gfx950 kernels for KVpop's running top-k ranking (App. B.3, App. C.2, Sec. 3.1
// eqs. eligible_set and teacher_label).
//
// Per (batch row, KV head) sequence of scores r_t:
//   * static priority (eq. static_priority_app, decay step 1), in float32:
//       prio_t = fl(r_t - fl(t * log_gamma));
//   * rank_t = position of t in descending priority order, ties to the earlier t;
//   * running cutoff: at query q the eligible set is E(q) = {t : s <= t <= q - w};
//     cutoff_q = the k-th smallest rank in E(q) once |E(q)| >= k, else T (all kept);
//   * teacher label of t_new = q - w (+1 kept, -1 dropped, 0 if E(q) is empty) and
//     the boundary token (the kept eligible token with the largest rank).
//
// The paper scans q with a Fenwick tree, one dependent tree walk per query. Here
// every query is answered independently: E(q) is a prefix of the positions s, s+1,
// ..., so cutoff_q is the k-th smallest value of a prefix of the array
// A_i = rank_{s+i}, which a wavelet matrix over A answers in ceil(log2 T) constant-
// time steps. The ranks come from chunks of 4096 positions, each sorted by one
// workgroup (a stable LSD radix sort of 32-bit priority keys, 8 bits per pass),
// and then merged: a key's rank is its rank in its own chunk plus, for every other
// chunk, the number of that chunk's keys ordered before it (a binary search), so
// a sequence of 32768 positions keeps 8 workgroups busy in each step. One workgroup
// per sequence then builds the wavelet matrix (one stable partition per bit level,
// most significant first): in LDS, one scan per level, when A has at most 32767
// entries and T <= 65536; otherwise in global memory, 1024 consecutive elements per
// round so that every access is coalesced. Then one thread per query walks the
// levels.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "kvpop.h"
#include "kvpop_internal.h"

namespace kvpop {
namespace {

constexpr int kPrepThreads = 1024;
constexpr int kPrepWaves = kPrepThreads / 64;

// Monotone map from float to uint32 such that larger floats give larger keys;
// inverted so that an ascending sort puts the highest priority first. -0.0 and
// +0.0 compare equal as numbers, so both map to the key of +0.0.
__device__ __forceinline__ uint32_t desc_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  const uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ~asc;
}

// fl(r - fl(t * lg)): two roundings, never fused into one fma, so that the ranking
// decided by these values is reproducible from their float32 definition.
__device__ __forceinline__ float static_priority(float r, float t, float lg) {
#pragma clang fp contract(off)
  const float d = t * lg;
  return r - d;
}

// Workgroup barrier after this wave's LDS operations have completed (lgkmcnt(0)),
// without waiting for its outstanding global stores as __syncthreads() does: for
// barriers that only exchange LDS data.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt at their maxima
  asm volatile("s_barrier" ::: "memory");
}

// Exclusive scan (sum or max) over the 1024 threads of the block. `sh` needs
// kPrepWaves + 1 ints. Returns the exclusive prefix; `total` gets the reduction.
template <bool MAX>
__device__ __forceinline__ int block_scan(int v, int* sh, int& total) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off);
    if (lane >= off) x = MAX ? max(x, y) : x + y;
  }
  if (lane == 63) sh[wid] = x;
  lds_barrier();
  if (wid == 0) {
    int s = lane < kPrepWaves ? sh[lane] : (MAX ? INT32_MIN : 0);
    int incl = s;
#pragma unroll
    for (int off = 1; off < kPrepWaves; off <<= 1) {
      const int y = __shfl_up(incl, off);
      if (lane >= off) incl = MAX ? max(incl, y) : incl + y;
    }
    if (lane < kPrepWaves) sh[lane] = incl;
  }
  lds_barrier();
  const int before_wave = wid > 0 ? sh[wid - 1] : (MAX ? INT32_MIN : 0);
  const int prev = __shfl_up(x, 1);  // inclusive value of lane - 1 (all lanes take part)
  const int excl = MAX ? (lane > 0 ? max(before_wave, prev) : before_wave) : before_wave + x - v;
  total = sh[kPrepWaves - 1];
  lds_barrier();
  return excl;
}

constexpr int kSortJ = 4;  // elements per thread in a sort round
// Positions per sorted chunk: one sort round of kSortJ x 1024 elements.
constexpr int kRankChunk = kSortJ * kPrepThreads;

// LDS of the chunk sort.
// A chunk is one round of the sort, so a destination never exceeds kRankChunk and
// the counts fit 16 bits; that leaves room in LDS for the chunk itself.
struct SortSmem {
  uint16_t cnt[kSortJ][kPrepWaves][256];  // per-(slot, wave) digit counts of a round (cleared after use)
  uint16_t pre[kSortJ][kPrepWaves][256];  // destinations: bucket base plus earlier (slot, wave)s
  int base[256];                          // next free slot of each bucket
  int sh[kPrepWaves + 1];                 // block_scan scratch
  uint32_t key[2][kRankChunk];            // the chunk's keys and positions, sorted from one
  uint32_t val[2][kRankChunk];            // buffer into the other by each pass
};

// Eligible positions whose wavelet levels are built in LDS: the array A and its
// partition, 16-bit values each (ranks below 65536). One below 2^15, so that a
// block's zero and one counts, and their sums, pack into the halves of an int.
constexpr int kLdsLevels = 32767;
constexpr int kLdsBlocks = (kLdsLevels + 63) / 64;  // 64-position blocks of a level
constexpr int kLdsPerThread = (kLdsLevels + kPrepThreads - 1) / kPrepThreads;  // 32

// LDS of the wavelet build.
struct PrepSmem {
  int sh[kPrepWaves + 1];        // block_scan scratch
  int wc[2][2][4 * kPrepWaves];  // wavelet rounds: [round parity][zeros, ones][j * 16 + wave]
  int bitcnt[32];                // elements of A with each bit set
  int blk[kLdsBlocks];           // LDS levels: (zeros << 16) | ones of each 64-position block
  int blkpre[kLdsBlocks];        // and their exclusive prefix sums
};

// One stable counting-sort pass on the 8-bit digit at `shift` (a pass of an LSD
// radix sort). A round moves 4096 elements: thread tid takes r0 + 1024 j + tid for
// j = 0..3, each placed at base[d] + (elements of digit d in earlier (j, wave)
// pairs of the round) + (earlier lanes of its wave with digit d), the last found
// with eight ballots. n <= kRankChunk (one round; the 16-bit destinations hold it).
__device__ __forceinline__ void sort_pass(const uint32_t* __restrict__ kin, const uint32_t* __restrict__ vin,
                                          uint32_t* __restrict__ kout, uint32_t* __restrict__ vout, int n, int shift,
                                          SortSmem& sm) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid < 256) sm.base[tid] = 0;
  __syncthreads();
  for (int i = tid; i < n; i += kPrepThreads) atomicAdd(&sm.base[(kin[i] >> shift) & 255u], 1);
  __syncthreads();
  int tot;
  const int ex = block_scan<false>(tid < 256 ? sm.base[tid] : 0, sm.sh, tot);
  if (tid < 256) sm.base[tid] = ex;
  __syncthreads();
  const uint64_t lt = (1ull << lane) - 1ull;
  for (int r0 = 0; r0 < n; r0 += kSortJ * kPrepThreads) {
    uint32_t k[kSortJ], v[kSortJ];
    int d[kSortJ], rk[kSortJ];
    bool valid[kSortJ];
#pragma unroll
    for (int j = 0; j < kSortJ; ++j) {
      const int i = r0 + 1024 * j + tid;
      valid[j] = i < n;
      k[j] = valid[j] ? kin[i] : 0u;
      v[j] = valid[j] ? vin[i] : 0u;
    }
#pragma unroll
    for (int j = 0; j < kSortJ; ++j) {
      d[j] = (int)((k[j] >> shift) & 255u);
      uint64_t mm = __builtin_amdgcn_ballot_w64(valid[j]);
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const bool bit = (d[j] >> b) & 1;
        const uint64_t bb = __builtin_amdgcn_ballot_w64(bit);
        mm &= bit ? bb : ~bb;
      }
      rk[j] = __popcll(mm & lt);
      if (valid[j] && rk[j] == 0) sm.cnt[j][wave][d[j]] = (uint16_t)__popcll(mm);
    }
    __syncthreads();
    if (tid < 256) {
      int run = sm.base[tid];
#pragma unroll
      for (int j = 0; j < kSortJ; ++j) {
        int c[kPrepWaves];
#pragma unroll
        for (int w = 0; w < kPrepWaves; ++w) c[w] = sm.cnt[j][w][tid];
#pragma unroll
        for (int w = 0; w < kPrepWaves; ++w) {
          sm.pre[j][w][tid] = (uint16_t)run;
          sm.cnt[j][w][tid] = 0;
          run += c[w];
        }
      }
      sm.base[tid] = run;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kSortJ; ++j) {
      if (valid[j]) {
        const int dst = sm.pre[j][wave][d[j]] + rk[j];
        kout[dst] = k[j];
        vout[dst] = v[j];
      }
    }
  }
  __syncthreads();
}

// One wavelet-matrix level: stable partition of ain by bit `bit` (zeros first) into
// aout, and the level's bit words bw[W + 1] and ones-before-word counts cw[W + 1].
// A round covers 4096 elements: thread tid takes r0 + 1024 j + tid for j = 0..3, so
// each (j, wave) ballot is 64 consecutive bits, i.e. two words of the level; the
// zeros and ones before each (j, wave) come from one exchange of the 64 counts and a
// scan across the lanes of every wave.
// total_ones: elements with bit `bit` set (a reordering does not change it).
__device__ __forceinline__ uint32_t wavelet_level(const uint32_t* __restrict__ ain, uint32_t* __restrict__ aout,
                                                  int n, int bit, int total_ones, uint32_t* __restrict__ bw,
                                                  uint32_t* __restrict__ cw, PrepSmem& sm) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int W = (n + 31) / 32;
  const uint64_t lt = (1ull << lane) - 1ull;
  int zrun = 0, orun = n - total_ones;  // next slots of zeros and ones
  int onesb = 0;                        // ones before this round
  for (int r0 = 0, par = 0; r0 < n; r0 += 4 * kPrepThreads, par ^= 1) {
    uint32_t x[4];
    bool one[4], valid[4];
    uint64_t ob[4], zb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = r0 + 1024 * j + tid;
      valid[j] = i < n;
      x[j] = valid[j] ? ain[i] : 0u;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      one[j] = valid[j] && ((x[j] >> bit) & 1u);
      ob[j] = __builtin_amdgcn_ballot_w64(one[j]);
      zb[j] = __builtin_amdgcn_ballot_w64(valid[j]) & ~ob[j];
    }
    int* zc = sm.wc[par][0];  // [j * 16 + wave]
    int* oc = sm.wc[par][1];
    if (lane == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        zc[j * kPrepWaves + wave] = __popcll(zb[j]);
        oc[j * kPrepWaves + wave] = __popcll(ob[j]);
      }
    }
    lds_barrier();
    // Exclusive scans of the 64 counts in (j, wave) order, one count per lane.
    int zi = zc[lane], oi = oc[lane];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int zy = __shfl_up(zi, off), oy = __shfl_up(oi, off);
      if (lane >= off) {
        zi += zy;
        oi += oy;
      }
    }
    const int ztot = __shfl(zi, 63), otot = __shfl(oi, 63);
    const int zex = zi - zc[lane], oex = oi - oc[lane];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int zpre = __shfl(zex, j * kPrepWaves + wave), opre = __shfl(oex, j * kPrepWaves + wave);
      if (valid[j]) aout[one[j] ? orun + opre + __popcll(ob[j] & lt) : zrun + zpre + __popcll(zb[j] & lt)] = x[j];
      const int p0 = r0 + 1024 * j + 64 * wave;
      if (lane == 0 && p0 < n) {
        const int wd = p0 >> 5;
        bw[wd] = (uint32_t)ob[j];
        cw[wd] = (uint32_t)(onesb + opre);
        if (wd + 1 < W) {
          bw[wd + 1] = (uint32_t)(ob[j] >> 32);
          cw[wd + 1] = (uint32_t)(onesb + opre + __popc((uint32_t)ob[j]));
        }
      }
    }
    zrun += ztot;
    orun += otot;
    onesb += otot;
  }
  if (tid == 0) {
    bw[W] = 0u;
    cw[W] = (uint32_t)total_ones;
  }
  __syncthreads();  // the next level reads aout
  return (uint32_t)(n - total_ones);
}

// One wavelet-matrix level for an array of at most kLdsLevels elements in LDS, the
// same result as wavelet_level. Thread tid holds the elements 1024 e + tid of all 32
// slots e in registers, so the level needs one scan, over the zero and one counts of
// its 64-position blocks (block 16 e + wave), instead of one per round: a pass of
// ballots, the scan, and a pass that scatters the elements. Both passes stop at the
// last slot that holds elements; within them the loads never branch (the buffers
// hold 32768 entries; those from n on are ignored). Each wave gathers its 32 block
// counts, prefixes and 64 bit words in lanes, so that each moves in one instruction.
__device__ __forceinline__ uint32_t wavelet_level_lds(const uint16_t* __restrict__ ain, uint16_t* __restrict__ aout,
                                                      int n, int bit, uint32_t* __restrict__ bw,
                                                      uint32_t* __restrict__ cw, PrepSmem& sm) {
  constexpr int E = kLdsPerThread;  // 32 slots of 1024 positions
  static_assert(2 * E == 64, "two bit words per slot fill a wave");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int W = (n + 31) / 32;
  const uint64_t lt = (1ull << lane) - 1ull;
  uint32_t x[E];
  int cntv = 0;  // lane e: (zeros << 16) | ones of slot e's block
  // An opaque copy of n: the 32 compares against it are then made at every level,
  // not hoisted out of the level loop as 32 masks that spill.
  int n1 = n;
  asm volatile("" : "+s"(n1));
#pragma unroll
  for (int e = 0; e < E; ++e) {
    if (e * kPrepThreads >= n1) break;  // slots past the array (a scalar branch)
    const int i = e * kPrepThreads + tid;
    x[e] = ain[i];
    const bool valid = i < n1, one = valid && ((x[e] >> bit) & 1u);
    const uint64_t ob = __builtin_amdgcn_ballot_w64(one);
    const uint64_t zb = __builtin_amdgcn_ballot_w64(valid) & ~ob;
    const int packed = (__popcll(zb) << 16) | __popcll(ob);
    cntv = lane == e ? packed : cntv;
  }
  if (lane < E) sm.blk[16 * lane + wave] = cntv;  // blocks past n count nothing
  lds_barrier();
  int tot;
  const int ex = block_scan<false>(tid < kLdsBlocks ? sm.blk[tid] : 0, sm.sh, tot);
  if (tid < kLdsBlocks) sm.blkpre[tid] = ex;
  lds_barrier();
  const int zeros = tot >> 16, ones = tot & 0xFFFF;
  const int prev = lane < E ? sm.blkpre[16 * lane + wave] : 0;  // lane e: slot e's prefix
  uint32_t wv = 0u, cv = 0u;  // lane 2 e + h: word h of slot e's block and the ones before it
  // The ballots are taken again rather than kept: held across the scan, the 64
  // masks would spill. (Opaque copies of bit and n keep the compiler from reusing
  // the first pass's masks.)
  int bit2 = bit, n2 = n;
  asm volatile("" : "+s"(bit2), "+s"(n2));
#pragma unroll
  for (int e = 0; e < E; ++e) {
    if (e * kPrepThreads >= n2) break;
    const int i = e * kPrepThreads + tid;
    const bool valid = i < n2, one = valid && ((x[e] >> bit2) & 1u);
    const uint64_t ob = __builtin_amdgcn_ballot_w64(one);
    const uint64_t zb = __builtin_amdgcn_ballot_w64(valid) & ~ob;
    const int pre = __builtin_amdgcn_readlane(prev, e);
    const int zpre = pre >> 16, opre = pre & 0xFFFF;
    if (valid) aout[one ? zeros + opre + __popcll(ob & lt) : zpre + __popcll(zb & lt)] = (uint16_t)x[e];
    const uint32_t lo = (uint32_t)ob;
    wv = lane == 2 * e ? lo : (lane == 2 * e + 1 ? (uint32_t)(ob >> 32) : wv);
    cv = lane == 2 * e ? (uint32_t)opre : (lane == 2 * e + 1 ? (uint32_t)(opre + __popc(lo)) : cv);
  }
  // Lane 2 e + h writes word 2 (16 e + wave) + h; words from W on belong to no block.
  const int wd = 2 * (16 * (lane >> 1) + wave) + (lane & 1);
  if (wd < W) {
    bw[wd] = wv;
    cw[wd] = cv;
  }
  if (tid == 0) {
    bw[W] = 0u;
    cw[W] = (uint32_t)ones;
  }
  lds_barrier();  // the next level reads aout
  return (uint32_t)zeros;
}

struct SegWork {
  uint32_t* ka;
  uint32_t* kb;
  uint32_t* va;
  uint32_t* vb;
  int32_t* ps;     // positions in rank order
  int32_t* pmax;   // prefix maximum of A
  uint32_t* bits;  // [L][W + 1] bit words of each level
  uint32_t* cnt;   // [L][W + 1] ones before each word
  uint32_t* zeros; // [L]
};

__device__ __forceinline__ SegWork seg_work(void* ws, size_t per_seg_words, int seg, int T, int L) {
  uint32_t* base = reinterpret_cast<uint32_t*>(ws) + (size_t)seg * per_seg_words;
  const size_t W1 = (size_t)(T + 31) / 32 + 1;
  SegWork s;
  s.ka = base;
  s.kb = s.ka + T;
  s.va = s.kb + T;
  s.vb = s.va + T;
  s.ps = reinterpret_cast<int32_t*>(s.vb + T);
  s.pmax = s.ps + T;
  s.bits = reinterpret_cast<uint32_t*>(s.pmax + T);
  s.cnt = s.bits + (size_t)L * W1;
  s.zeros = s.cnt + (size_t)L * W1;
  return s;
}

// One workgroup per (sequence, chunk of kRankChunk positions): the chunk's priority
// keys and positions, sorted by key in place in ka / va. The sort is stable and the
// positions enter in order, so equal keys stay in position order.
// With a single chunk (T <= kRankChunk) the sorted order is the ranking: the kernel
// then writes rank[t] and the positions in rank order itself, and no merge follows.
__global__ __launch_bounds__(kPrepThreads) void topk_chunk_sort_kernel(const float* __restrict__ scores,
                                                                       const float* __restrict__ log_gamma, int H,
                                                                       int T, int L, void* ws, size_t per_seg_words,
                                                                       int32_t* __restrict__ rank) {
  __shared__ SortSmem sm;
  const int tid = threadIdx.x;
  const int nch = (T + kRankChunk - 1) / kRankChunk;
  const int seg = (int)blockIdx.x / nch, c = (int)blockIdx.x - seg * nch;
  const int h = seg % H;
  SegWork w = seg_work(ws, per_seg_words, seg, T, L);
  const float lg = log_gamma ? log_gamma[h] : 0.f;
  const float* r = scores + (size_t)seg * T;
  const int t0 = c * kRankChunk, n = min(kRankChunk, T - t0);

  for (int i = tid; i < kSortJ * kPrepWaves * 256; i += kPrepThreads) (&sm.cnt[0][0][0])[i] = 0;
  // Keys and positions into LDS; no fma contraction, to match fl(r - fl(t * lg)).
  for (int i = tid; i < n; i += kPrepThreads) {
    const int t = t0 + i;
    sm.key[0][i] = desc_key(static_priority(r[t], (float)t, lg));
    sm.val[0][i] = (uint32_t)t;
  }
  __syncthreads();
  sort_pass(sm.key[0], sm.val[0], sm.key[1], sm.val[1], n, 0, sm);
  sort_pass(sm.key[1], sm.val[1], sm.key[0], sm.val[0], n, 8, sm);
  sort_pass(sm.key[0], sm.val[0], sm.key[1], sm.val[1], n, 16, sm);
  sort_pass(sm.key[1], sm.val[1], sm.key[0], sm.val[0], n, 24, sm);
  if (nch == 1) {
    for (int i = tid; i < n; i += kPrepThreads) {
      const int t = (int)sm.val[0][i];
      rank[(size_t)seg * T + t] = i;
      w.ps[i] = t;
    }
    return;
  }
  for (int i = tid; i < n; i += kPrepThreads) {
    w.ka[t0 + i] = sm.key[0][i];
    w.va[t0 + i] = sm.val[0][i];
  }
}

// For each key, the number of keys of a sorted chunk (m of them) ordered before it:
// those below it, and with LE (an earlier chunk) those equal to it too. The kSortJ
// searches advance together, so that their LDS reads overlap, and never branch.
template <bool LE>
__device__ __forceinline__ void count_before(const uint32_t* __restrict__ sorted, int m,
                                             const uint32_t (&key)[kSortJ], int (&rk)[kSortJ]) {
  int pos[kSortJ];
#pragma unroll
  for (int j = 0; j < kSortJ; ++j) pos[j] = 0;
#pragma unroll
  for (int step = kRankChunk; step > 0; step >>= 1) {
#pragma unroll
    for (int j = 0; j < kSortJ; ++j) {
      const int np = pos[j] + step;
      const uint32_t x = sorted[min(np, m) - 1];
      const bool before = LE ? x <= key[j] : x < key[j];
      pos[j] = ((np <= m) & before) ? np : pos[j];
    }
  }
#pragma unroll
  for (int j = 0; j < kSortJ; ++j) rk[j] += pos[j];
}

// One workgroup per (sequence, chunk): the rank of each of the chunk's keys (the
// descending priority order, ties to the earlier position) is its index in the
// sorted chunk plus, for every other chunk, the number of that chunk's keys ordered
// before it. An earlier chunk holds only earlier positions, so its equal keys count;
// a later chunk's do not. Writes rank[t] and the positions in rank order (ps).
// Chunks are staged in LDS kMergeGroup at a time, their loads all in flight at once.
constexpr int kMergeGroup = 8;
__global__ __launch_bounds__(kPrepThreads) void topk_merge_rank_kernel(int T, int L, void* ws, size_t per_seg_words,
                                                                       int32_t* __restrict__ rank) {
  __shared__ uint32_t other[kMergeGroup][kRankChunk];
  const int tid = threadIdx.x;
  const int nch = (T + kRankChunk - 1) / kRankChunk;
  const int seg = (int)blockIdx.x / nch, c = (int)blockIdx.x - seg * nch;
  SegWork w = seg_work(ws, per_seg_words, seg, T, L);
  const int t0 = c * kRankChunk, n = min(kRankChunk, T - t0);
  uint32_t key[kSortJ];
  int rk[kSortJ];
  bool valid[kSortJ];
#pragma unroll
  for (int j = 0; j < kSortJ; ++j) {
    const int i = j * kPrepThreads + tid;
    valid[j] = i < n;
    key[j] = valid[j] ? w.ka[t0 + i] : 0u;
    rk[j] = i;
  }
  for (int g0 = 0; g0 < nch; g0 += kMergeGroup) {
    __syncthreads();  // every thread is done with the previous group's keys
    uint32_t st[kMergeGroup][kSortJ];
#pragma unroll
    for (int g = 0; g < kMergeGroup; ++g)
#pragma unroll
      for (int j = 0; j < kSortJ; ++j) {
        const int c2 = g0 + g, i = j * kPrepThreads + tid;
        st[g][j] = c2 < nch && c2 != c && c2 * kRankChunk + i < T ? w.ka[c2 * kRankChunk + i] : 0u;
      }
#pragma unroll
    for (int g = 0; g < kMergeGroup; ++g)
#pragma unroll
      for (int j = 0; j < kSortJ; ++j) other[g][j * kPrepThreads + tid] = st[g][j];
    __syncthreads();
    for (int g = 0; g < kMergeGroup && g0 + g < nch; ++g) {
      const int c2 = g0 + g;
      if (c2 == c) continue;
      const int m = min(kRankChunk, T - c2 * kRankChunk);
      if (c2 < c) count_before<true>(other[g], m, key, rk);
      else count_before<false>(other[g], m, key, rk);
    }
  }
  int32_t* rkout = rank + (size_t)seg * T;
#pragma unroll
  for (int j = 0; j < kSortJ; ++j) {
    if (valid[j]) {
      const int t = (int)w.va[t0 + j * kPrepThreads + tid];
      rkout[t] = rk[j];
      w.ps[rk[j]] = t;
    }
  }
}

// One workgroup per sequence, after the ranks: prefix maxima and the wavelet matrix
// over A_i = rank_{s+i}. With LDSA (at most kLdsLevels eligible positions, T <=
// 65536) every level partitions A from one LDS buffer into the other
// (wavelet_level_lds), and only the levels' bit words and counts go to global
// memory.
template <bool LDSA>
__global__ __launch_bounds__(kPrepThreads) void topk_prepare_kernel(int T, int s, int L, void* ws,
                                                                    size_t per_seg_words,
                                                                    const int32_t* __restrict__ rank) {
  __shared__ PrepSmem sm;
  __shared__ uint16_t abuf[LDSA ? 2 : 1][LDSA ? kLdsPerThread * kPrepThreads : 1];
  const int tid = threadIdx.x;
  const int seg = blockIdx.x;
  SegWork w = seg_work(ws, per_seg_words, seg, T, L);
  const int32_t* rk = rank + (size_t)seg * T;

  const int n = T - s;  // eligible positions s .. T-1
  if (n <= 0) return;

  const int W = (n + 31) / 32;
  if constexpr (LDSA) {
    // A_i = rank_{s+i} into LDS, coalesced.
    for (int i = tid; i < n; i += kPrepThreads) abuf[0][i] = (uint16_t)rk[s + i];
    lds_barrier();
    // Prefix maxima of A (the boundary token before saturation): thread tid takes
    // positions kLdsPerThread tid .. + kLdsPerThread - 1, and one scan of the
    // threads' maxima gives each its running maximum before them.
    // (The loads never branch: the buffer holds 32768 entries.)
    const int i0 = tid * kLdsPerThread;
    int av[kLdsPerThread];
    int mx = INT32_MIN;
#pragma unroll
    for (int e = 0; e < kLdsPerThread; ++e) {
      av[e] = i0 + e < n ? (int)abuf[0][i0 + e] : INT32_MIN;
      mx = max(mx, av[e]);
    }
    int total;
    int run = block_scan<true>(mx, sm.sh, total);
#pragma unroll
    for (int e = 0; e < kLdsPerThread; ++e) {
      run = max(run, av[e]);
      if (i0 + e < n) w.pmax[i0 + e] = run;
    }
    // Wavelet matrix: level l splits on bit L-1-l of the current array (stable).
    uint16_t *ain = abuf[0], *aout = abuf[LDSA ? 1 : 0];
    for (int l = 0; l < L; ++l) {
      const uint32_t z = wavelet_level_lds(ain, aout, n, L - 1 - l, w.bits + (size_t)l * (W + 1),
                                           w.cnt + (size_t)l * (W + 1), sm);
      if (tid == 0) w.zeros[l] = z;
      uint16_t* t0 = ain;
      ain = aout;
      aout = t0;
    }
  } else {
    // A_i = rank_{s+i} and its prefix maxima (the boundary token before
    // saturation), one coalesced round of 1024 positions at a time; also the number
    // of A values with each bit set, which every wavelet level needs.
    if (tid < 32) sm.bitcnt[tid] = 0;
    int bits[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) bits[k] = 0;
    int run = INT32_MIN;
    for (int r0 = 0; r0 < n; r0 += kPrepThreads) {
      const int i = r0 + tid;
      const int av = i < n ? rk[s + i] : INT32_MIN;
      if (i < n) {
        w.ka[i] = (uint32_t)av;
#pragma unroll
        for (int k = 0; k < 32; ++k) bits[k] += (av >> k) & 1;
      }
      int total;
      const int ex = block_scan<true>(av, sm.sh, total);
      if (i < n) w.pmax[i] = max(run, max(ex, av));
      run = max(run, total);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 32; ++k) {
      int c = bits[k];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
      if ((tid & 63) == 0 && k < L) atomicAdd(&sm.bitcnt[k], c);
    }
    __syncthreads();
    // Wavelet matrix: level l splits on bit L-1-l of the current array (stable).
    uint32_t *ain = w.ka, *aout = w.kb;
    for (int l = 0; l < L; ++l) {
      const uint32_t z = wavelet_level(ain, aout, n, L - 1 - l, sm.bitcnt[L - 1 - l], w.bits + (size_t)l * (W + 1),
                                       w.cnt + (size_t)l * (W + 1), sm);
      if (tid == 0) w.zeros[l] = z;
      uint32_t* t0 = ain;
      ain = aout;
      aout = t0;
    }
  }
}

// Ones among the first i entries of level l.
__device__ __forceinline__ int rank1(const uint32_t* bw, const uint32_t* cw, int i) {
  const int wd = i >> 5, b = i & 31;
  const uint32_t mask = b ? (0xFFFFFFFFu >> (32 - b)) : 0u;
  return (int)cw[wd] + __popc(bw[wd] & mask);
}

// The answer to query q of a sequence: the cutoff, the label of t_new = q - w and the
// boundary token. bits, cnt: the wavelet levels' words and ones-before counts, W1
// per level; zeros: each level's zero count; in global memory or LDS.
__device__ __forceinline__ void answer_query(int q, int T, int s, int w_win, int k, int L, int W1,
                                             const uint32_t* bits, const uint32_t* cnt, const uint32_t* zeros,
                                             const int32_t* __restrict__ ps, const int32_t* __restrict__ pmax,
                                             const int32_t* __restrict__ rk, int& cut, int& lab, int& bnd) {
  const long long tnew = (long long)q - w_win;
  const long long p = tnew - s + 1;  // |E(q)|
  cut = T;
  lab = 0;
  bnd = -1;
  if (p >= 1) {
    if (p >= k) {
      // k-th smallest of A[0, p) by walking the wavelet levels.
      int lo = 0, hi = (int)p, kk = k, val = 0;
      for (int l = 0; l < L; ++l) {
        const uint32_t* bw = bits + (size_t)l * W1;
        const uint32_t* cw = cnt + (size_t)l * W1;
        const int o_lo = rank1(bw, cw, lo), o_hi = rank1(bw, cw, hi);
        const int z = (hi - o_hi) - (lo - o_lo);
        if (kk <= z) {
          lo -= o_lo;
          hi -= o_hi;
        } else {
          kk -= z;
          const int Z = (int)zeros[l];
          lo = Z + o_lo;
          hi = Z + o_hi;
          val |= 1 << (L - 1 - l);
        }
      }
      cut = val;
      bnd = ps[cut];
    } else {
      bnd = ps[pmax[p - 1]];
    }
    lab = rk[tnew] <= cut ? 1 : -1;
  }
}

// One thread per (sequence, query).
__global__ __launch_bounds__(256) void topk_query_kernel(int nseg, int T, int s, int w_win, int k, int L, void* ws,
                                                         size_t per_seg_words, const int32_t* __restrict__ rank,
                                                         int32_t* __restrict__ cutoff, int32_t* __restrict__ label,
                                                         int32_t* __restrict__ boundary) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (long long)nseg * T) return;
  const int seg = (int)(gid / T), q = (int)(gid - (long long)seg * T);
  SegWork w = seg_work(ws, per_seg_words, seg, T, L);
  const int W1 = (T - s + 31) / 32 + 1;
  int cut, lab, bnd;
  answer_query(q, T, s, w_win, k, L, W1, w.bits, w.cnt, w.zeros, w.ps, w.pmax, rank + (size_t)seg * T, cut, lab,
               bnd);
  cutoff[gid] = cut;
  if (label) label[gid] = lab;
  if (boundary) boundary[gid] = bnd;
}

// Words of LDS for a sequence's wavelet levels (bit words, counts and zero counts)
// in the query kernel below: 2 L W1 + L of them (T = 32768: 30765).
constexpr int kQueryLdsWords = 32768;
constexpr int kQueryPerThread = 4;

// One workgroup per (sequence, 4096 queries): the sequence's levels are copied into
// LDS once, and each thread answers 4 queries from there, so that the level walks
// read LDS instead of global memory.
__global__ __launch_bounds__(kPrepThreads) void topk_query_lds_kernel(int T, int s, int w_win, int k, int L,
                                                                      void* ws, size_t per_seg_words,
                                                                      const int32_t* __restrict__ rank,
                                                                      int32_t* __restrict__ cutoff,
                                                                      int32_t* __restrict__ label,
                                                                      int32_t* __restrict__ boundary) {
  __shared__ uint32_t wl[kQueryLdsWords];
  constexpr int QB = kQueryPerThread * kPrepThreads;
  const int tid = threadIdx.x;
  const int nqb = (T + QB - 1) / QB;
  const int seg = (int)blockIdx.x / nqb, qb = (int)blockIdx.x - seg * nqb;
  SegWork w = seg_work(ws, per_seg_words, seg, T, L);
  const int W1 = (T - s + 31) / 32 + 1;
  const int lw = L * W1;
  for (int i = tid; i < lw; i += kPrepThreads) {
    wl[i] = w.bits[i];
    wl[lw + i] = w.cnt[i];
  }
  for (int i = tid; i < L; i += kPrepThreads) wl[2 * lw + i] = w.zeros[i];
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kQueryPerThread; ++j) {
    const int q = qb * QB + j * kPrepThreads + tid;
    if (q < T) {
      int cut, lab, bnd;
      answer_query(q, T, s, w_win, k, L, W1, wl, wl + lw, wl + 2 * lw, w.ps, w.pmax, rank + (size_t)seg * T, cut,
                   lab, bnd);
      const size_t gid = (size_t)seg * T + q;
      cutoff[gid] = cut;
      if (label) label[gid] = lab;
      if (boundary) boundary[gid] = bnd;
    }
  }
}

// One thread per (sequence, token): the query at which the token leaves the mask.
// cutoff is non-increasing in q, so the first q with cutoff_q < rank_t is found by
// binary search.
__global__ __launch_bounds__(256) void topk_evict_kernel(int nseg, int T, int s, int w_win,
                                                         const int32_t* __restrict__ rank,
                                                         const int32_t* __restrict__ cutoff,
                                                         int32_t* __restrict__ evict) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (long long)nseg * T) return;
  const int seg = (int)(gid / T), t = (int)(gid - (long long)seg * T);
  int e = T;
  if (t >= s) {
    const int32_t* cut = cutoff + (size_t)seg * T;
    const int r = rank[gid];
    int lo = 0, hi = T;  // first q in [lo, hi) with cut[q] < r, or T
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (cut[mid] < r) hi = mid;
      else lo = mid + 1;
    }
    const long long leave = (long long)t + w_win;
    e = (int)(lo > leave ? lo : (leave < T ? leave : T));
  }
  evict[gid] = e;
}

}  // namespace

int topk_levels(int T) {
  int L = 1;
  while ((1 << L) < T) ++L;
  return L;
}

size_t topk_workspace_words_per_seq(int T) {
  const int L = topk_levels(T);
  const size_t W1 = (size_t)(T + 31) / 32 + 1;
  return 6 * (size_t)T + 2 * (size_t)L * W1 + (size_t)L + 4;
}

// Scratch of kvpop_running_topk_noalloc: the workspace of the ranking kernels in a
// file-scope device array instead of caller memory. Every GPU the library runs on
// holds its own copy until the process ends; all calls on one GPU share it.
static __device__ __align__(256) uint32_t scratch[KVPOP_NOALLOC_SCRATCH_BYTES / 4];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// Device address of `scratch` on the device of `stream` (the current device for
// the null stream), resolved once per device with that device current. In host
// code the array's name is only a handle for the runtime, never an address.
int noalloc_scratch(void* stream, void** ptr) {
  int dev = 0;
  hipError_t e = stream ? hipStreamGetDevice((hipStream_t)stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  if (dev < 0 || dev >= kMaxDevices) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = 0;
    e = hipGetDevice(&cur);
    if (e != hipSuccess) return (int)e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return (int)e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return (int)e;
    if (!p) return (int)hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return 0;
}

int launch_running_topk(const TopkLaunch& L) {
  const int nseg = L.B * L.H;
  const int levels = topk_levels(L.T);
  const size_t per = topk_workspace_words_per_seq(L.T);
  const long long n_elig = (long long)L.T - L.sinks;  // eligible positions s .. T-1
  const long long chunks = (long long)nseg * ((L.T + kRankChunk - 1) / kRankChunk);
  hipLaunchKernelGGL(topk_chunk_sort_kernel, dim3((unsigned)chunks), dim3(kPrepThreads), 0, (hipStream_t)L.stream,
                     L.scores, L.log_gamma, L.H, L.T, levels, L.workspace, per, L.rank);
  int e = (int)hipGetLastError();
  if (e) return e;
  if (L.T > kRankChunk) {
    hipLaunchKernelGGL(topk_merge_rank_kernel, dim3((unsigned)chunks), dim3(kPrepThreads), 0, (hipStream_t)L.stream,
                       L.T, levels, L.workspace, per, L.rank);
    e = (int)hipGetLastError();
    if (e) return e;
  }
  if (n_elig <= kLdsLevels && L.T <= 65536)
    hipLaunchKernelGGL(topk_prepare_kernel<true>, dim3(nseg), dim3(kPrepThreads), 0, (hipStream_t)L.stream, L.T,
                       L.sinks, levels, L.workspace, per, L.rank);
  else
    hipLaunchKernelGGL(topk_prepare_kernel<false>, dim3(nseg), dim3(kPrepThreads), 0, (hipStream_t)L.stream, L.T,
                       L.sinks, levels, L.workspace, per, L.rank);
  e = (int)hipGetLastError();
  if (e) return e;
  const long long total = (long long)nseg * L.T;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  // The query kernel with the levels in LDS when they fit and its grid (one
  // workgroup per 4096 queries) covers every compute unit: below that, the copies
  // into LDS cost more than they save (B = 2, T = 16384: 64 workgroups, 2% slower).
  const long long qw1 = n_elig > 0 ? (n_elig + 31) / 32 + 1 : 0;
  const long long qblocks = (long long)nseg * ((L.T + kQueryPerThread * kPrepThreads - 1) /
                                               (kQueryPerThread * kPrepThreads));
  const int ncu = stream_cus(L.stream);
  if (n_elig > 0 && 2 * levels * qw1 + levels <= kQueryLdsWords && ncu > 0 && qblocks >= ncu) {
    hipLaunchKernelGGL(topk_query_lds_kernel, dim3((unsigned)qblocks), dim3(kPrepThreads), 0, (hipStream_t)L.stream,
                       L.T, L.sinks, L.window, L.topk, levels, L.workspace, per, L.rank, L.cutoff, L.label,
                       L.boundary);
  } else {
    hipLaunchKernelGGL(topk_query_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)L.stream, nseg, L.T, L.sinks,
                       L.window, L.topk, levels, L.workspace, per, L.rank, L.cutoff, L.label, L.boundary);
  }
  e = (int)hipGetLastError();
  if (e || !L.evict) return e;
  hipLaunchKernelGGL(topk_evict_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)L.stream, nseg, L.T, L.sinks,
                     L.window, L.rank, L.cutoff, L.evict);
  return (int)hipGetLastError();
}

}  // namespace kvpop
