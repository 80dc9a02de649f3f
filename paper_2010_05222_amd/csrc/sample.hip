// Positive-preserving negative sampling and label remap on one class shard
// (Partial FC, Sec. 3.3.1-3.3.2, Eq. local_sampling).
//
// S = P  union  {the n_neg = max(b - |P|, 0) non-positive classes with the
// smallest 64-bit Philox keys, ties to the lower class id}, sorted ascending,
// then labels_mapped = searchsorted(S, y - a).
//
// Kernel sequence (no host synchronisation; every kernel reads the
// device-side mode and returns early when it has nothing to do):
//   clear -> mark positives (bitmap, |P|) -> plan (mode, n_neg)
//   -> keys + top-bit histogram (one Philox pass; only each key's top-bit
//      digit is kept, 2 bytes per class)
//   -> pick the top bucket holding the n_neg-th key -> collect that bucket
//      (its keys recomputed in full)
//   -> resolve the remaining key bits inside one workgroup (exact threshold)
//   -> count / scan / write compaction in class order (wavefront ballots),
//      which yields S already sorted -> remap by binary search.
// A class whose digit differs from the threshold's is decided by the digit
// alone; the few in the threshold's bucket compare their recomputed key.
#include "pfc_internal.h"

namespace pfc {
namespace {

// Philox4x64-10 (Salmon et al., SC'11): multipliers and Weyl key increments
// of the 4x64 variant.
constexpr uint64_t kPhiloxM0 = 0xD2E7470EE14C6C93ull;
constexpr uint64_t kPhiloxM1 = 0xCA5A826395121157ull;
constexpr uint64_t kPhiloxW0 = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kPhiloxW1 = 0xBB67AE8584CAA73Bull;

struct U64x4 {
  uint64_t v[4];
};

__device__ __forceinline__ U64x4 philox4x64_10(uint64_t c0, uint64_t seed) {
  uint64_t x0 = c0, x1 = 0, x2 = 0, x3 = 0;
  uint64_t k0 = seed, k1 = 0;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += kPhiloxW0;
      k1 += kPhiloxW1;
    }
    const uint64_t hi0 = __umul64hi(kPhiloxM0, x0);
    const uint64_t lo0 = kPhiloxM0 * x0;
    const uint64_t hi1 = __umul64hi(kPhiloxM1, x2);
    const uint64_t lo1 = kPhiloxM1 * x2;
    const uint64_t n0 = hi1 ^ x1 ^ k0;
    const uint64_t n2 = hi0 ^ x3 ^ k1;
    x0 = n0;
    x1 = lo1;
    x2 = n2;
    x3 = lo0;
  }
  U64x4 out;
  out.v[0] = x0;
  out.v[1] = x1;
  out.v[2] = x2;
  out.v[3] = x3;
  return out;
}

// Key of class c of the shard starting at global class a.  The word is
// picked with selects: indexing the block's words by a run-time value would
// place them in LDS, and that costs more than the generator here.
__device__ __forceinline__ uint64_t class_key(uint64_t seed, int64_t a, int64_t c) {
  const int64_t g = a + c;
  const U64x4 w = philox4x64_10((uint64_t)(g >> 2), seed);
  const int i = (int)(g & 3);
  return i == 0 ? w.v[0] : i == 1 ? w.v[1] : i == 2 ? w.v[2] : w.v[3];
}

// Digits of the 16 classes c0 .. c0 + 15 (c0 a multiple of 16; the digit
// array is padded to whole groups of 16): two 16-byte loads.
__device__ __forceinline__ void load_digits16(const uint16_t* digits, int64_t c0, uint32_t (&w)[8]) {
  const uint4 d0 = *reinterpret_cast<const uint4*>(digits + c0);
  const uint4 d1 = *reinterpret_cast<const uint4*>(digits + c0 + 8);
  w[0] = d0.x; w[1] = d0.y; w[2] = d0.z; w[3] = d0.w;
  w[4] = d1.x; w[5] = d1.y; w[6] = d1.z; w[7] = d1.w;
}
__device__ __forceinline__ uint32_t digit_of(const uint32_t (&w)[8], int i) {
  return (w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

__device__ __forceinline__ uint32_t popc_below(uint64_t mask) {
  const uint64_t below = (1ull << lane_id()) - 1ull;
  return (uint32_t)__popcll(mask & below);
}

// Exclusive prefix sum of `v` over the block (blockDim.x a multiple of 64,
// at most 1024 threads); `total` receives the block sum.  Uses `smem` of
// (blockDim.x / 64) entries.
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* smem, uint32_t* total) {
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  uint32_t incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  if (lane == 63) smem[wave] = incl;
  __syncthreads();
  uint32_t wave_off = 0, sum = 0;
  for (int w = 0; w < nwaves; ++w) {
    const uint32_t t = smem[w];
    if (w < wave) wave_off += t;
    sum += t;
  }
  __syncthreads();
  *total = sum;
  return wave_off + incl - v;
}

// Same for 64-bit sums.
__device__ uint64_t block_exclusive_scan64(uint64_t v, uint64_t* smem, uint64_t* total) {
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  uint64_t incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint64_t t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  if (lane == 63) smem[wave] = incl;
  __syncthreads();
  uint64_t wave_off = 0, sum = 0;
  for (int w = 0; w < nwaves; ++w) {
    const uint64_t t = smem[w];
    if (w < wave) wave_off += t;
    sum += t;
  }
  __syncthreads();
  *total = sum;
  return wave_off + incl - v;
}

// Find the bin holding the k-th (1-based) element of an LDS histogram of
// `nbins` bins (nbins a multiple of blockDim.x).  Returns through shared
// out[0] = bin, out[1] = count before the bin, out[2] = count of the bin
// (the last bin and zero counts if the histogram holds fewer than k).
__device__ void find_kth_bin(const uint32_t* hist, int nbins, int64_t k,
                             uint64_t* scan_smem, int64_t* out) {
  if (threadIdx.x == 0) {   // ordered before the writes below by the scan's barriers
    out[0] = nbins - 1;
    out[1] = 0;
    out[2] = 0;
  }
  const int per = nbins / blockDim.x;
  const int b0 = threadIdx.x * per;
  uint64_t local = 0;
  for (int i = 0; i < per; ++i) local += hist[b0 + i];
  uint64_t total;
  uint64_t before = block_exclusive_scan64(local, scan_smem, &total);
  if ((int64_t)before < k && k <= (int64_t)(before + local)) {
    for (int i = 0; i < per; ++i) {
      const uint64_t h = hist[b0 + i];
      if ((int64_t)(before + h) >= k) {
        out[0] = b0 + i;
        out[1] = (int64_t)before;
        out[2] = (int64_t)h;
        break;
      }
      before += h;
    }
  }
  __syncthreads();
}

// ----------------------------------------------------------------- kernels

__global__ void k_sample_clear(uint32_t* bitmap, int64_t nwords, uint32_t* hist,
                               SampleState* st) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = tid; i < nwords; i += stride) bitmap[i] = 0u;
  for (int64_t i = tid; i < (1 << kTopBitsMax); i += stride) hist[i] = 0u;
  if (tid == 0) {
    st->n_pos = 0;
    st->mode = kSelectNone;
    st->top_digit = 0;
    st->n_neg = 0;
    st->k_rem = 0;
    st->thresh = 0;
  }
}

// Marks the positives and counts them once each.  The key histogram counts
// non-positive classes only; the key pass adds every class, so each
// positive's digit is taken off here (unsigned counts: the sum is exact once
// both passes are done, whatever their order inside the histogram).
__global__ void k_mark_positives(const int64_t* labels, int64_t B, int64_t C,
                                 int64_t a, uint64_t seed, int top_bits, uint32_t* bitmap,
                                 uint32_t* hist, SampleState* st) {
  const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= B) return;
  const int64_t y = labels[n];
  if (y < a || y >= a + C) return;
  const int64_t c = y - a;
  const uint32_t bit = 1u << (c & 31);
  const uint32_t old = atomicOr(&bitmap[c >> 5], bit);
  if (!(old & bit)) {
    atomicAdd(&st->n_pos, 1u);
    atomicSub(&hist[(uint32_t)(class_key(seed, a, c) >> (64 - top_bits))], 1u);
  }
}

__global__ void k_sample_plan(SampleState* st, int64_t budget, int64_t C) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const int64_t n_pos = st->n_pos;
  const int64_t n_neg = budget > n_pos ? budget - n_pos : 0;
  const int64_t pool = C - n_pos;
  st->n_neg = n_neg;
  if (n_neg == 0) {
    st->mode = kSelectNone;
    st->thresh = 0;
    st->k_rem = 0;
  } else if (n_neg >= pool) {
    st->mode = kSelectAll;
    st->thresh = ~0ull;
    st->k_rem = INT64_MAX;
  } else {
    st->mode = kSelectKeys;
    st->k_rem = n_neg;
  }
}

// Digits of the four classes of Philox block q into `digits` and the
// workgroup's histogram.  With the shard starting on a block boundary the
// four digits are one 8-byte store.
__device__ __forceinline__ void keys_block(const U64x4& w, int64_t q, int64_t a, int64_t C,
                                           int top_bits, uint16_t* digits, uint32_t* lhist) {
  const int64_t c0 = 4 * q - a;
  uint32_t dg[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) dg[i] = (uint32_t)(w.v[i] >> (64 - top_bits));
  if ((a & 3) == 0 && c0 + 3 < C) {
    *reinterpret_cast<uint2*>(digits + c0) = make_uint2(dg[0] | (dg[1] << 16), dg[2] | (dg[3] << 16));
#pragma unroll
    for (int i = 0; i < 4; ++i) atomicAdd(&lhist[dg[i]], 1u);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t c = c0 + i;
      if (c < 0 || c >= C) continue;
      digits[c] = (uint16_t)dg[i];
      atomicAdd(&lhist[dg[i]], 1u);
    }
  }
}

// Grid-stride over the Philox blocks of the shard (global ids 4q .. 4q + 3),
// two independent blocks per thread and iteration; each workgroup builds one
// histogram of its share (every class; the positives were taken off before)
// and flushes it once.  The loop reads nothing from memory.
__global__ void __launch_bounds__(1024) k_keys_hist(uint64_t seed, int64_t a, int64_t C,
                                                    int top_bits, uint16_t* digits,
                                                    uint32_t* hist, const SampleState* st) {
  if (st->mode != kSelectKeys) return;
  __shared__ uint32_t lhist[1 << kTopBitsMax];
  const int nbins = 1 << top_bits;
  for (int i = threadIdx.x; i < nbins; i += blockDim.x) lhist[i] = 0u;
  __syncthreads();
  const int64_t q_hi = (a + C - 1) >> 2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t q = (a >> 2) + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; q + stride <= q_hi; q += 2 * stride) {
    const U64x4 w0 = philox4x64_10((uint64_t)q, seed);
    const U64x4 w1 = philox4x64_10((uint64_t)(q + stride), seed);
    keys_block(w0, q, a, C, top_bits, digits, lhist);
    keys_block(w1, q + stride, a, C, top_bits, digits, lhist);
  }
  if (q <= q_hi) keys_block(philox4x64_10((uint64_t)q, seed), q, a, C, top_bits, digits, lhist);
  __syncthreads();
  // Flush starting at a per-workgroup offset so that workgroups finishing
  // together hit different bins.
  const int rot = (int)((blockIdx.x * 97u) & (uint32_t)(nbins - 1));
  for (int i = threadIdx.x; i < nbins; i += blockDim.x) {
    const int b = (i + rot) & (nbins - 1);
    const uint32_t h = lhist[b];
    if (h) atomicAdd(&hist[b], h);
  }
}

// One workgroup of 1024 threads: the top bucket holding the n_neg-th key.
__global__ void __launch_bounds__(1024) k_select_top(const uint32_t* hist, int top_bits,
                                                     SampleState* st) {
  if (st->mode != kSelectKeys) return;
  __shared__ uint32_t lh[1 << kTopBitsMax];
  __shared__ uint64_t scan_smem[16];
  __shared__ int64_t found[3];
  const int nbins = 1 << top_bits;
  const int nb = nbins < (int)blockDim.x ? (int)blockDim.x : nbins;
  for (int i = threadIdx.x; i < nb; i += blockDim.x) lh[i] = i < nbins ? hist[i] : 0u;
  __syncthreads();
  find_kth_bin(lh, nb, st->k_rem, scan_smem, found);
  if (threadIdx.x == 0) {
    st->top_digit = (uint32_t)found[0];
    st->k_rem -= found[1];
  }
}

// One workgroup per compaction group (kCompactClasses classes, kCompactPer per
// thread).  Counts the group's classes that the top-bit digit already selects
// (positives, and non-positives below the threshold's bucket; every class when
// all are taken, the positives when no negative is), and writes the full keys
// of the group's non-positive classes in that bucket to the group's own part
// of cand_key (offsets from one workgroup scan, no atomics).  The bucket's
// classes are added to their groups' counts once the threshold is known
// (k_refine).
__global__ void __launch_bounds__(kCompactThreads) k_collect(
    const uint16_t* digits, const uint32_t* bitmap, int64_t C, uint64_t seed, int64_t a,
    const SampleState* st, uint64_t* cand_key, uint32_t* grp_sure, uint32_t* grp_tie) {
  __shared__ uint32_t smem[kCompactThreads / 64];
  const uint32_t mode = st->mode;
  const uint32_t digit = st->top_digit;
  const int64_t c0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kCompactPer;
  uint32_t take = 0, base_bits = 0;
  if (c0 < C) {
    // The digits are read whatever the mode (the array always holds whole
    // groups of 16), so that these loads need not wait for the state's.
    uint32_t w[8];
    load_digits16(digits, c0, w);
    const uint32_t pos = (bitmap[c0 >> 5] >> (c0 & 31)) & 0xFFFFu;
    const uint32_t live = C - c0 >= kCompactPer ? 0xFFFFu : (1u << (C - c0)) - 1u;
    uint32_t below = 0, equal = 0;
#pragma unroll
    for (int i = 0; i < kCompactPer; ++i) {
      const uint32_t dg = digit_of(w, i);
      below |= (uint32_t)(dg < digit) << i;
      equal |= (uint32_t)(dg == digit) << i;
    }
    if (mode == kSelectAll) {
      base_bits = live;
    } else if (mode == kSelectNone) {
      base_bits = pos & live;
    } else {
      base_bits = (below | pos) & live;
      take = equal & ~pos & live;
    }
  }
  // Both counts in one scan: selected classes in the low half, candidates in
  // the high half (each at most kCompactClasses per group, so no carry).
  uint32_t tot;
  const uint32_t pre = block_exclusive_scan(
      (uint32_t)__popc(base_bits) | ((uint32_t)__popc(take) << 16), smem, &tot);
  if (threadIdx.x == 0) {
    grp_sure[blockIdx.x] = tot & 0xFFFFu;
    grp_tie[blockIdx.x] = tot >> 16;
  }
  uint64_t* out = cand_key + (int64_t)blockIdx.x * kCompactClasses + (pre >> 16);
  while (take) {
    const int i = __ffs(take) - 1;
    take &= take - 1;
    *out++ = class_key(seed, a, c0 + i);
  }
}

// The refinement's workgroup and the candidates it keeps in LDS (32 KB of
// keys; more stay in memory).  It is small enough (40 KB of LDS, two waves
// per SIMD) to share a CU with one workgroup of the step's big kernels, so a
// sampler running beside a step does not wait for a whole kernel to drain.
constexpr int kRefineThreads = 512;
constexpr int kRefineLds = 4096;

// One workgroup: resolve the remaining 64 - top_bits bits of the threshold
// among the collected candidates, 11 bits per round.  Thread t owns groups
// t, t + kRefineThreads, ...; the candidates are first gathered in that
// order into LDS when they fit.
__global__ void __launch_bounds__(kRefineThreads) k_refine(const uint64_t* cand_key, int64_t n_groups,
                                                 int top_bits, SampleState* st,
                                                 uint32_t* grp_sure, uint32_t* grp_tie) {
  if (st->mode != kSelectKeys) return;
  constexpr int kBits = 11;
  __shared__ uint32_t lh[1 << kBits];
  __shared__ uint64_t lkeys[kRefineLds];
  __shared__ uint64_t scan_smem[16];
  __shared__ int64_t found[3];
  __shared__ uint64_t sole;
  uint64_t mine = 0;
  for (int64_t g = threadIdx.x; g < n_groups; g += blockDim.x) mine += grp_tie[g];
  uint64_t total;
  const uint64_t base = block_exclusive_scan64(mine, scan_smem, &total);
  const bool in_lds = total <= (uint64_t)kRefineLds;
  if (in_lds) {
    uint64_t p = base;
    for (int64_t g = threadIdx.x; g < n_groups; g += blockDim.x) {
      const uint32_t cnt = grp_tie[g];
      for (uint32_t j = 0; j < cnt; ++j) lkeys[p + j] = cand_key[g * kCompactClasses + j];
      p += cnt;
    }
  }
  __syncthreads();
  // Calls f on every candidate key once (across the workgroup).
  auto for_each_key = [&](auto&& f) {
    if (in_lds) {
      for (uint64_t i = threadIdx.x; i < total; i += blockDim.x) f(lkeys[i]);
    } else {
      for (int64_t g = threadIdx.x; g < n_groups; g += blockDim.x) {
        const uint32_t cnt = grp_tie[g];
        for (uint32_t j = 0; j < cnt; ++j) f(cand_key[g * kCompactClasses + j]);
      }
    }
  };
  uint64_t prefix = st->top_digit;
  int known = top_bits;
  int64_t k = st->k_rem;
  while (known < 64) {
    const int bits = (64 - known) < kBits ? (64 - known) : kBits;
    const int shift = 64 - known - bits;
    for (int i = threadIdx.x; i < (1 << kBits); i += blockDim.x) lh[i] = 0u;
    __syncthreads();
    for_each_key([&](uint64_t key) {
      if ((key >> (64 - known)) == prefix)
        atomicAdd(&lh[(key >> shift) & ((1u << bits) - 1u)], 1u);
    });
    __syncthreads();
    find_kth_bin(lh, 1 << kBits, k, scan_smem, found);
    prefix = (prefix << bits) | (uint64_t)found[0];
    k -= found[1];
    known += bits;
    if (found[2] == 1 && known < 64) {
      // The bin holds a single key (k is then 1): that key is the threshold.
      for_each_key([&](uint64_t key) {
        if ((key >> (64 - known)) == prefix) sole = key;
      });
      __syncthreads();
      prefix = sole;
      known = 64;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    st->thresh = prefix;
    st->k_rem = k;
  }
  // The bucket's classes join their groups' counts: below the threshold they
  // are selected, equal to it they are ties (taken in class order).  Each
  // thread updates only the groups it owns.
  uint64_t p = base;
  for (int64_t g = threadIdx.x; g < n_groups; g += blockDim.x) {
    const uint32_t cnt = grp_tie[g];
    uint32_t below = 0, equal = 0;
    for (uint32_t j = 0; j < cnt; ++j) {
      const uint64_t key = in_lds ? lkeys[p + j] : cand_key[g * kCompactClasses + j];
      below += key < prefix;
      equal += key == prefix;
    }
    p += cnt;
    if (cnt) {
      grp_sure[g] += below;
      grp_tie[g] = equal;
    }
  }
}

// Per class of one thread: bit i of `sure` / `tie` for class c0 + i
// (i < kCompactPer).  The threshold's top-bit digit decides every class
// outside its bucket; a class inside compares its recomputed key.
__device__ __forceinline__ void class_flags(const uint16_t* digits, const uint32_t* bitmap,
                                            int64_t C, uint64_t seed, int64_t a,
                                            const SampleState* st, int64_t c0, uint32_t* sure,
                                            uint32_t* tie) {
  const uint32_t mode = st->mode;
  const uint32_t top = st->top_digit;
  const uint64_t thresh = st->thresh;
  uint32_t s = 0, t = 0, need = 0;
  if (c0 >= C) {
    *sure = 0;
    *tie = 0;
    return;
  }
  // c0 is a multiple of 16: one bitmap word holds the classes' bits.  The
  // digits are read whatever the mode, beside the state's loads.
  uint32_t w[8];
  load_digits16(digits, c0, w);
  const uint32_t pos = (bitmap[c0 >> 5] >> (c0 & 31)) & 0xFFFFu;
  const uint32_t live = C - c0 >= kCompactPer ? 0xFFFFu : (1u << (C - c0)) - 1u;
  uint32_t below = 0, equal = 0;
#pragma unroll
  for (int i = 0; i < kCompactPer; ++i) {
    const uint32_t dg = digit_of(w, i);
    below |= (uint32_t)(dg < top) << i;
    equal |= (uint32_t)(dg == top) << i;
  }
  if (mode == kSelectAll) {
    s = live;
  } else if (mode == kSelectKeys) {
    s = (below | pos) & live;
    need = equal & ~pos & live;
  } else {
    s = pos & live;
  }
  // Classes in the threshold's bucket (rare): one key generator in a loop.
  if (need) {
    do {
      const int i = __ffs(need) - 1;
      need &= need - 1;
      const uint64_t key = class_key(seed, a, c0 + i);
      if (key < thresh) s |= 1u << i;
      else if (key == thresh) t |= 1u << i;
    } while (need);
  }
  *sure = s;
  *tie = t;
}

// One workgroup of 1024 threads: per-group tie offsets, selected counts and
// output offsets; n_active.  The groups go in tiles of four per thread
// (independent, coalesced loads), with running totals carried across tiles.
__global__ void __launch_bounds__(1024) k_compact_scan(const uint32_t* grp_sure,
                                                       const uint32_t* grp_tie,
                                                       int64_t n_groups, const SampleState* st,
                                                       int64_t cap, uint32_t* grp_out,
                                                       uint32_t* grp_tie_off,
                                                       int32_t* n_active) {
  constexpr int PER = 4;
  __shared__ uint64_t smem[16];
  const int64_t k_rem = st->k_rem;
  const int64_t tile = (int64_t)blockDim.x * PER;
  uint64_t carry_tie = 0, carry_sel = 0;
  for (int64_t base = 0; base < n_groups; base += tile) {
    const int64_t g0 = base + (int64_t)threadIdx.x * PER;
    uint32_t t[PER], sr[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int64_t g = g0 + i;
      t[i] = g < n_groups ? grp_tie[g] : 0u;
      sr[i] = g < n_groups ? grp_sure[g] : 0u;
    }
    // Ties before each group.
    uint64_t tile_tie;
    uint64_t tb = carry_tie +
                  block_exclusive_scan64((uint64_t)t[0] + t[1] + t[2] + t[3], smem, &tile_tie);
    // Selected count of each group: sure + the ties whose class-order rank is below k_rem.
    uint32_t sel[PER];
    uint64_t tie_off[PER];
    uint64_t local_sel = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      int64_t take = k_rem - (int64_t)tb;
      take = take < 0 ? 0 : (take > (int64_t)t[i] ? (int64_t)t[i] : take);
      sel[i] = sr[i] + (uint32_t)take;
      tie_off[i] = tb;
      local_sel += sel[i];
      tb += t[i];
    }
    uint64_t tile_sel;
    uint64_t ob = carry_sel + block_exclusive_scan64(local_sel, smem, &tile_sel);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int64_t g = g0 + i;
      if (g < n_groups) {
        grp_tie_off[g] = (uint32_t)tie_off[i];
        grp_out[g] = (uint32_t)ob;
      }
      ob += sel[i];
    }
    carry_tie += tile_tie;
    carry_sel += tile_sel;
  }
  // |S| <= cap by construction; the clamp keeps every later index in bounds.
  if (threadIdx.x == 0) *n_active = (int32_t)(carry_sel < (uint64_t)cap ? carry_sel : cap);
}

__global__ void __launch_bounds__(kCompactThreads) k_compact_write(
    const uint16_t* digits, const uint32_t* bitmap, int64_t C, uint64_t seed, int64_t a,
    const SampleState* st, const uint32_t* grp_out, const uint32_t* grp_tie_off, int64_t cap,
    int32_t* active) {
  __shared__ uint32_t smem[kCompactThreads / 64];
  const int64_t c0 = ((int64_t)blockIdx.x * kCompactThreads + threadIdx.x) * kCompactPer;
  const int64_t tie_off = grp_tie_off[blockIdx.x];
  const int64_t out_off = grp_out[blockIdx.x];
  const int64_t k_rem = st->k_rem;
  uint32_t s, t;
  class_flags(digits, bitmap, C, seed, a, st, c0, &s, &t);
  // Class-order ranks: thread t owns classes kCompactPer t .. + kCompactPer - 1,
  // so a class's rank is the block's exclusive prefix of the per-thread
  // counts plus the bits below it in the thread.
  uint32_t ttot;
  const uint32_t tpre = block_exclusive_scan((uint32_t)__popc(t), smem, &ttot);
  const int64_t tie_base = tie_off + tpre;
  uint32_t sel = s;
#pragma unroll
  for (int i = 0; i < kCompactPer; ++i)
    if (((t >> i) & 1u) && tie_base + __popc(t & ((1u << i) - 1u)) < k_rem) sel |= 1u << i;
  uint32_t stot;
  const uint32_t spre = block_exclusive_scan((uint32_t)__popc(sel), smem, &stot);
  const int64_t out_base = out_off + spre;
  uint32_t rest = sel;
  while (rest) {
    const int i = __ffs(rest) - 1;
    rest &= rest - 1;
    const int64_t o = out_base + __popc(sel & ((1u << i) - 1u));
    if (o < cap) active[o] = (int32_t)(c0 + i);
  }
}

// One wave per batch row.  S is written group by group, so a class of
// compaction group g can only sit in [grp_out[g], grp_out[g + 1]) (clamped to
// |S|).  The wave finds the first index f there whose id is >= the label
// (searchsorted): [lo, hi) is the part not yet decided (ids before lo are
// < the label, ids from hi on are >=); 64 probes per round shrink it to under
// 64 entries (one round for a group's at most 4,096), and one read of those
// plus index hi gives f and the id found there.
__global__ void __launch_bounds__(256) k_remap(const int64_t* labels, int64_t B, int64_t C,
                                               int64_t a, const int32_t* active,
                                               const int32_t* n_active, const uint32_t* grp_out,
                                               int64_t n_groups, int32_t* labels_mapped) {
  const int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = lane_id();
  if (n >= B) return;   // wave-uniform
  const int64_t y = labels[n];
  if (y < a || y >= a + C) {
    if (lane == 0) labels_mapped[n] = -1;
    return;
  }
  const int32_t c = (int32_t)(y - a);
  const int64_t k = *n_active;
  const int64_t g = c / kCompactClasses;
  const int64_t g_lo = grp_out[g];
  const int64_t g_hi = g + 1 < n_groups ? (int64_t)grp_out[g + 1] : k;
  const int64_t end = g_hi < k ? g_hi : k;
  int64_t lo = g_lo < end ? g_lo : end;
  int64_t hi = end;
  while (hi - lo > 63) {
    const int64_t len = hi - lo;
    const int64_t p = lo + (len * lane) / 64;   // strictly increasing in [lo, hi), p_0 = lo
    const int nl = __popcll(__ballot(active[p] < c));   // sorted: true on lanes 0 .. nl - 1
    const int64_t p_last = __shfl(p, nl > 0 ? nl - 1 : 0, 64);
    const int64_t p_next = __shfl(p, nl < 64 ? nl : 63, 64);
    if (nl == 0) {
      hi = lo;
    } else {
      lo = p_last + 1;
      if (nl < 64) hi = p_next;
    }
  }
  const int64_t m = (hi < end ? hi + 1 : end) - lo;   // <= 64
  const int32_t v = lane < m ? active[lo + lane] : INT32_MAX;
  const int f = __popcll(__ballot(lane < m && v < c));
  const int32_t vf = __shfl(v, f < 64 ? f : 63, 64);
  // Every in-shard label is a positive, which the sampler always keeps; a
  // label not found in S is nevertheless mapped to -1 (unowned), never to a
  // position whose id is another class or lies past |S|.
  if (lane == 0) labels_mapped[n] = (f < m && vf == c) ? (int32_t)(lo + f) : -1;
}

}  // namespace

hipError_t launch_sample(const int64_t* labels, int64_t B, int64_t C, int64_t a,
                         int64_t budget, uint64_t seed, int top_bits, int64_t n_groups,
                         const SampleWs& w, int32_t* active, int64_t cap, int32_t* n_active,
                         int32_t* labels_mapped, hipStream_t stream) {
  timing_start(0, stream);
  const int64_t nwords = ceil_div(C, 32);
  const int clear_blocks = (int)(ceil_div(nwords, 256) < 4096 ? ceil_div(nwords, 256) : 4096);
  hipLaunchKernelGGL(k_sample_clear, dim3(clear_blocks > 0 ? clear_blocks : 1), dim3(256), 0,
                     stream, w.bitmap, nwords, w.hist, w.state);
  hipLaunchKernelGGL(k_mark_positives, dim3((unsigned)ceil_div(B, 256)), dim3(256), 0, stream,
                     labels, B, C, a, seed, top_bits, w.bitmap, w.hist, w.state);
  hipLaunchKernelGGL(k_sample_plan, dim3(1), dim3(64), 0, stream, w.state, budget, C);
  const int64_t n_blocks_philox = ((a + C - 1) >> 2) - (a >> 2) + 1;
  // One workgroup of 1024 threads per CU at most: each flushes a histogram.
  const int64_t hist_wgs = ceil_div(n_blocks_philox, 1024);
  hipLaunchKernelGGL(k_keys_hist, dim3((unsigned)(hist_wgs < 256 ? hist_wgs : 256)), dim3(1024), 0,
                     stream, seed, a, C, top_bits, w.digits, w.hist, w.state);
  hipLaunchKernelGGL(k_select_top, dim3(1), dim3(1024), 0, stream, w.hist, top_bits, w.state);
  hipLaunchKernelGGL(k_collect, dim3((unsigned)n_groups), dim3(kCompactThreads), 0, stream,
                     w.digits, w.bitmap, C, seed, a, w.state, w.cand_key, w.grp_sure, w.grp_tie);
  hipLaunchKernelGGL(k_refine, dim3(1), dim3(kRefineThreads), 0, stream, w.cand_key, n_groups, top_bits,
                     w.state, w.grp_sure, w.grp_tie);
  hipLaunchKernelGGL(k_compact_scan, dim3(1), dim3(1024), 0, stream, w.grp_sure, w.grp_tie,
                     n_groups, w.state, cap, w.grp_out, w.grp_tie_off, n_active);
  hipLaunchKernelGGL(k_compact_write, dim3((unsigned)n_groups), dim3(kCompactThreads), 0, stream,
                     w.digits, w.bitmap, C, seed, a, w.state, w.grp_out, w.grp_tie_off, cap,
                     active);
  hipLaunchKernelGGL(k_remap, dim3((unsigned)ceil_div(B, 4)), dim3(256), 0, stream, labels, B,
                     C, a, active, n_active, w.grp_out, n_groups, labels_mapped);
  timing_stop(0, stream);
  return hipGetLastError();
}

}  // namespace pfc
