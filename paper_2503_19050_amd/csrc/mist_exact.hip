// Exact time-vs-memory frontier (the staircase without memory buckets), second stage.  The
// candidates of every group are sorted by memory (a non-negative double orders like its bit
// pattern) by a segmented sort of this file: a block per group sorts up to kSortCap candidates
// in LDS (bitonic), and a larger group as sorted chunks merged pairwise (merge path).  In
// (mem, obj, id) order a candidate is on the frontier exactly when its objective is below that of
// every candidate before it; within a run of equal memory only the run's (obj, id) minimum can be,
// and it is when its objective is below the minima of every earlier run.  So the sort by memory
// alone suffices (the order inside a run of equal memory does not matter): one wave per group
// walks its candidates in chunks of 64, reduces each run to its minimum (a segmented scan across
// the lanes, carried over chunk boundaries) and keeps the runs that lower the running minimum.
#include <hip/hip_runtime.h>

#include <utility>

#include "mist_internal.h"

namespace mist {
namespace {

constexpr uint64_t kNoKey = ~0ull;  // no memory value has this bit pattern (it is a NaN)

// ---------------------------------------------------------------------------------------
// Segmented sort by memory key: keys [b, e) of cand_key, one block of kSortBlock threads per
// group.  Output: key_out[b..e) ascending and idx_out[b..e) = the slots the keys came from.
// ---------------------------------------------------------------------------------------
constexpr int kSortBlock = 256;
constexpr int kSortCap = 4096;  // keys sorted in LDS at once (48 KB with their slots)

// Bitonic sort of the block's LDS keys [0, N) (N a power of two, padding keys kNoKey) with
// their slots.
__device__ __forceinline__ void lds_bitonic(uint64_t* sk, uint32_t* si, int N) {
  for (int k = 2; k <= N; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = (int)threadIdx.x; i < N / 2; i += kSortBlock) {
        const int lo = ((i & ~(j - 1)) << 1) | (i & (j - 1));
        const int hi = lo + j;
        const bool asc = (lo & k) == 0;
        const uint64_t a = sk[lo], c = sk[hi];
        if ((a > c) == asc) {
          sk[lo] = c;
          sk[hi] = a;
          const uint32_t t = si[lo];
          si[lo] = si[hi];
          si[hi] = t;
        }
      }
      __syncthreads();
    }
}

// Sorts keys [b, b + n) (n <= kSortCap) in LDS and writes them with their slots at out + b.
__device__ __forceinline__ void sort_chunk(const uint64_t* __restrict__ key, int64_t b, int n, uint64_t* sk,
                                           uint32_t* si, uint64_t* __restrict__ key_out, uint32_t* __restrict__ idx_out) {
  int N = 1;
  while (N < n) N <<= 1;
  for (int i = (int)threadIdx.x; i < N; i += kSortBlock) {
    sk[i] = i < n ? key[b + i] : kNoKey;
    si[i] = (uint32_t)i;
  }
  __syncthreads();
  lds_bitonic(sk, si, N);
  for (int i = (int)threadIdx.x; i < n; i += kSortBlock) {
    key_out[b + i] = sk[i];
    idx_out[b + i] = (uint32_t)(b + si[i]);
  }
  __syncthreads();
}

// Merges the sorted runs A = [a0, a1) and B = [a1, b1) of (ks, is) into (kd, id) at a0, by the
// whole block: thread t produces its share of the output from the split of its diagonal
// (merge path: the number of A's keys among the first d outputs, ties taken from A first).
__device__ __forceinline__ void merge_runs(const uint64_t* __restrict__ ks, const uint32_t* __restrict__ is,
                                           uint64_t* __restrict__ kd, uint32_t* __restrict__ id, int64_t a0,
                                           int64_t a1, int64_t b1) {
  const int64_t na = a1 - a0, nb = b1 - a1, L = na + nb;
  const int64_t per = (L + kSortBlock - 1) / kSortBlock;
  const int64_t d0 = min((int64_t)threadIdx.x * per, L), d1 = min(d0 + per, L);
  if (d0 >= d1) return;
  // i = keys of A among the first d0 outputs: the largest i with A[i-1] <= B[d0-i].
  int64_t lo = max((int64_t)0, d0 - nb), hi = min(d0, na);
  while (lo < hi) {
    const int64_t i = (lo + hi) / 2;  // is A[i] <= B[d0-i-1]?  then more of A comes first
    if (ks[a0 + i] <= ks[a1 + d0 - i - 1]) lo = i + 1;
    else hi = i;
  }
  int64_t i = lo, j = d0 - lo;
  for (int64_t d = d0; d < d1; ++d) {
    const bool take_a = j >= nb || (i < na && ks[a0 + i] <= ks[a1 + j]);
    const int64_t src = take_a ? a0 + i : a1 + j;
    kd[a0 + d] = ks[src];
    id[a0 + d] = is[src];
    if (take_a) ++i;
    else ++j;
  }
}

__global__ __launch_bounds__(kSortBlock) void k_seg_sort(const uint64_t* __restrict__ key, const int64_t* __restrict__ seg,
                                                        const int64_t* __restrict__ seg_end, uint64_t* __restrict__ key_out,
                                                        uint32_t* __restrict__ idx_out, uint64_t* __restrict__ key_tmp,
                                                        uint32_t* __restrict__ idx_tmp) {
  __shared__ uint64_t sk[kSortCap];
  __shared__ uint32_t si[kSortCap];
  const int64_t g = blockIdx.x;
  const int64_t b = seg[g], e = seg_end[g], n = e - b;
  if (n <= 0) return;
  if (n <= kSortCap) {
    sort_chunk(key, b, (int)n, sk, si, key_out, idx_out);
    return;
  }
  // Sorted chunks of kSortCap, then pairwise merges, alternating between (key_out, idx_out)
  // and (key_tmp, idx_tmp) (both indexed by slot).
  for (int64_t c0 = 0; c0 < n; c0 += kSortCap)
    sort_chunk(key, b + c0, (int)min((int64_t)kSortCap, n - c0), sk, si, key_out, idx_out);
  uint64_t* ks = key_out;
  uint32_t* is = idx_out;
  uint64_t* kd = key_tmp;
  uint32_t* id = idx_tmp;
  for (int64_t w = kSortCap; w < n; w <<= 1) {
    for (int64_t s0 = 0; s0 < n; s0 += 2 * w) {
      const int64_t a1 = min(s0 + w, n), b1 = min(s0 + 2 * w, n);
      merge_runs(ks, is, kd, id, b + s0, b + a1, b + b1);
    }
    __syncthreads();
    uint64_t* const tk = ks;
    ks = kd;
    kd = tk;
    uint32_t* const ti = is;
    is = id;
    id = ti;
  }
  if (ks != key_out) {
    for (int64_t i = threadIdx.x; i < n; i += kSortBlock) {
      key_out[b + i] = ks[b + i];
      idx_out[b + i] = is[b + i];
    }
  }
}

__device__ __forceinline__ bool lex_less(double o1, uint64_t i1, double o2, uint64_t i2) {
  return o1 < o2 || (o1 == o2 && i1 < i2);
}

// A wave takes a group's sorted candidates 512 at a time, eight consecutive ones per lane.
constexpr int kScanItems = 8;
constexpr int kScanStep = 64 * kScanItems;

struct ScanKeys {  // a step's memory keys and candidate slots
  uint64_t key[kScanItems];
  uint32_t ord[kScanItems];
};
struct ScanVals {  // and its candidates' objectives and ids
  double obj[kScanItems];
  uint64_t id[kScanItems];
};

// The lane's items i0..i0+7 (past e: no key).
__device__ __forceinline__ void scan_keys(ScanKeys& k, const uint32_t* __restrict__ order,
                                          const uint64_t* __restrict__ sorted_key, int64_t i0, int64_t e) {
#pragma unroll
  for (int q = 0; q < kScanItems; ++q) {
    const bool valid = i0 + q < e;
    k.key[q] = valid ? sorted_key[i0 + q] : kNoKey;
    k.ord[q] = valid ? order[i0 + q] : 0u;
  }
}

__device__ __forceinline__ void scan_vals(ScanVals& v, const ScanKeys& k, const double* __restrict__ cand_obj,
                                          const uint64_t* __restrict__ cand_id, int64_t i0, int64_t e) {
#pragma unroll
  for (int q = 0; q < kScanItems; ++q) {
    const bool valid = i0 + q < e;
    v.obj[q] = valid ? cand_obj[k.ord[q]] : __builtin_huge_val();
    v.id[q] = valid ? cand_id[k.ord[q]] : kNoKey;
  }
}

// One wave per group: candidates [seg_begin[g], seg_end[g]) sorted by memory (keys in sorted_key, the
// candidates' slots in order).  Per step: each run of equal memory is reduced to its (obj, id)
// minimum by a segmented scan (within the lane over its items, then across the lanes, with the
// run that crosses into the step carried in); a run's minimum is on the frontier when its
// objective is below the minima of every earlier run (a prefix minimum over the run ends,
// within the lane, across the lanes, and over the earlier steps).  Loads run ahead of the
// scan: keys and slots two steps, objectives and ids one step.
__global__ __launch_bounds__(256) void k_front_scan(const uint32_t* __restrict__ order,
                                                    const uint64_t* __restrict__ sorted_key,
                                                    const double* __restrict__ cand_obj,
                                                    const uint64_t* __restrict__ cand_id,
                                                    const int64_t* __restrict__ seg_begin,
                                                    const int64_t* __restrict__ seg_end, int64_t n_groups,
                                                    uint64_t* __restrict__ front_key, double* __restrict__ front_obj,
                                                    uint64_t* __restrict__ front_id, int64_t* __restrict__ front_cnt) {
  const int lane = threadIdx.x & 63;
  const int64_t g = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (g >= n_groups) return;
  const int64_t b = seg_begin[g], e = seg_end[g];
  const int64_t li = (int64_t)lane * kScanItems;
  int64_t w = b;
  double carry = __builtin_huge_val();  // minimum objective of the completed runs before
  uint64_t run_key = kNoKey;            // a run continuing from the previous step: its memory
  double run_obj = __builtin_huge_val();  // and its minimum so far
  uint64_t run_id = kNoKey;
  ScanKeys k0, k1;
  ScanVals v0;
  if (b < e) {
    scan_keys(k0, order, sorted_key, b + li, e);
    scan_vals(v0, k0, cand_obj, cand_id, b + li, e);
    if (b + kScanStep < e) scan_keys(k1, order, sorted_key, b + kScanStep + li, e);
  }
  for (int64_t c = b; c < e; c += kScanStep) {
    const bool more = c + kScanStep < e;
    ScanVals v1;
    ScanKeys k2;
    if (more) scan_vals(v1, k1, cand_obj, cand_id, c + kScanStep + li, e);
    if (c + 2 * kScanStep < e) scan_keys(k2, order, sorted_key, c + 2 * kScanStep + li, e);
    const int64_t i0 = c + li;

    // Runs: an item starts one when its memory differs from the item before it (for lane 0's
    // first item: from the run carried in); it ends one when the item after it differs.
    const uint64_t before_key = __shfl_up(k0.key[kScanItems - 1], 1, 64);
    const uint64_t after_key = __shfl_down(k0.key[0], 1, 64);
    const uint64_t next_step_key = more ? __shfl(k1.key[0], 0, 64) : kNoKey;
    bool st[kScanItems], en[kScanItems];
    double o[kScanItems];
    uint64_t id[kScanItems];
#pragma unroll
    for (int q = 0; q < kScanItems; ++q) {
      const bool valid = i0 + q < e;
      const uint64_t prev = q > 0 ? k0.key[q - 1] : (lane == 0 ? run_key : before_key);
      const uint64_t next = q + 1 < kScanItems ? k0.key[q + 1] : (lane == 63 ? next_step_key : after_key);
      st[q] = valid && k0.key[q] != prev;
      en[q] = valid && k0.key[q] != next;
      o[q] = v0.obj[q];
      id[q] = v0.id[q];
    }
    if (lane == 0 && i0 < e && !st[0] && lex_less(run_obj, run_id, o[0], id[0])) {
      o[0] = run_obj;  // the carried run goes on
      id[0] = run_id;
    }
    // Within the lane: each item's run minimum from the run's start (or from the lane's first
    // item).
    bool any_start = st[0];
#pragma unroll
    for (int q = 1; q < kScanItems; ++q) {
      if (!st[q] && lex_less(o[q - 1], id[q - 1], o[q], id[q])) {
        o[q] = o[q - 1];
        id[q] = id[q - 1];
      }
      any_start = any_start || st[q];
    }
    // Across the lanes: segmented inclusive scan of (a run starts in the lane, the lane's last
    // minimum), then the exclusive value from the lane before.
    bool sf = any_start;
    double so = o[kScanItems - 1];
    uint64_t si = id[kScanItems - 1];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int pf = __shfl_up((int)sf, off, 64);
      const double po = __shfl_up(so, off, 64);
      const uint64_t pi = __shfl_up(si, off, 64);
      if (lane >= off) {
        if (!sf && lex_less(po, pi, so, si)) {
          so = po;
          si = pi;
        }
        sf = sf || pf != 0;
      }
    }
    double in_o = __shfl_up(so, 1, 64);
    uint64_t in_i = __shfl_up(si, 1, 64);
    if (lane == 0) {
      in_o = __builtin_huge_val();
      in_i = kNoKey;
    }
    // Items before the lane's first start continue the run coming from the lanes before.
    bool open = true;
#pragma unroll
    for (int q = 0; q < kScanItems; ++q) {
      open = open && !st[q];
      if (open && lex_less(in_o, in_i, o[q], id[q])) {
        o[q] = in_o;
        id[q] = in_i;
      }
    }
    // Prefix minimum over the run ends: within the lane, then across the lanes and steps.
    double lp[kScanItems];
#pragma unroll
    for (int q = 0; q < kScanItems; ++q) {
      const double v = en[q] ? o[q] : __builtin_huge_val();
      lp[q] = q > 0 ? __builtin_fmin(lp[q - 1], v) : v;
    }
    double pm = lp[kScanItems - 1];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const double v = __shfl_up(pm, off, 64);
      if (lane >= off) pm = __builtin_fmin(pm, v);
    }
    double lane_before = __shfl_up(pm, 1, 64);
    lane_before = lane == 0 ? carry : __builtin_fmin(carry, lane_before);
    bool on[kScanItems];
    unsigned int below = 0;  // frontier items of the lanes before this one
    unsigned int total = 0;
#pragma unroll
    for (int q = 0; q < kScanItems; ++q) {
      const double before = q > 0 ? __builtin_fmin(lane_before, lp[q - 1]) : lane_before;
      on[q] = en[q] && o[q] < before;
      const unsigned long long m = __builtin_amdgcn_ballot_w64(on[q]);
      below += __builtin_amdgcn_mbcnt_hi((unsigned int)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned int)m, 0u));
      total += (unsigned int)__builtin_popcountll(m);
    }
    int64_t slot = w + below;
#pragma unroll
    for (int q = 0; q < kScanItems; ++q) {
      if (on[q]) {
        front_key[slot] = k0.key[q];
        front_obj[slot] = o[q];
        front_id[slot] = id[q];
        ++slot;
      }
    }
    w += total;
    carry = __builtin_fmin(carry, __shfl(pm, 63, 64));
    // The step's last run goes on into the next step unless it ended here.
    const bool last_open = __shfl((int)!en[kScanItems - 1], 63, 64) != 0;
    run_key = last_open ? __shfl(k0.key[kScanItems - 1], 63, 64) : kNoKey;
    run_obj = __shfl(o[kScanItems - 1], 63, 64);
    run_id = __shfl(id[kScanItems - 1], 63, 64);
    if (more) {
      k0 = k1;
      v0 = v1;
      k1 = k2;
    }
  }
  if (lane == 0) front_cnt[g] = w - b;
}

// Exact pre-filter, one block per group: a candidate with at least as large an objective as a
// candidate of strictly smaller memory is not on the frontier.  The group's memory range is cut
// into kSub sub-ranges by a monotone map, so every candidate of a lower sub-range has strictly
// smaller memory; the candidates whose objective is not below the minimum of all lower
// sub-ranges are dropped, and the others are moved to the front of the group's slots in
// order.  seg_end[g] receives the end of the survivors.
constexpr int kSub = 4096;

__device__ __forceinline__ int sub_range(uint64_t key, double lo, double kap) {
  const double m = __longlong_as_double((long long)key);
  return min((int)((m - lo) * kap), kSub - 1);
}

__global__ __launch_bounds__(256) void k_prefilter(uint64_t* __restrict__ key, double* __restrict__ obj,
                                                   uint64_t* __restrict__ id, const int64_t* __restrict__ seg,
                                                   int64_t* __restrict__ seg_end) {
  constexpr int kPf = 4;               // items per thread and step: four loads in flight
  constexpr int kPfStep = 256 * kPf;
  __shared__ unsigned long long s_min[kSub];
  __shared__ double s_lo[4], s_hi[4], s_wmin[4];
  __shared__ int s_cnt[4][kPf];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t g = blockIdx.x;
  const int64_t b = seg[g], e = seg[g + 1];
  if (b == e) {
    if (tid == 0) seg_end[g] = e;
    return;
  }
  // The group's memory range.
  double lo = __builtin_huge_val(), hi = 0.0;
  for (int64_t c = b; c < e; c += kPfStep) {
    uint64_t k[kPf];
#pragma unroll
    for (int q = 0; q < kPf; ++q) {
      const int64_t i = c + q * 256 + tid;
      k[q] = i < e ? key[i] : kNoKey;
    }
#pragma unroll
    for (int q = 0; q < kPf; ++q) {
      if (k[q] == kNoKey) continue;
      const double m = __longlong_as_double((long long)k[q]);
      lo = __builtin_fmin(lo, m);
      hi = __builtin_fmax(hi, m);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    lo = __builtin_fmin(lo, __shfl_xor(lo, off, 64));
    hi = __builtin_fmax(hi, __shfl_xor(hi, off, 64));
  }
  if (lane == 0) {
    s_lo[wave] = lo;
    s_hi[wave] = hi;
  }
  for (int j = tid; j < kSub; j += 256) s_min[j] = kNoKey;
  __syncthreads();
  lo = __builtin_fmin(__builtin_fmin(s_lo[0], s_lo[1]), __builtin_fmin(s_lo[2], s_lo[3]));
  hi = __builtin_fmax(__builtin_fmax(s_hi[0], s_hi[1]), __builtin_fmax(s_hi[2], s_hi[3]));
  const double kap = hi > lo ? (double)kSub / (hi - lo) : 0.0;
  // Minimum objective per sub-range (a non-negative double orders like its bits).
  for (int64_t c = b; c < e; c += kPfStep) {
    uint64_t k[kPf], o[kPf];
#pragma unroll
    for (int q = 0; q < kPf; ++q) {
      const int64_t i = c + q * 256 + tid;
      k[q] = i < e ? key[i] : kNoKey;
      o[q] = i < e ? (unsigned long long)__double_as_longlong(obj[i]) : 0ull;
    }
#pragma unroll
    for (int q = 0; q < kPf; ++q)
      if (k[q] != kNoKey) atomicMin(&s_min[sub_range(k[q], lo, kap)], o[q]);
  }
  __syncthreads();
  // Exclusive prefix minimum over the sub-ranges: thread t holds sub-ranges [16t, 16t + 16).
  constexpr int kPer = kSub / 256;
  double run = __builtin_huge_val();
  double own[kPer];
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const unsigned long long v = s_min[tid * kPer + q];
    own[q] = v == kNoKey ? __builtin_huge_val() : __longlong_as_double((long long)v);
    run = __builtin_fmin(run, own[q]);
  }
  double incl = run;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double v = __shfl_up(incl, off, 64);
    if (lane >= off) incl = __builtin_fmin(incl, v);
  }
  if (lane == 63) s_wmin[wave] = incl;
  __syncthreads();
  double before = __shfl_up(incl, 1, 64);
  if (lane == 0) before = __builtin_huge_val();
  for (int w = 0; w < wave; ++w) before = __builtin_fmin(before, s_wmin[w]);
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    s_min[tid * kPer + q] = (unsigned long long)__double_as_longlong(before);
    before = __builtin_fmin(before, own[q]);
  }
  __syncthreads();
  // Keep the candidates below every lower sub-range's minimum, in order, at the front.  A
  // step's writes land below its own start, after every thread of the block read the step.
  int64_t wp = b;
  for (int64_t c = b; c < e; c += kPfStep) {
    uint64_t k[kPf], d[kPf];
    double o[kPf];
    bool keep[kPf];
#pragma unroll
    for (int q = 0; q < kPf; ++q) {
      const int64_t i = c + q * 256 + tid;
      const bool valid = i < e;
      k[q] = valid ? key[i] : 0ull;
      o[q] = valid ? obj[i] : 0.0;
      d[q] = valid ? id[i] : 0ull;
      keep[q] = valid && o[q] < __longlong_as_double((long long)s_min[sub_range(k[q], lo, kap)]);
    }
    unsigned long long m[kPf];
#pragma unroll
    for (int q = 0; q < kPf; ++q) {
      m[q] = __builtin_amdgcn_ballot_w64(keep[q]);
      if (lane == 0) s_cnt[wave][q] = __builtin_popcountll(m[q]);
    }
    __syncthreads();
    // Item (q, tid) follows every item of the steps' earlier rows q' < q, then the earlier
    // waves' items of row q, then the earlier lanes of its wave.
    int base = 0, total = 0;
#pragma unroll
    for (int q = 0; q < kPf; ++q) {
      const int row = s_cnt[0][q] + s_cnt[1][q] + s_cnt[2][q] + s_cnt[3][q];
      if (keep[q]) {
        int rank = base + __builtin_amdgcn_mbcnt_hi((unsigned int)(m[q] >> 32),
                                                    __builtin_amdgcn_mbcnt_lo((unsigned int)m[q], 0u));
        for (int w = 0; w < wave; ++w) rank += s_cnt[w][q];
        key[wp + rank] = k[q];
        obj[wp + rank] = o[q];
        id[wp + rank] = d[q];
      }
      base += row;
      total += row;
    }
    wp += total;
    __syncthreads();
  }
  if (tid == 0) seg_end[g] = wp;
}

// One wave per tile: its window's candidates (its first ones, in order) to the tile's place in
// group order; the rest of an overflowing tile comes from the pool.
__global__ __launch_bounds__(256) void k_compact(const uint64_t* __restrict__ slab_key,
                                                 const double* __restrict__ slab_obj,
                                                 const uint64_t* __restrict__ slab_id,
                                                 const int64_t* __restrict__ slab_begin,
                                                 const int32_t* __restrict__ cnt,
                                                 const uint8_t* __restrict__ tile_drop,
                                                 const int64_t* __restrict__ tile_off, int32_t n_tiles,
                                                 uint64_t* __restrict__ cand_key, double* __restrict__ cand_obj,
                                                 uint64_t* __restrict__ cand_id) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_tiles) return;
  if (tile_drop[t]) return;  // a candidate found no place: the tile is evaluated again
  const int64_t src = slab_begin[t], dst = tile_off[t];
  const int64_t win = slab_begin[t + 1] - src;
  const int64_t n = cnt[t] < win ? (int64_t)cnt[t] : win;
  for (int64_t i = lane; i < n; i += 64) {
    cand_key[dst + i] = slab_key[src + i];
    cand_obj[dst + i] = slab_obj[src + i];
    cand_id[dst + i] = slab_id[src + i];
  }
}

// One thread per pool slot: the overflowing candidate to its tile's place plus its rank (slots
// that a wave's chunk left unused hold tile -1).
__global__ __launch_bounds__(256) void k_pool_place(const uint64_t* __restrict__ pool_key,
                                                    const double* __restrict__ pool_obj,
                                                    const uint64_t* __restrict__ pool_id,
                                                    const int32_t* __restrict__ pool_tile,
                                                    const int32_t* __restrict__ pool_rank, int64_t n,
                                                    const uint8_t* __restrict__ tile_drop,
                                                    const int64_t* __restrict__ tile_off,
                                                    uint64_t* __restrict__ cand_key, double* __restrict__ cand_obj,
                                                    uint64_t* __restrict__ cand_id) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  const int32_t t = pool_tile[p];
  if (t < 0 || tile_drop[t]) return;  // an unused slot of a chunk, or a tile evaluated again
  const int64_t dst = tile_off[t] + pool_rank[p];
  cand_key[dst] = pool_key[p];
  cand_obj[dst] = pool_obj[p];
  cand_id[dst] = pool_id[p];
}

int last_error() {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace

int exact_sort(const uint64_t* cand_key, uint64_t* key_out, uint32_t* idx_out, uint64_t* key_tmp, uint32_t* idx_tmp,
               int64_t n_groups, const int64_t* seg_begin, const int64_t* seg_end, void* stream) {
  if (n_groups <= 0) return 0;
  hipLaunchKernelGGL(k_seg_sort, dim3((unsigned)n_groups), dim3(kSortBlock), 0, (hipStream_t)stream, cand_key,
                     seg_begin, seg_end, key_out, idx_out, key_tmp, idx_tmp);
  return last_error();
}

int launch_compact(const uint64_t* slab_key, const double* slab_obj, const uint64_t* slab_id,
                   const int64_t* slab_begin, const int32_t* cnt, const uint8_t* tile_drop, const int64_t* tile_off,
                   int32_t n_tiles, uint64_t* cand_key, double* cand_obj, uint64_t* cand_id, void* stream) {
  if (n_tiles <= 0) return 0;
  hipLaunchKernelGGL(k_compact, dim3((unsigned)((n_tiles + 3) / 4)), dim3(256), 0, (hipStream_t)stream, slab_key,
                     slab_obj, slab_id, slab_begin, cnt, tile_drop, tile_off, n_tiles, cand_key, cand_obj, cand_id);
  return last_error();
}

int launch_pool_place(const uint64_t* pool_key, const double* pool_obj, const uint64_t* pool_id,
                      const int32_t* pool_tile, const int32_t* pool_rank, int64_t n, const uint8_t* tile_drop,
                      const int64_t* tile_off, uint64_t* cand_key, double* cand_obj, uint64_t* cand_id,
                      void* stream) {
  if (n <= 0) return 0;
  hipLaunchKernelGGL(k_pool_place, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, (hipStream_t)stream, pool_key,
                     pool_obj, pool_id, pool_tile, pool_rank, n, tile_drop, tile_off, cand_key, cand_obj, cand_id);
  return last_error();
}

int launch_prefilter(uint64_t* cand_key, double* cand_obj, uint64_t* cand_id, const int64_t* seg,
                     int64_t n_groups, int64_t* seg_end, void* stream) {
  if (n_groups <= 0) return 0;
  hipLaunchKernelGGL(k_prefilter, dim3((unsigned)n_groups), dim3(256), 0, (hipStream_t)stream, cand_key, cand_obj,
                     cand_id, seg, seg_end);
  return last_error();
}

int launch_front_scan(const uint32_t* order, const uint64_t* sorted_key, const double* cand_obj,
                      const uint64_t* cand_id, const int64_t* seg_begin, const int64_t* seg_end, int64_t n_groups,
                      uint64_t* front_key, double* front_obj, uint64_t* front_id, int64_t* front_cnt, void* stream) {
  if (n_groups <= 0) return 0;
  hipLaunchKernelGGL(k_front_scan, dim3((unsigned)((n_groups + 3) / 4)), dim3(256), 0, (hipStream_t)stream, order,
                     sorted_key, cand_obj, cand_id, seg_begin, seg_end, n_groups, front_key, front_obj, front_id,
                     front_cnt);
  return last_error();
}

}  // namespace mist
