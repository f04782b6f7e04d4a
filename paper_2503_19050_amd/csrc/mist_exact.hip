// Exact time-vs-memory frontier (the staircase without memory buckets), second stage.  The
// candidates of every group are sorted by memory with one segmented radix sort (rocPRIM; a
// non-negative double orders like its bit pattern).  In (mem, obj, id) order a candidate is on the
// frontier exactly when its objective is below that of every candidate before it; within a run of
// equal memory only the run's (obj, id) minimum can be, and it is when its objective is below the
// minima of every earlier run.  So the sort by memory alone suffices: one wave per group walks
// its candidates in chunks of 64, reduces each run to its minimum (a segmented scan across the
// lanes, carried over chunk boundaries) and keeps the runs that lower the running minimum.
#include <hip/hip_runtime.h>

#include <rocprim/device/device_segmented_radix_sort.hpp>

#include <utility>

#include "mist_internal.h"

namespace mist {
namespace {

__global__ __launch_bounds__(256) void k_iota(uint32_t* __restrict__ idx, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) idx[i] = (uint32_t)i;
}

constexpr uint64_t kNoKey = ~0ull;  // no memory value has this bit pattern (it is a NaN)

__device__ __forceinline__ bool lex_less(double o1, uint64_t i1, double o2, uint64_t i2) {
  return o1 < o2 || (o1 == o2 && i1 < i2);
}

// One wave per group: candidates [seg[g], seg[g+1]) sorted by memory (keys in sorted_key, the
// candidates' slots in order).
__global__ __launch_bounds__(256) void k_front_scan(const uint32_t* __restrict__ order,
                                                    const uint64_t* __restrict__ sorted_key,
                                                    const double* __restrict__ cand_obj,
                                                    const uint64_t* __restrict__ cand_id,
                                                    const int64_t* __restrict__ seg, int64_t n_groups,
                                                    uint64_t* __restrict__ front_key, double* __restrict__ front_obj,
                                                    uint64_t* __restrict__ front_id, int64_t* __restrict__ front_cnt) {
  const int lane = threadIdx.x & 63;
  const int64_t g = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (g >= n_groups) return;
  const int64_t b = seg[g], e = seg[g + 1];
  int64_t w = b;
  double carry = __builtin_huge_val();  // minimum objective of the completed runs before
  uint64_t run_key = kNoKey;            // a run continuing from the previous chunk: its memory
  double run_obj = __builtin_huge_val();  // and its minimum so far
  uint64_t run_id = kNoKey;
  for (int64_t c = b; c < e; c += 64) {
    const int64_t i = c + lane;
    const bool valid = i < e;
    const uint32_t k = valid ? order[i] : 0u;
    const uint64_t key = valid ? sorted_key[i] : kNoKey;
    const uint64_t next = i + 1 < e ? sorted_key[i + 1] : kNoKey;
    double o = valid ? cand_obj[k] : __builtin_huge_val();
    uint64_t id = valid ? cand_id[k] : kNoKey;
    uint64_t prev = __shfl_up(key, 1, 64);
    if (lane == 0) prev = run_key;
    const bool start = valid && key != prev;
    if (lane == 0 && valid && !start && lex_less(run_obj, run_id, o, id)) {
      o = run_obj;
      id = run_id;
    }
    // First lane of this lane's run in the chunk (0 for the run carried in), then the run's
    // (obj, id) minimum up to this lane.
    int head = start ? lane : 0;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int h = __shfl_up(head, off, 64);
      if (lane >= off) head = max(head, h);
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const double vo = __shfl_up(o, off, 64);
      const uint64_t vi = __shfl_up(id, off, 64);
      if (lane - off >= head && lex_less(vo, vi, o, id)) {
        o = vo;
        id = vi;
      }
    }
    const bool end = valid && next != key;  // last candidate of its run: (o, id) is the run's minimum
    double pm = end ? o : __builtin_huge_val();  // inclusive prefix minimum over the run ends
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const double v = __shfl_up(pm, off, 64);
      if (lane >= off) pm = __builtin_fmin(pm, v);
    }
    double before = __shfl_up(pm, 1, 64);
    before = lane == 0 ? carry : __builtin_fmin(carry, before);
    const bool on = end && o < before;
    const unsigned long long m = __builtin_amdgcn_ballot_w64(on);
    if (on) {
      const unsigned int rank =
          __builtin_amdgcn_mbcnt_hi((unsigned int)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned int)m, 0u));
      front_key[w + rank] = key;
      front_obj[w + rank] = o;
      front_id[w + rank] = id;
    }
    w += __builtin_popcountll(m);
    carry = __builtin_fmin(carry, __shfl(pm, 63, 64));
    // The last lane's run goes on into the next chunk unless it ended here.
    const bool open = __shfl((int)(valid && !end), 63, 64) != 0;
    run_key = open ? __shfl(key, 63, 64) : kNoKey;
    run_obj = __shfl(o, 63, 64);
    run_id = __shfl(id, 63, 64);
  }
  if (lane == 0) front_cnt[g] = w - b;
}

// One wave per tile: its window's candidates, in order, to the tile's place in group order.
__global__ __launch_bounds__(256) void k_compact(const uint64_t* __restrict__ slab_key,
                                                 const double* __restrict__ slab_obj,
                                                 const uint64_t* __restrict__ slab_id,
                                                 const int64_t* __restrict__ slab_begin,
                                                 const int32_t* __restrict__ cnt,
                                                 const int64_t* __restrict__ tile_off, int32_t n_tiles,
                                                 uint64_t* __restrict__ cand_key, double* __restrict__ cand_obj,
                                                 uint64_t* __restrict__ cand_id) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_tiles) return;
  const int64_t src = slab_begin[t], n = cnt[t], dst = tile_off[t];
  if (n > slab_begin[t + 1] - src) return;  // overflowed: the tile is evaluated again
  for (int64_t i = lane; i < n; i += 64) {
    cand_key[dst + i] = slab_key[src + i];
    cand_obj[dst + i] = slab_obj[src + i];
    cand_id[dst + i] = slab_id[src + i];
  }
}

int last_error() {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace

int exact_sort(const uint64_t* cand_key, uint64_t* key_out, uint32_t* idx_in, uint32_t* idx_out, int64_t n,
               int64_t n_groups, const int64_t* seg, void* temp, size_t* temp_bytes, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const unsigned int un = (unsigned int)n, ug = (unsigned int)n_groups;
  if (!temp) {  // storage query
    const hipError_t e = rocprim::segmented_radix_sort_pairs(nullptr, *temp_bytes, cand_key, key_out, idx_in,
                                                             idx_out, un, ug, seg, seg + 1, 0, 64, st);
    return e == hipSuccess ? 0 : (int)e;
  }
  if (n == 0) return 0;
  hipLaunchKernelGGL(k_iota, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, idx_in, n);
  int rc = last_error();
  if (!rc) {
    const hipError_t e = rocprim::segmented_radix_sort_pairs(temp, *temp_bytes, cand_key, key_out, idx_in, idx_out,
                                                             un, ug, seg, seg + 1, 0, 64, st);
    if (e != hipSuccess) rc = (int)e;
  }
  return rc;
}

int launch_compact(const uint64_t* slab_key, const double* slab_obj, const uint64_t* slab_id,
                   const int64_t* slab_begin, const int32_t* cnt, const int64_t* tile_off, int32_t n_tiles,
                   uint64_t* cand_key, double* cand_obj, uint64_t* cand_id, void* stream) {
  if (n_tiles <= 0) return 0;
  hipLaunchKernelGGL(k_compact, dim3((unsigned)((n_tiles + 3) / 4)), dim3(256), 0, (hipStream_t)stream, slab_key,
                     slab_obj, slab_id, slab_begin, cnt, tile_off, n_tiles, cand_key, cand_obj, cand_id);
  return last_error();
}

int launch_front_scan(const uint32_t* order, const uint64_t* sorted_key, const double* cand_obj,
                      const uint64_t* cand_id, const int64_t* seg, int64_t n_groups, uint64_t* front_key,
                      double* front_obj, uint64_t* front_id, int64_t* front_cnt, void* stream) {
  if (n_groups <= 0) return 0;
  hipLaunchKernelGGL(k_front_scan, dim3((unsigned)((n_groups + 3) / 4)), dim3(256), 0, (hipStream_t)stream, order,
                     sorted_key, cand_obj, cand_id, seg, n_groups, front_key, front_obj, front_id, front_cnt);
  return last_error();
}

}  // namespace mist
