// Exact time-vs-memory frontier (the staircase without memory buckets), second stage.  The
// candidates of every group are put in (mem, obj, id) order by three stable segmented radix
// sorts (rocPRIM), least significant key first: id, then the objective's bit pattern, then the
// memory's (non-negative doubles order like their bit patterns).  In that order a candidate is
// on the frontier exactly when its objective is below the minimum of every candidate before
// it, a segmented prefix minimum: one wave per group walks its candidates in chunks of 64.
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

// key[i] = src[idx[i]] (the next sort key in the current order).
__global__ __launch_bounds__(256) void k_gather(const uint64_t* __restrict__ src, const uint32_t* __restrict__ idx,
                                                uint64_t* __restrict__ key, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) key[i] = src[idx[i]];
}

// One wave per group: candidates [seg[g], seg[g+1]) in (mem, obj, id) order.
__global__ __launch_bounds__(256) void k_front_scan(const uint32_t* __restrict__ order,
                                                    const uint64_t* __restrict__ cand_key,
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
  double carry = __builtin_huge_val();  // minimum objective of the earlier chunks
  for (int64_t c = b; c < e; c += 64) {
    const int64_t i = c + lane;
    const bool valid = i < e;
    const uint32_t k = valid ? order[i] : 0u;
    const double o = valid ? cand_obj[k] : __builtin_huge_val();
    double pm = o;  // inclusive prefix minimum over the chunk's lanes
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const double v = __shfl_up(pm, off, 64);
      if (lane >= off) pm = __builtin_fmin(pm, v);
    }
    double before = __shfl_up(pm, 1, 64);
    before = lane == 0 ? carry : __builtin_fmin(carry, before);
    const bool on = valid && o < before;
    const unsigned long long m = __builtin_amdgcn_ballot_w64(on);
    if (on) {
      const unsigned int rank =
          __builtin_amdgcn_mbcnt_hi((unsigned int)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned int)m, 0u));
      front_key[w + rank] = cand_key[k];
      front_obj[w + rank] = o;
      front_id[w + rank] = cand_id[k];
    }
    w += __builtin_popcountll(m);
    carry = __builtin_fmin(carry, __shfl(pm, 63, 64));
  }
  if (lane == 0) front_cnt[g] = w - b;
}

int last_error() {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace

int exact_sort(const uint64_t* cand_key, const double* cand_obj, const uint64_t* cand_id, uint64_t* key_tmp,
               uint64_t* key_out, uint32_t* idx_a, uint32_t* idx_b, int64_t n, int64_t n_groups, const int64_t* seg,
               void* temp, size_t* temp_bytes, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const unsigned int un = (unsigned int)n, ug = (unsigned int)n_groups;
  if (!temp) {  // storage query (the three passes sort the same number of 64-bit keys)
    const hipError_t e = rocprim::segmented_radix_sort_pairs(nullptr, *temp_bytes, key_tmp, key_out, idx_a, idx_b,
                                                             un, ug, seg, seg + 1, 0, 64, st);
    return e == hipSuccess ? 0 : (int)e;
  }
  if (n == 0) return 0;
  const dim3 grid((unsigned)((n + 255) / 256)), block(256);
  hipLaunchKernelGGL(k_iota, grid, block, 0, st, idx_a, n);
  int rc = last_error();
  // Each pass: key_tmp = the next key in the current order idx_a, stable sort into idx_b.
  const uint64_t* keys[3] = {cand_id, reinterpret_cast<const uint64_t*>(cand_obj), cand_key};
  for (int pass = 0; pass < 3 && !rc; ++pass) {
    hipLaunchKernelGGL(k_gather, grid, block, 0, st, keys[pass], idx_a, key_tmp, n);
    rc = last_error();
    if (rc) break;
    const hipError_t e = rocprim::segmented_radix_sort_pairs(temp, *temp_bytes, key_tmp, key_out, idx_a, idx_b, un,
                                                             ug, seg, seg + 1, 0, 64, st);
    if (e != hipSuccess) rc = (int)e;
    std::swap(idx_a, idx_b);
  }
  return rc;  // the final order is in the buffer passed as idx_b (three swaps)
}

int launch_front_scan(const uint32_t* order, const uint64_t* cand_key, const double* cand_obj,
                      const uint64_t* cand_id, const int64_t* seg, int64_t n_groups, uint64_t* front_key,
                      double* front_obj, uint64_t* front_id, int64_t* front_cnt, void* stream) {
  if (n_groups <= 0) return 0;
  hipLaunchKernelGGL(k_front_scan, dim3((unsigned)((n_groups + 3) / 4)), dim3(256), 0, (hipStream_t)stream, order,
                     cand_key, cand_obj, cand_id, seg, n_groups, front_key, front_obj, front_id, front_cnt);
  return last_error();
}

}  // namespace mist
