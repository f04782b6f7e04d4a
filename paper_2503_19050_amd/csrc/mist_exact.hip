// Exact time-vs-memory frontier (the staircase without memory buckets), second stage: the
// candidates of every group sorted by memory (rocPRIM's segmented radix sort on the bit
// patterns of the non-negative memory values, which order like the values), then one scan
// per group.  A group's frontier, in the definition's (mem, obj, id) order, keeps a
// configuration when its objective is strictly below every earlier one's; among equal memory
// only the run's lexicographic (obj, id) minimum can qualify.

#include <hip/hip_runtime.h>

#include <rocprim/device/device_segmented_radix_sort.hpp>

#include "mist_internal.h"

namespace mist {
namespace {

__global__ __launch_bounds__(256) void k_iota(uint32_t* __restrict__ idx, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) idx[i] = (uint32_t)i;
}

// One thread per group: candidates [seg[g], seg[g+1]) in increasing memory.
__global__ __launch_bounds__(256) void k_front_scan(const uint64_t* __restrict__ key_sorted,
                                                    const uint32_t* __restrict__ idx_sorted,
                                                    const double* __restrict__ cand_obj,
                                                    const uint64_t* __restrict__ cand_id,
                                                    const int64_t* __restrict__ seg, int64_t n_groups,
                                                    uint64_t* __restrict__ front_key, double* __restrict__ front_obj,
                                                    uint64_t* __restrict__ front_id, int64_t* __restrict__ front_cnt) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= n_groups) return;
  const int64_t b = seg[g], e = seg[g + 1];
  int64_t w = b;
  double run = __builtin_huge_val();
  for (int64_t i = b; i < e;) {
    const uint64_t key = key_sorted[i];
    double bo = __builtin_huge_val();
    uint64_t bi = ~0ull;
    int64_t j = i;
    for (; j < e && key_sorted[j] == key; ++j) {
      const uint32_t k = idx_sorted[j];
      const double o = cand_obj[k];
      const uint64_t id = cand_id[k];
      if (o < bo || (o == bo && id < bi)) {
        bo = o;
        bi = id;
      }
    }
    if (bo < run) {
      front_key[w] = key;
      front_obj[w] = bo;
      front_id[w] = bi;
      ++w;
      run = bo;
    }
    i = j;
  }
  front_cnt[g] = w - b;
}

int last_error() {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace

int exact_sort(const uint64_t* key_in, uint64_t* key_out, uint32_t* idx_in, uint32_t* idx_out, int64_t n,
               int64_t n_groups, const int64_t* seg, void* temp, size_t* temp_bytes, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  if (!temp) {  // storage query
    const hipError_t e = rocprim::segmented_radix_sort_pairs(
        nullptr, *temp_bytes, key_in, key_out, idx_in, idx_out, (unsigned int)n, (unsigned int)n_groups, seg,
        seg + 1, 0, 64, st);
    return e == hipSuccess ? 0 : (int)e;
  }
  if (n > 0) {
    hipLaunchKernelGGL(k_iota, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, idx_in, n);
    const int rc = last_error();
    if (rc) return rc;
  }
  const hipError_t e = rocprim::segmented_radix_sort_pairs(temp, *temp_bytes, key_in, key_out, idx_in, idx_out,
                                                           (unsigned int)n, (unsigned int)n_groups, seg, seg + 1,
                                                           0, 64, st);
  return e == hipSuccess ? 0 : (int)e;
}

int launch_front_scan(const uint64_t* key_sorted, const uint32_t* idx_sorted, const double* cand_obj,
                      const uint64_t* cand_id, const int64_t* seg, int64_t n_groups, uint64_t* front_key,
                      double* front_obj, uint64_t* front_id, int64_t* front_cnt, void* stream) {
  if (n_groups <= 0) return 0;
  hipLaunchKernelGGL(k_front_scan, dim3((unsigned)((n_groups + 255) / 256)), dim3(256), 0, (hipStream_t)stream,
                     key_sorted, idx_sorted, cand_obj, cand_id, seg, n_groups, front_key, front_obj, front_id,
                     front_cnt);
  return last_error();
}

}  // namespace mist
