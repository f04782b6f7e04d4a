// FP64 instruction-mix probe.  Each kernel issues a known number of one FP64 VALU instruction
// (add, mul, fma, min, max or compare) and nothing else of FP64 type, so that the profiler's
// per-type FP64 instruction counters can be read against a known count: which counter (if any)
// a v_min_f64, v_max_f64 or v_cmp_*_f64 lands in decides how an instruction-counter FLOP figure
// of the evaluation kernel is to be read.  Measurement support only; not on the tuner's path.

#include <hip/hip_runtime.h>

#include <string>

#include "mist.h"

namespace mist {
__attribute__((visibility("hidden"))) mist_status lib_fail(mist_status code, const std::string& msg);  // sets the thread's error
}

namespace {

constexpr int kProbeBlock = 256;
constexpr int kPerRep = 8;  // instructions of the probed kind per repetition

// One repetition: eight dependent instructions of the kind on x with operand y (the asm keeps
// the compiler from folding, reordering or fusing them).
template <int KIND>
__device__ __forceinline__ void rep(double& x, double y, unsigned long long& acc) {
  if constexpr (KIND == MIST_PROBE_ADD) {
    asm volatile(
        "v_add_f64 %0, %0, %1\n v_add_f64 %0, %0, %1\n v_add_f64 %0, %0, %1\n v_add_f64 %0, %0, %1\n"
        "v_add_f64 %0, %0, %1\n v_add_f64 %0, %0, %1\n v_add_f64 %0, %0, %1\n v_add_f64 %0, %0, %1"
        : "+v"(x) : "v"(y));
  } else if constexpr (KIND == MIST_PROBE_MUL) {
    asm volatile(
        "v_mul_f64 %0, %0, %1\n v_mul_f64 %0, %0, %1\n v_mul_f64 %0, %0, %1\n v_mul_f64 %0, %0, %1\n"
        "v_mul_f64 %0, %0, %1\n v_mul_f64 %0, %0, %1\n v_mul_f64 %0, %0, %1\n v_mul_f64 %0, %0, %1"
        : "+v"(x) : "v"(y));
  } else if constexpr (KIND == MIST_PROBE_FMA) {
    asm volatile(
        "v_fma_f64 %0, %0, %1, %1\n v_fma_f64 %0, %0, %1, %1\n v_fma_f64 %0, %0, %1, %1\n"
        "v_fma_f64 %0, %0, %1, %1\n v_fma_f64 %0, %0, %1, %1\n v_fma_f64 %0, %0, %1, %1\n"
        "v_fma_f64 %0, %0, %1, %1\n v_fma_f64 %0, %0, %1, %1"
        : "+v"(x) : "v"(y));
  } else if constexpr (KIND == MIST_PROBE_MIN) {
    asm volatile(
        "v_min_f64 %0, %0, %1\n v_min_f64 %0, %0, %1\n v_min_f64 %0, %0, %1\n v_min_f64 %0, %0, %1\n"
        "v_min_f64 %0, %0, %1\n v_min_f64 %0, %0, %1\n v_min_f64 %0, %0, %1\n v_min_f64 %0, %0, %1"
        : "+v"(x) : "v"(y));
  } else if constexpr (KIND == MIST_PROBE_MAX) {
    asm volatile(
        "v_max_f64 %0, %0, %1\n v_max_f64 %0, %0, %1\n v_max_f64 %0, %0, %1\n v_max_f64 %0, %0, %1\n"
        "v_max_f64 %0, %0, %1\n v_max_f64 %0, %0, %1\n v_max_f64 %0, %0, %1\n v_max_f64 %0, %0, %1"
        : "+v"(x) : "v"(y));
  } else {  // compare: a lane mask per instruction, folded into the accumulator by the SALU
    unsigned long long m[kPerRep];
#pragma unroll
    for (int k = 0; k < kPerRep; ++k) {
      asm volatile("v_cmp_lt_f64_e64 %0, %1, %2" : "=s"(m[k]) : "v"(x), "v"(y));
      acc ^= m[k] + (unsigned long long)k;
    }
  }
}

template <int KIND>
__global__ __launch_bounds__(kProbeBlock) void k_probe(const double* __restrict__ in, unsigned long long* __restrict__ out,
                                                       int reps) {
  const size_t i = (size_t)blockIdx.x * kProbeBlock + threadIdx.x;
  double x = in[2 * i];
  const double y = in[2 * i + 1];
  unsigned long long acc = 0;
  for (int r = 0; r < reps; ++r) rep<KIND>(x, y, acc);
  out[i] = (unsigned long long)__double_as_longlong(x) ^ acc;
}

}  // namespace

extern "C" mist_status mist_probe_fp64(int32_t kind, const double* in, uint64_t* out, int64_t n_threads, int32_t reps,
                                       uint64_t* n_instructions, void* stream) {
  if (!in || !out || n_threads <= 0 || n_threads % kProbeBlock || n_threads / kProbeBlock > INT32_MAX || reps < 1)
    return mist::lib_fail(MIST_E_INVALID, "probe: null buffer, reps < 1, or n_threads not a positive multiple of 256");
  const dim3 grid((unsigned)(n_threads / kProbeBlock)), block(kProbeBlock);
  hipStream_t st = (hipStream_t)stream;
  unsigned long long* o = (unsigned long long*)out;
  switch (kind) {
    case MIST_PROBE_ADD: hipLaunchKernelGGL(k_probe<MIST_PROBE_ADD>, grid, block, 0, st, in, o, reps); break;
    case MIST_PROBE_MUL: hipLaunchKernelGGL(k_probe<MIST_PROBE_MUL>, grid, block, 0, st, in, o, reps); break;
    case MIST_PROBE_FMA: hipLaunchKernelGGL(k_probe<MIST_PROBE_FMA>, grid, block, 0, st, in, o, reps); break;
    case MIST_PROBE_MIN: hipLaunchKernelGGL(k_probe<MIST_PROBE_MIN>, grid, block, 0, st, in, o, reps); break;
    case MIST_PROBE_MAX: hipLaunchKernelGGL(k_probe<MIST_PROBE_MAX>, grid, block, 0, st, in, o, reps); break;
    case MIST_PROBE_CMP: hipLaunchKernelGGL(k_probe<MIST_PROBE_CMP>, grid, block, 0, st, in, o, reps); break;
    default: return mist::lib_fail(MIST_E_INVALID, "probe: unknown kind");
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return mist::lib_fail(MIST_E_DEVICE, std::string("probe launch: ") + hipGetErrorString(e));
  if (n_instructions) *n_instructions = (uint64_t)(n_threads / 64) * (uint64_t)reps * kPerRep;
  return MIST_OK;
}
