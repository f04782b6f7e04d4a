// Device side of the calibration: the co-run benchmark behind the fitted slowdown factors of
// Algorithm 1 (Sec. 5.2.2) and the operator database that replaces the efficiency formula
// (Sec. 5.2.1).  The compute stream runs rocBLAS bf16 GEMMs (the library GEMMs that training's
// linear layers run), the host streams run pinned-memory copies on the copy engines, and the
// GPU-GPU stream, which one device cannot drive over a link, runs a device-to-device copy kernel
// on a few workgroups, the footprint of a collective's kernel on the CUs and HBM.
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include <algorithm>
#include <cmath>
#include <new>
#include <string>
#include <vector>

#include "mist.h"

namespace mist {
__attribute__((visibility("hidden"))) mist_status lib_fail(mist_status code, const std::string& msg);  // sets the thread's error
}

namespace {

using mist::lib_fail;

constexpr int kCopyThreads = 256;
constexpr double kStartDelay = 0.025;   // seconds the first stream waits before the common start,
                                        // long enough for the host to enqueue every unit
constexpr uint32_t kSpinCap = 4000000;  // bound of the wait loop (each pass sleeps ~2 us)

// Pseudo-random bf16 values in [-1, 1) from a counter hash (operands of realistic magnitude, so
// that the GEMMs draw realistic power).
__global__ void k_fill_bf16(uint16_t* __restrict__ p, int64_t n, uint32_t seed) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    uint32_t x = (uint32_t)i * 0x9E3779B1u ^ seed;
    x ^= x >> 15;
    x *= 0x2C1B3C6Du;
    x ^= x >> 12;
    const float v = (float)(x >> 8) * (1.0f / 8388608.0f) - 1.0f;
    p[i] = (uint16_t)(__float_as_uint(v) >> 16);
  }
}

// The GPU-GPU stand-in: a grid-stride copy of n 16-byte words.
__global__ __launch_bounds__(kCopyThreads) void k_copy16(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                         int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * kCopyThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kCopyThreads)
    dst[i] = src[i];
}

// Holds its stream for `ticks` of the constant-rate wall clock (at most kSpinCap passes).
__global__ void k_spin(int64_t ticks) {
  const long long t0 = wall_clock64();
  for (uint32_t i = 0; i < kSpinCap; ++i) {
    if (wall_clock64() - t0 >= ticks) break;
    __builtin_amdgcn_s_sleep(64);
  }
}

mist_status hip_fail(hipError_t e, const char* what) {
  return lib_fail(MIST_E_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIP_TRY(call, what)              \
  do {                                   \
    const hipError_t e_ = (call);        \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

mist_status fill(uint16_t* p, int64_t n, uint32_t seed, hipStream_t s) {
  if (n <= 0) return MIST_OK;
  const int64_t blocks = std::min<int64_t>(4096, (n + 255) / 256);
  hipLaunchKernelGGL(k_fill_bf16, dim3((unsigned)blocks), dim3(256), 0, s, p, n, seed);
  HIP_TRY(hipGetLastError(), "fill kernel");
  return MIST_OK;
}

// D (m x n) = A^T B with A (k x m) and B (k x n), column-major bf16, fp32 accumulation.
mist_status gemm(rocblas_handle h, int64_t m, int64_t n, int64_t k, const uint16_t* A, const uint16_t* B,
                 uint16_t* D) {
  const float alpha = 1.0f, beta = 0.0f;
  const rocblas_status st = rocblas_gemm_ex(
      h, rocblas_operation_transpose, rocblas_operation_none, (rocblas_int)m, (rocblas_int)n, (rocblas_int)k, &alpha,
      A, rocblas_datatype_bf16_r, (rocblas_int)k, B, rocblas_datatype_bf16_r, (rocblas_int)k, &beta, D,
      rocblas_datatype_bf16_r, (rocblas_int)m, D, rocblas_datatype_bf16_r, (rocblas_int)m, rocblas_datatype_f32_r,
      rocblas_gemm_algo_standard, 0, 0);
  if (st != rocblas_status_success)
    return lib_fail(MIST_E_DEVICE, "rocblas_gemm_ex failed with status " + std::to_string((int)st));
  return MIST_OK;
}

bool gemm_dims_ok(int64_t m, int64_t n, int64_t k) {
  const int64_t lim = 0x7FFFFFFF;
  return m >= 1 && n >= 1 && k >= 1 && m <= lim && n <= lim && k <= lim;
}

}  // namespace

struct mist_corun {
  int device = 0;
  hipStream_t s[4] = {};
  hipEvent_t go = nullptr;
  hipEvent_t ev[4][MIST_CORUN_MAX_UNITS + 1] = {};
  rocblas_handle blas = nullptr;
  mist_corun_shape max{};
  int32_t g2g_blocks = 0;
  double clock_hz = 0.0;  // wall clock of k_spin
  uint16_t *A = nullptr, *B = nullptr, *D = nullptr;
  void *g_src = nullptr, *g_dst = nullptr, *d_h2d = nullptr, *d_d2h = nullptr;
  void *h_h2d = nullptr, *h_d2h = nullptr;  // pinned
};

namespace {

void release(mist_corun* C) {
  if (!C) return;
  int cur = 0;
  if (hipGetDevice(&cur) == hipSuccess && cur != C->device) (void)hipSetDevice(C->device);
  for (int j = 0; j < 4; ++j)
    if (C->s[j]) (void)hipStreamSynchronize(C->s[j]);
  if (C->blas) rocblas_destroy_handle(C->blas);
  for (int j = 0; j < 4; ++j)
    for (int i = 0; i <= MIST_CORUN_MAX_UNITS; ++i)
      if (C->ev[j][i]) (void)hipEventDestroy(C->ev[j][i]);
  if (C->go) (void)hipEventDestroy(C->go);
  for (void* p : {(void*)C->A, (void*)C->B, (void*)C->D, C->g_src, C->g_dst, C->d_h2d, C->d_d2h})
    if (p) (void)hipFree(p);
  if (C->h_h2d) (void)hipHostFree(C->h_h2d);
  if (C->h_d2h) (void)hipHostFree(C->h_d2h);
  for (int j = 0; j < 4; ++j)
    if (C->s[j]) (void)hipStreamDestroy(C->s[j]);
  if (cur != C->device) (void)hipSetDevice(cur);
  delete C;
}

bool shape_ok(const mist_corun_shape& s) {
  return gemm_dims_ok(s.gemm_m, s.gemm_n, s.gemm_k) && s.g2g_bytes > 0 && s.g2g_bytes % 16 == 0 &&
         s.h2d_bytes > 0 && s.d2h_bytes > 0;
}

bool shape_fits(const mist_corun_shape& s, const mist_corun_shape& max) {
  return s.gemm_m * s.gemm_k <= max.gemm_m * max.gemm_k && s.gemm_k * s.gemm_n <= max.gemm_k * max.gemm_n &&
         s.gemm_m * s.gemm_n <= max.gemm_m * max.gemm_n && s.g2g_bytes <= max.g2g_bytes &&
         s.h2d_bytes <= max.h2d_bytes && s.d2h_bytes <= max.d2h_bytes;
}

mist_status unit(mist_corun* C, int j, const mist_corun_shape& sh) {
  switch (j) {
    case 0:
      return gemm(C->blas, sh.gemm_m, sh.gemm_n, sh.gemm_k, C->A, C->B, C->D);
    case 1:
      hipLaunchKernelGGL(k_copy16, dim3((unsigned)C->g2g_blocks), dim3(kCopyThreads), 0, C->s[1],
                         (const uint4*)C->g_src, (uint4*)C->g_dst, sh.g2g_bytes / 16);
      HIP_TRY(hipGetLastError(), "copy kernel");
      return MIST_OK;
    case 2:
      HIP_TRY(hipMemcpyAsync(C->d_h2d, C->h_h2d, (size_t)sh.h2d_bytes, hipMemcpyHostToDevice, C->s[2]), "host->device copy");
      return MIST_OK;
    default:
      HIP_TRY(hipMemcpyAsync(C->h_d2h, C->d_d2h, (size_t)sh.d2h_bytes, hipMemcpyDeviceToHost, C->s[3]), "device->host copy");
      return MIST_OK;
  }
}

int popcount4(int v) { return (v & 1) + (v >> 1 & 1) + (v >> 2 & 1) + (v >> 3 & 1); }

}  // namespace

extern "C" {

mist_status mist_corun_create(const mist_corun_shape* max, int32_t g2g_blocks, mist_corun** out) {
  if (!max || !out) return lib_fail(MIST_E_INVALID, "null argument");
  *out = nullptr;
  if (!shape_ok(*max)) return lib_fail(MIST_E_INVALID, "shape fields must be positive (GEMM sizes < 2^31, GPU-GPU bytes a multiple of 16)");
  if (g2g_blocks < 1 || g2g_blocks > 1024) return lib_fail(MIST_E_INVALID, "g2g_blocks must be in 1..1024");
  mist_corun* C = new (std::nothrow) mist_corun();
  if (!C) return lib_fail(MIST_E_NOMEM, "host allocation failed");
  C->max = *max;
  C->g2g_blocks = g2g_blocks;
  auto bad = [&](mist_status st) {
    release(C);
    return st;
  };
  hipError_t e = hipGetDevice(&C->device);
  if (e != hipSuccess) return bad(hip_fail(e, "hipGetDevice"));
  int khz = 0;
  e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, C->device);
  if (e != hipSuccess || khz <= 0) return bad(e != hipSuccess ? hip_fail(e, "wall clock rate") : lib_fail(MIST_E_DEVICE, "no wall clock"));
  C->clock_hz = 1000.0 * khz;
  for (int j = 0; j < 4; ++j) {
    e = hipStreamCreateWithFlags(&C->s[j], hipStreamNonBlocking);
    if (e != hipSuccess) return bad(hip_fail(e, "hipStreamCreate"));
  }
  e = hipEventCreate(&C->go);
  if (e != hipSuccess) return bad(hip_fail(e, "hipEventCreate"));
  for (int j = 0; j < 4; ++j)
    for (int i = 0; i <= MIST_CORUN_MAX_UNITS; ++i) {
      e = hipEventCreate(&C->ev[j][i]);
      if (e != hipSuccess) return bad(hip_fail(e, "hipEventCreate"));
    }
  const size_t a = (size_t)(max->gemm_m * max->gemm_k), b = (size_t)(max->gemm_k * max->gemm_n),
               d = (size_t)(max->gemm_m * max->gemm_n);
  struct {
    void** p;
    size_t bytes;
  } dev[] = {{(void**)&C->A, a * 2}, {(void**)&C->B, b * 2}, {(void**)&C->D, d * 2}, {&C->g_src, (size_t)max->g2g_bytes},
             {&C->g_dst, (size_t)max->g2g_bytes}, {&C->d_h2d, (size_t)max->h2d_bytes}, {&C->d_d2h, (size_t)max->d2h_bytes}};
  for (auto& x : dev) {
    e = hipMalloc(x.p, x.bytes);
    if (e != hipSuccess) return bad(e == hipErrorOutOfMemory ? lib_fail(MIST_E_NOMEM, "device allocation failed") : hip_fail(e, "hipMalloc"));
  }
  e = hipHostMalloc(&C->h_h2d, (size_t)max->h2d_bytes, hipHostMallocDefault);
  if (e == hipSuccess) e = hipHostMalloc(&C->h_d2h, (size_t)max->d2h_bytes, hipHostMallocDefault);
  if (e != hipSuccess) return bad(lib_fail(MIST_E_NOMEM, std::string("pinned host allocation failed: ") + hipGetErrorString(e)));
  std::fill((char*)C->h_h2d, (char*)C->h_h2d + max->h2d_bytes, 1);
  mist_status st = fill(C->A, (int64_t)a, 1u, C->s[0]);
  if (!st) st = fill(C->B, (int64_t)b, 2u, C->s[0]);
  if (!st) st = fill((uint16_t*)C->g_src, max->g2g_bytes / 2, 3u, C->s[0]);
  if (!st) st = fill((uint16_t*)C->d_d2h, max->d2h_bytes / 2, 4u, C->s[0]);
  if (st) return bad(st);
  if (rocblas_create_handle(&C->blas) != rocblas_status_success) return bad(lib_fail(MIST_E_DEVICE, "rocblas_create_handle failed"));
  if (rocblas_set_stream(C->blas, C->s[0]) != rocblas_status_success) return bad(lib_fail(MIST_E_DEVICE, "rocblas_set_stream failed"));
  // Warm-up: the first GEMM loads its kernels, the first copies set up the copy engines.
  e = hipStreamSynchronize(C->s[0]);
  if (e != hipSuccess) return bad(hip_fail(e, "initial fill"));
  for (int j = 0; j < 4; ++j) {
    st = unit(C, j, *max);
    if (st) return bad(st);
  }
  for (int j = 0; j < 4; ++j) {
    e = hipStreamSynchronize(C->s[j]);
    if (e != hipSuccess) return bad(hip_fail(e, "warm-up"));
  }
  *out = C;
  return MIST_OK;
}

mist_status mist_corun_run(mist_corun* C, int32_t mask, const mist_corun_shape* sh, const int32_t* units, double* t,
                           int32_t stride) {
  if (!C || !sh || !units || !t) return lib_fail(MIST_E_INVALID, "null argument");
  if (mask < 1 || mask > 15) return lib_fail(MIST_E_INVALID, "mask must be in 1..15");
  if (!shape_ok(*sh) || !shape_fits(*sh, C->max)) return lib_fail(MIST_E_INVALID, "shape invalid or larger than at creation");
  for (int j = 0; j < 4; ++j)
    if ((mask >> j & 1) && (units[j] < 1 || units[j] > MIST_CORUN_MAX_UNITS || stride <= units[j]))
      return lib_fail(MIST_E_INVALID, "units must be in 1..MIST_CORUN_MAX_UNITS and below stride");
  int cur = 0;
  HIP_TRY(hipGetDevice(&cur), "hipGetDevice");
  if (cur != C->device) return lib_fail(MIST_E_INVALID, "the benchmark belongs to another device");
  // The first member holds its stream for kStartDelay, then records the common start that every
  // member waits for; meanwhile the host enqueues all units.
  int first = 0;
  while (!(mask >> first & 1)) ++first;
  hipLaunchKernelGGL(k_spin, dim3(1), dim3(64), 0, C->s[first], (int64_t)(kStartDelay * C->clock_hz));
  HIP_TRY(hipGetLastError(), "start kernel");
  HIP_TRY(hipEventRecord(C->go, C->s[first]), "hipEventRecord");
  for (int j = 0; j < 4; ++j) {
    if (!(mask >> j & 1)) continue;
    if (j != first) HIP_TRY(hipStreamWaitEvent(C->s[j], C->go, 0), "hipStreamWaitEvent");
    HIP_TRY(hipEventRecord(C->ev[j][0], C->s[j]), "hipEventRecord");
  }
  // Units are enqueued round-robin over the members so that no stream's queue runs dry early.
  int most = 0;
  for (int j = 0; j < 4; ++j)
    if (mask >> j & 1) most = std::max(most, units[j]);
  for (int i = 0; i < most; ++i)
    for (int j = 0; j < 4; ++j) {
      if (!(mask >> j & 1) || i >= units[j]) continue;
      const mist_status st = unit(C, j, *sh);
      if (st) {
        for (int q = 0; q < 4; ++q) (void)hipStreamSynchronize(C->s[q]);
        return st;
      }
      HIP_TRY(hipEventRecord(C->ev[j][i + 1], C->s[j]), "hipEventRecord");
    }
  for (int j = 0; j < 4; ++j)
    if (mask >> j & 1) HIP_TRY(hipStreamSynchronize(C->s[j]), "co-run");
  for (int j = 0; j < 4; ++j) {
    if (!(mask >> j & 1)) continue;
    for (int i = 0; i <= units[j]; ++i) {
      float ms = 0.0f;
      HIP_TRY(hipEventElapsedTime(&ms, C->go, C->ev[j][i]), "hipEventElapsedTime");
      t[(int64_t)j * stride + i] = 1e-3 * (double)ms;
    }
  }
  return MIST_OK;
}

mist_status mist_corun_measure(mist_corun* C, const mist_corun_shape* shapes, int32_t n_shapes, double target_s,
                               mist_corun_sample* out, int32_t cap, int32_t* n_out) {
  if (!C || !shapes || !n_out || n_shapes < 1) return lib_fail(MIST_E_INVALID, "bad argument");
  if (!(target_s > 0.0) || !(target_s <= 10.0)) return lib_fail(MIST_E_INVALID, "target_s must be in (0, 10]");
  const int64_t need = (int64_t)n_shapes * MIST_CORUN_SAMPLES_PER_SHAPE;
  *n_out = (int32_t)std::min<int64_t>(need, INT32_MAX);
  if (need > INT32_MAX) return lib_fail(MIST_E_INVALID, "too many shapes");
  if (!out || cap < need) return lib_fail(MIST_E_RANGE, "output capacity too small");
  const int32_t stride = MIST_CORUN_MAX_UNITS + 1;
  std::vector<double> t((size_t)4 * stride);
  double mean[4];
  int32_t count[4];
  int32_t n = 0;
  for (int32_t k = 0; k < n_shapes; ++k) {
    const mist_corun_shape& sh = shapes[k];
    int32_t U[4] = {3, 3, 3, 3};
    double solo[4];
    // Alone: a short run sizes each stream's unit count for target_s, then the measured run.
    for (int pass = 0; pass < 2; ++pass) {
      for (int j = 0; j < 4; ++j) {
        mist_status st = mist_corun_run(C, 1 << j, &sh, U, t.data(), stride);
        if (!st) st = mist_corun_reduce(1 << j, t.data(), stride, U, mean, count);
        if (st) return st;
        if (!(mean[j] > 0.0)) return lib_fail(MIST_E_STATE, "a unit took no measurable time");
        solo[j] = mean[j];
      }
      if (pass == 0)
        for (int j = 0; j < 4; ++j)
          U[j] = (int32_t)std::min<double>(MIST_CORUN_MAX_UNITS, std::max(3.0, std::ceil(target_s / solo[j])));
    }
    for (int mask = 3; mask < 16; ++mask) {
      if (popcount4(mask) < 2) continue;
      int32_t V[4] = {U[0], U[1], U[2], U[3]};
      for (int attempt = 0; attempt < 2; ++attempt) {
        if (attempt) {  // a member had no whole unit inside the window: once more, twice as long
          bool grown = false;
          for (int j = 0; j < 4; ++j) {
            const int32_t v = std::min(MIST_CORUN_MAX_UNITS, 2 * V[j]);
            grown = grown || v != V[j];
            V[j] = v;
          }
          if (!grown) break;
        }
        mist_status st = mist_corun_run(C, mask, &sh, V, t.data(), stride);
        if (!st) st = mist_corun_reduce(mask, t.data(), stride, V, mean, count);
        if (st) return st;
        bool ok = true;
        for (int j = 0; j < 4; ++j)
          if ((mask >> j & 1) && !(count[j] > 0 && mean[j] > 0.0)) ok = false;
        if (ok) break;
      }
      // A member starved for the whole window (its one unit there spans it) gets the window's
      // length: a lower bound of its co-run unit time.
      double lo = -HUGE_VAL, hi = HUGE_VAL;
      for (int j = 0; j < 4; ++j) {
        if (!(mask >> j & 1)) continue;
        lo = std::max(lo, t[(size_t)j * stride]);
        hi = std::min(hi, t[(size_t)j * stride + V[j]]);
      }
      for (int j = 0; j < 4; ++j) {
        if (!(mask >> j & 1)) continue;
        mist_corun_sample& x = out[n++];
        x.mask = mask;
        x.stream = j;
        x.shape = k;
        x.units = count[j];
        x.solo_s = solo[j];
        x.corun_s = count[j] > 0 ? mean[j] : hi - lo;
        if (!(x.corun_s > 0.0))
          return lib_fail(MIST_E_STATE, "shape " + std::to_string(k) + ", mask " + std::to_string(mask) +
                                            ": the streams never ran together");
      }
    }
  }
  *n_out = n;
  return MIST_OK;
}

mist_status mist_corun_destroy(mist_corun* C) {
  release(C);
  return MIST_OK;
}

mist_status mist_measure_eta(const mist_model_desc* m, const int32_t* mb, int32_t n_mb, int32_t tp, double peak_flops,
                             int32_t reps, double* eta, double* sec) {
  if (!m || !mb || !eta || !sec) return lib_fail(MIST_E_INVALID, "null argument");
  if (n_mb < 1 || n_mb > MIST_MAX_MB || reps < 1 || reps > 1000 || !(peak_flops > 0.0) || !std::isfinite(peak_flops))
    return lib_fail(MIST_E_INVALID, "n_mb, reps or peak_flops out of range");
  if (m->hidden < 1 || m->heads < 1 || m->kv_heads < 1 || m->ffn < 1 || m->seq < 1 || m->hidden % m->heads ||
      m->heads % m->kv_heads || (m->arch != MIST_ARCH_GPT && m->arch != MIST_ARCH_LLAMA))
    return lib_fail(MIST_E_INVALID, "invalid model");
  if (tp < 1 || m->heads % tp || m->hidden % tp || m->ffn % tp) return lib_fail(MIST_E_INVALID, "tp must divide heads, hidden and ffn");
  for (int32_t i = 0; i < n_mb; ++i)
    if (mb[i] < 1) return lib_fail(MIST_E_INVALID, "microbatch sizes must be positive");
  const int64_t h = m->hidden, f = m->ffn, dh = m->hidden / m->heads;
  const int64_t kv = m->arch == MIST_ARCH_GPT ? m->heads : m->kv_heads;
  const int64_t kv_r = tp <= kv ? kv / tp : 1;  // KV heads per rank (replicated past kv_heads)
  // (out, in) of each forward GEMM of one layer on one TP rank.
  std::vector<std::pair<int64_t, int64_t>> g = {{h / tp + 2 * kv_r * dh, h}, {h, h / tp}};
  if (m->arch == MIST_ARCH_GPT)
    g.push_back({f / tp, h});
  else
    g.push_back({2 * f / tp, h});
  g.push_back({h, f / tp});
  int64_t max_in = 0, max_out = 0, w = 0, max_tok = 0;
  for (auto& x : g) {
    max_out = std::max(max_out, x.first);
    max_in = std::max(max_in, x.second);
    w = std::max(w, x.first * x.second);
  }
  for (int32_t i = 0; i < n_mb; ++i) max_tok = std::max<int64_t>(max_tok, (int64_t)mb[i] * m->seq);
  if (!gemm_dims_ok(max_out, max_tok, max_in)) return lib_fail(MIST_E_INVALID, "GEMM sizes reach 2^31");
  uint16_t *X = nullptr, *W = nullptr, *Y = nullptr;
  hipStream_t s = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  rocblas_handle blas = nullptr;
  mist_status st = MIST_OK;
  auto cleanup = [&]() {
    if (s) (void)hipStreamSynchronize(s);
    if (blas) rocblas_destroy_handle(blas);
    for (void* p : {(void*)X, (void*)W, (void*)Y})
      if (p) (void)hipFree(p);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    if (s) (void)hipStreamDestroy(s);
  };
  hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) e = hipMalloc((void**)&X, (size_t)(max_tok * max_in) * 2);
  if (e == hipSuccess) e = hipMalloc((void**)&W, (size_t)w * 2);
  if (e == hipSuccess) e = hipMalloc((void**)&Y, (size_t)(max_tok * max_out) * 2);
  if (e != hipSuccess) {
    st = e == hipErrorOutOfMemory ? lib_fail(MIST_E_NOMEM, "device allocation failed") : hip_fail(e, "set-up");
    cleanup();
    return st;
  }
  st = fill(X, max_tok * max_in, 5u, s);
  if (!st) st = fill(W, w, 6u, s);
  if (!st && (rocblas_create_handle(&blas) != rocblas_status_success || rocblas_set_stream(blas, s) != rocblas_status_success))
    st = lib_fail(MIST_E_DEVICE, "rocBLAS handle set-up failed");
  for (int32_t i = 0; i < n_mb && !st; ++i) {
    const int64_t tok = (int64_t)mb[i] * m->seq;
    double flops = 0.0;
    for (auto& x : g) flops += 2.0 * (double)tok * (double)x.first * (double)x.second;
    std::vector<double> times;
    for (int32_t r = -1; r < reps && !st; ++r) {  // r = -1: warm-up
      e = hipEventRecord(e0, s);
      for (auto& x : g) {
        if (st || e != hipSuccess) break;
        st = gemm(blas, x.first, tok, x.second, W, X, Y);
      }
      if (!st && e == hipSuccess) e = hipEventRecord(e1, s);
      if (!st && e == hipSuccess) e = hipEventSynchronize(e1);
      float ms = 0.0f;
      if (!st && e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
      if (!st && e != hipSuccess) st = hip_fail(e, "timing");
      if (!st && r >= 0) times.push_back(1e-3 * (double)ms);
    }
    if (st) break;
    std::sort(times.begin(), times.end());
    const size_t q = times.size();
    const double med = q % 2 ? times[q / 2] : 0.5 * (times[q / 2 - 1] + times[q / 2]);
    sec[i] = med;
    eta[i] = flops / med / peak_flops;
  }
  cleanup();
  return st;
}

}  // extern "C"
