// Achievable-peak probes (measurement only; not part of the method).
//
// A roofline fraction against a vendor figure says how far a kernel is from
// the datasheet; these two probes measure what this chip reaches in practice
// under the same conditions (clock under load, HBM refresh, fabric), so that
// the fractions can also be quoted against an achievable ceiling:
//
//   wam_probe_mfma_bf16  chains of independent bf16 MFMAs on register
//                        operands, several waves per SIMD: the matrix-core
//                        issue rate with no memory traffic at all;
//   wam_probe_copy       a streaming device-to-device copy (one 16-byte load and
//                        store per thread): the HBM rate of a plain kernel.
#include "wam_internal.h"

namespace wam {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kProbeThreads = 256;

// SHAPE 0: v_mfma_f32_16x16x32_bf16, eight independent accumulators of 4
// floats.  SHAPE 1: v_mfma_f32_32x32x16_bf16, four of 16 floats.  Both issue
// 131072 FLOP per wave per iteration.
template <int SHAPE>
__global__ __launch_bounds__(kProbeThreads) void probe_mfma_kernel(int iters, float* sink) {
  const int t = threadIdx.x;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = static_cast<bf16>(0.001f * (float)((t + i) & 15));
    b[i] = static_cast<bf16>(0.002f * (float)((t * 3 + i) & 7));
  }
  float s = 0.f;
  if constexpr (SHAPE == 0) {
    f32x4 acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[j], 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
  } else {
    f32x16 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) s += acc[j][r];
  }
  sink[(size_t)blockIdx.x * kProbeThreads + t] = s;
}

// One 16-byte element per thread, one pass: with every element's load in
// flight at once this form measured 6.2 TB/s on 1 GiB, where grid-stride
// loops over 1-16 Ki blocks (plain or non-temporal, 4 or 8 elements per
// iteration) stayed at 4.2-5.2 TB/s.
__global__ __launch_bounds__(kProbeThreads) void probe_copy_kernel(const f32x4* __restrict__ src,
                                                                   f32x4* __restrict__ dst, int64_t n4) {
  const int64_t i = (int64_t)blockIdx.x * kProbeThreads + threadIdx.x;
  if (i < n4) dst[i] = src[i];
}

// Times fn() (which enqueues on s) with an event pair; returns WAM_OK or WAM_E_HIP.
template <typename F>
int time_on_stream(hipStream_t s, F&& fn, double* ms_out) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
    if (e0) (void)hipEventDestroy(e0);
    return WAM_E_HIP;
  }
  int rc = WAM_OK;
  float ms = 0.f;
  if (hipEventRecord(e0, s) != hipSuccess) rc = WAM_E_HIP;
  if (rc == WAM_OK) fn();
  if (rc == WAM_OK && hipGetLastError() != hipSuccess) rc = WAM_E_HIP;
  if (rc == WAM_OK && hipEventRecord(e1, s) != hipSuccess) rc = WAM_E_HIP;
  if (rc == WAM_OK && hipEventSynchronize(e1) != hipSuccess) rc = WAM_E_HIP;
  if (rc == WAM_OK && hipEventElapsedTime(&ms, e0, e1) != hipSuccess) rc = WAM_E_HIP;
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (rc == WAM_OK) *ms_out = ms;
  return rc;
}

}  // namespace
}  // namespace wam

extern "C" {

int wam_probe_mfma_bf16(void* hip_stream, int shape, int n_blocks, int iters, float* sink, double* tflops,
                        double* ms) {
  using namespace wam;
  if ((shape != 0 && shape != 1) || n_blocks <= 0 || iters <= 0 || !sink || !tflops || !ms)
    return WAM_E_ARG;
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  auto launch = [&] {
    if (shape == 0)
      probe_mfma_kernel<0><<<n_blocks, kProbeThreads, 0, s>>>(iters, sink);
    else
      probe_mfma_kernel<1><<<n_blocks, kProbeThreads, 0, s>>>(iters, sink);
  };
  launch();  // warm-up (clocks ramp, code object loaded)
  if (hipGetLastError() != hipSuccess) return WAM_E_HIP;
  double t = 0.0;
  const int rc = time_on_stream(s, launch, &t);
  if (rc != WAM_OK) return rc;
  const double flop = (double)n_blocks * (kProbeThreads / kWave) * (double)iters * 131072.0;
  *ms = t;
  *tflops = flop / (t * 1e-3) / 1e12;
  return WAM_OK;
}

int wam_probe_copy(void* hip_stream, const void* src, void* dst, size_t bytes, int reps, double* gbs,
                   double* ms) {
  using namespace wam;
  if (!src || !dst || bytes == 0 || bytes % 16 != 0 || reps <= 0 || !gbs || !ms) return WAM_E_ARG;
  if (((uintptr_t)src | (uintptr_t)dst) % 16 != 0) return WAM_E_ARG;
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  const int64_t n4 = (int64_t)(bytes / 16);
  const int64_t nblk = (n4 + kProbeThreads - 1) / kProbeThreads;
  if (nblk > INT32_MAX) return WAM_E_ARG;
  const unsigned blocks = (unsigned)nblk;
  auto once = [&] {
    probe_copy_kernel<<<blocks, kProbeThreads, 0, s>>>(static_cast<const f32x4*>(src), static_cast<f32x4*>(dst),
                                                       n4);
  };
  once();
  if (hipGetLastError() != hipSuccess) return WAM_E_HIP;
  double t = 0.0;
  const int rc = time_on_stream(s, [&] { for (int r = 0; r < reps; ++r) once(); }, &t);
  if (rc != WAM_OK) return rc;
  *ms = t / reps;
  *gbs = 2.0 * (double)bytes / (*ms * 1e-3) / 1e9;
  return WAM_OK;
}

}  // extern "C"
