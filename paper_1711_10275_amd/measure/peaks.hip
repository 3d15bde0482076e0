// Measured ceilings of the GPU the library runs on, for the roofline
// denominators reported beside the datasheet figures: the HBM bandwidth a
// plain streaming copy reaches, and the rate of register-only MFMA loops
// (fp32 16x16x4 and bf16 16x16x32, the two instructions the contraction
// kernels issue).  Measurement infrastructure, not part of the layer path;
// built as libsscn_measure.so.
#include <hip/hip_runtime.h>

#include <cstdint>

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

namespace {

constexpr int kChains = 4;  // independent accumulators per wavefront

__global__ __launch_bounds__(256) void k_mfma_f32(float* out, int iters) {
  f32x4 d[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) d[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float a = threadIdx.x * 1e-3f, b = 1.0f + threadIdx.x * 1e-4f;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) d[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, d[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c) s += d[c][0] + d[c][1] + d[c][2] + d[c][3];
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void k_mfma_bf16(float* out, int iters) {
  f32x4 d[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) d[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 a, b;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    a[j] = (__bf16)(threadIdx.x * 1e-3f);
    b[j] = (__bf16)1.0f;
  }
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) d[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, d[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c) s += d[c][0] + d[c][1] + d[c][2] + d[c][3];
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void k_copy(const uint4* __restrict__ a, uint4* __restrict__ b, size_t n) {
  const size_t step = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += step) b[i] = a[i];
}

template <typename F>
int time_ms(F launch, int reps, float* ms) {
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess) return 1;
  if (hipEventCreate(&e1) != hipSuccess) return 1;
  launch();  // warm-up
  if (hipDeviceSynchronize() != hipSuccess) return 1;
  hipEventRecord(e0, nullptr);
  for (int r = 0; r < reps; ++r) launch();
  hipEventRecord(e1, nullptr);
  if (hipEventSynchronize(e1) != hipSuccess) return 1;
  float t = 0.f;
  hipEventElapsedTime(&t, e0, e1);
  hipEventDestroy(e0);
  hipEventDestroy(e1);
  *ms = t / reps;
  return hipGetLastError() == hipSuccess ? 0 : 1;
}

}  // namespace

// Bandwidth of a device-to-device copy of `bytes` (read + write bytes over
// the kernel time), GB/s.  Returns 0 on success.
extern "C" int sscn_measure_copy(int64_t bytes, int reps, double* gbs) {
  const size_t n = (size_t)bytes / sizeof(uint4);
  if (n == 0 || reps < 1 || !gbs) return 1;
  uint4 *a = nullptr, *b = nullptr;
  if (hipMalloc(&a, n * sizeof(uint4)) != hipSuccess) return 1;
  if (hipMalloc(&b, n * sizeof(uint4)) != hipSuccess) {
    hipFree(a);
    return 1;
  }
  hipMemset(a, 0, n * sizeof(uint4));
  int cus = 256;
  hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0);
  float ms = 0.f;
  const int rc = time_ms([&] { k_copy<<<cus * 16, 256>>>(a, b, n); }, reps, &ms);
  hipFree(a);
  hipFree(b);
  if (rc) return rc;
  *gbs = 2.0 * (double)(n * sizeof(uint4)) / (ms * 1e-3) / 1e9;
  return 0;
}

// Rate of a register-only MFMA loop filling every CU (8 workgroups of 4
// wavefronts per CU), TFLOP/s.  kind 0: fp32 16x16x4 (2048 flops per
// instruction); kind 1: bf16 16x16x32 (16384 flops).
extern "C" int sscn_measure_mfma(int kind, int reps, double* tflops) {
  if ((kind != 0 && kind != 1) || reps < 1 || !tflops) return 1;
  int cus = 256;
  hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0);
  const int blocks = cus * 8, iters = 4096;
  float* out = nullptr;
  if (hipMalloc(&out, (size_t)blocks * 256 * sizeof(float)) != hipSuccess) return 1;
  float ms = 0.f;
  const int rc = kind == 0 ? time_ms([&] { k_mfma_f32<<<blocks, 256>>>(out, iters); }, reps, &ms)
                           : time_ms([&] { k_mfma_bf16<<<blocks, 256>>>(out, iters); }, reps, &ms);
  hipFree(out);
  if (rc) return rc;
  const double per = kind == 0 ? 2048.0 : 16384.0;
  const double flops = (double)blocks * 4 /* wavefronts */ * iters * kChains * per;
  *tflops = flops / (ms * 1e-3) / 1e12;
  return 0;
}
