// Row-wise operations on the active sites only (Sec. 4.1 "Other operators"):
// batch normalisation in inference form + ReLU, and the column concatenation
// that merges a skip connection in the U-Net of Sec. 5.  Both stream the
// n x C matrices once (HBM-bound): 16-byte vector accesses when the row
// length allows, one row element per lane otherwise.
#include "internal.h"

namespace sscn {

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__global__ void k_affine_relu_f32(const float* __restrict__ x, const float* __restrict__ scale,
                                  const float* __restrict__ shift, int64_t total, int c, float* y) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int ch = (int)(i % c);
    y[i] = fmaxf(0.f, fmaf(x[i], scale[ch], shift[ch]));
  }
}

__global__ void k_affine_relu_bf16(const uint16_t* __restrict__ x, const float* __restrict__ scale,
                                   const float* __restrict__ shift, int64_t total, int c, uint16_t* y) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int ch = (int)(i % c);
    y[i] = f32_to_bf16_bits(fmaxf(0.f, fmaf(bf16_bits_to_f32(x[i]), scale[ch], shift[ch])));
  }
}

// The same with 16 bytes per lane (4 fp32 or 8 bf16 channels): c % V == 0,
// x and y 16-byte aligned, fewer than 2^31 chunks (32-bit index arithmetic that cannot wrap).
__device__ __forceinline__ void affine8(const uint4 v, const float* __restrict__ sc, const float* __restrict__ sh,
                                        uint4& out, float) {
  const float* f = reinterpret_cast<const float*>(&v);
  float r[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) r[i] = fmaxf(0.f, fmaf(f[i], sc[i], sh[i]));
  out = make_uint4(__float_as_uint(r[0]), __float_as_uint(r[1]), __float_as_uint(r[2]), __float_as_uint(r[3]));
}
__device__ __forceinline__ void affine8(const uint4 v, const float* __restrict__ sc, const float* __restrict__ sh,
                                        uint4& out, uint16_t) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float lo = fmaxf(0.f, fmaf(bf16_bits_to_f32((uint16_t)(w[i] & 0xffffu)), sc[2 * i], sh[2 * i]));
    const float hi = fmaxf(0.f, fmaf(bf16_bits_to_f32((uint16_t)(w[i] >> 16)), sc[2 * i + 1], sh[2 * i + 1]));
    o[i] = (uint32_t)f32_to_bf16_bits(lo) | ((uint32_t)f32_to_bf16_bits(hi) << 16);
  }
  out = make_uint4(o[0], o[1], o[2], o[3]);
}
template <typename T>
__global__ void k_affine_relu_x16(const uint4* __restrict__ x, const float* __restrict__ scale,
                                  const float* __restrict__ shift, uint32_t n_chunks, uint32_t per_row,
                                  uint4* __restrict__ y) {
  constexpr int V = 16 / sizeof(T);
  for (uint32_t q = blockIdx.x * blockDim.x + threadIdx.x; q < n_chunks; q += gridDim.x * blockDim.x) {
    const uint32_t ch = (q % per_row) * V;
    uint4 out;
    affine8(x[q], scale + ch, shift + ch, out, T{});
    y[q] = out;
  }
}

// y[r] = [a[r] | b[r]] in 16-byte chunks (both row lengths whole chunks,
// pointers 16-byte aligned, fewer than 2^31 chunks).
__global__ void k_concat_x16(const uint4* __restrict__ a, uint32_t wa, const uint4* __restrict__ b, uint32_t wb,
                             uint32_t n_chunks, uint4* __restrict__ y) {
  const uint32_t w = wa + wb;
  for (uint32_t q = blockIdx.x * blockDim.x + threadIdx.x; q < n_chunks; q += gridDim.x * blockDim.x) {
    const uint32_t r = q / w, c = q - r * w;
    y[q] = c < wa ? a[(size_t)r * wa + c] : b[(size_t)r * wb + (c - wa)];
  }
}

// y[r] = [a[r] | b[r]] for element size `es` bytes, copied in 4-byte words
// when every row length is a whole number of words, else byte by byte.
__global__ void k_concat_words(const uint32_t* __restrict__ a, int wa, const uint32_t* __restrict__ b, int wb,
                               int64_t n, uint32_t* __restrict__ y) {
  const int w = wa + wb;
  const int64_t total = n * w;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / w;
    const int c = (int)(i % w);
    y[i] = c < wa ? a[r * wa + c] : b[r * wb + (c - wa)];
  }
}

__global__ void k_concat_u16(const uint16_t* __restrict__ a, int ca, const uint16_t* __restrict__ b, int cb,
                             int64_t n, uint16_t* __restrict__ y) {
  const int w = ca + cb;
  const int64_t total = n * w;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / w;
    const int c = (int)(i % w);
    y[i] = c < ca ? a[r * ca + c] : b[r * cb + (c - ca)];
  }
}

static unsigned grid_of(int64_t total) {
  int64_t b = ceil_div(total, 256);
  if (b > 16384) b = 16384;
  if (b < 1) b = 1;
  return (unsigned)b;
}

}  // namespace sscn

using namespace sscn;

extern "C" sscn_status sscn_affine_relu(const void* x, const float* scale, const float* shift, int64_t n,
                                        int32_t c, sscn_dtype dtype, void* y, hipStream_t stream) {
  if (n < 0 || c < 1) return fail(SSCN_ERR_INVALID_ARG, "n must be >= 0 and c >= 1");
  if (dtype != SSCN_F32 && dtype != SSCN_BF16) return fail(SSCN_ERR_INVALID_ARG, "unknown dtype");
  if (n == 0) return SSCN_OK;
  if (!x || !y || !scale || !shift) return fail(SSCN_ERR_INVALID_ARG, "NULL pointer");
  const int64_t total = n * (int64_t)c;
  const int es = dtype == SSCN_F32 ? 4 : 2;
  const int64_t chunks = total * es / 16;
  if (((int64_t)c * es) % 16 == 0 && (uintptr_t)x % 16 == 0 && (uintptr_t)y % 16 == 0 && chunks < (1ll << 31)) {
    const uint32_t per_row = (uint32_t)((int64_t)c * es / 16);
    if (dtype == SSCN_F32)
      k_affine_relu_x16<float><<<grid_of(chunks), 256, 0, stream>>>((const uint4*)x, scale, shift,
                                                                   (uint32_t)chunks, per_row, (uint4*)y);
    else
      k_affine_relu_x16<uint16_t><<<grid_of(chunks), 256, 0, stream>>>((const uint4*)x, scale, shift,
                                                                      (uint32_t)chunks, per_row, (uint4*)y);
    SSCN_HIP(hipGetLastError());
    return SSCN_OK;
  }
  if (dtype == SSCN_F32)
    k_affine_relu_f32<<<grid_of(total), 256, 0, stream>>>((const float*)x, scale, shift, total, c, (float*)y);
  else
    k_affine_relu_bf16<<<grid_of(total), 256, 0, stream>>>((const uint16_t*)x, scale, shift, total, c,
                                                           (uint16_t*)y);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

extern "C" sscn_status sscn_concat_cols(const void* a, int32_t ca, const void* b, int32_t cb, int64_t n,
                                        sscn_dtype dtype, void* y, hipStream_t stream) {
  if (n < 0 || ca < 1 || cb < 1) return fail(SSCN_ERR_INVALID_ARG, "n must be >= 0, ca and cb >= 1");
  if (dtype != SSCN_F32 && dtype != SSCN_BF16) return fail(SSCN_ERR_INVALID_ARG, "unknown dtype");
  if (n == 0) return SSCN_OK;
  if (!a || !b || !y) return fail(SSCN_ERR_INVALID_ARG, "NULL pointer");
  const int es = dtype == SSCN_F32 ? 4 : 2;
  const int64_t chunks = n * ((int64_t)(ca + cb) * es / 16);
  if (((int64_t)ca * es) % 16 == 0 && ((int64_t)cb * es) % 16 == 0 && (uintptr_t)a % 16 == 0 &&
      (uintptr_t)b % 16 == 0 && (uintptr_t)y % 16 == 0 && chunks < (1ll << 31)) {
    k_concat_x16<<<grid_of(chunks), 256, 0, stream>>>((const uint4*)a, (uint32_t)(ca * es / 16), (const uint4*)b,
                                                      (uint32_t)(cb * es / 16), (uint32_t)chunks, (uint4*)y);
    SSCN_HIP(hipGetLastError());
    return SSCN_OK;
  }
  const bool words = ((int64_t)ca * es) % 4 == 0 && ((int64_t)cb * es) % 4 == 0 && ((uintptr_t)a % 4 == 0) &&
                     ((uintptr_t)b % 4 == 0) && ((uintptr_t)y % 4 == 0);
  if (words) {
    const int wa = ca * es / 4, wb = cb * es / 4;
    k_concat_words<<<grid_of(n * (wa + wb)), 256, 0, stream>>>((const uint32_t*)a, wa, (const uint32_t*)b, wb, n,
                                                               (uint32_t*)y);
  } else {
    // bf16 with an odd channel count
    k_concat_u16<<<grid_of(n * (ca + cb)), 256, 0, stream>>>((const uint16_t*)a, ca, (const uint16_t*)b, cb, n,
                                                             (uint16_t*)y);
  }
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}
