// Sparse convolution arithmetic (Sec. 4.2 step 2 of the paper): per filter
// offset o, a gather of input rows, a dense (pairs x C_in) x (C_in x C_out)
// product with W^o, and a scatter-add into output rows.
//
// Forward and dgrad use one output-stationary kernel.  A workgroup owns a
// block of output rows (tiles of 64 rows, see the rule-book layout) and a
// block of output columns; each wavefront of it owns 16 columns.  For each
// offset the workgroup walks its contiguous segment of pairs 16 at a time:
// every lane gathers 16 contiguous input channels of one pair's input row
// and 16 contiguous weights of its output column, the wavefront issues
// 16x16 MFMAs (fp32 16x16x4, or bf16 16x16x32 with fp32 accumulation), and
// the 16x16 result is added into an fp32 accumulator tile in LDS at the
// pairs' output rows.  Within one offset an output row occurs at most once
// and wavefronts own disjoint columns, so the LDS adds need no atomics and
// the summation order (offset by offset) is fixed.  The tile is written to
// HBM once, after the last offset.
//
// wgrad: dW^o = X[in_o]^T dY[out_o].  A workgroup takes one offset and a
// chunk of its pairs, stages the gathered X and dY rows in LDS (fp32) and
// accumulates 16x16 blocks of dW^o over the chunk with fp32 MFMAs; partial
// blocks are added into dW with fp32 atomics.
#include <algorithm>

#include "internal.h"

namespace sscn {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round to nearest, ties to even; NaN stays NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float* p) { return *p; }
  static __device__ __forceinline__ void store(float* p, float v) { *p = v; }
};
template <> struct Elem<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t* p) { return bf16_to_f32(p->bits); }
  static __device__ __forceinline__ void store(bf16_t* p, float v) { p->bits = f32_to_bf16(v); }
};

// ------------------------------------------------------------------ gathers
// 16 consecutive fp32 values row[k0 .. k0+16), zero beyond kmax.
__device__ __forceinline__ void load16(const float* __restrict__ row, int k0, int kmax, bool vec,
                                       float (&v)[16]) {
  if (vec && k0 + 16 <= kmax) {
    const float4* p = reinterpret_cast<const float4*>(row + k0);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float4 x = p[q];
      v[4 * q + 0] = x.x; v[4 * q + 1] = x.y; v[4 * q + 2] = x.z; v[4 * q + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = (k0 + i < kmax) ? row[k0 + i] : 0.f;
  }
}

// 16 consecutive bf16 values as two 8-wide MFMA operands, zero beyond kmax.
__device__ __forceinline__ void load16(const bf16_t* __restrict__ row, int k0, int kmax, bool vec,
                                       bf16x8 (&v)[2]) {
  if (vec && k0 + 16 <= kmax) {
    const uint4* p = reinterpret_cast<const uint4*>(row + k0);
    uint4 a = p[0], b = p[1];
    v[0] = __builtin_bit_cast(bf16x8, a);
    v[1] = __builtin_bit_cast(bf16x8, b);
  } else {
    uint16_t t[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) t[i] = (k0 + i < kmax) ? row[k0 + i].bits : (uint16_t)0;
    uint4 a, b;
    a.x = t[0] | ((uint32_t)t[1] << 16);   a.y = t[2] | ((uint32_t)t[3] << 16);
    a.z = t[4] | ((uint32_t)t[5] << 16);   a.w = t[6] | ((uint32_t)t[7] << 16);
    b.x = t[8] | ((uint32_t)t[9] << 16);   b.y = t[10] | ((uint32_t)t[11] << 16);
    b.z = t[12] | ((uint32_t)t[13] << 16); b.w = t[14] | ((uint32_t)t[15] << 16);
    v[0] = __builtin_bit_cast(bf16x8, a);
    v[1] = __builtin_bit_cast(bf16x8, b);
  }
}

// D += A B^T over 64 reduction indices held 16 per lane.
// Lane l supplies row (l % 16) of A and of B; its 16 values are the
// reduction indices 16*(l/16) + [0, 16) of a 64-wide chunk.  Any fixed
// assignment of reduction indices to (instruction, lane group) gives the
// same sum, so each instruction takes one index (fp32) or eight (bf16) per
// lane group.
__device__ __forceinline__ f32x4 mma64(const float (&a)[16], const float (&b)[16], f32x4 d) {
#pragma unroll
  for (int i = 0; i < 16; ++i) d = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[i], d, 0, 0, 0);
  return d;
}
__device__ __forceinline__ f32x4 mma64(const bf16x8 (&a)[2], const bf16x8 (&b)[2], f32x4 d) {
  d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[0], b[0], d, 0, 0, 0);
  d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[1], b[1], d, 0, 0, 0);
  return d;
}

template <typename T> struct Frag;
template <> struct Frag<float> { typedef float type[16]; };
template <> struct Frag<bf16_t> { typedef bf16x8 type[2]; };

// ---------------------------------------------------------- forward / dgrad
// X   : n_in x cin rows (the gathered operand)
// Bt  : K x cout x cin  (row n of Bt[o] = the cin weights feeding output column n)
// Y   : n_out x cout, fully written for the workgroup's rows and columns
template <typename T, int NW>
__global__ __launch_bounds__(NW * 64) void k_gather_mma(
    const T* __restrict__ X, const T* __restrict__ Bt, const int64_t* __restrict__ seg,
    const int32_t* __restrict__ in_rows, const int32_t* __restrict__ out_rows, int64_t n_tiles, int K,
    int mirror, int cin, int cout, int64_t n_out, int tpw, int vec, T* __restrict__ Y) {
  extern __shared__ float acc[];
  constexpr int WCOLS = 16 * NW;
  constexpr int LDW = WCOLS + 1;  // padded row stride of the accumulator tile
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int64_t t0 = (int64_t)blockIdx.x * tpw;
  const int64_t t1 = min<int64_t>(t0 + tpw, n_tiles);
  const int64_t row0 = t0 * kTile;
  const int rows = tpw * kTile;
  const int col_base = blockIdx.y * WCOLS;
  const int col = col_base + wave * 16 + m;  // this lane's output column (B row)
  const bool col_ok = col < cout;

  for (int i = threadIdx.x; i < rows * LDW; i += blockDim.x) acc[i] = 0.f;
  __syncthreads();

  for (int o = 0; o < K; ++o) {
    const int so = mirror ? K - 1 - o : o;
    const int64_t s = seg[(int64_t)so * n_tiles + t0];
    const int64_t e = seg[(int64_t)so * n_tiles + t1];
    if (s == e) continue;
    const T* __restrict__ brow = Bt + ((int64_t)o * cout + (col_ok ? col : 0)) * cin;
    for (int64_t p0 = s; p0 < e; p0 += 16) {
      const int64_t p = p0 + m;
      const bool pv = p < e;
      const int32_t irow = pv ? in_rows[p] : 0;
      const int32_t orow = pv ? (int32_t)(out_rows[p] - row0) : -1;
      const T* __restrict__ arow = X + (int64_t)irow * cin;
      f32x4 d = {0.f, 0.f, 0.f, 0.f};
      for (int kb = 0; kb < cin; kb += 64) {
        typename Frag<T>::type a, b;
        load16(arow, kb + 16 * g, pv ? cin : 0, vec, a);
        load16(brow, kb + 16 * g, col_ok ? cin : 0, vec, b);
        d = mma64(a, b, d);
      }
      // lane holds D[4g + r][m]: pair 4g + r, column m
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ol = __shfl(orow, 4 * g + r, 64);
        if (ol >= 0) acc[ol * LDW + wave * 16 + m] += d[r];
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < rows * WCOLS; i += blockDim.x) {
    const int r = i / WCOLS, c = i % WCOLS;
    const int64_t row = row0 + r;
    const int cc = col_base + c;
    if (row < n_out && cc < cout) Elem<T>::store(Y + row * cout + cc, acc[r * LDW + c]);
  }
}

// Bt[o][n][k] = W[o][k][n]
template <typename T>
__global__ void k_transpose_w(const T* __restrict__ W, int K, int cin, int cout, T* __restrict__ Bt) {
  const int64_t total = (int64_t)K * cin * cout;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t o = i / ((int64_t)cin * cout);
    const int64_t r = i % ((int64_t)cin * cout);
    const int k = (int)(r / cout), n = (int)(r % cout);
    Bt[(o * cout + n) * cin + k] = W[i];
  }
}

// ------------------------------------------------------------------- wgrad
// Workgroup (chunk, o, z): pairs [start_o + chunk*pch, ...) of offset o;
// z selects a block of up to 64 input channels (wave w: channels
// 16*(4*zc + w) + [0,16)) and up to MAXCO*16 output channels.
constexpr int kWgradPairs = 64;   // pairs staged in LDS per step
template <typename T, int MAXCO>
__global__ __launch_bounds__(256) void k_wgrad(const T* __restrict__ X, const T* __restrict__ dY,
                                               const int64_t* __restrict__ seg, int64_t n_tiles,
                                               const int32_t* __restrict__ in_rows,
                                               const int32_t* __restrict__ out_rows, int K, int mirror,
                                               int cin, int cout, int pch, int nzc, float* __restrict__ dW) {
  const int o = blockIdx.y;
  const int so = mirror ? K - 1 - o : o;  // storage slot of offset o
  const int64_t start = seg[(int64_t)so * n_tiles], end = seg[(int64_t)(so + 1) * n_tiles];
  const int64_t pb = start + (int64_t)blockIdx.x * pch;
  if (pb >= end) return;
  const int64_t pe = min<int64_t>(pb + pch, end);
  const int zc = blockIdx.z % nzc, zo = blockIdx.z / nzc;
  const int ci_base = zc * 64, co_base = zo * MAXCO * 16;
  const int ci_n = min(64, cin - ci_base), co_n = min(MAXCO * 16, cout - co_base);
  constexpr int LDX = 64 + 1, LDY = MAXCO * 16 + 1;
  __shared__ float xs[kWgradPairs * LDX];
  __shared__ float ys[kWgradPairs * LDY];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int ci_w = wave * 16;  // wave's channel block inside the 64-block
  f32x4 d[MAXCO];
#pragma unroll
  for (int c = 0; c < MAXCO; ++c) d[c] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int64_t q0 = pb; q0 < pe; q0 += kWgradPairs) {
    const int np = (int)min<int64_t>(kWgradPairs, pe - q0);
    __syncthreads();
    for (int i = threadIdx.x; i < kWgradPairs * 64; i += 256) {
      const int pr = i / 64, c = i % 64;
      float v = 0.f;
      if (pr < np && c < ci_n) v = Elem<T>::load(X + (int64_t)in_rows[q0 + pr] * cin + ci_base + c);
      xs[pr * LDX + c] = v;
    }
    for (int i = threadIdx.x; i < kWgradPairs * MAXCO * 16; i += 256) {
      const int pr = i / (MAXCO * 16), c = i % (MAXCO * 16);
      float v = 0.f;
      if (pr < np && c < co_n) v = Elem<T>::load(dY + (int64_t)out_rows[q0 + pr] * cout + co_base + c);
      ys[pr * LDY + c] = v;
    }
    __syncthreads();
    if (ci_w < ci_n) {
#pragma unroll 4
      for (int i = 0; i < kWgradPairs / 4; ++i) {
        const int pr = 4 * i + g;  // reduction index of this lane group
        const float a = xs[pr * LDX + ci_w + m];
#pragma unroll
        for (int c = 0; c < MAXCO; ++c) {
          const float b = ys[pr * LDY + c * 16 + m];
          d[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, d[c], 0, 0, 0);
        }
      }
    }
  }
  if (ci_w >= ci_n) return;
  // lane holds D[4g + r][m]: input channel ci_w + 4g + r, output channel c*16 + m
#pragma unroll
  for (int c = 0; c < MAXCO; ++c) {
    const int co = co_base + c * 16 + m;
    if (c * 16 + m >= co_n) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ci = ci_base + ci_w + 4 * g + r;
      if (ci_w + 4 * g + r < ci_n) atomicAdd(dW + ((int64_t)o * cin + ci) * cout + co, d[c][r]);
    }
  }
}

// ---------------------------------------------------------------- launchers
template <typename T, int NW>
static sscn_status launch_gather_mma_nw(const T* X, const T* Bt, const View& v, int cin, int cout,
                                        int grid_y, T* Y, hipStream_t s) {
  // accumulator tile (tpw * 64 rows x (16 NW + 1) fp32) kept within 64 KiB of LDS
  const int tpw = NW >= 8 ? 1 : 2;
  const int64_t blocks = ceil_div(v.st->n_tiles, tpw);
  const size_t lds = sizeof(float) * tpw * kTile * (16 * NW + 1);
  constexpr int VEC = sizeof(T) == 4 ? 4 : 8;  // elements per 16-byte load
  const int vec = (cin % VEC == 0) && ((uintptr_t)X % 16 == 0) && ((uintptr_t)Bt % 16 == 0);
  k_gather_mma<T, NW><<<dim3((unsigned)blocks, (unsigned)grid_y), NW * 64, lds, s>>>(
      X, Bt, v.st->seg, v.st->in_rows, v.st->out_rows, v.st->n_tiles, v.K, v.mirror ? 1 : 0, cin, cout,
      v.n_out, tpw, vec, Y);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

template <typename T>
static sscn_status launch_gather_mma(const T* X, const T* Bt, const View& v, int cin, int cout, T* Y,
                                     hipStream_t s) {
  const int ncb = (cout + 15) / 16;
  const int grid_y = (ncb + 7) / 8;
  const int nw = (ncb + grid_y - 1) / grid_y;
  switch (nw) {
    case 1: return launch_gather_mma_nw<T, 1>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 2: return launch_gather_mma_nw<T, 2>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 3: return launch_gather_mma_nw<T, 3>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 4: return launch_gather_mma_nw<T, 4>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 5: return launch_gather_mma_nw<T, 5>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 6: return launch_gather_mma_nw<T, 6>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 7: return launch_gather_mma_nw<T, 7>(X, Bt, v, cin, cout, grid_y, Y, s);
    default: return launch_gather_mma_nw<T, 8>(X, Bt, v, cin, cout, grid_y, Y, s);
  }
}

template <typename T>
static sscn_status launch_wgrad(const T* X, const T* dY, const View& v, int cin, int cout, float* dW,
                                hipStream_t s, int64_t max_pairs_per_offset, int64_t n_pairs) {
  constexpr int MAXCO = 4;
  int64_t pch = ceil_div(n_pairs, 2048);
  pch = ceil_div(pch, kWgradPairs) * kWgradPairs;
  pch = std::min<int64_t>(std::max<int64_t>(pch, 256), 16384);
  const int nzc = (cin + 63) / 64;
  const int nzo = (cout + MAXCO * 16 - 1) / (MAXCO * 16);
  const int64_t gx = std::max<int64_t>(1, ceil_div(max_pairs_per_offset, pch));
  k_wgrad<T, MAXCO><<<dim3((unsigned)gx, (unsigned)v.K, (unsigned)(nzc * nzo)), 256, 0, s>>>(
      X, dY, v.st->seg, v.st->n_tiles, v.st->in_rows, v.st->out_rows, v.K, v.mirror ? 1 : 0, cin, cout,
      (int)pch, nzc, dW);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

static View transposed_view(const sscn_rulebook_s* rb) {
  sscn_rulebook_s t{rb->d, !rb->transposed};
  return view_of(&t);
}

static sscn_status check_conv_args(sscn_rulebook rb, int32_t c_in, int32_t c_out, sscn_dtype dtype) {
  if (!rb) return fail(SSCN_ERR_INVALID_ARG, "NULL rule book");
  if (c_in < 1 || c_out < 1) return fail(SSCN_ERR_INVALID_ARG, "channel counts must be >= 1");
  if (c_in > 65536 || c_out > 65536) return fail(SSCN_ERR_INVALID_ARG, "channel counts must be <= 65536");
  if (dtype != SSCN_F32 && dtype != SSCN_BF16) return fail(SSCN_ERR_INVALID_ARG, "unknown dtype");
  return SSCN_OK;
}

template <typename T>
static sscn_status forward_t(const T* X, const T* W, const View& v, int cin, int cout, T* Y, hipStream_t s) {
  const int64_t K = v.K;
  T* Bt = nullptr;
  sscn_status st = dev_alloc((void**)&Bt, sizeof(T) * K * cin * cout, s);
  if (st != SSCN_OK) return st;
  const int64_t total = K * cin * cout;
  k_transpose_w<T><<<(unsigned)std::min<int64_t>(ceil_div(total, 256), 4096), 256, 0, s>>>(W, (int)K, cin,
                                                                                            cout, Bt);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) st = launch_gather_mma<T>(X, Bt, v, cin, cout, Y, s);
  dev_free(Bt, s);
  if (e != hipSuccess) return hip_fail(e, "transpose launch");
  return st;
}

}  // namespace sscn

using namespace sscn;

extern "C" sscn_status sparse_conv_forward(const void* features, const void* weights, sscn_rulebook rb,
                                           int32_t c_in, int32_t c_out, sscn_dtype dtype, void* out,
                                           hipStream_t stream) {
  sscn_status st = check_conv_args(rb, c_in, c_out, dtype);
  if (st != SSCN_OK) return st;
  const View v = view_of(rb);
  if (v.n_out == 0) return SSCN_OK;
  if (!out || !weights || (v.n_in > 0 && !features))
    return fail(SSCN_ERR_INVALID_ARG, "NULL features, weights or out");
  if (dtype == SSCN_F32)
    return forward_t<float>((const float*)features, (const float*)weights, v, c_in, c_out, (float*)out, stream);
  return forward_t<bf16_t>((const bf16_t*)features, (const bf16_t*)weights, v, c_in, c_out, (bf16_t*)out,
                           stream);
}

extern "C" sscn_status sparse_conv_backward(const void* features, const void* weights, const void* dout,
                                            sscn_rulebook rb, int32_t c_in, int32_t c_out, sscn_dtype dtype,
                                            void* dgrad, float* wgrad, hipStream_t stream) {
  sscn_status st = check_conv_args(rb, c_in, c_out, dtype);
  if (st != SSCN_OK) return st;
  const View v = view_of(rb);
  if (dgrad && v.n_in > 0) {
    if (!weights || (v.n_out > 0 && !dout)) return fail(SSCN_ERR_INVALID_ARG, "NULL weights or dout");
    // dgrad = forward over the transposed rule book with B = W^o (as stored:
    // row ci of W[o] holds the c_out weights feeding input channel ci)
    const View vt = transposed_view(rb);
    if (dtype == SSCN_F32)
      st = launch_gather_mma<float>((const float*)dout, (const float*)weights, vt, c_out, c_in, (float*)dgrad,
                                    stream);
    else
      st = launch_gather_mma<bf16_t>((const bf16_t*)dout, (const bf16_t*)weights, vt, c_out, c_in,
                                     (bf16_t*)dgrad, stream);
    if (st != SSCN_OK) return st;
  }
  if (wgrad) {
    const int64_t total = (int64_t)v.K * c_in * c_out;
    st = fill_f32(wgrad, 0.f, total, stream);
    if (st != SSCN_OK) return st;
    const RulebookData* d = rb->d;
    if (d->n_pairs > 0) {
      if (!features || !dout) return fail(SSCN_ERR_INVALID_ARG, "NULL features or dout");
      int64_t mx = 0;
      for (int64_t c : d->pairs_per_offset) mx = std::max(mx, c);
      if (dtype == SSCN_F32)
        st = launch_wgrad<float>((const float*)features, (const float*)dout, v, c_in, c_out, wgrad, stream, mx,
                                 d->n_pairs);
      else
        st = launch_wgrad<bf16_t>((const bf16_t*)features, (const bf16_t*)dout, v, c_in, c_out, wgrad, stream,
                                  mx, d->n_pairs);
    }
  }
  return st;
}
