// Training pieces of a submanifold network (Sec. 4.1 "Other operators":
// batch normalisation as regular batch normalisation over the set of
// active sites, activation functions on the active sites; Sec. 5: the final
// linear layer and softmax on each active site; Sec. 6.2: negative
// log-likelihood, SGD with Nesterov momentum and L2 weight decay).
//
// Batch statistics and their gradients are column reductions over the n
// active rows.  They run in two deterministic passes: a grid of workgroups
// each sums a fixed set of rows into fp64 partials (one per workgroup and
// channel), and one thread per channel then adds the partials in workgroup
// order.  No atomics, so every result is reproducible bit for bit.  The
// passes stream the n x c matrix once (HBM-bound).
#include <algorithm>
#include <initializer_list>
#include <utility>

#include "internal.h"
#include "numeric.h"

namespace sscn {

namespace {

constexpr int kColChunk = 64;       // channels per workgroup (one per lane)
constexpr int kMaxPartials = 1024;  // workgroups over the rows

enum ColOp { kSums = 0, kSumSquares = 1, kBnBack = 2 };

// The normalised, scaled and shifted value before the ReLU, as the forward
// computes it: (x - mean) * (gamma * invstd) + beta.  (Subtracting the mean
// first keeps the result accurate when the variance is tiny next to the
// mean; the backward's ReLU mask evaluates the same expression.)
__device__ __forceinline__ float bn_pre(float x, float mean, float scale, float beta) {
  return fmaf(x - mean, scale, beta);
}

// Per channel: a0 = sum of v, a1 = sum of v^2 (kSumSquares) or of v * xhat
// (kBnBack, where v = dA masked by the forward's ReLU and xhat the
// normalised input); kSums: a0 only.  partial[(blk * 2 + i) * c + col].
template <typename T, int OP>
__global__ __launch_bounds__(256) void k_colreduce(const T* __restrict__ x, int64_t ldx, const T* __restrict__ da,
                                                   int64_t ldd, int64_t n, int c, const float* __restrict__ scale,
                                                   const float* __restrict__ beta, const float* __restrict__ mean,
                                                   const float* __restrict__ invstd, double* __restrict__ partial) {
  __shared__ double red[2][4][kColChunk];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = blockIdx.y * kColChunk + lane;
  const bool live = col < c;
  double a0 = 0.0, a1 = 0.0;
  if (live) {
    float sc = 0.f, be = 0.f, mu = 0.f, is = 0.f;
    if constexpr (OP == kBnBack) {
      sc = scale[col]; be = beta[col]; mu = mean[col]; is = invstd[col];
    }
    // U rows in flight per wavefront (one at a time left the pass bound by
    // load latency); the sums still run over the rows in order
    constexpr int U = 8;
    const int64_t stride = (int64_t)gridDim.x * 4;
    for (int64_t r0 = (int64_t)blockIdx.x * 4 + wave; r0 < n; r0 += U * stride) {
      float vx[U], vd[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t r = r0 + u * stride;
        vx[u] = r < n ? ld(x + r * ldx + col) : 0.f;
        vd[u] = 0.f;
        if constexpr (OP == kBnBack) vd[u] = r < n ? ld(da + r * ldd + col) : 0.f;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (r0 + u * stride >= n) break;
        const float v = vx[u];
        if constexpr (OP == kBnBack) {
          const float dz = bn_pre(v, mu, sc, be) > 0.f ? vd[u] : 0.f;
          a0 += dz;
          a1 += (double)dz * (double)((v - mu) * is);
        } else {
          a0 += v;
          if constexpr (OP == kSumSquares) a1 += (double)v * (double)v;
        }
      }
    }
  }
  red[0][wave][lane] = a0;
  red[1][wave][lane] = a1;
  __syncthreads();
  if (wave == 0 && live) {
    double s0 = 0.0, s1 = 0.0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      s0 += red[0][w][lane];
      s1 += red[1][w][lane];
    }
    partial[((int64_t)blockIdx.x * 2) * c + col] = s0;
    partial[((int64_t)blockIdx.x * 2 + 1) * c + col] = s1;
  }
}

// The same reductions for rows of whole 16-byte pieces (c e a multiple of
// 16 and at most 1024 bytes, rows 16-byte aligned): lane l of a wavefront
// loads piece l % LPR of row l / LPR (LPR = pieces per row) of RPW = 64 / LPR
// rows at once, VPL = 16 / e channels, and keeps fp64 sums for them; a
// workgroup takes a contiguous range of rows, U row groups in flight per
// wavefront.  (One channel per lane and one row per wavefront load, as in
// k_colreduce, left the passes latency-bound: 0.3-0.4 ms for 2M x 32 bf16.)
// The lanes' sums are then added in a fixed order through LDS, so the result
// is reproducible.
template <typename T, int OP>
__global__ __launch_bounds__(256) void k_colreduce_vec(const T* __restrict__ x, int64_t ldx, const T* __restrict__ da,
                                                       int64_t ldd, int64_t n, int c, int64_t rows_per_block,
                                                       const float* __restrict__ scale,
                                                       const float* __restrict__ beta,
                                                       const float* __restrict__ mean,
                                                       const float* __restrict__ invstd,
                                                       double* __restrict__ partial) {
  constexpr int VPL = 16 / (int)sizeof(T);  // channels per lane
  constexpr int U = 4;                      // row groups in flight per wavefront
  __shared__ double red[4][64][2 * VPL];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lpr = c / VPL;                  // pieces per row
  const int rpw = 64 / lpr;                 // rows per wavefront load
  const int cg = lane % lpr, ro = lane / lpr;
  const bool live = ro < rpw;
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block, r1 = min<int64_t>(n, r0 + rows_per_block);
  double a0[VPL], a1[VPL];
  float mu[VPL], sc[VPL], be[VPL], is[VPL];
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    a0[v] = 0.0;
    a1[v] = 0.0;
    mu[v] = sc[v] = be[v] = is[v] = 0.f;
  }
  if constexpr (OP == kBnBack) {
    if (live) {
#pragma unroll
      for (int v = 0; v < VPL; ++v) {
        const int col = cg * VPL + v;
        mu[v] = mean[col];
        sc[v] = scale[col];
        be[v] = beta[col];
        is[v] = invstd[col];
      }
    }
  }
  auto vals = [](const uint4& q, float (&f)[VPL]) {
    if constexpr (sizeof(T) == 4) {
      f[0] = __uint_as_float(q.x); f[1] = __uint_as_float(q.y); f[2] = __uint_as_float(q.z); f[3] = __uint_as_float(q.w);
    } else {
      const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f[2 * i] = __uint_as_float(w[i] << 16);
        f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
      }
    }
  };
  const int64_t step = 4 * (int64_t)rpw;  // rows per workgroup load
  for (int64_t base = r0 + (int64_t)wave * rpw + ro; base < r1; base += U * step) {
    uint4 qx[U], qd[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t r = base + u * step;
      const bool ok = live && r < r1;
      qx[u] = ok ? *reinterpret_cast<const uint4*>(x + r * ldx + cg * VPL) : make_uint4(0, 0, 0, 0);
      if constexpr (OP == kBnBack)
        qd[u] = ok ? *reinterpret_cast<const uint4*>(da + r * ldd + cg * VPL) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (!(live && base + u * step < r1)) continue;
      float fx[VPL];
      vals(qx[u], fx);
      if constexpr (OP == kBnBack) {
        float fd[VPL];
        vals(qd[u], fd);
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
          const float dz = bn_pre(fx[v], mu[v], sc[v], be[v]) > 0.f ? fd[v] : 0.f;
          a0[v] += dz;
          a1[v] += (double)dz * (double)((fx[v] - mu[v]) * is[v]);
        }
      } else {
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
          a0[v] += fx[v];
          if constexpr (OP == kSumSquares) a1[v] += (double)fx[v] * (double)fx[v];
        }
      }
    }
  }
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    red[wave][lane][v] = a0[v];
    red[wave][lane][VPL + v] = a1[v];
  }
  __syncthreads();
  // value t: sum (t < c) or second sum (c <= t < 2 c) of channel t % c
  for (int t = threadIdx.x; t < 2 * c; t += blockDim.x) {
    const int kind = t / c, col = t % c, g = col / VPL, v = col % VPL;
    double sum = 0.0;
    for (int w = 0; w < 4; ++w)
      for (int q = 0; q < rpw; ++q) sum += red[w][q * lpr + g][kind * VPL + v];
    partial[((int64_t)blockIdx.x * 2 + kind) * c + col] = sum;
  }
}

// Sums of the partials of the `blocks` workgroups for channel col: one
// workgroup of kFinThreads threads per 64 channels, wavefront w adding
// blocks w, w + 16, .. in order, then the sixteen wavefronts' sums added
// pairwise in a fixed tree (a fixed order: reproducible).  (One thread
// adding all blocks in turn took ~0.25 ms for 1024 blocks; four wavefronts
// ~15 us.)
constexpr int kFinThreads = 1024;
__device__ __forceinline__ bool sum_partials(const double* __restrict__ partial, int blocks, int c, double& s0,
                                             double& s1, int& col) {
  constexpr int NW = kFinThreads / 64;
  __shared__ double red[2][NW][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  col = blockIdx.x * 64 + lane;
  double a0 = 0.0, a1 = 0.0;
  if (col < c) {
#pragma unroll 4
    for (int b = wave; b < blocks; b += NW) {
      a0 += partial[((int64_t)b * 2) * c + col];
      a1 += partial[((int64_t)b * 2 + 1) * c + col];
    }
  }
  red[0][wave][lane] = a0;
  red[1][wave][lane] = a1;
  __syncthreads();
#pragma unroll
  for (int h = NW / 2; h >= 1; h /= 2) {
    if (wave < h) {
      red[0][wave][lane] += red[0][wave + h][lane];
      red[1][wave][lane] += red[1][wave + h][lane];
    }
    __syncthreads();
  }
  if (wave != 0 || col >= c) return false;
  s0 = red[0][0][lane];
  s1 = red[1][0][lane];
  return true;
}

// Batch statistics -> the affine map of the normalisation, and the running
// (inference) statistics: mean, biased variance for the map, unbiased for
// the running variance.
__global__ __launch_bounds__(kFinThreads) void k_bn_finalize(const double* __restrict__ partial, int blocks, int c,
                                                     int64_t n, const float* __restrict__ gamma,
                                                     const float* __restrict__ beta, float eps, float momentum,
                                                     float* running_mean, float* running_var,
                                                     float* __restrict__ mean, float* __restrict__ invstd,
                                                     float* __restrict__ scale, float* __restrict__ shift) {
  double s0, s1;
  int col;
  if (!sum_partials(partial, blocks, c, s0, s1, col)) return;
  const double mu = s0 / (double)n;
  const double var = fmax(s1 / (double)n - mu * mu, 0.0);
  const float is = (float)(1.0 / sqrt(var + (double)eps));
  const float sc = gamma[col] * is;
  mean[col] = (float)mu;
  invstd[col] = is;
  scale[col] = sc;
  shift[col] = beta[col] - (float)mu * sc;
  if (running_mean) {
    const double unbiased = n > 1 ? var * (double)n / (double)(n - 1) : var;
    running_mean[col] = (1.f - momentum) * running_mean[col] + momentum * (float)mu;
    running_var[col] = (1.f - momentum) * running_var[col] + momentum * (float)unbiased;
  }
}

__global__ __launch_bounds__(kFinThreads) void k_two_sums(const double* __restrict__ partial, int blocks, int c,
                                                  float* __restrict__ out0, float* __restrict__ out1) {
  double s0, s1;
  int col;
  if (!sum_partials(partial, blocks, c, s0, s1, col)) return;
  out0[col] = (float)s0;
  if (out1) out1[col] = (float)s1;
}

// dx = gamma invstd (dz - dbeta / n - xhat dgamma / n) (+ add), dz = dA where
// the forward's ReLU passed, else 0.
template <typename T>
__global__ void k_bn_back_input(const T* __restrict__ da, int64_t ldd, const T* __restrict__ x, int64_t ldx,
                                int64_t n, int c, const float* __restrict__ gamma, const float* __restrict__ scale,
                                const float* __restrict__ beta, const float* __restrict__ mean,
                                const float* __restrict__ invstd, const float* __restrict__ dgamma,
                                const float* __restrict__ dbeta, const T* __restrict__ add, int64_t lda,
                                T* __restrict__ dx, int64_t ldo) {
  const int64_t total = n * c;
  const float inv_n = 1.f / (float)n;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / c;
    const int col = (int)(i - r * c);
    const float v = ld(x + r * ldx + col);
    const float g = ld(da + r * ldd + col);
    const float dz = bn_pre(v, mean[col], scale[col], beta[col]) > 0.f ? g : 0.f;
    const float xhat = (v - mean[col]) * invstd[col];
    float out = gamma[col] * invstd[col] * (dz - dbeta[col] * inv_n - xhat * (dgamma[col] * inv_n));
    if (add) out += ld(add + r * lda + col);
    st(dx + r * ldo + col, out);
  }
}

// relu((x - mean) * scale + beta), strided rows.
template <typename T>
__global__ void k_bn_relu_apply(const T* __restrict__ x, int64_t ldx, int64_t n, int c,
                                const float* __restrict__ mean, const float* __restrict__ scale,
                                const float* __restrict__ beta, T* __restrict__ y, int64_t ldy) {
  const int64_t total = n * c;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / c;
    const int col = (int)(i - r * c);
    st(y + r * ldy + col, fmaxf(0.f, bn_pre(ld(x + r * ldx + col), mean[col], scale[col], beta[col])));
  }
}

// y = a + b, strided rows.
template <typename T>
__global__ void k_add(const T* __restrict__ a, int64_t lda, const T* __restrict__ b, int64_t ldb, int64_t n, int c,
                      T* __restrict__ y, int64_t ldy) {
  const int64_t total = n * c;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / c;
    const int col = (int)(i - r * c);
    st(y + r * ldy + col, ld(a + r * lda + col) + ld(b + r * ldb + col));
  }
}

// The row-wise passes for rows of whole 16-byte pieces (the layout of
// k_colreduce_vec: lane l handles VPL = 16 / e channels of row l / LPR of
// each wavefront's group of RPW = 64 / LPR rows), 16 bytes per load and
// store; MODE 0: relu((x - mean) * scale + beta), 1: the input gradient of
// that (as k_bn_back_input), 2: a + b.  (One element per lane with a 64-bit
// division per element ran the 2M x 32 bf16 passes at ~30% of HBM.)
template <typename T, int MODE>
__global__ __launch_bounds__(256) void k_rows_vec(const T* __restrict__ a, int64_t lda, const T* __restrict__ b,
                                                  int64_t ldb, const T* __restrict__ add, int64_t ldadd, int64_t n,
                                                  int c, const float* __restrict__ gamma,
                                                  const float* __restrict__ mean, const float* __restrict__ scale,
                                                  const float* __restrict__ beta, const float* __restrict__ invstd,
                                                  const float* __restrict__ dgamma, const float* __restrict__ dbeta,
                                                  T* __restrict__ y, int64_t ldy) {
  constexpr int VPL = 16 / (int)sizeof(T);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lpr = c / VPL, rpw = 64 / lpr;
  const int cg = lane % lpr, ro = lane / lpr;
  if (ro >= rpw) return;
  // per-channel constants: k0 = mean, k1 = scale, k2 = beta, k3 = invstd,
  // k4 = dbeta / n, k5 = dgamma / n, k6 = gamma invstd
  float k0[VPL], k1[VPL], k2[VPL], k3[VPL], k4[VPL], k5[VPL], k6[VPL];
  const float inv_n = 1.f / (float)max<int64_t>(n, 1);
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    const int col = cg * VPL + v;
    k0[v] = k1[v] = k2[v] = k3[v] = k4[v] = k5[v] = k6[v] = 0.f;
    if constexpr (MODE == 0) {
      k0[v] = mean[col]; k1[v] = scale[col]; k2[v] = beta[col];
    } else if constexpr (MODE == 1) {
      k0[v] = mean[col]; k1[v] = scale[col]; k2[v] = beta[col]; k3[v] = invstd[col];
      k4[v] = dbeta[col] * inv_n; k5[v] = dgamma[col] * inv_n; k6[v] = gamma[col] * invstd[col];
    }
  }
  auto unpack = [](const uint4& q, float (&f)[VPL]) {
    if constexpr (sizeof(T) == 4) {
      f[0] = __uint_as_float(q.x); f[1] = __uint_as_float(q.y); f[2] = __uint_as_float(q.z); f[3] = __uint_as_float(q.w);
    } else {
      const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f[2 * i] = __uint_as_float(w[i] << 16);
        f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
      }
    }
  };
  auto pack = [](const float (&f)[VPL]) {
    uint4 q;
    if constexpr (sizeof(T) == 4) {
      q.x = __float_as_uint(f[0]); q.y = __float_as_uint(f[1]); q.z = __float_as_uint(f[2]); q.w = __float_as_uint(f[3]);
    } else {
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = (uint32_t)f32_bf16_bits(f[2 * i]) | ((uint32_t)f32_bf16_bits(f[2 * i + 1]) << 16);
      q.x = w[0]; q.y = w[1]; q.z = w[2]; q.w = w[3];
    }
    return q;
  };
  const int64_t step = (int64_t)gridDim.x * 4 * rpw;
  for (int64_t r = ((int64_t)blockIdx.x * 4 + wave) * rpw + ro; r < n; r += step) {
    float fa[VPL], fo[VPL];
    unpack(*reinterpret_cast<const uint4*>(a + r * lda + cg * VPL), fa);
    if constexpr (MODE == 0) {
#pragma unroll
      for (int v = 0; v < VPL; ++v) fo[v] = fmaxf(0.f, bn_pre(fa[v], k0[v], k1[v], k2[v]));
    } else if constexpr (MODE == 1) {
      float fx[VPL];  // a = dA, b = x
      unpack(*reinterpret_cast<const uint4*>(b + r * ldb + cg * VPL), fx);
#pragma unroll
      for (int v = 0; v < VPL; ++v) {
        const float dz = bn_pre(fx[v], k0[v], k1[v], k2[v]) > 0.f ? fa[v] : 0.f;
        const float xhat = (fx[v] - k0[v]) * k3[v];
        fo[v] = k6[v] * (dz - k4[v] - xhat * k5[v]);
      }
      if (add) {
        float fd[VPL];
        unpack(*reinterpret_cast<const uint4*>(add + r * ldadd + cg * VPL), fd);
#pragma unroll
        for (int v = 0; v < VPL; ++v) fo[v] += fd[v];
      }
    } else {
      float fb[VPL];
      unpack(*reinterpret_cast<const uint4*>(b + r * ldb + cg * VPL), fb);
#pragma unroll
      for (int v = 0; v < VPL; ++v) fo[v] = fa[v] + fb[v];
    }
    *reinterpret_cast<uint4*>(y + r * ldy + cg * VPL) = pack(fo);
  }
}

// Whether matrices of c channels suit k_rows_vec (each pointer 16-byte
// aligned with a row stride of whole 16-byte pieces; nullptr is fine).
bool rows_vec_ok(sscn_dtype dtype, int c, std::initializer_list<std::pair<const void*, int64_t>> mats) {
  const int e = dtype == SSCN_F32 ? 4 : 2;
  if ((int64_t)c * e % 16 != 0 || (int64_t)c * e > 1024) return false;
  for (const auto& m : mats)
    if (m.first && (reinterpret_cast<uintptr_t>(m.first) % 16 != 0 || m.second * e % 16 != 0)) return false;
  return true;
}

template <int MODE>
sscn_status rows_vec(sscn_dtype dtype, const void* a, int64_t lda, const void* b, int64_t ldb, const void* add,
                     int64_t ldadd, int64_t n, int c, const float* gamma, const float* mean, const float* scale,
                     const float* beta, const float* invstd, const float* dgamma, const float* dbeta, void* y,
                     int64_t ldy, hipStream_t s);

unsigned rows_vec_grid(int64_t n, int c, sscn_dtype dtype) {
  const int vpl = dtype == SSCN_F32 ? 4 : 8;
  const int64_t rpw = 64 / (c / vpl);
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(ceil_div(n, 4 * rpw), 4096));
}

template <int MODE>
sscn_status rows_vec(sscn_dtype dtype, const void* a, int64_t lda, const void* b, int64_t ldb, const void* add,
                     int64_t ldadd, int64_t n, int c, const float* gamma, const float* mean, const float* scale,
                     const float* beta, const float* invstd, const float* dgamma, const float* dbeta, void* y,
                     int64_t ldy, hipStream_t s) {
  const unsigned g = rows_vec_grid(n, c, dtype);
  if (dtype == SSCN_F32)
    k_rows_vec<float, MODE><<<g, 256, 0, s>>>((const float*)a, lda, (const float*)b, ldb, (const float*)add, ldadd, n,
                                              c, gamma, mean, scale, beta, invstd, dgamma, dbeta, (float*)y, ldy);
  else
    k_rows_vec<uint16_t, MODE><<<g, 256, 0, s>>>((const uint16_t*)a, lda, (const uint16_t*)b, ldb,
                                                 (const uint16_t*)add, ldadd, n, c, gamma, mean, scale, beta, invstd,
                                                 dgamma, dbeta, (uint16_t*)y, ldy);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

// Softmax and negative log-likelihood, one wavefront per row (lanes over
// the classes).  dlogits = (softmax - onehot) / n; the row losses go to
// per-workgroup fp64 partials (summed in order by k_loss_finalize).  A label
// outside [0, classes) makes that row's loss NaN (its gradient is the
// softmax alone).
template <typename T>
__global__ __launch_bounds__(256) void k_softmax_nll(const T* __restrict__ z, int64_t n, int classes,
                                                     const int32_t* __restrict__ labels, T* __restrict__ dz,
                                                     double* __restrict__ partial) {
  __shared__ double red[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float inv_n = 1.f / (float)n;
  double acc = 0.0;
  for (int64_t r = (int64_t)blockIdx.x * 4 + wave; r < n; r += (int64_t)gridDim.x * 4) {
    const T* row = z + r * classes;
    float m = -INFINITY;
    for (int k = lane; k < classes; k += 64) m = fmaxf(m, ld(row + k));
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) m = fmaxf(m, __shfl_xor(m, d, 64));
    // s: the sum of exp(z - max) over all classes, so: over all but the
    // label.  The label's gradient p - 1 = -so / s and the loss
    // log(s / e_label) = log1p(so / e_label) are formed from so, which
    // keeps them accurate when the label's probability is close to 1.
    const int lab = labels[r];
    const bool ok = lab >= 0 && lab < classes;
    float s = 0.f, so = 0.f;
    for (int k = lane; k < classes; k += 64) {
      const float e = expf(ld(row + k) - m);
      s += e;
      if (k != lab) so += e;
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
      s += __shfl_xor(s, d, 64);
      so += __shfl_xor(so, d, 64);
    }
    for (int k = lane; k < classes; k += 64) {
      const float g = k == lab ? -so / s : expf(ld(row + k) - m) / s;
      st(dz + r * classes + k, g * inv_n);
    }
    if (lane == 0) {
      double l = (double)NAN;
      if (ok) {
        const float zl = ld(row + lab);
        const float el = expf(zl - m);
        l = el > 0.f ? (double)log1pf(so / el) : (double)(m - zl) + (double)logf(s);
      }
      acc += l;
    }
  }
  if (lane == 0) red[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) partial[blockIdx.x] = red[0] + red[1] + red[2] + red[3];
}

// The same for at most kSoftmaxRowMax classes, one thread per row: a
// wavefront then reads 64 consecutive rows (one wavefront per row left most
// lanes idle and took 1.1 ms for 2M rows of 20 classes).  The row losses
// are added per thread, then per workgroup in thread order.
constexpr int kSoftmaxRowMax = 64;
template <typename T>
__global__ __launch_bounds__(256) void k_softmax_nll_rows(const T* __restrict__ z, int64_t n, int classes,
                                                          const int32_t* __restrict__ labels, T* __restrict__ dz,
                                                          double* __restrict__ partial) {
  __shared__ double red[256];
  const float inv_n = 1.f / (float)n;
  double acc = 0.0;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n; r += (int64_t)gridDim.x * blockDim.x) {
    const T* row = z + r * classes;
    float m = -INFINITY;
    for (int k = 0; k < classes; ++k) m = fmaxf(m, ld(row + k));
    const int lab = labels[r];
    const bool ok = lab >= 0 && lab < classes;
    float s = 0.f, so = 0.f;  // as in k_softmax_nll
    for (int k = 0; k < classes; ++k) {
      const float e = expf(ld(row + k) - m);
      s += e;
      if (k != lab) so += e;
    }
    for (int k = 0; k < classes; ++k) {
      const float g = k == lab ? -so / s : expf(ld(row + k) - m) / s;
      st(dz + r * classes + k, g * inv_n);
    }
    double l = (double)NAN;
    if (ok) {
      const float zl = ld(row + lab);
      const float el = expf(zl - m);
      l = el > 0.f ? (double)log1pf(so / el) : (double)(m - zl) + (double)logf(s);
    }
    acc += l;
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double sum = 0.0;
    for (int i = 0; i < (int)blockDim.x; ++i) sum += red[i];
    partial[blockIdx.x] = sum;
  }
}

// One wavefront: lane l adds blocks l, l + 64, .. in order, then lane 0 adds
// the 64 lane sums in order.
__global__ __launch_bounds__(64) void k_loss_finalize(const double* __restrict__ partial, int blocks, int64_t n,
                                                      float* __restrict__ loss) {
  __shared__ double red[64];
  const int l = threadIdx.x;
  double a = 0.0;
  for (int b = l; b < blocks; b += 64) a += partial[b];
  red[l] = a;
  __syncthreads();
  if (l != 0) return;
  double s = 0.0;
  for (int i = 0; i < 64; ++i) s += red[i];
  loss[0] = (float)(s / (double)n);
}

// g' = g + wd p; buf = momentum buf + g'; p -= lr (g' + momentum buf).
__global__ void k_sgd_nesterov(float* __restrict__ p, const float* __restrict__ g, float* __restrict__ buf,
                               int64_t count, float lr, float momentum, float wd, uint16_t* __restrict__ p_bf16) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x) {
    const float gi = g[i] + wd * p[i];
    const float b = momentum * buf[i] + gi;
    buf[i] = b;
    const float np = p[i] - lr * (gi + momentum * b);
    p[i] = np;
    if (p_bf16) p_bf16[i] = f32_bf16_bits(np);
  }
}

unsigned grid_1d(int64_t total) {
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, 256), 8192));
}

int row_blocks(int64_t n) { return (int)std::max<int64_t>(1, std::min<int64_t>(ceil_div(n, 64), kMaxPartials)); }

sscn_status check_mat(const void* p, int64_t ld, int64_t n, int c, const char* what) {
  if (n < 0 || c < 1) return fail(SSCN_ERR_INVALID_ARG, std::string(what) + ": n must be >= 0 and c >= 1");
  if (n > 0 && !p) return fail(SSCN_ERR_INVALID_ARG, std::string(what) + " is NULL");
  if (ld < c) return fail(SSCN_ERR_INVALID_ARG, std::string(what) + ": row stride below the channel count");
  return SSCN_OK;
}

sscn_status check_dtype(sscn_dtype dtype) {
  if (dtype != SSCN_F32 && dtype != SSCN_BF16) return fail(SSCN_ERR_INVALID_ARG, "unknown dtype");
  return SSCN_OK;
}

// Whether the rows suit k_colreduce_vec: whole 16-byte pieces, at most 1024
// bytes, 16-byte aligned (both matrices).
bool colreduce_vec_ok(sscn_dtype dtype, const void* x, int64_t ldx, const void* da, int64_t ldd, int c) {
  const int e = dtype == SSCN_F32 ? 4 : 2;
  auto al = [&](const void* p, int64_t ld) { return !p || (reinterpret_cast<uintptr_t>(p) % 16 == 0 && ld * e % 16 == 0); };
  return (int64_t)c * e % 16 == 0 && (int64_t)c * e <= 1024 && al(x, ldx) && al(da, ldd);
}

template <int OP>
sscn_status colreduce(sscn_dtype dtype, const void* x, int64_t ldx, const void* da, int64_t ldd, int64_t n, int c,
                      const float* scale, const float* beta, const float* mean, const float* invstd, double* partial,
                      int blocks, hipStream_t s) {
  if (colreduce_vec_ok(dtype, x, ldx, da, ldd, c)) {
    const int64_t rpb = ceil_div(std::max<int64_t>(n, 1), blocks);
    if (dtype == SSCN_F32)
      k_colreduce_vec<float, OP><<<(unsigned)blocks, 256, 0, s>>>((const float*)x, ldx, (const float*)da, ldd, n, c,
                                                                  rpb, scale, beta, mean, invstd, partial);
    else
      k_colreduce_vec<uint16_t, OP><<<(unsigned)blocks, 256, 0, s>>>((const uint16_t*)x, ldx, (const uint16_t*)da,
                                                                     ldd, n, c, rpb, scale, beta, mean, invstd,
                                                                     partial);
    SSCN_HIP(hipGetLastError());
    return SSCN_OK;
  }
  const dim3 grid((unsigned)blocks, (unsigned)ceil_div(c, kColChunk));
  if (dtype == SSCN_F32)
    k_colreduce<float, OP><<<grid, 256, 0, s>>>((const float*)x, ldx, (const float*)da, ldd, n, c, scale, beta, mean,
                                                invstd, partial);
  else
    k_colreduce<uint16_t, OP><<<grid, 256, 0, s>>>((const uint16_t*)x, ldx, (const uint16_t*)da, ldd, n, c, scale,
                                                   beta, mean, invstd, partial);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

struct Partials {
  double* p = nullptr;
  hipStream_t s;
  explicit Partials(hipStream_t st) : s(st) {}
  sscn_status alloc(int blocks, int c) { return dev_alloc((void**)&p, sizeof(double) * 2 * (size_t)blocks * c, s); }
  ~Partials() { dev_free(p, s); }
};

}  // namespace
}  // namespace sscn

using namespace sscn;

extern "C" sscn_status sscn_batchnorm_forward(const void* x, int64_t ldx, int64_t n, int32_t c, sscn_dtype dtype,
                                              const float* gamma, const float* beta, float eps, float momentum,
                                              float* running_mean, float* running_var, float* mean, float* invstd,
                                              float* scale, float* shift, hipStream_t stream) {
  SSCN_TRY(check_dtype(dtype));
  SSCN_TRY(check_mat(x, ldx, n, c, "x"));
  if (n < 1) return fail(SSCN_ERR_INVALID_ARG, "batch statistics need at least one active site");
  if (!gamma || !beta || !mean || !invstd || !scale || !shift)
    return fail(SSCN_ERR_INVALID_ARG, "NULL gamma, beta, mean, invstd, scale or shift");
  if ((running_mean == nullptr) != (running_var == nullptr))
    return fail(SSCN_ERR_INVALID_ARG, "running_mean and running_var go together");
  if (!(eps > 0.f)) return fail(SSCN_ERR_INVALID_ARG, "eps must be positive");
  const int blocks = row_blocks(n);
  Partials part(stream);
  SSCN_TRY(part.alloc(blocks, c));
  SSCN_TRY(colreduce<kSumSquares>(dtype, x, ldx, nullptr, 0, n, c, nullptr, nullptr, nullptr, nullptr, part.p, blocks,
                                  stream));
  k_bn_finalize<<<(unsigned)ceil_div(c, 64), kFinThreads, 0, stream>>>(part.p, blocks, c, n, gamma, beta, eps, momentum,
                                                                running_mean, running_var, mean, invstd, scale, shift);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

extern "C" sscn_status sscn_batchnorm_relu_apply(const void* x, int64_t ldx, int64_t n, int32_t c, sscn_dtype dtype,
                                                 const float* mean, const float* scale, const float* beta, void* y,
                                                 int64_t ldy, hipStream_t stream) {
  SSCN_TRY(check_dtype(dtype));
  SSCN_TRY(check_mat(x, ldx, n, c, "x"));
  SSCN_TRY(check_mat(y, ldy, n, c, "y"));
  if (!mean || !scale || !beta) return fail(SSCN_ERR_INVALID_ARG, "NULL mean, scale or beta");
  if (n == 0) return SSCN_OK;
  if (rows_vec_ok(dtype, c, {{x, ldx}, {y, ldy}}))
    return rows_vec<0>(dtype, x, ldx, nullptr, 0, nullptr, 0, n, c, nullptr, mean, scale, beta, nullptr, nullptr,
                       nullptr, y, ldy, stream);
  const unsigned g = grid_1d(n * c);
  if (dtype == SSCN_F32)
    k_bn_relu_apply<float><<<g, 256, 0, stream>>>((const float*)x, ldx, n, c, mean, scale, beta, (float*)y, ldy);
  else
    k_bn_relu_apply<uint16_t><<<g, 256, 0, stream>>>((const uint16_t*)x, ldx, n, c, mean, scale, beta, (uint16_t*)y,
                                                     ldy);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

extern "C" sscn_status sscn_batchnorm_relu_backward_params(const void* da, int64_t ldd, const void* x, int64_t ldx,
                                                           int64_t n, int32_t c, sscn_dtype dtype, const float* mean,
                                                           const float* invstd, const float* scale, const float* beta,
                                                           float* dgamma, float* dbeta, hipStream_t stream) {
  SSCN_TRY(check_dtype(dtype));
  SSCN_TRY(check_mat(x, ldx, n, c, "x"));
  SSCN_TRY(check_mat(da, ldd, n, c, "dA"));
  if (!scale || !beta || !mean || !invstd || !dgamma || !dbeta)
    return fail(SSCN_ERR_INVALID_ARG, "NULL statistics or outputs");
  const int blocks = row_blocks(n);
  Partials part(stream);
  SSCN_TRY(part.alloc(blocks, c));
  SSCN_TRY(colreduce<kBnBack>(dtype, x, ldx, da, ldd, n, c, scale, beta, mean, invstd, part.p, blocks, stream));
  k_two_sums<<<(unsigned)ceil_div(c, 64), kFinThreads, 0, stream>>>(part.p, blocks, c, dbeta, dgamma);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

extern "C" sscn_status sscn_batchnorm_relu_backward_input(const void* da, int64_t ldd, const void* x, int64_t ldx,
                                                          int64_t n, int32_t c, sscn_dtype dtype, const float* gamma,
                                                          const float* beta, const float* mean, const float* invstd,
                                                          const float* scale, const float* dgamma, const float* dbeta,
                                                          const void* add, int64_t ld_add, void* dx, int64_t ldx_out,
                                                          hipStream_t stream) {
  SSCN_TRY(check_dtype(dtype));
  SSCN_TRY(check_mat(x, ldx, n, c, "x"));
  SSCN_TRY(check_mat(da, ldd, n, c, "dA"));
  SSCN_TRY(check_mat(dx, ldx_out, n, c, "dx"));
  if (add) SSCN_TRY(check_mat(add, ld_add, n, c, "add"));
  if (!gamma || !scale || !beta || !mean || !invstd || !dgamma || !dbeta)
    return fail(SSCN_ERR_INVALID_ARG, "NULL parameters or statistics");
  if (n == 0) return SSCN_OK;
  if (rows_vec_ok(dtype, c, {{da, ldd}, {x, ldx}, {add, ld_add}, {dx, ldx_out}}))
    return rows_vec<1>(dtype, da, ldd, x, ldx, add, ld_add, n, c, gamma, mean, scale, beta, invstd, dgamma, dbeta, dx,
                       ldx_out, stream);
  const unsigned g = grid_1d(n * c);
  if (dtype == SSCN_F32)
    k_bn_back_input<float><<<g, 256, 0, stream>>>((const float*)da, ldd, (const float*)x, ldx, n, c, gamma, scale,
                                                  beta, mean, invstd, dgamma, dbeta, (const float*)add, ld_add,
                                                  (float*)dx, ldx_out);
  else
    k_bn_back_input<uint16_t><<<g, 256, 0, stream>>>((const uint16_t*)da, ldd, (const uint16_t*)x, ldx, n, c, gamma,
                                                     scale, beta, mean, invstd, dgamma, dbeta, (const uint16_t*)add,
                                                     ld_add, (uint16_t*)dx, ldx_out);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

extern "C" sscn_status sscn_column_sum(const void* x, int64_t ldx, int64_t n, int32_t c, sscn_dtype dtype, float* out,
                                       hipStream_t stream) {
  SSCN_TRY(check_dtype(dtype));
  SSCN_TRY(check_mat(x, ldx, n, c, "x"));
  if (!out) return fail(SSCN_ERR_INVALID_ARG, "NULL out");
  const int blocks = row_blocks(n);
  Partials part(stream);
  SSCN_TRY(part.alloc(blocks, c));
  SSCN_TRY(colreduce<kSums>(dtype, x, ldx, nullptr, 0, n, c, nullptr, nullptr, nullptr, nullptr, part.p, blocks,
                            stream));
  k_two_sums<<<(unsigned)ceil_div(c, 64), kFinThreads, 0, stream>>>(part.p, blocks, c, out, nullptr);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

extern "C" sscn_status sscn_add(const void* a, int64_t lda, const void* b, int64_t ldb, int64_t n, int32_t c,
                                sscn_dtype dtype, void* y, int64_t ldy, hipStream_t stream) {
  SSCN_TRY(check_dtype(dtype));
  SSCN_TRY(check_mat(a, lda, n, c, "a"));
  SSCN_TRY(check_mat(b, ldb, n, c, "b"));
  SSCN_TRY(check_mat(y, ldy, n, c, "y"));
  if (n == 0) return SSCN_OK;
  if (rows_vec_ok(dtype, c, {{a, lda}, {b, ldb}, {y, ldy}}))
    return rows_vec<2>(dtype, a, lda, b, ldb, nullptr, 0, n, c, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                       nullptr, y, ldy, stream);
  const unsigned g = grid_1d(n * c);
  if (dtype == SSCN_F32)
    k_add<float><<<g, 256, 0, stream>>>((const float*)a, lda, (const float*)b, ldb, n, c, (float*)y, ldy);
  else
    k_add<uint16_t><<<g, 256, 0, stream>>>((const uint16_t*)a, lda, (const uint16_t*)b, ldb, n, c, (uint16_t*)y, ldy);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

extern "C" sscn_status sscn_softmax_nll(const void* logits, int64_t n, int32_t classes, sscn_dtype dtype,
                                        const int32_t* labels, float* loss, void* dlogits, hipStream_t stream) {
  SSCN_TRY(check_dtype(dtype));
  SSCN_TRY(check_mat(logits, classes, n, classes, "logits"));
  if (n < 1) return fail(SSCN_ERR_INVALID_ARG, "the loss needs at least one active site");
  if (!labels || !loss || !dlogits) return fail(SSCN_ERR_INVALID_ARG, "NULL labels, loss or dlogits");
  const bool per_row = classes <= kSoftmaxRowMax;
  const int blocks = (int)std::max<int64_t>(1, std::min<int64_t>(ceil_div(n, per_row ? 256 : 4), kMaxPartials));
  Partials part(stream);
  SSCN_TRY(part.alloc(blocks, 1));
  if (per_row) {
    if (dtype == SSCN_F32)
      k_softmax_nll_rows<float><<<(unsigned)blocks, 256, 0, stream>>>((const float*)logits, n, classes, labels,
                                                                      (float*)dlogits, part.p);
    else
      k_softmax_nll_rows<uint16_t><<<(unsigned)blocks, 256, 0, stream>>>((const uint16_t*)logits, n, classes, labels,
                                                                         (uint16_t*)dlogits, part.p);
  } else if (dtype == SSCN_F32)
    k_softmax_nll<float><<<(unsigned)blocks, 256, 0, stream>>>((const float*)logits, n, classes, labels,
                                                               (float*)dlogits, part.p);
  else
    k_softmax_nll<uint16_t><<<(unsigned)blocks, 256, 0, stream>>>((const uint16_t*)logits, n, classes, labels,
                                                                  (uint16_t*)dlogits, part.p);
  SSCN_HIP(hipGetLastError());
  k_loss_finalize<<<1, 64, 0, stream>>>(part.p, blocks, n, loss);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

extern "C" sscn_status sscn_sgd_nesterov(float* params, const float* grads, float* momentum_buf, int64_t count,
                                         float lr, float momentum, float weight_decay, void* params_bf16,
                                         hipStream_t stream) {
  if (count < 0) return fail(SSCN_ERR_INVALID_ARG, "count must be >= 0");
  if (count == 0) return SSCN_OK;
  if (!params || !grads || !momentum_buf) return fail(SSCN_ERR_INVALID_ARG, "NULL params, grads or momentum buffer");
  k_sgd_nesterov<<<grid_1d(count), 256, 0, stream>>>(params, grads, momentum_buf, count, lr, momentum, weight_decay,
                                                     (uint16_t*)params_bf16);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}
