// Pooling and upsampling over SC(f, s) connections (Sec. 4.1 "Other
// operators": MP takes the maximum of the zero vector and the active input
// vectors of a receptive field, AP f^-d times their sum; Sec. 5: the FCN
// upsamples by nearest neighbour).  All of them, and their gradients, are
// reductions over the pairs of a rule book direction:
//
//   AP forward      sum over the SC direction, scale f^-d (1 / K)
//   AP backward     sum over the transposed direction, scale f^-d
//   MP forward      max over the SC direction (records the winning offset)
//   MP backward     over the transposed direction: the gradient of an
//                   output element goes to the input at its winning offset
//   upsample        sum over the transposed direction (one pair per row, f = s)
//   its backward    sum over the SC direction
//
// One output-stationary kernel covers all of them: a workgroup owns 64
// output rows (one tile of the direction's storage) and 64 channels, keeps
// them in LDS, and walks the direction's offsets in order; within one
// offset every output row has at most one pair, so the four wavefronts
// take the offset's pairs in turn without conflicts, with one barrier per
// offset.  Each output element is written once: no atomics, deterministic.
// Memory-bound: every pair reads one input row piece (256 B per wavefront
// for fp32), every output row is written once.
#include "internal.h"
#include "numeric.h"

namespace sscn {

namespace {

enum PoolMode { kSum = 0, kMax = 1, kMaxBack = 2 };
constexpr int kPoolCols = 64;
constexpr uint8_t kNoArg = 255;  // the zero vector is the maximum

// X: rows of the direction's input side (n_in x c); arg_in (kMaxBack): the
// forward's winning offsets, indexed like X.  Y: n_out x c; arg_out (kMax):
// n_out x c winning offsets.
template <typename T, int MODE>
__global__ __launch_bounds__(256) void k_pool(const T* __restrict__ X, const uint8_t* __restrict__ arg_in,
                                              const int64_t* __restrict__ seg, int64_t n_tiles,
                                              const int32_t* __restrict__ in_rows, const int32_t* __restrict__ out_rows,
                                              int K, int mirror, int64_t n_out, int c, float scale, T* __restrict__ Y,
                                              uint8_t* __restrict__ arg_out) {
  __shared__ float acc[kPlanRows][kPoolCols];
  __shared__ uint8_t arg[kPlanRows][kPoolCols];
  const int64_t t = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = blockIdx.y * kPoolCols + lane;
  const bool live = col < c;
  const int64_t row0 = t * kPlanRows;
  for (int r = wave; r < kPlanRows; r += 4) {
    acc[r][lane] = 0.f;
    arg[r][lane] = kNoArg;
  }
  __syncthreads();
  for (int o = 0; o < K; ++o) {
    const int so = mirror ? K - 1 - o : o;
    const int64_t p0 = seg[(int64_t)so * n_tiles + t], p1 = seg[(int64_t)so * n_tiles + t + 1];
    for (int64_t p = p0 + wave; p < p1; p += 4) {
      const int64_t j = in_rows[p];
      const int r = (int)(out_rows[p] - row0);
      if (!live) continue;
      const float v = ld(X + j * c + col);
      if constexpr (MODE == kSum) {
        acc[r][lane] += v;
      } else if constexpr (MODE == kMax) {
        if (v > acc[r][lane]) {
          acc[r][lane] = v;
          arg[r][lane] = (uint8_t)o;
        }
      } else {
        if (arg_in[j * c + col] == (uint8_t)o) acc[r][lane] += v;
      }
    }
    __syncthreads();
  }
  if (!live) return;
  for (int r = wave; r < kPlanRows; r += 4) {
    const int64_t row = row0 + r;
    if (row >= n_out) break;
    st(Y + row * c + col, MODE == kSum ? acc[r][lane] * scale : acc[r][lane]);
    if constexpr (MODE == kMax) arg_out[row * c + col] = arg[r][lane];
  }
}

template <typename T, int MODE>
sscn_status launch_pool(const View& v, const void* X, const uint8_t* arg_in, int c, float scale, void* Y,
                        uint8_t* arg_out, hipStream_t s) {
  const int64_t tiles = v.st->n_tiles;
  if (tiles == 0) return SSCN_OK;
  if (tiles > 0x7fffffff) return fail(SSCN_ERR_INVALID_ARG, "too many output rows");
  const dim3 grid((unsigned)tiles, (unsigned)ceil_div(c, kPoolCols));
  k_pool<T, MODE><<<grid, 256, 0, s>>>((const T*)X, arg_in, v.st->seg, tiles, v.st->in_rows, v.st->out_rows, v.K,
                                       v.mirror ? 1 : 0, v.n_out, c, scale, (T*)Y, arg_out);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

template <int MODE>
sscn_status launch_pool_t(sscn_dtype dtype, const View& v, const void* X, const uint8_t* arg_in, int c, float scale,
                          void* Y, uint8_t* arg_out, hipStream_t s) {
  if (dtype == SSCN_F32) return launch_pool<float, MODE>(v, X, arg_in, c, scale, Y, arg_out, s);
  return launch_pool<uint16_t, MODE>(v, X, arg_in, c, scale, Y, arg_out, s);
}

sscn_status check_pool(sscn_rulebook rb, int32_t c, sscn_dtype dtype) {
  if (!rb) return fail(SSCN_ERR_INVALID_ARG, "NULL rule book");
  if (c < 1 || c > 65536) return fail(SSCN_ERR_INVALID_ARG, "channel count must be in [1, 65536]");
  if (dtype != SSCN_F32 && dtype != SSCN_BF16) return fail(SSCN_ERR_INVALID_ARG, "unknown dtype");
  if (rb->d->submanifold) return fail(SSCN_ERR_INVALID_ARG, "pooling and upsampling take an SC(f, s) rule book");
  if (rb->transposed) return fail(SSCN_ERR_INVALID_ARG, "pass the SC rule book itself, not its transpose");
  return SSCN_OK;
}

View direction(sscn_rulebook rb, bool transposed) {
  sscn_rulebook_s t{rb->d, transposed};
  return view_of(&t);
}

}  // namespace
}  // namespace sscn

using namespace sscn;

extern "C" sscn_status sscn_pool_forward(const void* features, sscn_rulebook rb, int32_t c, sscn_dtype dtype,
                                         sscn_pool_mode mode, void* out, uint8_t* argmax, hipStream_t stream) {
  SSCN_TRY(check_pool(rb, c, dtype));
  if (mode != SSCN_POOL_MAX && mode != SSCN_POOL_AVG) return fail(SSCN_ERR_INVALID_ARG, "unknown pooling mode");
  const RulebookData* d = rb->d;
  if (mode == SSCN_POOL_MAX && d->K >= kNoArg) return fail(SSCN_ERR_INVALID_ARG, "max pooling takes at most 254 offsets");
  if (d->n_out == 0) return SSCN_OK;
  if (!out || (d->n_in > 0 && !features) || (mode == SSCN_POOL_MAX && !argmax))
    return fail(SSCN_ERR_INVALID_ARG, "NULL features, out or argmax");
  UseNote note{rb->d, stream};
  const View v = direction(rb, false);
  if (mode == SSCN_POOL_AVG)
    return launch_pool_t<kSum>(dtype, v, features, nullptr, c, 1.0f / (float)d->K, out, nullptr, stream);
  return launch_pool_t<kMax>(dtype, v, features, nullptr, c, 1.0f, out, argmax, stream);
}

extern "C" sscn_status sscn_pool_backward(const void* dout, const uint8_t* argmax, sscn_rulebook rb, int32_t c,
                                          sscn_dtype dtype, sscn_pool_mode mode, void* dgrad, hipStream_t stream) {
  SSCN_TRY(check_pool(rb, c, dtype));
  if (mode != SSCN_POOL_MAX && mode != SSCN_POOL_AVG) return fail(SSCN_ERR_INVALID_ARG, "unknown pooling mode");
  const RulebookData* d = rb->d;
  if (mode == SSCN_POOL_MAX && d->K >= kNoArg) return fail(SSCN_ERR_INVALID_ARG, "max pooling takes at most 254 offsets");
  if (d->n_in == 0) return SSCN_OK;
  if (!dgrad || (d->n_out > 0 && !dout) || (mode == SSCN_POOL_MAX && d->n_out > 0 && !argmax))
    return fail(SSCN_ERR_INVALID_ARG, "NULL dout, dgrad or argmax");
  UseNote note{rb->d, stream};
  const View v = direction(rb, true);
  if (mode == SSCN_POOL_AVG)
    return launch_pool_t<kSum>(dtype, v, dout, nullptr, c, 1.0f / (float)d->K, dgrad, nullptr, stream);
  return launch_pool_t<kMaxBack>(dtype, v, dout, argmax, c, 1.0f, dgrad, nullptr, stream);
}

extern "C" sscn_status sscn_upsample_forward(const void* features, sscn_rulebook rb, int32_t c, sscn_dtype dtype,
                                             void* out, hipStream_t stream) {
  SSCN_TRY(check_pool(rb, c, dtype));
  const RulebookData* d = rb->d;
  if (d->f != d->stride) return fail(SSCN_ERR_INVALID_ARG, "nearest-neighbour upsampling inverts an SC(s, s) rule book");
  if (d->n_in == 0) return SSCN_OK;
  if (!out || (d->n_out > 0 && !features)) return fail(SSCN_ERR_INVALID_ARG, "NULL features or out");
  UseNote note{rb->d, stream};
  return launch_pool_t<kSum>(dtype, direction(rb, true), features, nullptr, c, 1.0f, out, nullptr, stream);
}

extern "C" sscn_status sscn_upsample_backward(const void* dout, sscn_rulebook rb, int32_t c, sscn_dtype dtype,
                                              void* dgrad, hipStream_t stream) {
  SSCN_TRY(check_pool(rb, c, dtype));
  const RulebookData* d = rb->d;
  if (d->f != d->stride) return fail(SSCN_ERR_INVALID_ARG, "nearest-neighbour upsampling inverts an SC(s, s) rule book");
  if (d->n_out == 0) return SSCN_OK;
  if (!dgrad || (d->n_in > 0 && !dout)) return fail(SSCN_ERR_INVALID_ARG, "NULL dout or dgrad");
  UseNote note{rb->d, stream};
  return launch_pool_t<kSum>(dtype, direction(rb, false), dout, nullptr, c, 1.0f, dgrad, nullptr, stream);
}
