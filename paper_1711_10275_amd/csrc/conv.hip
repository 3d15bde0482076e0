// Sparse convolution arithmetic (Sec. 4.2 step 2 of the paper): per filter
// offset o, a gather of input rows, a dense (pairs x C_in) x (C_in x C_out)
// product with W^o, and a scatter-add into output rows.
//
// Forward and dgrad share one output-stationary kernel (k_conv_quad).  A
// workgroup owns one 64-row output tile and 64 output columns; the tile's
// pairs are processed in chunks of 16 pairs of one offset, and every
// chunk's 16x64 result is added into an fp32 accumulator tile in LDS at the
// pairs' output rows (within one offset an output row occurs at most once).
// The tile is written to HBM once, after its last chunk.  A generic kernel
// (k_gather_mma) covers channel counts the main kernel does not.
//
// wgrad: dW^o = X[in_o]^T dY[out_o], per-offset gathered contractions with
// fp32 MFMAs, split over pairs and reduced with fp32 atomics.
#include <algorithm>
#include <cstdlib>

#include <hip/hip_ext.h>

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

// Destinations of a layer's output: up to two, each with its own row stride
// and an optional per-column affine map followed by ReLU (the next unit's
// pre-activation), rounded once to T.
template <typename T>
struct Heads {
  T* out[2];
  int64_t ld[2];
  const float* scale[2];
  const float* shift[2];
  int n;
  // a buffer the row kernel clears on the side (the backward's dW, which the
  // wgrad kernel after it accumulates into), n_zero floats; 0: none
  float* zero;
  int64_t n_zero;
  // the layer's bias (c_out fp32, nullable) and a residual (n_out x c_out in
  // T, row stride res_ld, nullable): added to every output row before the
  // heads map it
  const float* bias;
  const T* res;
  int64_t res_ld;
  __device__ __forceinline__ void store(int64_t row, int col, float v) const {
    if (bias) v += bias[col];
    if (res) v += Elem<T>::load(res + row * res_ld + col);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (h < n) {
        const float a = scale[h] ? fmaxf(0.f, v * scale[h][col] + shift[h][col]) : v;
        Elem<T>::store(out[h] + row * ld[h] + col, a);
      }
    }
  }
};
template <typename T>
static Heads<T> plain_heads(T* Y, int cout) {
  Heads<T> h{};
  h.out[0] = Y;
  h.ld[0] = cout;
  h.n = 1;
  return h;
}

// ------------------------------------------------------- generic fallback
// 16 consecutive values of a row (zero beyond kmax) as MFMA operands.
__device__ __forceinline__ void load16(const float* __restrict__ row, int k0, int kmax, float (&v)[16]) {
#pragma unroll
  for (int i = 0; i < 16; ++i) v[i] = (k0 + i < kmax) ? row[k0 + i] : 0.f;
}
__device__ __forceinline__ void load16(const bf16_t* __restrict__ row, int k0, int kmax, bf16x8 (&v)[2]) {
  uint32_t t[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) t[i] = (k0 + i < kmax) ? row[k0 + i].bits : 0u;
  uint4 a, b;
  a.x = t[0] | (t[1] << 16);   a.y = t[2] | (t[3] << 16);
  a.z = t[4] | (t[5] << 16);   a.w = t[6] | (t[7] << 16);
  b.x = t[8] | (t[9] << 16);   b.y = t[10] | (t[11] << 16);
  b.z = t[12] | (t[13] << 16); b.w = t[14] | (t[15] << 16);
  v[0] = __builtin_bit_cast(bf16x8, a);
  v[1] = __builtin_bit_cast(bf16x8, b);
}

// D += A B^T over 64 reduction indices held 16 per lane.  Lane l supplies
// row (l % 16) of A and of B; its 16 values are the reduction indices
// 16*(l/16) + [0, 16) of a 64-wide block.  Any fixed assignment of
// reduction indices to (instruction, lane group) gives the same sum.
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

// Any channel counts.  Workgroup = NW wavefronts over 128 output rows; each
// wavefront owns 16 output columns and walks all of the tile's pairs 16 at a
// time, accumulating into an LDS tile (rows x (16 NW + 1)).
// X: n_in x cin rows; Bt: K x cout x cin (row n = the cin weights feeding
// output column n); Y: n_out x cout.
template <typename T, int NW>
__global__ __launch_bounds__(NW * 64) void k_gather_mma(
    const T* __restrict__ X, const T* __restrict__ Bt, const int64_t* __restrict__ seg,
    const int32_t* __restrict__ in_rows, const int32_t* __restrict__ out_rows, int64_t n_tiles, int K,
    int mirror, int cin, int cout, int64_t n_out, int tpw, Heads<T> Y) {
  extern __shared__ float acc[];
  constexpr int WCOLS = 16 * NW;
  constexpr int LDW = WCOLS + 1;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int64_t t0 = (int64_t)blockIdx.x * tpw;
  const int64_t t1 = min<int64_t>(t0 + tpw, n_tiles);
  const int64_t row0 = t0 * kTile;
  const int rows = tpw * kTile;
  const int col_base = blockIdx.y * WCOLS;
  const int col = col_base + wave * 16 + m;
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
        load16(arow, kb + 16 * g, pv ? cin : 0, a);
        load16(brow, kb + 16 * g, col_ok ? cin : 0, b);
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
    if (row < n_out && cc < cout) Y.store(row, cc, acc[r * LDW + c]);
  }
}

// ------------------------------------------------------------- main path
// Raw buffer loads: a 32-bit offset from a scalar base, with out-of-range
// offsets reading as zero (used to mask lanes without branches).
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOobOffset = 0x70000000u;  // >= any buffer size accepted on this path
// LDS bytes per row of a bf16 weight-part plane of the split row kernel
// (32 channels = 64 bytes, padded against bank conflicts).
// Weight tiles of the row kernel that arrive by direct-to-LDS loads: one
// row of CPR 16-byte chunks (4 or 8) per output column (and, for the split
// path, per bf16 plane), without padding; chunk k of row r is stored in slot
// k ^ swizzle(r mod 16).  An MFMA operand read takes the same chunk of 16
// consecutive rows.  The swizzles are the ones with the fewest LDS
// bank-conflict cycles in a sweep on the hardware (SQ_LDS_BANK_CONFLICT):
// for 8-chunk rows r mod 8 (0.02 conflict cycles per LDS cycle with the
// row tiles' 32-byte padding, against 2.55 unswizzled and 1.19 for
// (r ^ r / 8) mod 8), for 4-chunk rows (r / 2 ^ r / 4) mod 4 (0.25, against
// 1.66 for r mod 4).
template <int CPR>
__device__ __forceinline__ int tile_slot(int row, int chunk) {
  static_assert(CPR == 4 || CPR == 8, "chunks per tile row");
  const int m = row & 15;
  return chunk ^ (CPR == 4 ? ((m >> 1) ^ (m >> 2)) & 3 : m & 7);
}

__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// 8 consecutive channels of one row: a lane's operand for one column block.
template <typename T> struct Oct;
template <> struct Oct<float> {
  float v[8];
  __device__ __forceinline__ void load(rsrc_t r, uint32_t voff, uint32_t soff) {
    const auto a = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
    const auto b = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(voff + 16), (int)soff, 0);
    v[0] = __uint_as_float(a[0]); v[1] = __uint_as_float(a[1]); v[2] = __uint_as_float(a[2]); v[3] = __uint_as_float(a[3]);
    v[4] = __uint_as_float(b[0]); v[5] = __uint_as_float(b[1]); v[6] = __uint_as_float(b[2]); v[7] = __uint_as_float(b[3]);
  }
};
template <> struct Oct<bf16_t> {
  bf16x8 v;
  __device__ __forceinline__ void load(rsrc_t r, uint32_t voff, uint32_t soff) {
    const auto a = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
    uint4 u;
    u.x = a[0]; u.y = a[1]; u.z = a[2]; u.w = a[3];
    v = __builtin_bit_cast(bf16x8, u);
  }
};
// The same operand gathered with a stride of `step` bytes between the 8
// channels (weights stored [offset][c_in][c_out], read along c_in).
__device__ __forceinline__ void load_strided(Oct<float>& o, rsrc_t r, uint32_t voff, uint32_t step, uint32_t soff) {
#pragma unroll
  for (int i = 0; i < 8; ++i)
    o.v[i] = __uint_as_float((uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)(voff + i * step), (int)soff, 0));
}
__device__ __forceinline__ void load_strided(Oct<bf16_t>& o, rsrc_t r, uint32_t voff, uint32_t step, uint32_t soff) {
  uint32_t t[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) t[i] = (uint16_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)(voff + i * step), (int)soff, 0);
  uint4 u;
  u.x = t[0] | (t[1] << 16); u.y = t[2] | (t[3] << 16); u.z = t[4] | (t[5] << 16); u.w = t[6] | (t[7] << 16);
  o.v = __builtin_bit_cast(bf16x8, u);
}

__device__ __forceinline__ f32x4 mma_oct(const Oct<float>& a, const Oct<float>& b, f32x4 d) {
#pragma unroll
  for (int i = 0; i < 8; ++i) d = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[i], b.v[i], d, 0, 0, 0);
  return d;
}
__device__ __forceinline__ f32x4 mma_oct(const Oct<bf16_t>& a, const Oct<bf16_t>& b, f32x4 d) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, d, 0, 0, 0);
}

// An operand (8 channels) from LDS.
__device__ __forceinline__ void lds_oct(Oct<float>& o, const char* p) {
  const uint4 x = *reinterpret_cast<const uint4*>(p);
  const uint4 y = *reinterpret_cast<const uint4*>(p + 16);
  o.v[0] = __uint_as_float(x.x); o.v[1] = __uint_as_float(x.y); o.v[2] = __uint_as_float(x.z); o.v[3] = __uint_as_float(x.w);
  o.v[4] = __uint_as_float(y.x); o.v[5] = __uint_as_float(y.y); o.v[6] = __uint_as_float(y.z); o.v[7] = __uint_as_float(y.w);
}
// The same from two 16-byte chunks at p0 and p1 (bf16: p0 holds all 8).
__device__ __forceinline__ void lds_oct2(Oct<float>& o, const char* p0, const char* p1) {
  const uint4 x = *reinterpret_cast<const uint4*>(p0);
  const uint4 y = *reinterpret_cast<const uint4*>(p1);
  o.v[0] = __uint_as_float(x.x); o.v[1] = __uint_as_float(x.y); o.v[2] = __uint_as_float(x.z); o.v[3] = __uint_as_float(x.w);
  o.v[4] = __uint_as_float(y.x); o.v[5] = __uint_as_float(y.y); o.v[6] = __uint_as_float(y.z); o.v[7] = __uint_as_float(y.w);
}
__device__ __forceinline__ void lds_oct2(Oct<bf16_t>& o, const char* p0, const char*) {
  o.v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p0));
}
__device__ __forceinline__ void lds_oct(Oct<bf16_t>& o, const char* p) {
  o.v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

// LDS layout of k_conv_quad (bytes, each part 16-byte aligned).
struct QuadLds {
  size_t acc, prow, pacc, chof, seg_s, seg_n, seg_c0, total;
  __host__ __device__ QuadLds(int max_chunks, int K) {
    auto up = [](size_t x) __host__ __device__ { return (x + 15) & ~(size_t)15; };
    acc = 0;
    prow = up(acc + sizeof(float) * 2 * (kTile + 1) * 65);
    pacc = up(prow + sizeof(uint32_t) * max_chunks * 16);
    chof = up(pacc + sizeof(uint16_t) * max_chunks * 16);
    seg_s = up(chof + sizeof(int16_t) * max_chunks);
    seg_n = up(seg_s + sizeof(int64_t) * K);
    seg_c0 = up(seg_n + sizeof(int32_t) * K);
    total = up(seg_c0 + sizeof(int32_t) * K);
  }
};

// Main forward / dgrad kernel: c_in % 8 == 0, c_in <= 64 KB, any c_out
// (64 columns per workgroup row of the grid).
//
// Workgroup = 8 / NB wavefronts over one 64-row output tile and 64 output
// columns (NB = column blocks of 16 per wavefront; the library uses NB = 2,
// 4 wavefronts: with NB = 4 a workgroup has half the wavefronts for the same
// LDS, which halves occupancy).  Wavefront w takes input-channel half
// kh = w & 1 of every 64-channel block and, for NB = 2, output-column half
// ch = w >> 1: per chunk of 16 pairs it multiplies the pairs' gathered
// channels by a (32 KB) x 16 NB weight block.  At the start of a tile the workgroup lists its chunks
// (offset-major) and stores, per pair slot, the byte offset of the gathered
// row and the LDS offset of the output row, so the main loop does almost
// no address arithmetic.  Loads are raw buffer loads: a lane's offset
// within the row and its weight column are constants, the filter offset is
// a scalar offset, and masked lanes use an out-of-range offset that reads as
// zero.  Weights are read either from the stored layout W[o][c_in][c_out]
// (WT = false: a lane's 8 channels are c_out apart) or from a layout with
// c_in contiguous (WT = true, dgrad: W[o] read transposed).  The loop runs
// a RING-slot register ring with straight-line code:
// the gathered fragment of chunk c + RING - 1 is requested while chunk c is
// multiplied, and weights are requested only for the first chunk of each
// offset and kept in registers for the rest.  Partial sums of the two
// channel halves go to two LDS accumulators (each element has one writing
// wavefront, updated in chunk order) that are added at the end: the result
// is deterministic.  The workgroups are persistent.  The grid is a multiple
// of kTileGroups; workgroup b serves tile group b % kTileGroups (one group
// of contiguous tiles per XCD, as workgroups are dispatched round-robin over
// the XCDs), and the group's tiles, listed by decreasing work, are dealt to
// its workgroups in boustrophedon order (0..G-1, G-1..0, ...).
template <typename T, int RING, int KB, bool WT, int NB>
__global__ __launch_bounds__(256) void k_conv_quad(
    const T* __restrict__ X, uint32_t x_bytes, const T* __restrict__ W, uint32_t w_bytes,
    const int64_t* __restrict__ seg, const int32_t* __restrict__ in_rows, const int32_t* __restrict__ out_rows,
    const int32_t* __restrict__ order, int64_t n_tiles, int K, int mirror, int cin, int cout, int64_t n_out,
    int max_chunks, Heads<T> Y) {
  constexpr int LDW = 64 + 1;
  constexpr int ACC = (kTile + 1) * LDW;  // 64 rows + one dummy row for masked lanes
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const QuadLds L(max_chunks, K);
  float* acc_all = reinterpret_cast<float*>(smem + L.acc);     // [2][65][LDW]
  uint32_t* prow = reinterpret_cast<uint32_t*>(smem + L.prow);  // [max_chunks * 16] row byte offsets
  uint16_t* pacc = reinterpret_cast<uint16_t*>(smem + L.pacc);  // [max_chunks * 16] LDS row offsets
  int16_t* chof = reinterpret_cast<int16_t*>(smem + L.chof);    // [max_chunks] offset per chunk
  int64_t* seg_s = reinterpret_cast<int64_t*>(smem + L.seg_s);  // [K]
  int32_t* seg_n = reinterpret_cast<int32_t*>(smem + L.seg_n);  // [K]
  int32_t* seg_c0 = reinterpret_cast<int32_t*>(smem + L.seg_c0);  // [K]
  __shared__ int n_chunks_sh;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  constexpr int NWB = 8 / NB;             // wavefronts per workgroup
  constexpr int NT = 64 * NWB;             // threads per workgroup
  static_assert(NB == 2 || NB == 4, "2 or 4 column blocks per wavefront");
  const int kh = wave & 1, chf = NB == 2 ? wave >> 1 : 0;
  const int col_base = blockIdx.y * 64;
  const uint32_t row_bytes = (uint32_t)cin * (uint32_t)sizeof(T);
  // lane constants: channel octets of the gathered row, weight columns
  uint32_t a_lane[KB], b_lane[KB][NB];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
    const int k0 = kb * 64 + kh * 32 + 8 * g;
    const bool k_in = k0 + 8 <= cin;
    a_lane[kb] = k_in ? (uint32_t)k0 * sizeof(T) : kOobOffset;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int col = col_base + chf * 16 * NB + nb * 16 + m;
      const uint32_t e = WT ? (uint32_t)col * cin + k0 : (uint32_t)k0 * cout + col;  // element of W[o]
      b_lane[kb][nb] = (col < cout && k_in) ? e * (uint32_t)sizeof(T) : kOobOffset;
    }
  }
  const uint32_t w_stride = (uint32_t)cout * cin * sizeof(T);  // bytes per filter offset
  const uint32_t k_step = (uint32_t)cout * sizeof(T);           // bytes between channels (WT = false)
  const rsrc_t rx = make_rsrc(X, x_bytes), rb = make_rsrc(W, w_bytes);
  char* acc_lane = reinterpret_cast<char*>(acc_all + kh * ACC + chf * 16 * NB + m);

  const int64_t grp = blockIdx.x % kTileGroups;
  const int64_t G = gridDim.x / kTileGroups, b = blockIdx.x / kTileGroups;
  const int64_t first = (grp * n_tiles + kTileGroups - 1) / kTileGroups;
  const int64_t count = ((grp + 1) * n_tiles + kTileGroups - 1) / kTileGroups - first;
  for (int64_t idx = b, round = 0; idx < count; ++round, idx = round * G + ((round & 1) ? G - 1 - b : b)) {
    __syncthreads();  // the previous tile's LDS is free
    const int64_t t0 = order[first + idx];
    const int64_t row0 = t0 * kTile;

    // segment starts, pair counts and first chunk per offset; chunk -> offset
    if (wave == 0) {
      int base = 0;
      for (int ob = 0; ob < K; ob += 64) {
        const int o = ob + lane;
        int64_t s = 0, e = 0;
        int nc = 0;
        if (o < K) {
          const int so = mirror ? K - 1 - o : o;
          s = seg[(int64_t)so * n_tiles + t0];
          e = seg[(int64_t)so * n_tiles + t0 + 1];
          nc = (int)((e - s + 15) >> 4);
        }
        int x = nc;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
          const int y = __shfl_up(x, d, 64);
          if (lane >= d) x += y;
        }
        if (o < K) {
          const int c0 = base + x - nc;
          seg_s[o] = s;
          seg_n[o] = (int)(e - s);
          seg_c0[o] = c0;
          for (int c = 0; c < nc; ++c) chof[c0 + c] = (int16_t)o;
        }
        base += __shfl(x, 63, 64);
      }
      if (lane == 0) n_chunks_sh = base;
    }
    for (int i = threadIdx.x; i < 2 * ACC; i += blockDim.x) acc_all[i] = 0.f;
    __syncthreads();
    const int n_chunks = n_chunks_sh;
    // pair slots (16 per chunk): gathered-row byte offset (out of range when
    // the slot is empty) and LDS byte offset of the output row (dummy row when
    // empty).  Each thread issues all of its index loads before writing.
    {
      constexpr int PER = 8;
      for (int q0 = 0; q0 < n_chunks * 16; q0 += NT * PER) {
        int32_t vi[PER], vo[PER];
        bool ok[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const int q = q0 + u * NT + threadIdx.x;
          const bool live = q < n_chunks * 16;
          const int o = chof[live ? q >> 4 : 0];
          const int j = q - seg_c0[o] * 16;
          ok[u] = live && j < seg_n[o];
          const int64_t pp = ok[u] ? seg_s[o] + j : 0;
          vi[u] = in_rows[pp];
          vo[u] = out_rows[pp];
        }
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const int q = q0 + u * NT + threadIdx.x;
          if (q < n_chunks * 16) {
            prow[q] = ok[u] ? (uint32_t)vi[u] * row_bytes : kOobOffset;
            pacc[q] = (uint16_t)(((ok[u] ? (int)(vo[u] - row0) : kTile) * LDW) * 4);
          }
        }
      }
    }
    __syncthreads();

    if (n_chunks > 0) {
      Oct<T> a_ring[RING][KB], b_ring[RING][KB][NB], b_cur[KB][NB];
      // weights are requested only for the first chunk of each offset
      auto fresh_at = [&](int c) -> bool {
        const int cc = c < n_chunks ? c : n_chunks - 1;
        const int f = (cc == 0 || chof[cc - 1] != chof[cc]) ? 1 : 0;
        return __builtin_amdgcn_readfirstlane(f) != 0;
      };
      auto request = [&](int c, int slot) {
        const int cc = c < n_chunks ? c : n_chunks - 1;
        const uint32_t rowoff = prow[cc * 16 + m];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) a_ring[slot][kb].load(rx, rowoff + a_lane[kb], 0);
        if (fresh_at(c)) {
          const int o = __builtin_amdgcn_readfirstlane((int)chof[cc]);
          const uint32_t soff = (uint32_t)o * w_stride;
#pragma unroll
          for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
              if constexpr (WT)
                b_ring[slot][kb][nb].load(rb, b_lane[kb][nb], soff);
              else
                load_strided(b_ring[slot][kb][nb], rb, b_lane[kb][nb], k_step, soff);
            }
        }
      };
#pragma unroll
      for (int q = 0; q < RING - 1; ++q) request(q, q);
      // lane holds D[4g + r][m]: pair 4g + r, column chf*32 + nb*16 + m.  One
      // writer per element: plain read-modify-write; empty slots hit the dummy
      // row.  A chunk's sum is added one step later, after the next chunk's
      // MFMAs are issued, so the LDS round trip overlaps matrix work.
      constexpr uint32_t kDummy = (uint32_t)(kTile * LDW * 4);
      f32x4 dp[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) dp[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      uint2 rows_prev = make_uint2(kDummy | (kDummy << 16), kDummy | (kDummy << 16));
      auto add_prev = [&]() {
        const uint32_t ra[4] = {rows_prev.x & 0xffffu, rows_prev.x >> 16, rows_prev.y & 0xffffu,
                                rows_prev.y >> 16};
        float old[NB][4];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int r = 0; r < 4; ++r) old[nb][r] = *reinterpret_cast<const float*>(acc_lane + ra[r] + nb * 64);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int r = 0; r < 4; ++r) *reinterpret_cast<float*>(acc_lane + ra[r] + nb * 64) = old[nb][r] + dp[nb][r];
      };
      auto step = [&](int c, int slot) {
        request(c + RING - 1, (slot + RING - 1) % RING);
        if (fresh_at(c)) {
          // a real (uniform) branch: the copy runs only when the offset
          // changes, instead of a select per register on every chunk
          asm volatile("");
#pragma unroll
          for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) b_cur[kb][nb] = b_ring[slot][kb][nb];
        }
        f32x4 d[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) d[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) d[nb] = mma_oct(a_ring[slot][kb], b_cur[kb][nb], d[nb]);
        add_prev();
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) dp[nb] = d[nb];
        rows_prev = *reinterpret_cast<const uint2*>(&pacc[c * 16 + 4 * g]);
      };
      int c = 0;
      for (; c + RING <= n_chunks; c += RING) {
#pragma unroll
        for (int q = 0; q < RING; ++q) step(c + q, q);
      }
#pragma unroll
      for (int q = 0; q < RING - 1; ++q)
        if (c + q < n_chunks) step(c + q, q);
      add_prev();
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kTile * 64; i += blockDim.x) {
      const int r = i >> 6, cc = i & 63;
      const int64_t row = row0 + r;
      const int col = col_base + cc;
      if (row < n_out && col < cout)
        Y.store(row, col, acc_all[r * LDW + cc] + acc_all[ACC + r * LDW + cc]);
    }
  }
}

// ------------------------------------------------ fp32 as three bf16 terms
// An fp32 value x splits exactly into x = hi + mid + lo, each a bfloat16:
// hi keeps the leading 8 significant bits of x (truncated), mid the
// leading 8 of the remainder x - hi, and lo what is left, which has at
// most 8 significant bits (fp32 has 24).  A product x w is then the sum of
// the nine products of the parts; the six with hi/mid/lo "orders" adding up
// to at most 2 (hi hi, hi mid, mid hi, hi lo, mid mid, lo hi) keep every
// term down to about 2^-23 |x w|, fp32's own rounding, and bf16 MFMAs
// (16x16x32, exact products, fp32 accumulation) run them at 16 times the
// fp32 MFMA rate of this chip: the fp32 contraction costs 6 bf16 MFMAs per
// 32 reduction channels instead of 8 fp32 ones per 4.
__device__ __forceinline__ void split3(float x, uint32_t& h, uint32_t& m, uint32_t& l) {
  h = __float_as_uint(x) & 0xffff0000u;
  const float r1 = x - __uint_as_float(h);  // exact: x and h share their leading bits
  m = __float_as_uint(r1) & 0xffff0000u;
  l = __float_as_uint(r1 - __uint_as_float(m));  // exact, and its low 16 bits are zero
}

// Two values' parts packed as bfloat16 pairs (element 0 in the low half).
__device__ __forceinline__ uint32_t pack_hi16(uint32_t lo_elem, uint32_t hi_elem) {
  return __builtin_amdgcn_perm(hi_elem, lo_elem, 0x07060302u);
}

// The three part vectors of 8 consecutive fp32 channels (as bf16x8 each).
__device__ __forceinline__ void split8(const float (&v)[8], bf16x8& h8, bf16x8& m8, bf16x8& l8) {
  uint32_t h[8], m[8], l[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) split3(v[i], h[i], m[i], l[i]);
  uint4 a, b, c;
  a.x = pack_hi16(h[0], h[1]); a.y = pack_hi16(h[2], h[3]); a.z = pack_hi16(h[4], h[5]); a.w = pack_hi16(h[6], h[7]);
  b.x = pack_hi16(m[0], m[1]); b.y = pack_hi16(m[2], m[3]); b.z = pack_hi16(m[4], m[5]); b.w = pack_hi16(m[6], m[7]);
  c.x = pack_hi16(l[0], l[1]); c.y = pack_hi16(l[2], l[3]); c.z = pack_hi16(l[4], l[5]); c.w = pack_hi16(l[6], l[7]);
  h8 = __builtin_bit_cast(bf16x8, a);
  m8 = __builtin_bit_cast(bf16x8, b);
  l8 = __builtin_bit_cast(bf16x8, c);
}

// acc += a b^T over 32 reduction channels from the parts of both operands.
__device__ __forceinline__ f32x4 mma_split(const bf16x8& ah, const bf16x8& am, const bf16x8& al, const bf16x8& bh,
                                           const bf16x8& bm, const bf16x8& bl, f32x4 d) {
  d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, d, 0, 0, 0);
  d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, bm, d, 0, 0, 0);
  d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, d, 0, 0, 0);
  d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bm, d, 0, 0, 0);
  d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, bh, d, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, d, 0, 0, 0);
}

// Weight parts for the split row kernel: planes[p][o][n][k] (p = hi, mid,
// lo; bf16 bits) with n the output column and k the reduction channel of
// the launch: TR (forward) reads W[o][k][n], else (dgrad) W[o][n][k].
template <bool TR>
__global__ void k_split_w(const float* __restrict__ W, int K, int kdim, int ncols, uint16_t* __restrict__ planes) {
  const int64_t total = (int64_t)K * kdim * ncols;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    float w;
    if constexpr (TR) {
      const int64_t o = i / ((int64_t)kdim * ncols);
      const int64_t r = i - o * kdim * ncols;
      const int n = (int)(r / kdim), k = (int)(r % kdim);
      w = W[(o * kdim + k) * ncols + n];
    } else {
      w = W[i];
    }
    uint32_t h, m, l;
    split3(w, h, m, l);
    planes[i] = (uint16_t)(h >> 16);
    planes[total + i] = (uint16_t)(m >> 16);
    planes[2 * total + i] = (uint16_t)(l >> 16);
  }
}

// ---------------------------------------------------- row-block kernel
// Forward / dgrad over a row-block plan.  A workgroup owns one block of
// kPlanRows = 64 output rows (rows whose offset sets are alike) and 16 NB
// output columns; wavefront w owns rows 16 w .. 16 w + 15 with its
// accumulators in registers.  The workgroup walks the block's items (one
// offset each) in steps of WB bytes of reduction channels; per step every
// wavefront gathers its 16 rows' input rows (a row without a pair for the
// item reads zeros) and the workgroup stages the offset's weight tile, both
// through LDS, then multiplies.  Each output element is written once.
//
// Loads: gathers whose lanes follow the MFMA layout (consecutive lanes on
// consecutive rows) issue at about a third of the rate of loads in which
// several consecutive lanes read one contiguous piece of a row, so rows and
// weights are loaded WB bytes per row with WB / 16 lanes per row, put in
// LDS, and read back in the MFMA layout: lane (m, g) takes channels
// 32 j + 8 g + [0, 8) (j < S) of row m of the step's window (A) and of
// weight row m of each column block (B).  Each MFMA sums the channels of
// one item only (absent rows and channels past a row's end read zeros), in
// ascending item order, so a row's result does not depend on which rows
// share its block.  B is laid out [o][ncols][kdim] (a contiguous row of reduction
// channels per output column).  Row gathers run D - 1 steps ahead in
// registers and each wavefront's row tile is private to it; the weight
// tile goes straight from memory into one of two LDS buffers (a buffer
// load with LDS destination: no registers, no LDS writes), one barrier per
// step.  Taking the weight tile through registers and LDS writes had cost
// about a quarter of the fp32 kernel's time.  The plan entries are read
// from global memory (L2) a step ahead of their use.
// TB: B is stored [o][kdim][ncols] instead (the forward's weights as given);
// a thread then loads 16 bytes of one reduction channel (4 output columns)
// and writes them to the 4 columns' rows of the weight tile, which spares
// the forward a transposed copy of W.
// Bytes of one weight-tile buffer of the row kernel: COLS rows of the
// step's window (TB: padded rows written from registers; else unpadded rows
// of direct loads), or (SP) three planes of COLS rows of 32 bf16 channels.
// Bytes per row of the row tiles and of the TB weight tile (bank spread:
// +16 had 1.2 conflict cycles per LDS cycle in bf16 layers, +32 0.02).
template <int WB>
constexpr int rows_pitch() {
  return WB + 32;
}
template <int WB, int NB, bool SP, bool TB>
constexpr int rows_b_bytes() {
  return TB ? 16 * NB * rows_pitch<WB>() : (SP ? 3 * 16 * NB * 64 : 16 * NB * WB);
}
// LDS of the row kernel: the four wavefronts' row tiles, then the two weight
// buffers; the bf16 epilogue reuses all of it.
template <int WB, int NB, bool SP, bool TB>
struct RowsLds {
  static constexpr int PITCH = rows_pitch<WB>();  // bytes per row-tile row
  static constexpr int A_BYTES = 4 * 16 * PITCH;
  static constexpr int B_BYTES = rows_b_bytes<WB, NB, SP, TB>();
  static constexpr int BYTES = A_BYTES + 2 * B_BYTES;
};

template <typename T, int WB, int NB, int D, int PK, bool TB = false, bool SP = false>
__device__ __forceinline__ void conv_rows_block(
    const T* __restrict__ X, uint32_t x_bytes, const void* __restrict__ B, uint32_t b_bytes,
    const int32_t* __restrict__ perm, const uint32_t* __restrict__ items, int64_t blk, int first, int n_items,
    int K, int mirror, int kdim, int ncols, const Heads<T>& Y, char* smem, int tid, int wave, int lane, int m, int g,
    int col0) {
  static_assert(!SP || (sizeof(T) == 4 && WB == 128 && PK == 1 && !TB), "split path: fp32, whole windows");
  constexpr int LPR = WB / 16;              // lanes per row window
  constexpr int RPI = 64 / LPR;             // rows per wavefront load
  constexpr int NA = 16 / RPI;              // row loads per wavefront and step
  constexpr int COLS = 16 * NB;             // output columns per workgroup
  // The weight tile (TROWS rows of CPR chunks) arrives by direct-to-LDS
  // loads (except TB): NI wave loads of 64 chunks per step, loads j = wave,
  // wave + 4, .. by each wavefront; slot c = row * CPR + (slot within the
  // row) sits at byte 16 c of the tile.  TB: weight pieces (16 bytes) per
  // thread and step, written to LDS from registers.
  constexpr bool DB = !TB;
  constexpr int CPR = SP ? 4 : LPR;
  constexpr int TROWS = SP ? 3 * COLS : COLS;
  constexpr int NI = DB ? TROWS * CPR / 64 : 0;
  constexpr int NJ = (NI + 3) / 4;
  constexpr int NBP = DB ? 1 : (COLS * LPR + 255) / 256;
  using L = RowsLds<WB, NB, SP, TB>;
  constexpr int PITCH = L::PITCH;
  constexpr int S = WB / (32 * (int)sizeof(T));  // 32-channel MFMA groups per step
  char* const As = smem + wave * 16 * PITCH;     // this wavefront's row tile
  auto Bs = [&](int buf) { return smem + L::A_BYTES + buf * L::B_BYTES; };
  const uint32_t row_bytes = (uint32_t)kdim * sizeof(T);
  // PK > 1: rows of WB / PK bytes, PK items per step side by side in the
  // window (their products simply add up over the window's channels)
  const int ks_n = PK > 1 ? 1 : (int)((row_bytes + WB - 1) / WB);  // steps per item
  const int n_steps = PK > 1 ? (n_items + PK - 1) / PK : n_items * ks_n;
  // bytes per offset of B (SP: of one bf16 plane)
  const uint32_t w_stride = (uint32_t)ncols * (SP ? (uint32_t)kdim * 2u : row_bytes);
  const rsrc_t rx = make_rsrc(X, x_bytes), rb = make_rsrc(B, b_bytes);

  f32x4 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (n_steps > 0) {
    const uint32_t* ents = items + (int64_t)first * kPlanRows;  // the block's entries

    // lane constants of the coalesced loads
    const uint32_t a_byte = (uint32_t)(lane % LPR) * 16;  // within the window
    const int a_u = PK > 1 ? (int)(a_byte / row_bytes) : 0;  // item of the step (packed)
    const uint32_t a_in = a_byte - (uint32_t)a_u * row_bytes;  // byte within its row
    int a_row[NA];                                          // row within the wavefront's 16
#pragma unroll
    for (int i = 0; i < NA; ++i) a_row[i] = lane / LPR + RPI * i;
    int b_col[NBP], b_u[NBP];
    uint32_t b_byte[NBP], b_base[NBP];
#pragma unroll
    for (int q = 0; q < NBP; ++q) {
      const int p = tid + 256 * q;
      if constexpr (SP) {
        (void)p;
        b_col[q] = 0;
        b_byte[q] = 0;
        b_u[q] = 0;
        b_base[q] = kOobOffset;
      } else if constexpr (TB) {
        static_assert(PK == 1, "TB reads one item per step");
        constexpr int PPC = COLS / 4;  // 16-byte pieces per reduction channel
        const int ch = p / PPC;        // reduction channel within the window
        b_col[q] = (p % PPC) * 4;
        b_byte[q] = (uint32_t)ch * sizeof(T);
        b_u[q] = 0;
        const int col = col0 + b_col[q];
        b_base[q] = (ch < WB / (int)sizeof(T) && col < ncols) ? (uint32_t)col * sizeof(T) : kOobOffset;
      } else {
        (void)p;
        b_col[q] = 0;
        b_byte[q] = 0;
        b_u[q] = 0;
        b_base[q] = kOobOffset;
      }
    }

    // this lane's chunk of each of its wavefront's weight loads: byte offset
    // in B without the offset's part and the window's (SP: in the planes),
    // the chunk's byte within the window, and (PK > 1) its item of the step
    uint32_t d_voff[NJ > 0 ? NJ : 1], d_ch[NJ > 0 ? NJ : 1];
    int d_u[NJ > 0 ? NJ : 1];
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) {
      const int c = (wave + 4 * jj) * 64 + lane;
      const int row = c / CPR, chunk = tile_slot<CPR>(row, c % CPR);
      const int col = row % COLS, plane = row / COLS;
      d_ch[jj] = (uint32_t)chunk * 16;
      d_u[jj] = PK > 1 ? (int)(d_ch[jj] / row_bytes) : 0;
      const bool in = wave + 4 * jj < NI && col0 + col < ncols;
      if constexpr (SP)
        d_voff[jj] = in ? (uint32_t)plane * (uint32_t)K * w_stride + (uint32_t)(col0 + col) * (uint32_t)kdim * 2u +
                              d_ch[jj]
                        : kOobOffset;
      else
        d_voff[jj] = in ? (uint32_t)(col0 + col) * row_bytes + d_ch[jj] - (uint32_t)d_u[jj] * row_bytes : kOobOffset;
    }

    uint4 ga[D][NA], gb[D][NBP];  // global loads in flight
    int ld_item = 0, ld_ks = 0, ld_step = 0;
    // per ring slot, the weight tile's offset byte (PK > 1: per item, or
    // kOobOffset past the last), window byte, whether the step exists (its
    // tile is loaded a step after its rows), and whether this wavefront's 16
    // rows have no pair in it (its MFMAs are skipped; wavefront-uniform: the
    // lanes' entries cover the 16 rows and the step's items)
    uint32_t dm_off[D][PK], dm_win[D];
    bool dm_live[D], dm_skip[D];
    // entries of the next step to be issued, read one step ahead (every
    // entry of an item carries the item's offset)
    uint32_t nx_r[NA];
    auto fetch_ent = [&]() {
      const int it = min(ld_item + a_u, n_items - 1);
#pragma unroll
      for (int i = 0; i < NA; ++i) nx_r[i] = ents[it * kPlanRows + wave * 16 + a_row[i]];
    };
    fetch_ent();
    auto issue = [&](int slot) {
      const bool live = ld_step < n_steps;
      if constexpr (PK > 1) {
        // offset of each of the step's items, from a lane that holds its entries
        uint32_t soff[PK];
#pragma unroll
        for (int u = 0; u < PK; ++u) {
          const int o = (int)((uint32_t)__builtin_amdgcn_readlane((int)nx_r[0], u * (int)(row_bytes / 16)) >>
                              kPlanRowBits);
          soff[u] = (uint32_t)(mirror ? K - 1 - o : o) * w_stride;
        }
        bool any = false;
#pragma unroll
        for (int i = 0; i < NA; ++i) {
          const uint32_t r = nx_r[i] & kPlanNoRow;
          const bool ok = live && ld_item + a_u < n_items && r != kPlanNoRow;
          any = any || ok;
          const auto v = __builtin_amdgcn_raw_buffer_load_b128(rx, (int)(ok ? r * row_bytes + a_in : kOobOffset), 0, 0);
          ga[slot][i] = make_uint4(v[0], v[1], v[2], v[3]);
        }
        dm_skip[slot] = __ballot(any) == 0;
#pragma unroll
        for (int u = 0; u < PK; ++u) dm_off[slot][u] = ld_item + u < n_items ? soff[u] : kOobOffset;
        dm_win[slot] = 0;
        dm_live[slot] = live;
        ld_item += PK;
        ++ld_step;
        fetch_ent();
        return;
      }
      const int o = (int)((uint32_t)__builtin_amdgcn_readfirstlane((int)nx_r[0]) >> kPlanRowBits);
      const int ow = mirror ? K - 1 - o : o;
      const uint32_t win = (uint32_t)ld_ks * WB;
      if constexpr (DB) {
        dm_off[slot][0] = (uint32_t)ow * w_stride;
        dm_win[slot] = SP ? win / 2u : win;  // SP: 32 channels are 64 bytes of each bf16 plane row
        dm_live[slot] = live;
      }
      bool any = false;
#pragma unroll
      for (int i = 0; i < NA; ++i) {
        const uint32_t r = nx_r[i] & kPlanNoRow;
        any = any || (live && r != kPlanNoRow);
        const bool ok = live && r != kPlanNoRow && win + a_byte < row_bytes;
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(rx, (int)(ok ? r * row_bytes + win + a_byte : kOobOffset),
                                                             0, 0);
        ga[slot][i] = make_uint4(v[0], v[1], v[2], v[3]);
      }
      dm_skip[slot] = __ballot(any) == 0;
#pragma unroll
      for (int q = 0; q < (DB ? 0 : NBP); ++q) {
        const uint32_t bwin = win;
        const bool ok = live && bwin + b_byte[q] < (SP ? (uint32_t)kdim * 2u : row_bytes) && b_base[q] != kOobOffset;
        // TB: row (win + b_byte) / sizeof(T) of the offset's kdim x ncols matrix
        const uint32_t off = TB ? (win + b_byte[q]) / (uint32_t)sizeof(T) * ((uint32_t)ncols * sizeof(T)) + b_base[q]
                                : b_base[q] + bwin + b_byte[q];
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(rb, (int)(ok ? off : kOobOffset),
                                                             (int)((uint32_t)ow * w_stride), 0);
        gb[slot][q] = make_uint4(v[0], v[1], v[2], v[3]);
      }
      if (++ld_ks == ks_n) { ld_ks = 0; ++ld_item; }
      ++ld_step;
      fetch_ent();
    };
    auto stage = [&](int slot, int buf) {
#pragma unroll
      for (int i = 0; i < NA; ++i)
        *reinterpret_cast<uint4*>(&As[a_row[i] * PITCH + a_byte]) = ga[slot][i];
      if constexpr (TB) {
#pragma unroll
        for (int q = 0; q < NBP; ++q) {
          // 4 consecutive columns of one channel: one element in each column's row
          if (b_byte[q] >= (uint32_t)WB) continue;  // (never, when the pieces fill the threads exactly)
          char* dst = &Bs(buf)[b_col[q] * PITCH + b_byte[q]];
          *reinterpret_cast<uint32_t*>(dst) = gb[slot][q].x;
          *reinterpret_cast<uint32_t*>(dst + PITCH) = gb[slot][q].y;
          *reinterpret_cast<uint32_t*>(dst + 2 * PITCH) = gb[slot][q].z;
          *reinterpret_cast<uint32_t*>(dst + 3 * PITCH) = gb[slot][q].w;
        }
      }
    };
    // the step in ring slot sl, with its weight tile in LDS buffer buf
    auto multiply = [&](int sl, int buf) {
      // a wavefront whose 16 rows have no pair for the item(s) skips the MFMAs
      if (dm_skip[sl]) return;
      if constexpr (SP) {
        // the row tile's 8 channels of this lane, split; the weights' parts
        // were split once, before the launch
        Oct<float> a;
        lds_oct(a, &As[m * PITCH + 32 * g]);
        bf16x8 ah, am, al;
        split8(a.v, ah, am, al);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int col = nb * 16 + m;
          const char* bp = &Bs(buf)[(col * CPR + tile_slot<CPR>(col, g)) * 16];
          const bf16x8 bh = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(bp));
          const bf16x8 bm = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(bp + COLS * 64));
          const bf16x8 bl = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(bp + 2 * COLS * 64));
          acc[nb] = mma_split(ah, am, al, bh, bm, bl, acc[nb]);
        }
        return;
      }
      Oct<T> a[S], b[S][NB];
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int byte = (32 * j + 8 * g) * (int)sizeof(T);
        lds_oct(a[j], &As[m * PITCH + byte]);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int col = nb * 16 + m;
          if constexpr (TB) {
            lds_oct(b[j][nb], &Bs(buf)[col * PITCH + byte]);
          } else {
            // chunk byte / 16 (fp32: and the next) of the column's row
            const char* row = &Bs(buf)[col * CPR * 16];
            lds_oct2(b[j][nb], row + 16 * tile_slot<CPR>(col, byte / 16),
                     row + 16 * tile_slot<CPR>(col, (byte / 16 + 1) % CPR));
          }
        }
      }
#pragma unroll
      for (int j = 0; j < S; ++j)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[nb] = mma_oct(a[j], b[j][nb], acc[nb]);
    };

    // the weight tile of the step in ring slot sl into buffer buf
    auto dma_b = [&](int sl, int buf) {
      if constexpr (DB) {
        if (!dm_live[sl]) return;
        const uint32_t rowlen = SP ? (uint32_t)kdim * 2u : row_bytes;  // bytes of a row of B (SP: of a plane)
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
          if (wave + 4 * jj >= NI) break;
          auto* dst = (__attribute__((address_space(3))) void*)&Bs(buf)[(wave + 4 * jj) * 1024];
          if constexpr (PK > 1) {
            // the chunk's item of the step: its own offset, folded into the lane's address
            uint32_t so = dm_off[sl][0];
#pragma unroll
            for (int u = 1; u < PK; ++u) so = d_u[jj] == u ? dm_off[sl][u] : so;
            const bool ok = d_voff[jj] != kOobOffset && so != kOobOffset;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, dst, 16, (int)(ok ? d_voff[jj] + so : kOobOffset), 0, 0, 0);
          } else {
            const bool ok = d_voff[jj] != kOobOffset && dm_win[sl] + d_ch[jj] < rowlen;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, dst, 16, (int)(ok ? d_voff[jj] + dm_win[sl] : kOobOffset),
                                                     (int)dm_off[sl][0], 0, 0);
          }
        }
      }
    };
    // all of this wavefront's loads issued so far have landed (the direct
    // weight loads, which the compiler's own waits do not cover)
    auto wait_loads = [&]() {
      if constexpr (DB) __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    };
    // step t: its row loads are issued at step t - D (ring slot t % D) and
    // staged into LDS at step t - 1, its weight tile is loaded straight into
    // LDS buffer t % 2 at the start of step t - 1 (TB: staged there from
    // registers), and it is multiplied at step t.  (Row gathers loaded
    // straight into LDS the same way took bf16 layers 41 -> 61 us: the row
    // tiles stay staged from registers.)
#pragma unroll
    for (int q = 0; q < D; ++q) issue(q);
    dma_b(0, 0);
    stage(0, 0);
    wait_loads();
    __syncthreads();
    // u = t % (2 D) keeps the ring positions compile-time constants; the row
    // tile of step t is read before step t + 1's rows overwrite it, and the
    // weight buffer of step t + 1 was last read at step t - 1 (so its loads
    // can start before step t's multiplications)
    auto step = [&](int u) {
      dma_b((u + 1) % D, (u + 1) % 2);
      multiply(u % D, u % 2);
      stage((u + 1) % D, (u + 1) % 2);
      wait_loads();
      issue(u % D);  // loads of step t + D
      __syncthreads();
    };
    int t0 = 0;
    for (; t0 + 2 * D <= n_steps; t0 += 2 * D) {
#pragma unroll
      for (int u = 0; u < 2 * D; ++u) step(u);
    }
#pragma unroll
    for (int u = 0; u < 2 * D - 1; ++u)
      if (t0 + u < n_steps) step(u);
  }
  // lane holds rows 4 g + r of the wavefront's 16, column m of each column block
  const int32_t* wrows = perm + blk * kPlanRows + wave * 16;
  // bf16: 16-byte row pieces when every destination allows them: the
  // wavefront's 16 x COLS result goes through its quarter of the weight
  // buffers (free after the last step's barrier) and leaves as whole row
  // pieces instead of one 2-byte element per lane and row.  (fp32 rows take
  // 4 bytes per lane already; there the extra registers cost more.)
  constexpr int RB = COLS * (int)sizeof(T) + 16;  // tile row pitch (bank spread)
  static_assert(sizeof(T) == 4 || 4 * 16 * RB <= L::BYTES, "output tiles fit the LDS");
  bool vec = sizeof(T) == 2 && (ncols * (int)sizeof(T)) % 16 == 0;
#pragma unroll
  for (int h = 0; h < 2; ++h)
    if (h < Y.n)
      vec = vec && reinterpret_cast<uintptr_t>(Y.out[h]) % 16 == 0 && (Y.ld[h] * (int64_t)sizeof(T)) % 16 == 0;
  if constexpr (sizeof(T) == 2) if (vec) {
    char* tile = smem + wave * 16 * RB;
    constexpr int PIECES = COLS * (int)sizeof(T) / 16;  // 16-byte pieces per tile row
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (h >= Y.n) break;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int col = col0 + nb * 16 + m;
        const bool ok = col < ncols;
        const float sc = ok && Y.scale[h] ? Y.scale[h][col] : 1.f;
        const float sh = ok && Y.scale[h] ? Y.shift[h][col] : 0.f;
        const float bi = ok && Y.bias ? Y.bias[col] : 0.f;
        float rv[4] = {0.f, 0.f, 0.f, 0.f};
        if (Y.res) {  // uniform: layers without a residual skip the row reads
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int32_t rrow = wrows[4 * g + r];
            if (ok && rrow >= 0) rv[r] = Elem<T>::load(Y.res + rrow * Y.res_ld + col);
          }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float y = acc[nb][r] + bi + rv[r];
          const float v = Y.scale[h] ? fmaxf(0.f, y * sc + sh) : y;
          Elem<T>::store(reinterpret_cast<T*>(tile + (4 * g + r) * RB) + nb * 16 + m, v);
        }
      }
      // the wavefront reads back what other lanes wrote
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int q = lane; q < 16 * PIECES; q += 64) {
        const int row_in = q / PIECES, piece = q % PIECES;
        const int col = col0 + piece * (16 / (int)sizeof(T));
        const int32_t grow = wrows[row_in];
        if (grow >= 0 && col < ncols)
          *reinterpret_cast<uint4*>(Y.out[h] + grow * Y.ld[h] + col) =
              *reinterpret_cast<const uint4*>(tile + row_in * RB + piece * 16);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    return;
  }
  const int4 rows = *reinterpret_cast<const int4*>(wrows + 4 * g);
  const int rr[4] = {rows.x, rows.y, rows.z, rows.w};
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int col = col0 + nb * 16 + m;
    if (col < ncols)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (rr[r] >= 0) Y.store(rr[r], col, acc[nb][r]);
  }
}

template <typename T, int WB, int NB, int D, int PK, bool TB, bool SP>
__device__ __forceinline__ void conv_rows_run(
    const T* __restrict__ X, uint32_t x_bytes, const void* __restrict__ B, uint32_t b_bytes,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ b_first, const int4* __restrict__ b_rec,
    const uint32_t* __restrict__ items, int64_t n_blocks, int K, int mirror, int kdim, int ncols, const Heads<T>& Y) {
  constexpr int RPI = 64 / (WB / 16);       // rows per wavefront load
  constexpr int COLS = 16 * NB;             // output columns per workgroup
  static_assert(WB / (32 * (int)sizeof(T)) >= 1 && 16 % RPI == 0, "window");
  __shared__ __attribute__((aligned(16))) char smem[RowsLds<WB, NB, SP, TB>::BYTES];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int m = lane & 15, g = lane >> 4;
  const int col0 = blockIdx.y * COLS;
  const int64_t G = gridDim.x, wg = blockIdx.x;
  // persistent: the blocks, longest first, are dealt to the workgroups in
  // boustrophedon order (0 .. G-1, G-1 .. 0, ...)
  auto next = [&](int64_t round) { return round * G + ((round & 1) ? G - 1 - wg : wg); };
  {
    // Workgroups with more than their share of the items issue first (wave
    // priority), so that the ones that finish last are the ones that started
    // with the most work.
    int mine = 0;
    for (int64_t idx = wg, round = 0; idx < n_blocks; idx = next(++round)) mine += b_rec[idx].z;
    const float share = (float)mine * (float)G / (float)max(b_first[n_blocks], 1);
    if (share > 1.1f) __builtin_amdgcn_s_setprio(3);
    else if (share > 1.0f) __builtin_amdgcn_s_setprio(2);
    else if (share > 0.9f) __builtin_amdgcn_s_setprio(1);
  }
  if (Y.n_zero > 0) {
    const int64_t stride = (int64_t)gridDim.x * gridDim.y * 256;
    for (int64_t i = ((int64_t)blockIdx.y * gridDim.x + wg) * 256 + tid; i < Y.n_zero; i += stride) Y.zero[i] = 0.f;
  }
  for (int64_t idx = wg, round = 0; idx < n_blocks; idx = next(++round)) {
    const int4 rec = b_rec[idx];  // (block, first item, items): one load, no chain
    __syncthreads();  // the previous block's LDS is free
    conv_rows_block<T, WB, NB, D, PK, TB, SP>(X, x_bytes, B, b_bytes, perm, items, rec.x, rec.y, rec.z, K, mirror,
                                              kdim, ncols, Y, smem, tid, wave, lane, m, g, col0);
  }
}

#define SSCN_ROWS_ARGS                                                                                          \
  const T *__restrict__ X, uint32_t x_bytes, const void *__restrict__ B, uint32_t b_bytes,                     \
      const int32_t *__restrict__ perm, const int32_t *__restrict__ b_first, const int4 *__restrict__ b_rec,     \
      const uint32_t *__restrict__ items, int64_t n_blocks, int K, int mirror, int kdim, int ncols, Heads<T> Y

// Forward (and DC) launches.  SP: fp32 through bf16 parts (B holds the
// weight planes of k_split_w).
// Resident workgroups per CU the row kernel is compiled for (its LDS and
// registers): 6 for 64-byte windows, 5 for 128-byte ones, 4 for the split
// path (its three weight planes take 40 KB of LDS).
template <int WB, bool SP>
constexpr int rows_min_blocks() {
  return SP ? 4 : (WB == 64 ? 6 : 5);
}

template <typename T, int WB, int NB, int D, int PK, bool TB = false, bool SP = false>
__global__ __launch_bounds__(256, (rows_min_blocks<WB, SP>())) void k_conv_rows(SSCN_ROWS_ARGS) {
  conv_rows_run<T, WB, NB, D, PK, TB, SP>(X, x_bytes, B, b_bytes, perm, b_first, b_rec, items, n_blocks, K, mirror,
                                          kdim, ncols, Y);
}

// The dgrad launches of sparse_conv_backward: the same kernel under its own
// name, so that kernel traces tell the two directions apart.
template <typename T, int WB, int NB, int D, int PK, bool TB = false, bool SP = false>
__global__ __launch_bounds__(256, (rows_min_blocks<WB, SP>())) void k_dgrad_rows(SSCN_ROWS_ARGS) {
  conv_rows_run<T, WB, NB, D, PK, TB, SP>(X, x_bytes, B, b_bytes, perm, b_first, b_rec, items, n_blocks, K, mirror,
                                          kdim, ncols, Y);
}
#undef SSCN_ROWS_ARGS

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
// wgrad without LDS staging.  dW^o[ci][co] = sum_p X[in_p][ci] dY[out_p][co].
// MFMA row i of block a stands for input channel ci0 + CA*i + a, column j of
// block b for output channel co0 + CB*j + b, so a lane's CA (CB) operand
// values are contiguous channels of one gathered row: one 8/16-byte load
// each.  One MFMA step consumes 4 pairs (one per lane group).  Each
// wavefront accumulates the whole CA*16 x CB*16 block over a quarter of
// the workgroup's pairs, with pair indices and rows fetched one iteration
// (4 pairs) ahead; the four partial blocks are summed through LDS and
// added to dW with fp32 atomics.  A workgroup's pairs are those of one
// offset whose output rows lie in a range of `tr` consecutive tiles, so the
// rows it gathers are spatially close; workgroups are numbered so that each
// XCD takes contiguous tile ranges (L2 locality).
template <int N>
__device__ __forceinline__ void load_n(const float* __restrict__ p, bool ok, float (&v)[N]) {
  if (!ok) {
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = 0.f;
    return;
  }
  if constexpr (N == 4) {
    const float4 x = *reinterpret_cast<const float4*>(p);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  } else if constexpr (N == 2) {
    const float2 x = *reinterpret_cast<const float2*>(p);
    v[0] = x.x; v[1] = x.y;
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = p[i];
  }
}
template <int N>
__device__ __forceinline__ void load_n(const bf16_t* __restrict__ p, bool ok, float (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = ok ? bf16_to_f32(p[i].bits) : 0.f;
}

template <typename T, int CA, int CB>
__global__ __launch_bounds__(256) void k_wgrad_reg(const T* __restrict__ X, const T* __restrict__ dY,
                                                   const int64_t* __restrict__ seg, int64_t n_tiles,
                                                   const int32_t* __restrict__ in_rows,
                                                   const int32_t* __restrict__ out_rows, int K, int mirror,
                                                   int cin, int cout, int tr, int nzc, float* __restrict__ dW) {
  constexpr int STEPS = 1;  // MFMA steps (4 pairs each) per iteration (more costs occupancy)
  const int64_t item = xcd_remap(blockIdx.x, gridDim.x);
  const int o = (int)(item % K);
  const int64_t r = item / K;
  const int so = mirror ? K - 1 - o : o;
  const int64_t t_lo = r * tr, t_hi = min<int64_t>(t_lo + tr, n_tiles);
  const int64_t pb = seg[(int64_t)so * n_tiles + t_lo];
  const int64_t pe = seg[(int64_t)so * n_tiles + t_hi];
  if (pb >= pe) return;
  const int ci0 = (blockIdx.y % nzc) * 16 * CA, co0 = (blockIdx.y / nzc) * 16 * CB;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  // a lane's channels are fully inside or fully outside [0, cin) / [0, cout)
  const bool a_ok = ci0 + CA * m + CA <= cin, b_ok = co0 + CB * m + CB <= cout;
  const int64_t per = ((pe - pb + 3) / 4 + 3) / 4 * 4;
  const int64_t wb = pb + wave * per, we = min<int64_t>(wb + per, pe);

  f32x4 d[CA][CB];
#pragma unroll
  for (int a = 0; a < CA; ++a)
#pragma unroll
    for (int b = 0; b < CB; ++b) d[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  struct Rows {
    int32_t irow[STEPS], orow[STEPS];
    bool ok[STEPS];
  };
  auto fetch_rows = [&](int64_t p, Rows& r) {
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
      const int64_t q = p + 4 * st + g;
      r.ok[st] = q < we;
      r.irow[st] = r.ok[st] ? in_rows[q] : 0;
      r.orow[st] = r.ok[st] ? out_rows[q] : 0;
    }
  };
  auto fetch_data = [&](const Rows& r, float (&xa)[STEPS][CA], float (&yb)[STEPS][CB]) {
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
      load_n<CA>(X + (int64_t)r.irow[st] * cin + ci0 + CA * m, r.ok[st] && a_ok, xa[st]);
      load_n<CB>(dY + (int64_t)r.orow[st] * cout + co0 + CB * m, r.ok[st] && b_ok, yb[st]);
    }
  };

  if (wb < we) {
    Rows r_cur, r_nxt;
    float xa[STEPS][CA], yb[STEPS][CB], xa_n[STEPS][CA], yb_n[STEPS][CB];
    fetch_rows(wb, r_cur);
    fetch_data(r_cur, xa, yb);
    fetch_rows(wb + 4 * STEPS, r_nxt);
    for (int64_t p = wb; p < we; p += 4 * STEPS) {
      const bool more = p + 4 * STEPS < we;
      Rows r_nn;
      if (more) {
        fetch_data(r_nxt, xa_n, yb_n);
        fetch_rows(p + 8 * STEPS, r_nn);
      }
#pragma unroll
      for (int st = 0; st < STEPS; ++st)
#pragma unroll
        for (int a = 0; a < CA; ++a)
#pragma unroll
          for (int b = 0; b < CB; ++b)
            d[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(xa[st][a], yb[st][b], d[a][b], 0, 0, 0);
      if (more) {
#pragma unroll
        for (int st = 0; st < STEPS; ++st) {
#pragma unroll
          for (int a = 0; a < CA; ++a) xa[st][a] = xa_n[st][a];
#pragma unroll
          for (int b = 0; b < CB; ++b) yb[st][b] = yb_n[st][b];
        }
        r_nxt = r_nn;
      }
    }
  }
  // sum the four wavefronts' partial blocks, then add the block to dW.
  // Waves 0 and 1 store theirs in two LDS copies, waves 2 and 3 add theirs
  // (plain loads and stores: LDS float atomics are several times slower),
  // and every thread adds the two copies of its elements to dW.
  // D[4g + r][m] of block (a, b) is dW[ci0 + CA (4g + r) + a][co0 + CB m + b].
  constexpr int NE = CA * CB * 4;  // values per lane
  __shared__ float part[2][NE][64];
  float(*mine)[64] = part[wave & 1];
  if (wave < 2) {
#pragma unroll
    for (int a = 0; a < CA; ++a)
#pragma unroll
      for (int b = 0; b < CB; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) mine[(a * CB + b) * 4 + r][lane] = d[a][b][r];
  }
  __syncthreads();
  if (wave >= 2) {
#pragma unroll
    for (int a = 0; a < CA; ++a)
#pragma unroll
      for (int b = 0; b < CB; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) mine[(a * CB + b) * 4 + r][lane] += d[a][b][r];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < NE * 64; e += 256) {
    const int v = e / 64, l = e % 64;
    const float sum = part[0][v][l] + part[1][v][l];
    const int a = v / (CB * 4), b = (v / 4) % CB, r = v % 4;
    const int mm = l & 15, gg = l >> 4;
    const int ci = ci0 + CA * (4 * gg + r) + a, co = co0 + CB * mm + b;
    if (ci < cin && co < cout && sum != 0.f) atomicAdd(dW + ((int64_t)o * cin + ci) * cout + co, sum);
  }
}

// ------------------------------------------------- column-owner kernel
// One lane's operand for one 64-channel block: 16 channels as NJ b128
// loads of EPB elements; load j of lane group g covers channels
// 4 EPB j + EPB g .. + EPB - 1, so that the four lane groups of one load
// read 64 contiguous bytes of a row (one instruction touches half as many
// cache lines as with 16 contiguous channels per lane).
template <typename T> struct Frag16;
template <> struct Frag16<float> {
  static constexpr int kLoads = 4;
  float v[16];
  __device__ __forceinline__ void load(rsrc_t r, uint32_t base, const uint32_t (&lo)[4], uint32_t soff) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const auto q = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(base + lo[j]), (int)soff, 0);
      v[4 * j + 0] = __uint_as_float(q[0]); v[4 * j + 1] = __uint_as_float(q[1]);
      v[4 * j + 2] = __uint_as_float(q[2]); v[4 * j + 3] = __uint_as_float(q[3]);
    }
  }
  __device__ __forceinline__ void select(bool take, const Frag16& o) {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = take ? o.v[i] : v[i];
  }
};
template <> struct Frag16<bf16_t> {
  static constexpr int kLoads = 2;
  bf16x8 v[2];
  __device__ __forceinline__ void load(rsrc_t r, uint32_t base, const uint32_t (&lo)[4], uint32_t soff) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const auto q = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(base + lo[j]), (int)soff, 0);
      uint4 u;
      u.x = q[0]; u.y = q[1]; u.z = q[2]; u.w = q[3];
      v[j] = __builtin_bit_cast(bf16x8, u);
    }
  }
  __device__ __forceinline__ void select(bool take, const Frag16& o) {
#pragma unroll
    for (int j = 0; j < 2; ++j) v[j] = take ? o.v[j] : v[j];
  }
};
__device__ __forceinline__ f32x4 mma16(const Frag16<float>& a, const Frag16<float>& b, f32x4 d) {
#pragma unroll
  for (int i = 0; i < 16; ++i) d = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[i], b.v[i], d, 0, 0, 0);
  return d;
}
__device__ __forceinline__ f32x4 mma16(const Frag16<bf16_t>& a, const Frag16<bf16_t>& b, f32x4 d) {
  d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v[0], b.v[0], d, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v[1], b.v[1], d, 0, 0, 0);
}

constexpr int kColLdw = 17;                               // LDS row stride (floats) of a wave's tile
constexpr int kColRegion = (kChunkRows + 1) * kColLdw;    // floats per wave (one padding row)

// Forward / dgrad over the padded chunk table.  Every wavefront owns 16
// output columns and all input channels: per chunk (16 pairs of one
// offset) it multiplies the 16 gathered rows by the offset's weight block
// and adds the 16 x 16 result into a private fp32 tile of kChunkRows rows
// in LDS, at the pairs' output rows (a row occurs at most once per chunk).
// When the last chunk of a tile has been added, the wavefront writes its
// columns of the tile to Y and clears them.  No LDS location is shared
// between wavefronts, so there are no barriers, and the chunk stream of a
// workgroup runs across its tiles: chunk records (input rows, output rows)
// are loaded 2 RING chunks ahead, gathered rows RING chunks ahead and the
// weight block (only when the offset changes) together with the rows, into
// register rings with compile-time slots.  Record and row loads are issued
// unconditionally (a row that is not needed reads an out-of-range offset,
// which returns zeros without touching memory), so the compiler's wait
// counts stay close to exact and the loads of later chunks remain in
// flight; only the tile write-out, once per tile, waits for everything.
//
// Workgroups serve tile groups (one contiguous range of tiles per XCD, as
// workgroups are dispatched round-robin over XCDs); a group's tiles are
// dealt to its workgroups in boustrophedon order.  blockIdx.y selects a
// range of 16 * (blockDim.x / 64) output columns.
//
// Wt is the weight block with the reduction index contiguous:
// Wt[o][n][k], n < cout, k < cin.
template <typename T, int KB, int RING>
__global__ __launch_bounds__(256) void k_conv_col(
    const T* __restrict__ X, uint32_t x_bytes, const T* __restrict__ Wt, uint32_t w_bytes,
    const int32_t* __restrict__ ctile, const int32_t* __restrict__ c_in, const uint32_t* __restrict__ c_out,
    const int32_t* __restrict__ c_off, int n_ct, int K, int mirror, int cin, int cout, int n_out,
    Heads<T> Y) {
  constexpr int IR = 2 * RING;                 // chunk-record ring
  constexpr int TR = kChunkRows;
  constexpr int EPB = 16 / sizeof(T);          // elements per b128 load
  constexpr uint32_t kPadRows = (uint32_t)TR * 0x01010101u;
  constexpr int kNoOff = 0xffff;               // meta of a chunk past the end
  extern __shared__ float lds_col[];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int ncol = blockDim.x >> 6;
  const int col0 = (blockIdx.y * ncol + wave) * 16;
  if (col0 >= cout) return;                    // wave-uniform; nothing is shared across waves
  float* acc = lds_col + wave * kColRegion;
  for (int i = lane; i < kColRegion; i += 64) acc[i] = 0.f;

  // lane constants
  const uint32_t row_bytes = (uint32_t)cin * sizeof(T);
  const int col = col0 + m;
  uint32_t a_lo[KB][4], b_lo[KB][4];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k0 = kb * 64 + 4 * EPB * j + EPB * g;
      const bool ok = k0 + EPB <= cin;
      a_lo[kb][j] = ok ? (uint32_t)k0 * sizeof(T) : kOobOffset;
      b_lo[kb][j] = (ok && col < cout) ? ((uint32_t)col * cin + k0) * sizeof(T) : kOobOffset;
    }
  const uint32_t w_stride = (uint32_t)cout * cin * sizeof(T);
  const rsrc_t rx = make_rsrc(X, x_bytes), rw = make_rsrc(Wt, w_bytes);
  float* acc_lane = acc + m;

  // this workgroup's tiles
  const int ngrp = min((int)gridDim.x, kTileGroups);
  const int grp = blockIdx.x % ngrp;
  const int G = ((int)gridDim.x - grp + ngrp - 1) / ngrp, bi = blockIdx.x / ngrp;
  const int t_first = (int)((int64_t)grp * n_ct / ngrp);
  const int t_count = (int)((int64_t)(grp + 1) * n_ct / ngrp) - t_first;
  auto tile_of = [&](int r) -> int {
    const int idx = r * G + ((r & 1) ? G - 1 - bi : bi);
    return idx < t_count ? t_first + idx : -1;
  };
  int n_stream = 0;
  for (int r = 0;; ++r) {
    const int t = tile_of(r);
    if (t < 0) break;
    n_stream += ctile[(t + 1) * K] - ctile[t * K];
  }

  // record cursor over (tile, chunk); compute-side tile
  int cur_r = 0, cur_t = tile_of(0), cur_c = 0, cur_e = 0;
  if (cur_t >= 0) { cur_c = ctile[cur_t * K]; cur_e = ctile[(cur_t + 1) * K]; }
  int comp_r = 0;

  // Chunk records (loaded 2 RING chunks ahead) are read once, when the
  // chunk's operands are requested (RING chunks ahead): the output rows and
  // the offset then move into the operand ring.  A record slot is never read
  // in the step that refills it, so every slot keeps one register across the
  // loop and no wait lands on the loop's back edge.  The weight block of a
  // chunk is requested together with its gathered rows (same distance: loads
  // complete in order, so a later request would shorten the effective
  // prefetch distance of everything before it).
  int32_t r_in[IR];
  uint32_t r_out[IR];
  int r_meta[IR];         // stored offset (kNoOff past the end) | last chunk of its tile << 16
  uint32_t o_ring[RING];  // output rows of the chunk in operand slot
  int m_ring[RING];       // meta of the chunk in operand slot
  bool f_ring[RING];      // its weight block differs from the previous chunk's
  Frag16<T> a_ring[RING][KB], b_ring[RING][KB], b_cur[KB];
  int req_off = -1;       // offset of the last real chunk whose operands were requested

  auto fetch_record = [&](int slot) {
    const bool valid = cur_t >= 0;
    const int c = valid ? cur_c : 0;         // chunk 0 always exists: loads stay unconditional
    r_in[slot] = c_in[(int64_t)c * 16 + m];
    r_out[slot] = c_out[(int64_t)c * 4 + g];
    if (valid) {
      r_meta[slot] = c_off[c] | ((c + 1 == cur_e) ? (1 << 16) : 0);
      if (++cur_c == cur_e) {
        cur_t = tile_of(++cur_r);
        if (cur_t >= 0) { cur_c = ctile[cur_t * K]; cur_e = ctile[(cur_t + 1) * K]; }
      }
    } else {
      r_meta[slot] = kNoOff;
    }
  };
  auto fetch_operands = [&](int rs, int as) {
    const int meta = r_meta[rs];
    const int off = meta & 0xffff;
    const bool valid = off != kNoOff;
    const int32_t irow = r_in[rs];
    const uint32_t base = (valid && irow >= 0) ? (uint32_t)irow * row_bytes : kOobOffset;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) a_ring[as][kb].load(rx, base, a_lo[kb], 0);
    const bool fresh = valid && off != req_off;
    if (valid) req_off = off;
    const int ow = mirror ? K - 1 - off : off;
    const uint32_t soff = (uint32_t)ow * w_stride;
    if (fresh) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) b_ring[as][kb].load(rw, 0u, b_lo[kb], soff);
    }
    f_ring[as] = fresh;
    o_ring[as] = valid ? r_out[rs] : kPadRows;
    asm volatile("" : "+v"(o_ring[as]));  // keep the read of the record slot here
    m_ring[as] = meta;
  };

#pragma unroll
  for (int sl = 0; sl < IR; ++sl) fetch_record(sl);
#pragma unroll
  for (int sl = 0; sl < RING; ++sl) fetch_operands(sl, sl);

  f32x4 d_prev = {0.f, 0.f, 0.f, 0.f};
  uint32_t out_prev = kPadRows;
  bool last_prev = false;
  for (int i0 = 0; i0 <= n_stream; i0 += IR) {
#pragma unroll
    for (int sl = 0; sl < IR; ++sl) {
      const int as = sl % RING;
      // 1. this chunk's product
      const int meta = m_ring[as];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) b_cur[kb].select(f_ring[as], b_ring[as][kb]);
      f32x4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) d = mma16(a_ring[as][kb], b_cur[kb], d);
      // 2. add the previous chunk into its tile
      {
        float* q0 = acc_lane + ((out_prev >> 0) & 0xff) * kColLdw;
        float* q1 = acc_lane + ((out_prev >> 8) & 0xff) * kColLdw;
        float* q2 = acc_lane + ((out_prev >> 16) & 0xff) * kColLdw;
        float* q3 = acc_lane + ((out_prev >> 24) & 0xff) * kColLdw;
        const float v0 = *q0, v1 = *q1, v2 = *q2, v3 = *q3;
        *q0 = v0 + d_prev[0];
        *q1 = v1 + d_prev[1];
        *q2 = v2 + d_prev[2];
        *q3 = v3 + d_prev[3];
      }
      // ... and write the tile out after its last chunk (once per tile)
      if (last_prev) {
        const int64_t row0 = (int64_t)tile_of(comp_r++) * TR;
        for (int r = g; r < TR; r += 4) {
          float* q = acc_lane + r * kColLdw;
          const float v = *q;
          *q = 0.f;
          const int64_t row = row0 + r;
          if (row < n_out && col < cout) Y.store(row, col, v);
        }
        __builtin_amdgcn_s_waitcnt(0);
      }
      d_prev = d;
      out_prev = o_ring[as];
      last_prev = (meta >> 16) & 1;
      // 3. operands RING chunks ahead, record 2 RING chunks ahead
      fetch_operands((sl + RING) % IR, as);
      fetch_record(sl);
    }
  }
}

// ---------------------------------------------------------------- launchers
// Workgroups that fit on the device at once, capped by the work and rounded
// up to a multiple of kTileGroups (every tile group gets workgroups).
static unsigned persistent_grid(const void* kern, size_t lds, int64_t n_items, int block = 256) {
  int cus = 256, per_cu = 1;
  occupancy(kern, block, lds, &per_cu, &cus);
  int64_t g = std::min<int64_t>((int64_t)cus * per_cu, std::max<int64_t>(n_items, 1));
  g = ceil_div(g, kTileGroups) * kTileGroups;
  return (unsigned)g;
}

template <typename T, int RING, int KB, bool WT, int NB = 2>
static sscn_status launch_quad(const T* X, uint32_t x_bytes, const T* W, uint32_t w_bytes, const View& v, int cin,
                               int cout, const Heads<T>& Y, hipStream_t s) {
  SSCN_TRY(ensure_order(v, s));
  const int max_chunks = v.K * (kTile / 16 + 1);
  const QuadLds L(max_chunks, v.K);
  const int groups = (cout + 63) / 64;
  constexpr int NT = 64 * (8 / NB);
  auto kern = k_conv_quad<T, RING, KB, WT, NB>;
  const unsigned g = persistent_grid((const void*)kern, L.total, v.st->n_tiles, NT);
  kern<<<dim3(g, (unsigned)groups), NT, L.total, s>>>(X, x_bytes, W, w_bytes, v.st->seg, v.st->in_rows,
                                                       v.st->out_rows, v.st->order, v.st->n_tiles, v.K,
                                                       v.mirror ? 1 : 0, cin, cout, v.n_out, max_chunks, Y);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

template <typename T, int NW>
static sscn_status launch_generic_nw(const T* X, const T* Bt, const View& v, int cin, int cout, int grid_y, const Heads<T>& Y,
                                     hipStream_t s) {
  // accumulator tile (tpw * 64 rows x (16 NW + 1) fp32) within 64 KiB of LDS
  const int tpw = NW >= 8 ? 1 : 2;
  const int64_t blocks = ceil_div(v.st->n_tiles, tpw);
  const size_t lds = sizeof(float) * tpw * kTile * (16 * NW + 1);
  k_gather_mma<T, NW><<<dim3((unsigned)blocks, (unsigned)grid_y), NW * 64, lds, s>>>(
      X, Bt, v.st->seg, v.st->in_rows, v.st->out_rows, v.st->n_tiles, v.K, v.mirror ? 1 : 0, cin, cout, v.n_out, tpw,
      Y);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

template <typename T>
static sscn_status launch_generic(const T* X, const T* Bt, const View& v, int cin, int cout, const Heads<T>& Y, hipStream_t s) {
  const int ncb = (cout + 15) / 16;
  const int grid_y = (ncb + 7) / 8;
  const int nw = (ncb + grid_y - 1) / grid_y;
  switch (nw) {
    case 1: return launch_generic_nw<T, 1>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 2: return launch_generic_nw<T, 2>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 3: return launch_generic_nw<T, 3>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 4: return launch_generic_nw<T, 4>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 5: return launch_generic_nw<T, 5>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 6: return launch_generic_nw<T, 6>(X, Bt, v, cin, cout, grid_y, Y, s);
    case 7: return launch_generic_nw<T, 7>(X, Bt, v, cin, cout, grid_y, Y, s);
    default: return launch_generic_nw<T, 8>(X, Bt, v, cin, cout, grid_y, Y, s);
  }
}

// Y (n_out x cout) = forward of X (n_in x cin) over view v.  W holds the
// K (cin x cout) weight matrices, stored [o][cin][cout] (WT = false,
// forward) or [o][cout][cin] (WT = true, dgrad reads W^o transposed).  The
// generic fallback needs the [o][cout][cin] layout and receives it in Bt
// (a transposed copy made by the caller when WT = false).
// Column-owner kernel over the chunk table: Bt = weights with the
// reduction index contiguous ([o][cout][cin]).  Returns SSCN_ERR_SHAPE
// (without launching) when the shape is outside what the kernel covers.
template <typename T, int KB, int RING>
static sscn_status launch_col_kb(const T* X, uint32_t xb, const T* Bt, uint32_t wb, const View& v, int cin,
                                 int cout, const Heads<T>& Y, hipStream_t s) {
  const Storage& st = *v.st;
  const int ng = (cout + 15) / 16;
  int ncol = std::min(ng, 4);
  for (int c : {4, 3, 2})
    if (ng % c == 0) { ncol = c; break; }
  const int gy = (ng + ncol - 1) / ncol;
  const size_t lds = sizeof(float) * kColRegion * ncol;
  auto kern = k_conv_col<T, KB, RING>;
  int cus = 256, per_cu = 1;
  occupancy((const void*)kern, 64 * ncol, lds, &per_cu, &cus);
  const int64_t gx = std::min<int64_t>(st.n_ctiles, std::max<int64_t>(1, (int64_t)cus * per_cu / gy));
  kern<<<dim3((unsigned)gx, (unsigned)gy), 64 * ncol, lds, s>>>(
      X, xb, Bt, wb, st.ctile, st.c_in, reinterpret_cast<const uint32_t*>(st.c_out), st.c_off, (int)st.n_ctiles,
      v.K, v.mirror ? 1 : 0, cin, cout, (int)v.n_out, Y);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

// Which forward / dgrad kernel: the column kernel where its shape rules
// allow and either the output width is not a multiple of 64 (the quad
// kernel computes 64 columns per workgroup row) or output rows have few
// pairs (DC layers: one pair per output row; short chunks in 64-row tiles);
// the quad kernel otherwise.  Measured on the U-Net's layers.
template <typename T>
static bool quad_eligible(const View& v, int cin, int cout);
template <typename T>
static bool col_eligible(const View& v, int cin, int cout);
template <typename T>
static bool prefer_col(const View& v, int cin, int cout) {
  if (!col_eligible<T>(v, cin, cout)) return false;
  if (!quad_eligible<T>(v, cin, cout)) return true;
  return cout % 64 != 0 || v.n_pairs < 4 * v.n_out;
}

template <typename T>
static bool col_eligible(const View& v, int cin, int cout) {
  const uint64_t x_bytes = (uint64_t)std::max<int64_t>(v.n_in, 1) * cin * sizeof(T);
  const uint64_t w_bytes = (uint64_t)v.K * cout * cin * sizeof(T);
  const int kb = (cin + 63) / 64;
  return cin % (16 / (int)sizeof(T)) == 0 && kb <= (sizeof(T) == 4 ? 2 : 4) && x_bytes < kOobOffset &&
         w_bytes < kOobOffset && v.n_out < INT32_MAX &&
         ceil_div(v.n_out, kChunkRows) * (v.K + 1) + ceil_div(v.n_pairs, 16) < INT32_MAX;
}

template <typename T>
static sscn_status launch_col(const T* X, const T* Bt, const View& v, int cin, int cout, const Heads<T>& Y, hipStream_t s) {
  if (v.n_out == 0) return SSCN_OK;
  SSCN_TRY(ensure_chunks(v, s));
  const uint32_t xb = (uint32_t)((uint64_t)std::max<int64_t>(v.n_in, 1) * cin * sizeof(T));
  const uint32_t wb = (uint32_t)((uint64_t)v.K * cout * cin * sizeof(T));
  switch ((cin + 63) / 64) {
    case 1: return launch_col_kb<T, 1, 3>(X, xb, Bt, wb, v, cin, cout, Y, s);
    case 2: return launch_col_kb<T, 2, 2>(X, xb, Bt, wb, v, cin, cout, Y, s);
    default:
      if constexpr (sizeof(T) == 2) {
        if ((cin + 63) / 64 == 3) return launch_col_kb<T, 3, 2>(X, xb, Bt, wb, v, cin, cout, Y, s);
        return launch_col_kb<T, 4, 2>(X, xb, Bt, wb, v, cin, cout, Y, s);
      }
      return fail(SSCN_ERR_SHAPE, "channel count outside the column kernel");
  }
}

template <typename T>
static bool quad_eligible(const View& v, int cin, int cout) {
  const uint64_t x_bytes = (uint64_t)std::max<int64_t>(v.n_in, 1) * cin * sizeof(T);
  const uint64_t w_bytes = (uint64_t)v.K * cout * cin * sizeof(T);
  const int kb = (cin + 63) / 64;
  const int max_kb = sizeof(T) == 4 ? 2 : 4;  // register budget of the quad kernel
  return v.K <= 32767 && cin % 8 == 0 && kb <= max_kb && x_bytes < kOobOffset && w_bytes < kOobOffset;
}

// A temporary copy of the weights (K x c_in x c_out elements): from the
// block cache, or from the caller's region while a no-allocation entry point
// runs (then it is not released).
template <typename T>
static sscn_status temp_weights(T** p, int64_t count, hipStream_t s) {
  if (const NoAlloc* na = no_alloc()) {
    if ((size_t)count * sizeof(T) > na->bytes) return fail(SSCN_ERR_INVALID_ARG, "weights exceed the scratch region");
    *p = (T*)na->scratch;
    return SSCN_OK;
  }
  return dev_alloc((void**)p, sizeof(T) * count, s);
}

static void temp_release(void* p, hipStream_t s) {
  if (!no_alloc()) dev_free(p, s);
}

template <typename T, bool WT>
static sscn_status launch_conv(const T* X, const T* W, const View& v, int cin, int cout, const Heads<T>& Y, hipStream_t s) {
  if (v.st->n_tiles == 0) return SSCN_OK;
  if (WT && prefer_col<T>(v, cin, cout)) return launch_col<T>(X, W, v, cin, cout, Y, s);
  const uint64_t x_bytes = (uint64_t)std::max<int64_t>(v.n_in, 1) * cin * sizeof(T);
  const uint64_t w_bytes = (uint64_t)v.K * cout * cin * sizeof(T);
  const int kb = (cin + 63) / 64;
  if (quad_eligible<T>(v, cin, cout)) {
    const uint32_t xb = (uint32_t)x_bytes, wb = (uint32_t)w_bytes;
    switch (kb) {
      case 1: return launch_quad<T, 4, 1, WT>(X, xb, W, wb, v, cin, cout, Y, s);
      case 2: return launch_quad<T, 3, 2, WT>(X, xb, W, wb, v, cin, cout, Y, s);
      default:
        if constexpr (sizeof(T) == 2) {
          if (kb == 3) return launch_quad<T, 3, 3, WT>(X, xb, W, wb, v, cin, cout, Y, s);
          return launch_quad<T, 3, 4, WT>(X, xb, W, wb, v, cin, cout, Y, s);
        }
        break;
    }
  }
  const T* Bt = W;
  T* tmp = nullptr;
  if constexpr (!WT) {
    const int64_t total = (int64_t)v.K * cin * cout;
    SSCN_TRY(temp_weights(&tmp, total, s));
    k_transpose_w<T><<<(unsigned)std::min<int64_t>(ceil_div(total, 256), 4096), 256, 0, s>>>(W, v.K, cin, cout, tmp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
      temp_release(tmp, s);
      return hip_fail(e, "transpose launch");
    }
    Bt = tmp;
  }
  sscn_status st = launch_generic(X, Bt, v, cin, cout, Y, s);
  temp_release(tmp, s);
  return st;
}


// Row-block kernel: B laid out [o][ncols][kdim]; K <= kPlanMaxK (offset
// sets of up to three 32-bit words), whole 8-channel runs, 32-bit buffer
// offsets.
template <typename T>
static bool rows_eligible(const View& v, int kdim, int ncols) {
  const uint64_t x_bytes = (uint64_t)std::max<int64_t>(v.n_in, 1) * kdim * sizeof(T);
  const uint64_t b_bytes = (uint64_t)v.K * ncols * kdim * sizeof(T);
  return v.K <= kPlanMaxK && kdim % 8 == 0 && x_bytes < kOobOffset && b_bytes < kOobOffset &&
         std::max(v.n_in, v.n_out) < (int64_t)kPlanNoRow && ceil_div(v.n_out, kPlanRows) * v.K < INT32_MAX;
}

template <typename T, int WB, int NB, int PK = 1, bool TB = false, bool DG = false, bool SP = false>
static sscn_status launch_rows_nb(const T* X, const void* B, const View& v, int kdim, int ncols, const Heads<T>& Y,
                                  hipStream_t s) {
  const int64_t nb = v.st->n_blocks;
  if (nb == 0) return Y.n_zero > 0 ? fill_f32(Y.zero, 0.f, Y.n_zero, s) : SSCN_OK;
  const int gy = (ncols + 16 * NB - 1) / (16 * NB);
  const uint32_t xb = (uint32_t)((uint64_t)std::max<int64_t>(v.n_in, 1) * kdim * sizeof(T));
  // SP: three bf16 planes
  const uint32_t bb = (uint32_t)((uint64_t)v.K * ncols * kdim * (SP ? 6 : sizeof(T)));
  // loads two steps ahead for 64-byte windows (short steps), one otherwise;
  // six workgroups per CU for 64-byte windows (80 VGPRs), five otherwise
  constexpr int D = WB == 64 ? 3 : 2;
  auto kern = [] {
    if constexpr (DG) return k_dgrad_rows<T, WB, NB, D, PK, TB, SP>;
    else return k_conv_rows<T, WB, NB, D, PK, TB, SP>;
  }();
  int cus = 256, per_cu = 1;
  occupancy((const void*)kern, 256, 0, &per_cu, &cus);
  // persistent: one resident wave of workgroups per column group
  const int64_t gx = std::min<int64_t>(nb, std::max<int64_t>(1, (int64_t)cus * per_cu / gy));
  hipEvent_t t0, t1;
  if (take_launch_timer(&t0, &t1))
    hipExtLaunchKernelGGL(kern, dim3((unsigned)gx, (unsigned)gy), dim3(256), 0, s, t0, t1, 0, X, xb, B, bb, v.st->perm,
                          v.st->b_first, v.st->b_rec, v.st->items, nb, v.K, v.mirror ? 1 : 0, kdim, ncols, Y);
  else
    kern<<<dim3((unsigned)gx, (unsigned)gy), 256, 0, s>>>(X, xb, B, bb, v.st->perm, v.st->b_first, v.st->b_rec,
                                                           v.st->items, nb, v.K, v.mirror ? 1 : 0, kdim, ncols, Y);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

// Whether the forward hands launch_rows B as [o][kdim][ncols] (TB): fp32,
// whole 16-byte pieces of 4 columns, one item per step, and 32-column
// groups.  There the per-element LDS writes of the half-size weight tile
// cost less than the transposed copy (SC 64 -> 96 channels: 27.6 -> 24.8
// us); with 64-column groups they cost more (the 64-channel layer: 136 ->
// 152 us), and the copy is made.
template <typename T>
static bool rows_take_untransposed(int kdim, int ncols) {
  return sizeof(T) == 4 && ncols % 4 == 0 && ncols % 64 != 0 && kdim * sizeof(T) != 64;
}

// Whether an fp32 launch of the row kernel runs through bf16 parts (the
// weights handed over as the three planes of k_split_w): rows of 16 or at
// least 32 channels (one item per 32-channel window, channels past the
// row's end read as zeros; rows of 24 channels run faster on the fp32
// MFMAs), and the planes within 32-bit buffer offsets.
static bool rows_split(const View& v, int kdim, int ncols) {
  return (kdim == 16 || kdim >= 32) && (uint64_t)v.K * ncols * kdim * 6 < kOobOffset;
}

// DG: a dgrad launch (k_dgrad_rows), else a forward one (k_conv_rows).
// SP: fp32 through bf16 parts, B = the weight planes.
template <typename T, bool DG = false, bool SP = false>
static sscn_status launch_rows(const T* X, const void* B, const View& v, int kdim, int ncols, const Heads<T>& Y,
                               hipStream_t s, bool untransposed = false) {
  if (v.n_out == 0) return Y.n_zero > 0 ? fill_f32(Y.zero, 0.f, Y.n_zero, s) : SSCN_OK;
  SSCN_TRY(ensure_plan(v, s));
  if constexpr (SP) {
    static_assert(sizeof(T) == 4, "split path: fp32");
    return ncols % 64 == 0 ? launch_rows_nb<T, 128, 4, 1, false, DG, true>(X, B, v, kdim, ncols, Y, s)
                           : launch_rows_nb<T, 128, 2, 1, false, DG, true>(X, B, v, kdim, ncols, Y, s);
  }
  // 64 output columns per workgroup when they divide the width, else 32;
  // for bf16 (bound by loads and step latency rather than MFMAs) 64 unless
  // the width is at most 32: fewer column groups re-read the input rows
  // fewer times, and a partial last group costs less than a third group at
  // 96 or 160 columns.  128-byte windows (32 fp32 or 64 bf16 channels)
  // unless a bf16 row is not a multiple of 128 bytes.
  const bool wide_cols = sizeof(T) == 2 ? ncols > 32 : ncols % 64 == 0;
  if constexpr (sizeof(T) == 4 && !DG) {
    if (untransposed) {
      if (!rows_take_untransposed<T>(kdim, ncols)) return fail(SSCN_ERR_INVALID_ARG, "weights layout");
      return launch_rows_nb<T, 128, 2, 1, true, DG>(X, B, v, kdim, ncols, Y, s);
    }
  }
  // Rows of 32 bf16 channels (half a window): two items per step, each in
  // an MFMA of its own.  Rows of 16 bf16 channels take one item per 64-byte
  // window, half of it zeros, and fp32 rows one item per window: an MFMA
  // over two items' channels would round a row's sum by the pairing of its
  // block's items, and so by which rows share the block.
  const uint32_t row_bytes = (uint32_t)kdim * sizeof(T);
  if (sizeof(T) == 2 && row_bytes == 64)
    return wide_cols ? launch_rows_nb<T, 128, 4, 2, false, DG>(X, B, v, kdim, ncols, Y, s)
                     : launch_rows_nb<T, 128, 2, 2, false, DG>(X, B, v, kdim, ncols, Y, s);
  if constexpr (sizeof(T) == 2) {
    if (kdim % 64 != 0)
      return wide_cols ? launch_rows_nb<T, 64, 4, 1, false, DG>(X, B, v, kdim, ncols, Y, s)
                       : launch_rows_nb<T, 64, 2, 1, false, DG>(X, B, v, kdim, ncols, Y, s);
  }
  return wide_cols ? launch_rows_nb<T, 128, 4, 1, false, DG>(X, B, v, kdim, ncols, Y, s)
                   : launch_rows_nb<T, 128, 2, 1, false, DG>(X, B, v, kdim, ncols, Y, s);
}

// N contiguous channels of one row as fp32, one raw buffer load (an
// out-of-range offset reads zeros).
template <typename T, int N> struct RowLoad;
template <int N> struct RowLoad<float, N> {
  static __device__ __forceinline__ void load(rsrc_t r, uint32_t off, float (&v)[N]) {
    if constexpr (N == 4) {
      const auto q = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
      v[0] = __uint_as_float(q[0]); v[1] = __uint_as_float(q[1]); v[2] = __uint_as_float(q[2]); v[3] = __uint_as_float(q[3]);
    } else if constexpr (N == 2) {
      const auto q = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
      v[0] = __uint_as_float(q[0]); v[1] = __uint_as_float(q[1]);
    } else {
      v[0] = __uint_as_float((uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
    }
  }
};
template <int N> struct RowLoad<bf16_t, N> {
  static __device__ __forceinline__ void load(rsrc_t r, uint32_t off, float (&v)[N]) {
    if constexpr (N == 4) {
      const auto q = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
      v[0] = bf16_to_f32(q[0] & 0xffff); v[1] = bf16_to_f32(q[0] >> 16);
      v[2] = bf16_to_f32(q[1] & 0xffff); v[3] = bf16_to_f32(q[1] >> 16);
    } else if constexpr (N == 2) {
      const uint32_t q = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
      v[0] = bf16_to_f32(q & 0xffff); v[1] = bf16_to_f32(q >> 16);
    } else {
      v[0] = bf16_to_f32((uint16_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0));
    }
  }
};

// Work items of k_wgrad_ring: the output tiles are cut into ranges of `tr`
// tiles; within a range, offset o contributes sub[o] items that split its
// pairs in that range evenly (sub[o] ~ pairs of o / mean pairs per offset,
// so that items have similar sizes).  first[o] = sum of sub[q], q < o.
constexpr int kWgradMaxK = 128;
// wgrad on 16x16x32 bf16 MFMAs (see k_wgrad_ring)
constexpr bool kWgradM32 = true;
struct WgradItems {
  int32_t first[kWgradMaxK + 1];
};

// The same contraction as k_wgrad_reg with balanced items and a deeper
// pipeline.  Items are numbered range-major (all items of tile range r, then
// r + 1, ...) and renumbered so that each XCD takes a contiguous run of
// ranges (L2 locality across the offsets of one range).  Each wavefront
// walks its pairs 4 at a time (one MFMA step).  The pairs' row indices come
// in batches of 64 (one coalesced load per 16 steps, two batches ahead) and
// reach the lanes by shuffles; the rows are loaded R steps ahead into a
// register ring with compile-time slots.  Row loads are branch-free (a pair
// past the end reads out-of-range offsets, i.e. zeros), so the compiler's
// wait counts stay exact; a wave's last batch is padded with such empty
// steps.  Needs X and dY below kOobOffset bytes.
// M32: 16x16x32 bf16 MFMAs instead of 16x16x4 fp32 ones.  Such an MFMA
// takes 8 reduction values per lane; here the reduction runs over the
// pairs, and 8 consecutive steps give lane (m, g) the pairs 4 s + g, s < 8,
// of its channel -- exactly the operand layout (lane group g, element s),
// with the B lanes of group g holding the same 8 pairs.  So the values of 8
// steps are packed (bf16 in the high half of each 32-bit word, two words per
// register) and multiplied once per 8 steps.  bf16 inputs enter as they are
// (exact products); fp32 inputs are split into three bf16 parts and take
// six MFMAs (as in the row kernel).
template <typename T, int CA, int CB, int R, bool M32 = false>
__global__ __launch_bounds__(256) void k_wgrad_ring(const T* __restrict__ X, uint32_t x_bytes,
                                                    const T* __restrict__ dY, uint32_t y_bytes,
                                                    const int64_t* __restrict__ seg, int64_t n_tiles,
                                                    const int32_t* __restrict__ in_rows,
                                                    const int32_t* __restrict__ out_rows, int K, int mirror,
                                                    int cin, int cout, int tr, WgradItems items, int nzc,
                                                    float* __restrict__ dW, float* __restrict__ det) {
  static_assert(16 % R == 0, "ring depth must divide a batch");
  const int S = items.first[K];
  const int64_t item = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t r = item / S;
  const int w = (int)(item % S);
  int o = 0;
  while (items.first[o + 1] <= w) ++o;
  const int sub = w - items.first[o], n_sub = items.first[o + 1] - items.first[o];
  const int so = mirror ? K - 1 - o : o;
  const int64_t t_lo = r * tr, t_hi = min<int64_t>(t_lo + tr, n_tiles);
  const int64_t rb = seg[(int64_t)so * n_tiles + t_lo];
  const int64_t rn = seg[(int64_t)so * n_tiles + t_hi] - rb;
  const int64_t pb = rb + rn * sub / n_sub, pe = rb + rn * (sub + 1) / n_sub;
  // det: this item's block goes to its own slot of det (zeros when it has
  // no pairs) instead of being added to dW, for a fixed-order sum after.
  constexpr int NE = CA * CB * 4;
  float* const det_blk = det ? det + (item * gridDim.y + blockIdx.y) * (NE * 64) : nullptr;
  if (pb >= pe) {
    if (det_blk)
      for (int e = threadIdx.x; e < NE * 64; e += 256) det_blk[e] = 0.f;
    return;
  }
  const int ci0 = (blockIdx.y % nzc) * 16 * CA, co0 = (blockIdx.y / nzc) * 16 * CB;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  // a lane's channels are fully inside or fully outside [0, cin) / [0, cout)
  const uint32_t a_lane = ci0 + CA * m + CA <= cin ? (uint32_t)(ci0 + CA * m) * sizeof(T) : kOobOffset;
  const uint32_t b_lane = co0 + CB * m + CB <= cout ? (uint32_t)(co0 + CB * m) * sizeof(T) : kOobOffset;
  const uint32_t x_row = (uint32_t)cin * sizeof(T), y_row = (uint32_t)cout * sizeof(T);
  const rsrc_t rx = make_rsrc(X, x_bytes), ry = make_rsrc(dY, y_bytes);
  const int64_t per = ((pe - pb + 3) / 4 + 3) / 4 * 4;
  const int64_t wb = pb + wave * per, we = min<int64_t>(wb + per, pe);

  f32x4 d[CA][CB];
#pragma unroll
  for (int a = 0; a < CA; ++a)
#pragma unroll
    for (int b = 0; b < CB; ++b) d[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (wb < we) {
    // pair indices: one coalesced load per 64 pairs (16 steps), lane l
    // holding pair base + l; a step's pair for lane group g is taken from
    // lane 4 s + g of the batch by a shuffle
    int32_t bi_in[3], bi_out[3];   // batches k, k + 1, k + 2 (in flight)
    float xa[R][CA], yb[R][CB];
    auto load_batch = [&](int64_t base, int slot) {
      const int64_t q = min<int64_t>(base + lane, we - 1);
      bi_in[slot] = in_rows[q];
      bi_out[slot] = out_rows[q];
    };
    // rows of step t (t = 16 batch + s; `slot` holds that batch)
    const int n_mine = (int)(we - wb);  // pairs of this wavefront
    auto fetch_rows = [&](int t, int slot, int s16, int ds) {
      const int src = 4 * s16 + g;
      const int32_t irow = __shfl(bi_in[slot], src, 64);
      const int32_t orow = __shfl(bi_out[slot], src, 64);
      const bool ok = 4 * t + g < n_mine;
      const uint32_t xo = ok ? (uint32_t)irow * x_row : kOobOffset;
      const uint32_t yo = ok ? (uint32_t)orow * y_row : kOobOffset;
      RowLoad<T, CA>::load(rx, xo + a_lane, xa[ds]);
      RowLoad<T, CB>::load(ry, yo + b_lane, yb[ds]);
    };
    const int n_steps = (n_mine + 3) / 4;
    // M32: planes of the packed operands (3 for fp32 parts, 1 for bf16)
    constexpr int NP = sizeof(T) == 4 ? 3 : 1;
    uint32_t pa[M32 ? NP : 1][CA][4], pb[M32 ? NP : 1][CB][4];  // 8 steps, two per register
    uint32_t ea[M32 ? NP : 1][CA], eb[M32 ? NP : 1][CB];        // the even step's words
    auto words = [&](float v, uint32_t (&w)[M32 ? NP : 1]) {
      if constexpr (NP == 3) split3(v, w[0], w[1], w[2]);
      else w[0] = __float_as_uint(v);  // a bf16 value: its bits in the high half
    };
    load_batch(wb, 0);
    load_batch(wb + 64, 1);
#pragma unroll
    for (int sl = 0; sl < R; ++sl) fetch_rows(sl, 0, sl, sl);
    for (int b0 = 0; b0 < n_steps; b0 += 16) {
      load_batch(wb + 4 * (b0 + 32), 2);
#pragma unroll
      for (int s16 = 0; s16 < 16; ++s16) {
        const int ds = s16 % R;
        if constexpr (M32) {
          const int e = s16 % 8;  // element of the group's operands
#pragma unroll
          for (int a = 0; a < CA; ++a) {
            uint32_t w[NP];
            words(xa[ds][a], w);
#pragma unroll
            for (int pl = 0; pl < NP; ++pl) {
              if (e % 2 == 0) ea[pl][a] = w[pl];
              else pa[pl][a][e / 2] = pack_hi16(ea[pl][a], w[pl]);
            }
          }
#pragma unroll
          for (int b = 0; b < CB; ++b) {
            uint32_t w[NP];
            words(yb[ds][b], w);
#pragma unroll
            for (int pl = 0; pl < NP; ++pl) {
              if (e % 2 == 0) eb[pl][b] = w[pl];
              else pb[pl][b][e / 2] = pack_hi16(eb[pl][b], w[pl]);
            }
          }
          if (e == 7) {
            auto op = [](const uint32_t (&q)[4]) {
              uint4 u;
              u.x = q[0]; u.y = q[1]; u.z = q[2]; u.w = q[3];
              return __builtin_bit_cast(bf16x8, u);
            };
            if constexpr (NP == 3) {
              // the six part products, smallest first; one pass over all
              // blocks per product keeps the accumulator chains apart
              constexpr int PA[6] = {0, 1, 2, 0, 1, 0}, PB[6] = {2, 1, 0, 1, 0, 0};
#pragma unroll
              for (int pr = 0; pr < 6; ++pr)
#pragma unroll
                for (int a = 0; a < CA; ++a)
#pragma unroll
                  for (int b = 0; b < CB; ++b)
                    d[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(op(pa[PA[pr]][a]), op(pb[PB[pr]][b]), d[a][b],
                                                                      0, 0, 0);
            } else {
#pragma unroll
              for (int a = 0; a < CA; ++a)
#pragma unroll
                for (int b = 0; b < CB; ++b)
                  d[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(op(pa[0][a]), op(pb[0][b]), d[a][b], 0, 0, 0);
            }
          }
        } else {
#pragma unroll
          for (int a = 0; a < CA; ++a)
#pragma unroll
            for (int b = 0; b < CB; ++b)
              d[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(xa[ds][a], yb[ds][b], d[a][b], 0, 0, 0);
        }
        const int nx = s16 + R;  // step to request, relative to this batch
        if (nx < 16)
          fetch_rows(b0 + nx, 0, nx, ds);
        else
          fetch_rows(b0 + nx, 1, nx - 16, ds);
        // keep this step's row loads here: the compiler otherwise sinks them
        // towards their use R steps later, which empties the ring
        __builtin_amdgcn_sched_barrier(0);
      }
      bi_in[0] = bi_in[1]; bi_out[0] = bi_out[1];
      bi_in[1] = bi_in[2]; bi_out[1] = bi_out[2];
    }
  }
  // sum the four wavefronts' partial blocks, then add the block to dW
  // (as in k_wgrad_reg)
  __shared__ float part[2][NE][64];
  float(*mine)[64] = part[wave & 1];
  if (wave < 2) {
#pragma unroll
    for (int a = 0; a < CA; ++a)
#pragma unroll
      for (int b = 0; b < CB; ++b)
#pragma unroll
        for (int q = 0; q < 4; ++q) mine[(a * CB + b) * 4 + q][lane] = d[a][b][q];
  }
  __syncthreads();
  if (wave >= 2) {
#pragma unroll
    for (int a = 0; a < CA; ++a)
#pragma unroll
      for (int b = 0; b < CB; ++b)
#pragma unroll
        for (int q = 0; q < 4; ++q) mine[(a * CB + b) * 4 + q][lane] += d[a][b][q];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < NE * 64; e += 256) {
    const int v = e / 64, l = e % 64;
    const float sum = part[0][v][l] + part[1][v][l];
    const int a = v / (CB * 4), b = (v / 4) % CB, q = v % 4;
    const int mm = l & 15, gg = l >> 4;
    const int ci = ci0 + CA * (4 * gg + q) + a, co = co0 + CB * mm + b;
    if (det_blk) det_blk[e] = sum;
    else if (ci < cin && co < cout && sum != 0.f) atomicAdd(dW + ((int64_t)o * cin + ci) * cout + co, sum);
  }
}

// Deterministic mode of k_wgrad_ring: dW[o][ci][co] = the sum of the item
// blocks of offset o in a fixed order (tile ranges, then sub-items), from
// the blocks the items wrote (element e = v 64 + l of a block holds
// (ci, co) = (ci0 + CA (4 (l >> 4) + v % 4) + v / (4 CB), co0 + CB (l & 15)
// + (v / 4) % CB)).
template <int CA, int CB>
__global__ void k_wgrad_det_sum(const float* __restrict__ det, int K, int cin, int cout, int nzc, int gy,
                                int64_t ranges, WgradItems items, float* __restrict__ dW) {
  constexpr int NE = CA * CB * 4;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t per_o = (int64_t)cin * cout;
  if (t >= K * per_o) return;
  const int o = (int)(t / per_o);
  const int ci = (int)((t % per_o) / cout), co = (int)(t % cout);
  const int ib = ci / (16 * CA), jb = co / (16 * CB);
  const int by = jb * nzc + ib;
  const int dci = ci - ib * 16 * CA, dco = co - jb * 16 * CB;
  const int a = dci % CA, tt = dci / CA, gg = tt / 4, q = tt % 4;
  const int b = dco % CB, mm = dco / CB;
  const int e = ((a * CB + b) * 4 + q) * 64 + gg * 16 + mm;
  const int S = items.first[K];
  float sum = 0.f;
  for (int64_t r = 0; r < ranges; ++r)
    for (int w = items.first[o]; w < items.first[o + 1]; ++w)
      sum += det[((r * S + w) * gy + by) * (int64_t)(NE * 64) + e];
  dW[(int64_t)o * per_o + ci * cout + co] = sum;
}

template <typename T, int CA, int CB>
static sscn_status launch_wgrad_reg(bool zeroed, const T* X, const T* dY, const View& v, int cin, int cout, float* dW,
                                    hipStream_t s, int64_t max_ppo, int64_t n_pairs) {
  (void)max_ppo;
  (void)n_pairs;
  if (v.st->n_tiles == 0) return SSCN_OK;
  // about 1024 (tile range, offset) items
  const int64_t tr = std::max<int64_t>(1, ceil_div(v.st->n_tiles * v.K, 1024));
  const int64_t n_items = ceil_div(v.st->n_tiles, tr) * v.K;
  const int nzc = (cin + 16 * CA - 1) / (16 * CA);
  const int nzo = (cout + 16 * CB - 1) / (16 * CB);
  const uint64_t x_bytes = (uint64_t)std::max<int64_t>(v.n_in, 1) * cin * sizeof(T);
  const uint64_t y_bytes = (uint64_t)std::max<int64_t>(v.n_out, 1) * cout * sizeof(T);
  if (x_bytes < kOobOffset && y_bytes < kOobOffset && v.K <= kWgradMaxK) {
    // sub-items per offset ~ its share of the pairs; about one resident
    // round of workgroups in all (each item adds its block to dW with
    // atomics, so fewer, longer items cost less)
    const std::vector<int64_t>& ppo = v.owner->pairs_per_offset;
    const double mean = (double)std::max<int64_t>(v.n_pairs, 1) / v.K;
    WgradItems items{};
    items.first[0] = 0;
    for (int o = 0; o < v.K; ++o) {
      const double p = (double)ppo[v.mirror ? v.K - 1 - o : o];
      items.first[o + 1] = items.first[o] + std::max(1, (int)(p / mean + 0.5));
    }
    const int S = items.first[v.K];
    auto kern = k_wgrad_ring<T, CA, CB, 4, kWgradM32>;
    int cus = 256, per_cu = 1;
    occupancy((const void*)kern, 256, 0, &per_cu, &cus);
    const int64_t target = std::max<int64_t>(1, (int64_t)cus * per_cu / (nzc * nzo));
    // at most target / S tile ranges, so that the items fit one round
    // (a few items left for a second round would double the kernel's time)
    const int64_t ranges = std::max<int64_t>(1, target / S);
    const int64_t tr2 = std::max<int64_t>(1, ceil_div(v.st->n_tiles, ranges));
    const int64_t total = ceil_div(v.st->n_tiles, tr2) * S;
    // deterministic mode: every item block to its own slot, then a
    // fixed-order sum (no fill: the sum overwrites dW)
    const int gy = nzc * nzo;
    float* det = nullptr;
    if (deterministic()) {
      SSCN_TRY(dev_alloc((void**)&det, sizeof(float) * (size_t)total * gy * (CA * CB * 4 * 64), s));
    } else if (!zeroed) {
      SSCN_TRY(fill_f32(dW, 0.f, (int64_t)v.K * cin * cout, s));
    }
    hipEvent_t t0, t1;
    if (take_launch_timer(&t0, &t1))
      hipExtLaunchKernelGGL(kern, dim3((unsigned)total, (unsigned)gy), dim3(256), 0, s, t0, t1, 0, X,
                            (uint32_t)x_bytes, dY, (uint32_t)y_bytes, v.st->seg, v.st->n_tiles, v.st->in_rows,
                            v.st->out_rows, v.K, v.mirror ? 1 : 0, cin, cout, (int)tr2, items, nzc, dW, det);
    else
      kern<<<dim3((unsigned)total, (unsigned)gy), 256, 0, s>>>(
          X, (uint32_t)x_bytes, dY, (uint32_t)y_bytes, v.st->seg, v.st->n_tiles, v.st->in_rows, v.st->out_rows, v.K,
          v.mirror ? 1 : 0, cin, cout, (int)tr2, items, nzc, dW, det);
    if (det) {
      hipError_t e = hipGetLastError();
      if (e == hipSuccess) {
        const int64_t n_out = (int64_t)v.K * cin * cout;
        k_wgrad_det_sum<CA, CB><<<(unsigned)ceil_div(n_out, 256), 256, 0, s>>>(
            det, v.K, cin, cout, nzc, gy, total / items.first[v.K], items, dW);
        e = hipGetLastError();
      }
      dev_free(det, s);
      if (e != hipSuccess) return hip_fail(e, "deterministic wgrad");
    }
    SSCN_HIP(hipGetLastError());
    return SSCN_OK;
  }
  if (!zeroed) SSCN_TRY(fill_f32(dW, 0.f, (int64_t)v.K * cin * cout, s));
  k_wgrad_reg<T, CA, CB><<<dim3((unsigned)n_items, (unsigned)(nzc * nzo)), 256, 0, s>>>(
      X, dY, v.st->seg, v.st->n_tiles, v.st->in_rows, v.st->out_rows, v.K, v.mirror ? 1 : 0, cin, cout, (int)tr,
      nzc, dW);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

// Channel blocking: CA (CB) is the number of 16-row blocks per workgroup,
// chosen so a lane's channels are contiguous and the channel count is
// covered without wasted blocks.
static int wgrad_blocks(int c) {
  if (c % 4 == 0 && c >= 64) return 4;
  if (c % 2 == 0 && c >= 32) return 2;
  return 1;
}

// ------------------------------------------------ row-block wgrad (bf16)
// dW_o = sum over the pairs (j, k) of offset o of X[j]^T dY[k] for bf16
// layers of 32, 64, 96, 128 or 160 output channels and a multiple of 32
// input channels (a workgroup takes one tile of CI input channels and all
// CO output ones; wider inputs are split over several tiles, each with its
// own slice of the X rows and all of the dY rows).  A workgroup takes blocks of the
// row-block plan (64 output rows k with one item per offset of their
// union, as the forward walks them): the block's dY rows and each item's
// gathered X rows go straight into row-major LDS tiles (direct loads, 16
// bytes per lane; absent rows read zeros), and both MFMA operands are read
// from those tiles transposed (LDS transpose reads of four 16-bit elements
// per lane): a 16 x 16 x 32 bf16 MFMA then sums over 32 of the block's rows.
// Each wavefront keeps the output tiles of its workgroup's offset group
// (blockIdx.y) in registers over all its blocks; the workgroups' partial
// sums are added in a fixed order afterwards (k_wgrad_sum), so dW is
// bit-reproducible.  At these widths the per-pair wgrad gives a lane 4
// bytes of X and of dY per pair, and its load instructions bind.
typedef short wg_v4s __attribute__((ext_vector_type(4)));

// Lane (m, g) of a 16 x 16 x 32 operand from a row-major LDS tile of 64 rows
// (rb bytes each): rows 32 ks + 8 g .. + 7 of column 16 cb + m, through two
// transpose reads.  In a group of 16 lanes the read hands lane i element
// (i & 3) of the 8 bytes that lane 4 k + (i >> 2) addressed, as its element
// k: so lane j addresses row 8 g + 4 h + (j >> 2), columns 16 cb + 4 (j & 3)
// .. + 3, for the halves h = 0, 1.
__device__ __forceinline__ bf16x8 tile_operand_tr(const char* tile, int rb, int cb, int ks, int lane) {
  const int j = lane & 15, g = lane >> 4;
  const char* p = tile + (32 * ks + 8 * g + (j >> 2)) * rb + (16 * cb + 4 * (j & 3)) * 2;
  const wg_v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) wg_v4s*)p);
  const wg_v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) wg_v4s*)(p + 4 * rb));
  const uint2 a = __builtin_bit_cast(uint2, lo), b = __builtin_bit_cast(uint2, hi);
  return __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
}

// A tile of CI x CO channels; OPG offsets per group; grid.y = channel
// tiles x groups (y = tile * groups + group; tile = input-channel slice of
// CI channels, TILED: x_ld / (2 CI) of them, else one with x_ld = 2 CI);
// partials P[y][x][oo][CI][CO] (x < gridDim.x workgroups).  x_ld: bytes
// per row of X.  The 16 x 16 output tiles t = (ti, tj) are dealt TPW per
// wavefront in row-major order: either a wavefront's tiles share one row ti
// (TPW <= NTJ) or cover whole rows.
template <int CI, int CO, int OPG, bool TILED>
__global__ __launch_bounds__(256) void k_wgrad_rows(const bf16_t* __restrict__ X, uint32_t x_bytes, uint32_t x_ld,
                                                    const bf16_t* __restrict__ dY, uint32_t y_bytes,
                                                    const int32_t* __restrict__ perm,
                                                    const int4* __restrict__ b_rec,
                                                    const uint32_t* __restrict__ items, int64_t n_blocks, int K,
                                                    int groups, float* __restrict__ part) {
  constexpr int NTI = CI / 16, NTJ = CO / 16, TPW = NTI * NTJ / 4;
  constexpr bool ONE_ROW = TPW <= NTJ;               // the wavefront's tiles share ti
  constexpr int NA = ONE_ROW ? 1 : TPW / NTJ;        // tile rows (A operands) per wavefront
  constexpr int NB = ONE_ROW ? TPW : NTJ;            // tile columns (B operands) per wavefront
  static_assert(NTI * NTJ % 4 == 0 && (ONE_ROW ? NTJ % TPW == 0 : TPW % NTJ == 0), "tiles dealt evenly");
  constexpr int XB = CI * 2, YB = CO * 2;          // bytes per tile row
  constexpr int XCH = 64 * XB / 1024, YCH = 64 * YB / 1024;  // 1 KB load chunks per tile
  static_assert(XCH % 4 == 0 && YCH % 4 == 0, "whole chunks per wavefront");
  __shared__ __attribute__((aligned(16))) char Xs[2][64 * XB];
  __shared__ __attribute__((aligned(16))) char Ys[64 * YB];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int o_lo = (int)(TILED ? blockIdx.y % (unsigned)groups : blockIdx.y) * OPG, o_hi = min(K, o_lo + OPG);
  // the tile's bytes of an X row, and the row pitch
  const uint32_t x0 = TILED ? blockIdx.y / (unsigned)groups * (uint32_t)XB : 0u;
  const uint32_t xp = TILED ? x_ld : (uint32_t)XB;
  // this wavefront's tiles: t = TPW wave + q, (ti, tj) = (t / NTJ, t % NTJ):
  // rows ti0 + a (a < NA), columns tj0 + bq (bq < NB)
  const int ti0 = (TPW * wave) / NTJ, tj0 = ONE_ROW ? (TPW * wave) % NTJ : 0;
  const rsrc_t rx = make_rsrc(X, x_bytes), ry = make_rsrc(dY, y_bytes);
  f32x4 acc[OPG][TPW];
#pragma unroll
  for (int oo = 0; oo < OPG; ++oo)
#pragma unroll
    for (int q = 0; q < TPW; ++q) acc[oo][q] = f32x4{0.f, 0.f, 0.f, 0.f};

  // per chunk c this lane loads: tile row and 16-byte piece
  auto x_row = [&](int c) { return (c * 1024 + 16 * lane) / XB; };
  auto x_piece = [&](int c) { return (uint32_t)((c * 1024 + 16 * lane) % XB); };
  constexpr int NXC = XCH / 4;  // X chunks per wavefront
  uint32_t ent[NXC];            // entries of the next item's rows
  auto load_entries = [&](int64_t item) {
#pragma unroll
    for (int i = 0; i < NXC; ++i) ent[i] = items[item * kPlanRows + x_row(wave + 4 * i)];
  };
  auto dma_x = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NXC; ++i) {
      const int c = wave + 4 * i;
      const uint32_t r = ent[i] & kPlanNoRow;
      const uint32_t off = r != kPlanNoRow ? r * xp + x0 + x_piece(c) : kOobOffset;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (__attribute__((address_space(3))) void*)&Xs[buf][c * 1024], 16,
                                               (int)off, 0, 0, 0);
    }
  };

  const int64_t G = gridDim.x, wg = blockIdx.x;
  auto next = [&](int64_t round) { return round * G + ((round & 1) ? G - 1 - wg : wg); };
  for (int64_t idx = wg, round = 0; idx < n_blocks; idx = next(++round)) {
    const int4 rec = b_rec[idx];  // (block, first item, items)
    const int64_t b = rec.x;
    const int64_t first = rec.y;
    const int n_items = rec.z;
    // the items of this offset group: [j0, j1) (items are in increasing offset)
    const uint32_t oj = lane < n_items ? items[(first + lane) * kPlanRows] >> kPlanRowBits : 0xffu;
    const uint64_t below = __ballot(lane < n_items && (int)oj < o_lo);
    const uint64_t inside = __ballot(lane < n_items && (int)oj >= o_lo && (int)oj < o_hi);
    if (inside == 0) continue;  // uniform: no barrier skipped by some wavefronts only
    int j = __popcll(below);
    const int j1 = j + __popcll(inside);
    __syncthreads();  // the previous block's tiles are no longer read
    // the block's dY rows and the first item's X rows
#pragma unroll
    for (int i = 0; i < YCH / 4; ++i) {
      const int c = wave + 4 * i;
      const int row = (c * 1024 + 16 * lane) / YB;
      const int32_t k = perm[b * kPlanRows + row];
      const uint32_t off = k >= 0 ? (uint32_t)k * YB + (uint32_t)((c * 1024 + 16 * lane) % YB) : kOobOffset;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ry, (__attribute__((address_space(3))) void*)&Ys[c * 1024], 16,
                                               (int)off, 0, 0, 0);
    }
    load_entries(first + j);
    int buf = 0;
    dma_x(buf);
    if (j + 1 < j1) load_entries(first + j + 1);
    bf16x8 bop[NB][2];
    bool have_b = false;
    int o_cur = __builtin_amdgcn_readfirstlane((int)__shfl(oj, j, 64));
#pragma unroll
    for (int oo = 0; oo < OPG; ++oo) {
      if (j < j1 && o_cur == o_lo + oo) {  // uniform
        __syncthreads();  // item j's rows (and dY) landed; item j - 1's tile is free
        if (j + 1 < j1) {
          dma_x(buf ^ 1);
          if (j + 2 < j1) load_entries(first + j + 2);
        }
        if (!have_b) {
#pragma unroll
          for (int bq = 0; bq < NB; ++bq)
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) bop[bq][ks] = tile_operand_tr(Ys, YB, tj0 + bq, ks, lane);
          have_b = true;
        }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
          for (int a = 0; a < NA; ++a) {
            const bf16x8 av = tile_operand_tr(Xs[buf], XB, ti0 + a, ks, lane);
#pragma unroll
            for (int bq = 0; bq < NB; ++bq)
              acc[oo][a * NB + bq] =
                  __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bop[bq][ks], acc[oo][a * NB + bq], 0, 0, 0);
          }
        }
        buf ^= 1;
        ++j;
        o_cur = __builtin_amdgcn_readfirstlane((int)__shfl(oj, min(j, 63), 64));
      }
    }
  }
  // partial sums: lane (m, g) holds rows 4 g + r (c_in) of column m (c_out)
  const int m = lane & 15, g = lane >> 4;
  float* P = part + ((int64_t)blockIdx.y * gridDim.x + wg) * OPG * CI * CO;
#pragma unroll
  for (int oo = 0; oo < OPG; ++oo)
#pragma unroll
    for (int q = 0; q < TPW; ++q) {
      const int ti = ti0 + q / NB, tj = tj0 + q % NB;
#pragma unroll
      for (int r = 0; r < 4; ++r) P[((int64_t)oo * CI + 16 * ti + 4 * g + r) * CO + 16 * tj + m] = acc[oo][q][r];
    }
}

// dW[o'][ci][co] = the sum over the workgroups x of P[y][x][oo][ci'][co]
// for the stored offset o = g opg + oo and input channel ci = tile ti + ci'
// (y = tile groups + g; o' = K - 1 - o on a mirrored view), in a fixed
// order: a workgroup takes 64 consecutive outputs, its wavefront w the
// partials x = 4 i + w (four running sums, by i mod 4, eight loads in
// flight), and the sums are added in order of w and i mod 4.
__global__ __launch_bounds__(256) void k_wgrad_sum(const float* __restrict__ part, int K, int cin, int cout, int opg,
                                                   int ti, int groups, int64_t n_wg, int mirror,
                                                   float* __restrict__ dW) {
  __shared__ float red[4][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t per_o = (int64_t)cin * cout, per_t = (int64_t)ti * cout;
  const int64_t t = (int64_t)blockIdx.x * 64 + lane;
  const bool ok = t < K * per_o;
  const int o = ok ? (int)(t / per_o) : 0;
  const int64_t e = ok ? t % per_o : 0;
  const int tile = ti == cin ? 0 : (int)(e / cout) / ti;  // (uniform test: one tile needs no divisions)
  const int y = tile * groups + o / opg, oo = o % opg;
  const float* p = part + ((int64_t)y * n_wg * opg + oo) * per_t + e - (int64_t)tile * per_t;
  const int64_t xs = (int64_t)opg * per_t;  // from one workgroup's partials to the next
  float s[4] = {0.f, 0.f, 0.f, 0.f};
  int64_t x = wave;
  for (; x + 28 < n_wg; x += 32) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = ok ? p[(x + 4 * u) * xs] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) s[u % 4] += v[u];
  }
  for (int u = 0; x < n_wg; x += 4, ++u) s[u % 4] += ok ? p[x * xs] : 0.f;
  red[wave][lane] = (s[0] + s[1]) + (s[2] + s[3]);
  __syncthreads();
  if (wave == 0 && ok)
    dW[(int64_t)(mirror ? K - 1 - o : o) * per_o + e] = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
}

// Whether the row-block wgrad takes a bf16 layer: c_out one of 32, 64,
// 96, 128, 160 and c_in a multiple of 32 (at most 1024), and the plan's
// limits.
static bool wgrad_rows_eligible(const View& v, int cin, int cout) {
  const bool shape = (cout == 32 || cout == 64 || cout == 96 || cout == 128 || cout == 160) && cin % 32 == 0 &&
                     cin <= 1024;
  return shape && v.K <= 32 &&
         (uint64_t)std::max<int64_t>(v.n_in, 1) * cin * 2 < kOobOffset &&
         (uint64_t)std::max<int64_t>(v.n_out, 1) * cout * 2 < kOobOffset &&
         std::max(v.n_in, v.n_out) < (int64_t)kPlanNoRow;
}

template <int CI, int CO, int OPG>
static sscn_status launch_wgrad_rows_t(const bf16_t* X, const bf16_t* dY, const View& v, int cin, float* dW,
                                       hipStream_t s) {
  SSCN_TRY(ensure_plan(v, s));
  const int64_t nb = v.st->n_blocks;
  const int groups = (v.K + OPG - 1) / OPG, tiles = cin / CI;
  auto kern = tiles > 1 ? k_wgrad_rows<CI, CO, OPG, true> : k_wgrad_rows<CI, CO, OPG, false>;
  int cus = 256, per_cu = 1;
  occupancy((const void*)kern, 256, 0, &per_cu, &cus);
  // one resident wave of workgroups; at least 4 blocks each (fewer partial
  // sums to add on small layers)
  const int64_t gx = std::max<int64_t>(
      1, std::min<int64_t>(ceil_div(nb, 4), (int64_t)cus * per_cu / ((int64_t)groups * tiles)));
  float* part = nullptr;
  SSCN_TRY(dev_alloc((void**)&part, sizeof(float) * (size_t)gx * groups * tiles * OPG * CI * CO, s));
  const uint32_t xb = (uint32_t)((uint64_t)std::max<int64_t>(v.n_in, 1) * cin * 2);
  const uint32_t yb = (uint32_t)((uint64_t)std::max<int64_t>(v.n_out, 1) * CO * 2);
  const dim3 grid((unsigned)gx, (unsigned)(groups * tiles));
  hipEvent_t t0, t1;
  if (take_launch_timer(&t0, &t1))
    hipExtLaunchKernelGGL(kern, grid, dim3(256), 0, s, t0, t1, 0, X, xb, (uint32_t)cin * 2u, dY, yb, v.st->perm,
                          v.st->b_rec, v.st->items, nb, v.K, groups, part);
  else
    kern<<<grid, 256, 0, s>>>(X, xb, (uint32_t)cin * 2u, dY, yb, v.st->perm, v.st->b_rec, v.st->items, nb, v.K,
                              groups, part);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) {
    const int64_t total = (int64_t)v.K * cin * CO;
    k_wgrad_sum<<<(unsigned)ceil_div(total, 64), 256, 0, s>>>(part, v.K, cin, CO, OPG, CI, groups, gx,
                                                              v.mirror ? 1 : 0, dW);
    e = hipGetLastError();
  }
  dev_free(part, s);
  return e == hipSuccess ? SSCN_OK : hip_fail(e, "row-block wgrad");
}

static sscn_status launch_wgrad_rows(const bf16_t* X, const bf16_t* dY, const View& v, int cin, int cout, float* dW,
                                     hipStream_t s) {
  if (v.n_out == 0 || v.st->n_tiles == 0) return fill_f32(dW, 0.f, (int64_t)v.K * cin * cout, s);
  // Input-channel tiles of 128 (c_in = 128, c_out = 64), 64 where they
  // divide c_in, else 32; offsets per group: the wavefront's accumulators
  // (OPG x TPW x 4 VGPRs, TPW = CI CO / 1024) and operands within about 170
  // VGPRs; fewer where more resident workgroups paid off in the U-Net
  // training step (32 x 32: two groups of 14 instead of one of 27, 15.4 ->
  // 15.1 ms; 32 x 96 tiles 5 instead of 9, 64 x 96 tiles 2 instead of 4,
  // about 0.1 ms each).
  const bool t64 = cin % 64 == 0;
  switch (cout) {
    case 32:
      return t64 ? launch_wgrad_rows_t<64, 32, 14>(X, dY, v, cin, dW, s)
                 : launch_wgrad_rows_t<32, 32, 14>(X, dY, v, cin, dW, s);
    case 64:
      if (cin == 128) return launch_wgrad_rows_t<128, 64, 3>(X, dY, v, cin, dW, s);
      return t64 ? launch_wgrad_rows_t<64, 64, 6>(X, dY, v, cin, dW, s)
                 : launch_wgrad_rows_t<32, 64, 13>(X, dY, v, cin, dW, s);
    case 96:
      return t64 ? launch_wgrad_rows_t<64, 96, 2>(X, dY, v, cin, dW, s)
                 : launch_wgrad_rows_t<32, 96, 5>(X, dY, v, cin, dW, s);
    case 128:
      return t64 ? launch_wgrad_rows_t<64, 128, 3>(X, dY, v, cin, dW, s)
                 : launch_wgrad_rows_t<32, 128, 6>(X, dY, v, cin, dW, s);
    default:  // 160
      return t64 ? launch_wgrad_rows_t<64, 160, 2>(X, dY, v, cin, dW, s)
                 : launch_wgrad_rows_t<32, 160, 5>(X, dY, v, cin, dW, s);
  }
}

// zeroed: dW is already zero on stream s (cleared by the dgrad launch before it).
template <typename T>
static sscn_status launch_wgrad(const T* X, const T* dY, const View& v, int cin, int cout, float* dW,
                                hipStream_t s, int64_t max_ppo, int64_t n_pairs, bool zeroed = false) {
  const int ca = wgrad_blocks(cin), cb = wgrad_blocks(cout);
#define SSCN_WG(A, B) \
  if (ca == A && cb == B) return launch_wgrad_reg<T, A, B>(zeroed, X, dY, v, cin, cout, dW, s, max_ppo, n_pairs);
  SSCN_WG(4, 4) SSCN_WG(4, 2) SSCN_WG(4, 1) SSCN_WG(2, 4) SSCN_WG(2, 2) SSCN_WG(2, 1)
  SSCN_WG(1, 4) SSCN_WG(1, 2) SSCN_WG(1, 1)
#undef SSCN_WG
  return fail(SSCN_ERR_INVALID_ARG, "unsupported channel blocking");
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

// The row kernel takes W as stored where rows_take_untransposed says so (it
// transposes each weight tile while staging it); otherwise a transposed
// copy of W (one small kernel) gives it whole 16-byte pieces of each
// column's reduction channels.
template <typename T>
static sscn_status forward_t(const T* X, const T* W, const View& v, int cin, int cout, const Heads<T>& Y, hipStream_t s) {
  if (rows_eligible<T>(v, cin, cout)) {
    if (v.n_out == 0) return SSCN_OK;
    if constexpr (sizeof(T) == 4) {
      if (rows_split(v, cin, cout)) {
        const int64_t total = (int64_t)v.K * cin * cout;
        uint16_t* planes = nullptr;
        SSCN_TRY(temp_weights(&planes, 3 * total, s));
        k_split_w<true><<<(unsigned)std::min<int64_t>(ceil_div(total, 256), 4096), 256, 0, s>>>(W, v.K, cin, cout,
                                                                                               planes);
        hipError_t e = hipGetLastError();
        sscn_status st = e == hipSuccess ? launch_rows<T, false, true>(X, planes, v, cin, cout, Y, s)
                                         : hip_fail(e, "weight split");
        temp_release(planes, s);
        return st;
      }
    }
    if (rows_take_untransposed<T>(cin, cout)) return launch_rows<T>(X, W, v, cin, cout, Y, s, true);
    const int64_t total = (int64_t)v.K * cin * cout;
    T* Bt = nullptr;
    SSCN_TRY(temp_weights(&Bt, total, s));
    k_transpose_w<T><<<(unsigned)std::min<int64_t>(ceil_div(total, 256), 4096), 256, 0, s>>>(W, v.K, cin, cout, Bt);
    hipError_t e = hipGetLastError();
    sscn_status st = e == hipSuccess ? launch_rows<T>(X, Bt, v, cin, cout, Y, s) : hip_fail(e, "transpose");
    temp_release(Bt, s);
    return st;
  }
  if (prefer_col<T>(v, cin, cout)) {
    if (v.n_out == 0) return SSCN_OK;
    const int64_t total = (int64_t)v.K * cin * cout;
    T* Bt = nullptr;
    SSCN_TRY(temp_weights(&Bt, total, s));
    k_transpose_w<T><<<(unsigned)std::min<int64_t>(ceil_div(total, 256), 4096), 256, 0, s>>>(W, v.K, cin, cout, Bt);
    hipError_t e = hipGetLastError();
    sscn_status st = e == hipSuccess ? launch_col<T>(X, Bt, v, cin, cout, Y, s) : hip_fail(e, "transpose");
    temp_release(Bt, s);
    return st;
  }
  if constexpr (sizeof(T) == 2) {
    return launch_conv<T, false>(X, W, v, cin, cout, Y, s);
  } else {
    if (v.st->n_tiles == 0) return SSCN_OK;
    const int64_t total = (int64_t)v.K * cin * cout;
    T* Bt = nullptr;
    SSCN_TRY(temp_weights(&Bt, total, s));
    k_transpose_w<T><<<(unsigned)std::min<int64_t>(ceil_div(total, 256), 4096), 256, 0, s>>>(W, v.K, cin, cout, Bt);
    hipError_t e = hipGetLastError();
    sscn_status st = e == hipSuccess ? launch_conv<T, true>(X, Bt, v, cin, cout, Y, s) : hip_fail(e, "transpose");
    temp_release(Bt, s);
    return st;
  }
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
  UseNote note{rb->d, stream};
  if (!out || !weights || (v.n_in > 0 && !features))
    return fail(SSCN_ERR_INVALID_ARG, "NULL features, weights or out");
  if (dtype == SSCN_F32)
    return forward_t<float>((const float*)features, (const float*)weights, v, c_in, c_out,
                            plain_heads((float*)out, c_out), stream);
  return forward_t<bf16_t>((const bf16_t*)features, (const bf16_t*)weights, v, c_in, c_out,
                           plain_heads((bf16_t*)out, c_out),
                           stream);
}

template <typename T>
static Heads<T> heads_of(int n, const sscn_conv_output* h) {
  Heads<T> r{};
  r.n = n;
  for (int i = 0; i < n; ++i) {
    r.out[i] = (T*)h[i].data;
    r.ld[i] = h[i].row_stride;
    r.scale[i] = h[i].scale;
    r.shift[i] = h[i].shift;
  }
  return r;
}

static sscn_status forward_heads(const void* features, const void* weights, const float* bias, const void* residual,
                                 int64_t residual_ld, sscn_rulebook rb, int32_t c_in, int32_t c_out, sscn_dtype dtype,
                                 int32_t n_heads, const sscn_conv_output* heads, hipStream_t stream);

extern "C" sscn_status sparse_conv_forward_heads(const void* features, const void* weights, sscn_rulebook rb,
                                                 int32_t c_in, int32_t c_out, sscn_dtype dtype, int32_t n_heads,
                                                 const sscn_conv_output* heads, hipStream_t stream) {
  return forward_heads(features, weights, nullptr, nullptr, 0, rb, c_in, c_out, dtype, n_heads, heads, stream);
}

extern "C" sscn_status sparse_conv_forward_ex(const void* features, const void* weights, sscn_rulebook rb,
                                              int32_t c_in, int32_t c_out, sscn_dtype dtype, const float* bias,
                                              const void* residual, int64_t residual_ld, int32_t n_heads,
                                              const sscn_conv_output* heads, hipStream_t stream) {
  if (residual && residual_ld < c_out) return fail(SSCN_ERR_INVALID_ARG, "residual row stride < c_out");
  return forward_heads(features, weights, bias, residual, residual_ld, rb, c_in, c_out, dtype, n_heads, heads, stream);
}

static sscn_status forward_heads(const void* features, const void* weights, const float* bias, const void* residual,
                                 int64_t residual_ld, sscn_rulebook rb, int32_t c_in, int32_t c_out, sscn_dtype dtype,
                                 int32_t n_heads, const sscn_conv_output* heads, hipStream_t stream) {
  sscn_status st = check_conv_args(rb, c_in, c_out, dtype);
  if (st != SSCN_OK) return st;
  if (n_heads < 1 || n_heads > 2 || !heads) return fail(SSCN_ERR_INVALID_ARG, "1 or 2 output heads");
  for (int i = 0; i < n_heads; ++i) {
    if (!heads[i].data || heads[i].row_stride < c_out)
      return fail(SSCN_ERR_INVALID_ARG, "output head: NULL data or row stride < c_out");
    if ((heads[i].scale == nullptr) != (heads[i].shift == nullptr))
      return fail(SSCN_ERR_INVALID_ARG, "output head: scale and shift must both be set or both NULL");
  }
  const View v = view_of(rb);
  if (v.n_out == 0) return SSCN_OK;
  UseNote note{rb->d, stream};
  if (!weights || (v.n_in > 0 && !features)) return fail(SSCN_ERR_INVALID_ARG, "NULL features or weights");
  if (dtype == SSCN_F32) {
    Heads<float> h = heads_of<float>(n_heads, heads);
    h.bias = bias;
    h.res = (const float*)residual;
    h.res_ld = residual_ld;
    return forward_t<float>((const float*)features, (const float*)weights, v, c_in, c_out, h, stream);
  }
  Heads<bf16_t> h = heads_of<bf16_t>(n_heads, heads);
  h.bias = bias;
  h.res = (const bf16_t*)residual;
  h.res_ld = residual_ld;
  return forward_t<bf16_t>((const bf16_t*)features, (const bf16_t*)weights, v, c_in, c_out, h, stream);
}

extern "C" sscn_status sparse_conv_backward(const void* features, const void* weights, const void* dout,
                                            sscn_rulebook rb, int32_t c_in, int32_t c_out, sscn_dtype dtype,
                                            void* dgrad, float* wgrad, hipStream_t stream) {
  sscn_status st = check_conv_args(rb, c_in, c_out, dtype);
  if (st != SSCN_OK) return st;
  const View v = view_of(rb);
  UseNote note{rb->d, stream};
  const int64_t w_total = (int64_t)v.K * c_in * c_out;
  bool w_zeroed = false;  // the dgrad launch cleared wgrad on the side
  if (dgrad && v.n_in > 0) {
    if (!weights || (v.n_out > 0 && !dout)) return fail(SSCN_ERR_INVALID_ARG, "NULL weights or dout");
    // dgrad = forward over the transposed rule book with B = W^o (as stored:
    // row ci of W[o] holds the c_out weights feeding input channel ci)
    const View vt = transposed_view(rb);
    if (dtype == SSCN_F32) {
      Heads<float> h = plain_heads((float*)dgrad, c_in);
      if (rows_eligible<float>(vt, c_out, c_in)) {
        if (wgrad) { h.zero = wgrad; h.n_zero = w_total; w_zeroed = true; }
        if (rows_split(vt, c_out, c_in)) {
          // B[o][ci][co] = W[o][ci][co] as stored, in parts
          uint16_t* planes = nullptr;
          SSCN_TRY(temp_weights(&planes, 3 * w_total, stream));
          k_split_w<false><<<(unsigned)std::min<int64_t>(ceil_div(w_total, 256), 4096), 256, 0, stream>>>(
              (const float*)weights, vt.K, c_out, c_in, planes);
          hipError_t e = hipGetLastError();
          st = e == hipSuccess ? launch_rows<float, true, true>((const float*)dout, planes, vt, c_out, c_in, h, stream)
                               : hip_fail(e, "weight split");
          temp_release(planes, stream);
        } else {
          st = launch_rows<float, true>((const float*)dout, (const float*)weights, vt, c_out, c_in, h, stream);
        }
      } else {
        st = launch_conv<float, true>((const float*)dout, (const float*)weights, vt, c_out, c_in, h, stream);
      }
    } else {
      Heads<bf16_t> h = plain_heads((bf16_t*)dgrad, c_in);
      if (rows_eligible<bf16_t>(vt, c_out, c_in)) {
        if (wgrad) { h.zero = wgrad; h.n_zero = w_total; w_zeroed = true; }
        st = launch_rows<bf16_t, true>((const bf16_t*)dout, (const bf16_t*)weights, vt, c_out, c_in, h, stream);
      } else {
        st = launch_conv<bf16_t, true>((const bf16_t*)dout, (const bf16_t*)weights, vt, c_out, c_in, h, stream);
      }
    }
    if (st != SSCN_OK) return st;
  }
  if (wgrad) {
    const RulebookData* d = rb->d;
    if (d->n_pairs == 0) {
      if (!w_zeroed) st = fill_f32(wgrad, 0.f, w_total, stream);
      if (st != SSCN_OK) return st;
    } else {
      if (!features || !dout) return fail(SSCN_ERR_INVALID_ARG, "NULL features or dout");
      int64_t mx = 0;
      for (int64_t c : d->pairs_per_offset) mx = std::max(mx, c);
      if (dtype == SSCN_F32)
        st = launch_wgrad<float>((const float*)features, (const float*)dout, v, c_in, c_out, wgrad, stream, mx,
                                 d->n_pairs, w_zeroed);
      else if (wgrad_rows_eligible(v, c_in, c_out) && !no_alloc())
        st = launch_wgrad_rows((const bf16_t*)features, (const bf16_t*)dout, v, c_in, c_out, wgrad, stream);
      else
        st = launch_wgrad<bf16_t>((const bf16_t*)features, (const bf16_t*)dout, v, c_in, c_out, wgrad, stream,
                                  mx, d->n_pairs, w_zeroed);
    }
  }
  return st;
}

// ------------------------------------------------ no-allocation forward
// The forward's only temporary is the transposed copy of the weights.  For
// callers that cannot allocate device memory, it lives in a fixed region of
// the library's code object (one copy per device, kept until the process
// ends).  Host code uses the region only through the device address that
// hipGetSymbolAddress returns for the current device.
namespace {
constexpr size_t kScratchBytes = (size_t)8 << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

sscn_status scratch_address(void** out) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  SSCN_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(SSCN_ERR_INVALID_ARG, "device index out of range");
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    SSCN_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(SSCN_ERR_DEVICE, "no device address for the scratch region");
    addr[dev] = p;
  }
  *out = addr[dev];
  return SSCN_OK;
}

struct NoAllocScope {
  explicit NoAllocScope(const NoAlloc* na) { set_no_alloc(na); }
  ~NoAllocScope() { set_no_alloc(nullptr); }
};
}  // namespace

extern "C" sscn_status sparse_conv_forward_noalloc(const void* features, const void* weights, sscn_rulebook rb,
                                                   int32_t c_in, int32_t c_out, sscn_dtype dtype, void* out,
                                                   hipStream_t stream) {
  sscn_status st = check_conv_args(rb, c_in, c_out, dtype);
  if (st != SSCN_OK) return st;
  const View v = view_of(rb);
  // the weight copy: fp32 in three bf16 parts (6 bytes per weight), bf16 as is
  const size_t w_bytes = (size_t)v.K * c_in * c_out * (dtype == SSCN_F32 ? 6 : 2);
  if (w_bytes > kScratchBytes)
    return fail(SSCN_ERR_INVALID_ARG, "weights of " + std::to_string(w_bytes) + " bytes exceed the " +
                                          std::to_string(kScratchBytes) + "-byte scratch region of the "
                                          "no-allocation forward");
  if (v.n_out == 0) return SSCN_OK;
  if (!out || !weights || (v.n_in > 0 && !features))
    return fail(SSCN_ERR_INVALID_ARG, "NULL features, weights or out");
  NoAlloc na;
  SSCN_TRY(scratch_address(&na.scratch));
  na.bytes = kScratchBytes;
  NoAllocScope scope(&na);
  UseNote note{rb->d, stream};
  if (dtype == SSCN_F32)
    return forward_t<float>((const float*)features, (const float*)weights, v, c_in, c_out,
                            plain_heads((float*)out, c_out), stream);
  return forward_t<bf16_t>((const bf16_t*)features, (const bf16_t*)weights, v, c_in, c_out,
                           plain_heads((bf16_t*)out, c_out), stream);
}
