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
#include <cstdlib>

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

// Workgroups are dispatched round-robin over the 8 XCDs, each with its own
// L2.  Renumber them so that XCD x works on one contiguous range of tiles:
// neighbouring tiles gather overlapping input rows, which then stay in
// that XCD's L2.  A bijection on [0, nb).
constexpr int kNumXcd = 8;
__device__ __forceinline__ int64_t xcd_remap(int64_t b, int64_t nb) {
  const int64_t q = nb / kNumXcd, r = nb % kNumXcd;
  const int64_t x = b % kNumXcd, i = b / kNumXcd;
  return x * q + min(x, r) + i;
}

// d[nb] += A B_nb^T for NB column blocks sharing one A fragment; the loop
// order keeps consecutive MFMAs independent.
template <int NB, int KB>
__device__ __forceinline__ void mma64_multi(const float (&a)[16], const float (&b)[NB][KB][16], int kb,
                                            f32x4 (&d)[NB]) {
#pragma unroll
  for (int i = 0; i < 16; ++i)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) d[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[nb][kb][i], d[nb], 0, 0, 0);
}
template <int NB, int KB>
__device__ __forceinline__ void mma64_multi(const bf16x8 (&a)[2], const bf16x8 (&b)[NB][KB][2], int kb,
                                            f32x4 (&d)[NB]) {
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) d[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[h], b[nb][kb][h], d[nb], 0, 0, 0);
}

// Branch-free gathers.  `row` must point at a readable row even when the
// lane has nothing to load (callers pass row 0); masked lanes read it and
// select zero, so the loads of a chunk issue as one straight-line group.
// FAST: c % 16 == 0 and 16-byte aligned rows, so a lane's 16 values are
// either all inside the row or all past its end.
template <bool FAST>
__device__ __forceinline__ void gather16(const float* __restrict__ row, int k0, bool ok, int c,
                                         float (&v)[16]) {
  if constexpr (FAST) {
    const bool in = ok && k0 < c;
    const float4* p = reinterpret_cast<const float4*>(row + (in ? k0 : 0));
    float4 x[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) x[q] = p[q];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[4 * q + 0] = in ? x[q].x : 0.f;
      v[4 * q + 1] = in ? x[q].y : 0.f;
      v[4 * q + 2] = in ? x[q].z : 0.f;
      v[4 * q + 3] = in ? x[q].w : 0.f;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const bool in = ok && k0 + i < c;
      const float x = row[in ? k0 + i : 0];
      v[i] = in ? x : 0.f;
    }
  }
}
template <bool FAST>
__device__ __forceinline__ void gather16(const bf16_t* __restrict__ row, int k0, bool ok, int c,
                                         bf16x8 (&v)[2]) {
  if constexpr (FAST) {
    const bool in = ok && k0 < c;
    const uint4* p = reinterpret_cast<const uint4*>(row + (in ? k0 : 0));
    uint4 a = p[0], b = p[1];
    if (!in) a = b = make_uint4(0, 0, 0, 0);
    v[0] = __builtin_bit_cast(bf16x8, a);
    v[1] = __builtin_bit_cast(bf16x8, b);
  } else {
    uint32_t t[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const bool in = ok && k0 + i < c;
      const uint32_t x = row[in ? k0 + i : 0].bits;
      t[i] = in ? x : 0u;
    }
    uint4 a, b;
    a.x = t[0] | (t[1] << 16);   a.y = t[2] | (t[3] << 16);
    a.z = t[4] | (t[5] << 16);   a.w = t[6] | (t[7] << 16);
    b.x = t[8] | (t[9] << 16);   b.y = t[10] | (t[11] << 16);
    b.z = t[12] | (t[13] << 16); b.w = t[14] | (t[15] << 16);
    v[0] = __builtin_bit_cast(bf16x8, a);
    v[1] = __builtin_bit_cast(bf16x8, b);
  }
}

template <typename T> struct Frag;
template <> struct Frag<float> { typedef float type[16]; };
template <> struct Frag<bf16_t> { typedef bf16x8 type[2]; };

__device__ __forceinline__ void copy_frag(float (&d)[16], const float (&s)[16]) {
#pragma unroll
  for (int i = 0; i < 16; ++i) d[i] = s[i];
}
__device__ __forceinline__ void copy_frag(bf16x8 (&d)[2], const bf16x8 (&s)[2]) {
  d[0] = s[0];
  d[1] = s[1];
}

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

// Pipelined variant for c_in <= 64 * KBLK.  The workgroup first lists its
// chunks (offset, first pair, pair count) in LDS; each wavefront then streams
// the list with a two-deep software pipeline: pair indices two chunks ahead,
// the gathered A fragment (and, at an offset change, the B fragment) one
// chunk ahead, MFMAs on the current chunk.  B for the current offset stays
// in registers across that offset's chunks.
template <typename T, int NW, int KBLK>
__global__ __launch_bounds__(NW * 64) void k_gather_mma_pipe(
    const T* __restrict__ X, const T* __restrict__ Bt, const int64_t* __restrict__ seg,
    const int32_t* __restrict__ in_rows, const int32_t* __restrict__ out_rows, int64_t n_tiles, int K,
    int mirror, int cin, int cout, int64_t n_out, int tpw, int vec, int max_chunks, T* __restrict__ Y) {
  extern __shared__ float smem[];
  constexpr int WCOLS = 16 * NW;
  constexpr int LDW = WCOLS + 1;
  const int rows = tpw * kTile;
  float* acc = smem;
  int64_t* ch_p0 = reinterpret_cast<int64_t*>(smem + ((rows * LDW + 1) & ~1));
  int32_t* ch_info = reinterpret_cast<int32_t*>(ch_p0 + max_chunks);
  __shared__ int n_chunks_sh;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int64_t t0 = xcd_remap(blockIdx.x, gridDim.x) * tpw;
  const int64_t t1 = min<int64_t>(t0 + tpw, n_tiles);
  const int64_t row0 = t0 * kTile;
  const int col_base = blockIdx.y * WCOLS;
  const int col = col_base + wave * 16 + m;
  const bool col_ok = col < cout;

  // chunk list: offsets in order, 16 pairs per chunk
  if (wave == 0) {
    int base = 0;
    for (int ob = 0; ob < K; ob += 64) {
      const int o = ob + lane;
      int64_t s = 0, e = 0;
      int nc = 0;
      if (o < K) {
        const int so = mirror ? K - 1 - o : o;
        s = seg[(int64_t)so * n_tiles + t0];
        e = seg[(int64_t)so * n_tiles + t1];
        nc = (int)((e - s + 15) >> 4);
      }
      int x = nc;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
      }
      const int start = base + x - nc;
      for (int c = 0; c < nc; ++c) {
        const int64_t p0 = s + 16 * c;
        ch_p0[start + c] = p0;
        ch_info[start + c] = o | ((int)min<int64_t>(16, e - p0) << 16);
      }
      base += __shfl(x, 63, 64);
    }
    if (lane == 0) n_chunks_sh = base;
  }
  for (int i = threadIdx.x; i < rows * LDW; i += blockDim.x) acc[i] = 0.f;
  __syncthreads();
  const int n_chunks = n_chunks_sh;

  typedef typename Frag<T>::type F;
  struct Idx {
    int32_t irow, orow;
    int o;
    bool ok;
  };
  auto fetch_idx = [&](int c) {
    Idx r;
    r.irow = 0; r.orow = -1; r.o = -1; r.ok = false;
    if (c < n_chunks) {
      const int64_t p0 = ch_p0[c];
      const int info = ch_info[c];
      r.o = info & 0xffff;
      r.ok = m < (info >> 16);
      if (r.ok) {
        r.irow = in_rows[p0 + m];
        r.orow = (int32_t)(out_rows[p0 + m] - row0);
      }
    }
    return r;
  };
  auto load_a = [&](const Idx& ix, F (&a)[KBLK]) {
    const T* __restrict__ arow = X + (int64_t)ix.irow * cin;
#pragma unroll
    for (int kb = 0; kb < KBLK; ++kb) load16(arow, kb * 64 + 16 * g, ix.ok ? cin : 0, vec, a[kb]);
  };
  auto load_b = [&](int o, F (&b)[KBLK]) {
    const T* __restrict__ brow = Bt + ((int64_t)o * cout + (col_ok ? col : 0)) * cin;
#pragma unroll
    for (int kb = 0; kb < KBLK; ++kb) load16(brow, kb * 64 + 16 * g, col_ok ? cin : 0, vec, b[kb]);
  };

  if (n_chunks > 0) {
    F a_cur[KBLK], a_nxt[KBLK], b_cur[KBLK], b_nxt[KBLK];
    Idx ci_cur = fetch_idx(0);
    Idx ci_nxt = fetch_idx(1);
    load_a(ci_cur, a_cur);
    load_b(ci_cur.o, b_cur);
    int o_cur = ci_cur.o;
    for (int c = 0; c < n_chunks; ++c) {
      const Idx ci_nn = fetch_idx(c + 2);
      const bool have_next = c + 1 < n_chunks;
      const bool new_b = have_next && ci_nxt.o != o_cur;
      if (have_next) load_a(ci_nxt, a_nxt);
      if (new_b) load_b(ci_nxt.o, b_nxt);
      f32x4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < KBLK; ++kb) d = mma64(a_cur[kb], b_cur[kb], d);
      // lane holds D[4g + r][m]: pair 4g + r, column m
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ol = __shfl(ci_cur.orow, 4 * g + r, 64);
        if (ol >= 0) acc[ol * LDW + wave * 16 + m] += d[r];
      }
#pragma unroll
      for (int kb = 0; kb < KBLK; ++kb) {
        copy_frag(a_cur[kb], a_nxt[kb]);
        if (new_b) copy_frag(b_cur[kb], b_nxt[kb]);
      }
      if (new_b) o_cur = ci_nxt.o;
      ci_cur = ci_nxt;
      ci_nxt = ci_nn;
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

// Main forward / dgrad kernel for c_in <= 64 * KBLK.
//
// Workgroup = 4 wavefronts, one 64-row output tile, NB*16 output columns.
// The tile's pairs are listed as chunks of 16 (offset-major, as stored) and
// the list is cut into four equal contiguous ranges, one per wavefront, so
// every wavefront does the same number of chunks and meets each offset's
// weights once (twice at a range boundary).  A wavefront covers all NB
// column blocks of a chunk: the gathered A fragment (16 pairs x 64
// channels) feeds NB*16 fp32 MFMAs (or NB*2 bf16 ones), and the weights of
// the current offset stay in registers.  Each wavefront accumulates into a
// private LDS copy of the tile; the copies are summed in a fixed order at
// the end, so the result does not depend on scheduling.
template <typename T, int NB, int KBLK, bool FAST>
__global__ __launch_bounds__(256) void k_conv_tile(
    const T* __restrict__ X, const T* __restrict__ Bt, const int64_t* __restrict__ seg,
    const int32_t* __restrict__ in_rows, const int32_t* __restrict__ out_rows, int64_t n_tiles, int K,
    int mirror, int cin, int cout, int64_t n_out, int max_chunks, T* __restrict__ Y) {
  constexpr int WCOLS = 16 * NB;
  constexpr int LDW = WCOLS + 1;
  constexpr int ROWS = kTile;
  constexpr int ACC = (ROWS + 1) * LDW;  // floats per private accumulator (+ dummy row)
  extern __shared__ float smem[];
  float* acc_all = smem;
  int64_t* ch_p0 = reinterpret_cast<int64_t*>(smem + ((4 * ACC + 1) & ~1));
  int32_t* ch_info = reinterpret_cast<int32_t*>(ch_p0 + max_chunks);
  __shared__ int n_chunks_sh;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int64_t t0 = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t row0 = t0 * kTile;
  const int col_base = blockIdx.y * WCOLS;
  float* acc = acc_all + wave * ACC;

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
      const int start = base + x - nc;
      for (int c = 0; c < nc; ++c) {
        const int64_t p0 = s + 16 * c;
        ch_p0[start + c] = p0;
        ch_info[start + c] = o | ((int)min<int64_t>(16, e - p0) << 16);
      }
      base += __shfl(x, 63, 64);
    }
    if (lane == 0) n_chunks_sh = base;
  }
  for (int i = threadIdx.x; i < 4 * ACC; i += blockDim.x) acc_all[i] = 0.f;
  __syncthreads();
  const int n_all = n_chunks_sh;
  const int c_begin = (int)(((int64_t)n_all * wave) / 4);
  const int c_end = (int)(((int64_t)n_all * (wave + 1)) / 4);

  typedef typename Frag<T>::type F;
  struct Idx {
    int32_t irow, orow;
    int o;
    bool ok;
  };
  // chunk c of this wavefront's range (clamped into the range: past its end
  // the lane is simply masked)
  auto fetch_idx = [&](int c) {
    Idx r;
    const bool live = c < c_end;
    const int cc = live ? c : c_end - 1;
    const int64_t p0 = ch_p0[cc];
    const int info = ch_info[cc];
    r.o = info & 0xffff;
    r.ok = live && m < (info >> 16);
    const int64_t p = p0 + (r.ok ? m : 0);
    const int32_t ir = in_rows[p], orw = out_rows[p];
    r.irow = r.ok ? ir : 0;
    r.orow = r.ok ? (int32_t)(orw - row0) : -1;
    return r;
  };
  auto load_a = [&](const Idx& ix, F (&a)[KBLK]) {
    const T* __restrict__ arow = X + (int64_t)ix.irow * cin;
#pragma unroll
    for (int kb = 0; kb < KBLK; ++kb) gather16<FAST>(arow, kb * 64 + 16 * g, ix.ok, cin, a[kb]);
  };
  auto load_b = [&](int o, F (&b)[NB][KBLK]) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int col = col_base + nb * 16 + m;
      const bool ok = col < cout;
      const T* __restrict__ brow = Bt + ((int64_t)o * cout + (ok ? col : 0)) * cin;
#pragma unroll
      for (int kb = 0; kb < KBLK; ++kb) gather16<FAST>(brow, kb * 64 + 16 * g, ok, cin, b[nb][kb]);
    }
  };

  if (c_begin < c_end) {
    F a_cur[KBLK], a_nxt[KBLK];
    F b_cur[NB][KBLK], b_nxt[NB][KBLK];
    Idx ci_cur = fetch_idx(c_begin);
    Idx ci_nxt = fetch_idx(c_begin + 1);
    load_a(ci_cur, a_cur);
    load_b(ci_cur.o, b_cur);
    int o_cur = ci_cur.o;
    for (int c = c_begin; c < c_end; ++c) {
      const Idx ci_nn = fetch_idx(c + 2);
      const bool have_next = c + 1 < c_end;
      const bool new_b = have_next && ci_nxt.o != o_cur;
      if (have_next) load_a(ci_nxt, a_nxt);
      if (new_b) load_b(ci_nxt.o, b_nxt);
      int ol[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) ol[r] = __shfl(ci_cur.orow, 4 * g + r, 64);
      f32x4 d[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) d[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      // the NB accumulation chains are interleaved so consecutive MFMAs are independent
#pragma unroll
      for (int kb = 0; kb < KBLK; ++kb) mma64_multi<NB>(a_cur[kb], b_cur, kb, d);
      // lane holds D[4g + r][m]: pair 4g + r, column nb*16 + m.  The accumulator
      // is private to this wavefront: plain read-modify-write, masked lanes
      // on the dummy row.
      int addr[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) addr[r] = (ol[r] >= 0 ? ol[r] : ROWS) * LDW + m;
      float old[NB][4];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r) old[nb][r] = acc[addr[r] + nb * 16];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[addr[r] + nb * 16] = old[nb][r] + d[nb][r];
#pragma unroll
      for (int kb = 0; kb < KBLK; ++kb) copy_frag(a_cur[kb], a_nxt[kb]);
      if (new_b) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int kb = 0; kb < KBLK; ++kb) copy_frag(b_cur[nb][kb], b_nxt[nb][kb]);
        o_cur = ci_nxt.o;
      }
      ci_cur = ci_nxt;
      ci_nxt = ci_nn;
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < ROWS * WCOLS; i += blockDim.x) {
    const int r = i / WCOLS, c = i % WCOLS;
    const int64_t row = row0 + r;
    const int cc = col_base + c;
    const int a = r * LDW + c;
    const float v = ((acc_all[a] + acc_all[ACC + a]) + acc_all[2 * ACC + a]) + acc_all[3 * ACC + a];
    if (row < n_out && cc < cout) Elem<T>::store(Y + row * cout + cc, v);
  }
}

// Forward / dgrad for c_in <= 64, c_out <= 64 (fp32): the quad-split kernel.
//
// Workgroup = 4 wavefronts over one 64-row output tile and all (<= 64)
// output columns.  Wavefront w takes input-channel half kh = w & 1 and
// output-column half ch = w >> 1, so its weight fragment is 32 x 32 (16
// VGPRs) and its share of a gathered row is 32 contiguous channels.  Every
// wavefront walks the tile's whole chunk list (16 pairs per chunk,
// offset-major); per chunk it issues 16 MFMAs (2 column blocks x 8 steps of
// 4 channels).  The loop body is straight-line: pair indices two chunks
// ahead, the gathered fragment and the next chunk's weights one chunk
// ahead.  Weights are re-read every chunk, but when the offset does not
// change all lanes read one broadcast line and keep their registers.
// Partial sums of the two channel halves go to two LDS accumulators, each
// element written by one wavefront in chunk order, and are added at the
// end: the result is deterministic.
template <typename T>
__global__ __launch_bounds__(256) void k_conv_quad(
    const T* __restrict__ X, const T* __restrict__ Bt, const int64_t* __restrict__ seg,
    const int32_t* __restrict__ in_rows, const int32_t* __restrict__ out_rows, int64_t n_tiles, int K,
    int mirror, int cin, int cout, int64_t n_out, int max_chunks, T* __restrict__ Y) {
  constexpr int LDW = 64 + 1;
  constexpr int ACC = (kTile + 1) * LDW;  // 64 rows + one dummy row for masked lanes
  extern __shared__ float smem[];
  float* acc_all = smem;  // [2][65][LDW]
  int64_t* ch_p0 = reinterpret_cast<int64_t*>(smem + ((2 * ACC + 1) & ~1));
  int32_t* ch_info = reinterpret_cast<int32_t*>(ch_p0 + max_chunks);
  __shared__ int n_chunks_sh;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int kh = wave & 1, chf = wave >> 1;
  const int64_t t0 = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t row0 = t0 * kTile;
  float* acc = acc_all + kh * ACC;

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
      const int start = base + x - nc;
      for (int c = 0; c < nc; ++c) {
        const int64_t p0 = s + 16 * c;
        ch_p0[start + c] = p0;
        ch_info[start + c] = o | ((int)min<int64_t>(16, e - p0) << 16);
      }
      base += __shfl(x, 63, 64);
    }
    if (lane == 0) n_chunks_sh = base;
  }
  for (int i = threadIdx.x; i < 2 * ACC; i += blockDim.x) acc_all[i] = 0.f;
  __syncthreads();
  const int n_chunks = n_chunks_sh;

  // this lane's channel octet and output columns
  const int k0 = kh * 32 + 8 * g;
  const bool k_in = k0 + 8 <= cin;  // cin % 8 == 0 on this path
  int colv[2];
  bool col_in[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    colv[nb] = chf * 32 + nb * 16 + m;
    col_in[nb] = colv[nb] < cout && k_in;
  }

  struct Idx {
    int32_t irow, orow;
    int o;
    bool ok;
  };
  auto fetch_idx = [&](int c) {
    Idx r;
    const bool live = c < n_chunks;
    const int cc = live ? c : n_chunks - 1;
    const int64_t p0 = ch_p0[cc];
    const int info = ch_info[cc];
    r.o = live ? (info & 0xffff) : -1;
    r.ok = live && m < (info >> 16);
    const int64_t p = p0 + (r.ok ? m : 0);
    r.irow = in_rows[p];
    r.orow = out_rows[p];
    return r;
  };
  typedef float F8[8];
  auto load8 = [&](const T* __restrict__ p, F8& v) {
    const float4* q = reinterpret_cast<const float4*>(p);
    const float4 a = q[0], b = q[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  };
  auto load_a = [&](const Idx& ix, F8& a) {
    const bool in = ix.ok && k_in;
    load8(X + (int64_t)(in ? ix.irow : 0) * cin + (in ? k0 : 0), a);
#pragma unroll
    for (int i = 0; i < 8; ++i) a[i] = in ? a[i] : 0.f;
  };
  // weights of offset o for both column blocks; when `same`, every lane
  // reads the first line of Bt and the caller keeps its registers
  auto load_b = [&](int o, bool same, F8 (&b)[2]) {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const bool in = !same && col_in[nb];
      load8(Bt + (in ? ((int64_t)o * cout + colv[nb]) * cin + k0 : 0), b[nb]);
    }
  };

  if (n_chunks > 0) {
    F8 a_cur, a_nxt, b_cur[2], b_nxt[2];
    Idx ci_cur = fetch_idx(0);
    Idx ci_nxt = fetch_idx(1);
    load_a(ci_cur, a_cur);
    load_b(ci_cur.o, false, b_cur);
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int i = 0; i < 8; ++i) b_cur[nb][i] = col_in[nb] ? b_cur[nb][i] : 0.f;
    for (int c = 0; c < n_chunks; ++c) {
      const Idx ci_nn = fetch_idx(c + 2);
      const bool same = ci_nxt.o == ci_cur.o || ci_nxt.o < 0;
      load_a(ci_nxt, a_nxt);
      load_b(ci_nxt.o < 0 ? 0 : ci_nxt.o, same, b_nxt);
      int ol[4];
      const int32_t orow_local = ci_cur.ok ? (int32_t)(ci_cur.orow - row0) : -1;
#pragma unroll
      for (int r = 0; r < 4; ++r) ol[r] = __shfl(orow_local, 4 * g + r, 64);
      f32x4 d[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          d[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a_cur[i], b_cur[nb][i], d[nb], 0, 0, 0);
      // lane holds D[4g + r][m]: pair 4g + r, column chf*32 + nb*16 + m.  Each
      // accumulator element has one writer (this wavefront), so a plain
      // read-modify-write is exact; masked lanes use the dummy row.
      int addr[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) addr[r] = (ol[r] >= 0 ? ol[r] : kTile) * LDW + chf * 32 + m;
      float old[2][4];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r) old[nb][r] = acc[addr[r] + nb * 16];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[addr[r] + nb * 16] = old[nb][r] + d[nb][r];
#pragma unroll
      for (int i = 0; i < 8; ++i) a_cur[i] = a_nxt[i];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int i = 0; i < 8; ++i) b_cur[nb][i] = same ? b_cur[nb][i] : (col_in[nb] ? b_nxt[nb][i] : 0.f);
      ci_cur = ci_nxt;
      ci_nxt = ci_nn;
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kTile * 64; i += blockDim.x) {
    const int r = i >> 6, c = i & 63;
    const int64_t row = row0 + r;
    if (row < n_out && c < cout) Elem<T>::store(Y + row * cout + c, acc_all[r * LDW + c] + acc_all[ACC + r * LDW + c]);
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

// wgrad without LDS staging.  dW^o[ci][co] = sum_p X[in_p][ci] dY[out_p][co].
// MFMA row i of block a stands for input channel ci0 + CA*i + a, column j of
// block b for output channel co0 + CB*j + b, so a lane's CA (CB) operand
// values are contiguous channels of one gathered row: one 8/16-byte load
// each.  One MFMA step consumes 4 pairs (one per lane group).  Each
// wavefront accumulates the whole CA*16 x CB*16 block over a quarter of
// the workgroup's pairs, with pair indices and rows fetched one iteration
// (16 pairs) ahead; the four partial blocks are summed through LDS and
// added to dW with fp32 atomics.
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
                                                   int cin, int cout, int pch, int nzc, float* __restrict__ dW) {
  constexpr int STEPS = 4;  // MFMA steps (4 pairs each) per iteration
  const int o = blockIdx.y;
  const int so = mirror ? K - 1 - o : o;
  const int64_t start = seg[(int64_t)so * n_tiles], end = seg[(int64_t)(so + 1) * n_tiles];
  const int64_t pb = start + (int64_t)blockIdx.x * pch;
  if (pb >= end) return;
  const int64_t pe = min<int64_t>(pb + pch, end);
  const int ci0 = (blockIdx.z % nzc) * 16 * CA, co0 = (blockIdx.z / nzc) * 16 * CB;
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
  // sum the four wavefronts' partial blocks (LDS atomic adds into one
  // block), then add the block to dW.  D[4g + r][m] of block (a, b) is
  // dW[ci0 + CA (4g + r) + a][co0 + CB m + b].
  constexpr int NE = CA * CB * 4;  // values per lane
  __shared__ float part[NE][64];
  for (int e = threadIdx.x; e < NE * 64; e += 256) (&part[0][0])[e] = 0.f;
  __syncthreads();
#pragma unroll
  for (int a = 0; a < CA; ++a)
#pragma unroll
    for (int b = 0; b < CB; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) atomicAdd(&part[(a * CB + b) * 4 + r][lane], d[a][b][r]);
  __syncthreads();
  for (int e = threadIdx.x; e < NE * 64; e += 256) {
    const int v = e / 64, l = e % 64;
    const float sum = part[v][l];
    const int a = v / (CB * 4), b = (v / 4) % CB, r = v % 4;
    const int mm = l & 15, gg = l >> 4;
    const int ci = ci0 + CA * (4 * gg + r) + a, co = co0 + CB * mm + b;
    if (ci < cin && co < cout && sum != 0.f) atomicAdd(dW + ((int64_t)o * cin + ci) * cout + co, sum);
  }
}

// ---------------------------------------------------------------- launchers
static int tiles_per_wg() {
  static int tpw = [] {
    const char* e = getenv("SSCN_TILES_PER_WG");  // tuning knob: output tiles (64 rows) per workgroup
    int v = e ? atoi(e) : 1;
    return v < 1 ? 1 : (v > 4 ? 4 : v);
  }();
  return tpw;
}

template <typename T, int NW, int KBLK>
static sscn_status launch_pipe(const T* X, const T* Bt, const View& v, int cin, int cout, int grid_y, int tpw,
                               int vec, T* Y, hipStream_t s) {
  const int64_t blocks = ceil_div(v.st->n_tiles, tpw);
  const int rows = tpw * kTile;
  const int max_chunks = v.K * (rows / 16 + 1);
  const size_t lds = sizeof(float) * ((rows * (16 * NW + 1) + 1) & ~1) + max_chunks * (sizeof(int64_t) + sizeof(int32_t));
  k_gather_mma_pipe<T, NW, KBLK><<<dim3((unsigned)blocks, (unsigned)grid_y), NW * 64, lds, s>>>(
      X, Bt, v.st->seg, v.st->in_rows, v.st->out_rows, v.st->n_tiles, v.K, v.mirror ? 1 : 0, cin, cout,
      v.n_out, tpw, vec, max_chunks, Y);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

template <typename T, int NW>
static sscn_status launch_gather_mma_nw(const T* X, const T* Bt, const View& v, int cin, int cout,
                                        int grid_y, T* Y, hipStream_t s) {
  constexpr int VEC = sizeof(T) == 4 ? 4 : 8;  // elements per 16-byte load
  const int vec = (cin % VEC == 0) && ((uintptr_t)X % 16 == 0) && ((uintptr_t)Bt % 16 == 0);
  const int kblk = (cin + 63) / 64;
  const int tpw = NW >= 8 ? 1 : tiles_per_wg();
  switch (kblk) {
    case 1: return launch_pipe<T, NW, 1>(X, Bt, v, cin, cout, grid_y, tpw, vec, Y, s);
    case 2: return launch_pipe<T, NW, 2>(X, Bt, v, cin, cout, grid_y, tpw, vec, Y, s);
    case 3: return launch_pipe<T, NW, 3>(X, Bt, v, cin, cout, grid_y, tpw, vec, Y, s);
    case 4: return launch_pipe<T, NW, 4>(X, Bt, v, cin, cout, grid_y, tpw, vec, Y, s);
    default: break;
  }
  // wide inputs: unpipelined kernel, any c_in
  const int tpw_w = NW >= 8 ? 1 : 2;
  const int64_t blocks = ceil_div(v.st->n_tiles, tpw_w);
  const size_t lds = sizeof(float) * tpw_w * kTile * (16 * NW + 1);
  k_gather_mma<T, NW><<<dim3((unsigned)blocks, (unsigned)grid_y), NW * 64, lds, s>>>(
      X, Bt, v.st->seg, v.st->in_rows, v.st->out_rows, v.st->n_tiles, v.K, v.mirror ? 1 : 0, cin, cout,
      v.n_out, tpw_w, vec, Y);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

template <typename T, int NB, int KBLK>
static sscn_status launch_tile(const T* X, const T* Bt, const View& v, int cin, int cout, T* Y, hipStream_t s) {
  const int max_chunks = v.K * (kTile / 16 + 1);
  const size_t lds = sizeof(float) * ((4 * (kTile + 1) * (16 * NB + 1) + 1) & ~1) +
                     max_chunks * (sizeof(int64_t) + sizeof(int32_t));
  const int grid_y = (cout + 16 * NB - 1) / (16 * NB);
  const bool fast = (cin % 16 == 0) && ((uintptr_t)X % 16 == 0) && ((uintptr_t)Bt % 16 == 0);
  const dim3 grid((unsigned)v.st->n_tiles, (unsigned)grid_y);
  if (fast)
    k_conv_tile<T, NB, KBLK, true><<<grid, 256, lds, s>>>(X, Bt, v.st->seg, v.st->in_rows, v.st->out_rows,
                                                        v.st->n_tiles, v.K, v.mirror ? 1 : 0, cin, cout, v.n_out,
                                                        max_chunks, Y);
  else
    k_conv_tile<T, NB, KBLK, false><<<grid, 256, lds, s>>>(X, Bt, v.st->seg, v.st->in_rows, v.st->out_rows,
                                                         v.st->n_tiles, v.K, v.mirror ? 1 : 0, cin, cout, v.n_out,
                                                         max_chunks, Y);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

template <typename T>
static sscn_status launch_gather_mma(const T* X, const T* Bt, const View& v, int cin, int cout, T* Y,
                                     hipStream_t s) {
  if (v.st->n_tiles == 0) return SSCN_OK;
  constexpr int VEC = sizeof(T) == 4 ? 4 : 8;
  const int vec = (cin % VEC == 0) && ((uintptr_t)X % 16 == 0) && ((uintptr_t)Bt % 16 == 0);
  const char* mode = getenv("SSCN_FWD_KERNEL");  // tuning knob: "pipe" / "tile" / default "quad"
  const bool use_tile = !(mode && mode[0] == 'p');
  const bool use_quad = !(mode && (mode[0] == 'p' || mode[0] == 't'));
  if (use_quad && sizeof(T) == 4 && cin <= 64 && cout <= 64 && cin % 8 == 0 && (uintptr_t)X % 16 == 0 &&
      (uintptr_t)Bt % 16 == 0) {
    const int max_chunks = v.K * (kTile / 16 + 1);
    const size_t lds = sizeof(float) * ((2 * (kTile + 1) * 65 + 1) & ~1) + max_chunks * (sizeof(int64_t) + sizeof(int32_t));
    k_conv_quad<T><<<dim3((unsigned)v.st->n_tiles), 256, lds, s>>>(X, Bt, v.st->seg, v.st->in_rows, v.st->out_rows,
                                                                  v.st->n_tiles, v.K, v.mirror ? 1 : 0, cin, cout,
                                                                  v.n_out, max_chunks, Y);
    SSCN_HIP(hipGetLastError());
    return SSCN_OK;
  }
  if (use_tile && cin <= 64) {
    const int ncb = (cout + 15) / 16;
    if (ncb == 1) return launch_tile<T, 1, 1>(X, Bt, v, cin, cout, Y, s);
    if (ncb == 2) return launch_tile<T, 2, 1>(X, Bt, v, cin, cout, Y, s);
    if (ncb == 3) return launch_tile<T, 3, 1>(X, Bt, v, cin, cout, Y, s);
    return launch_tile<T, 4, 1>(X, Bt, v, cin, cout, Y, s);
  }
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

template <typename T, int CA, int CB>
static sscn_status launch_wgrad_reg(const T* X, const T* dY, const View& v, int cin, int cout, float* dW,
                                    hipStream_t s, int64_t max_ppo, int64_t n_pairs) {
  // about 1024 workgroups over all offsets, each a multiple of 64 pairs
  int64_t pch = ceil_div(n_pairs, 1024);
  pch = std::min<int64_t>(std::max<int64_t>(ceil_div(pch, 64) * 64, 256), 1 << 20);
  const int nzc = (cin + 16 * CA - 1) / (16 * CA);
  const int nzo = (cout + 16 * CB - 1) / (16 * CB);
  const int64_t gx = std::max<int64_t>(1, ceil_div(max_ppo, pch));
  k_wgrad_reg<T, CA, CB><<<dim3((unsigned)gx, (unsigned)v.K, (unsigned)(nzc * nzo)), 256, 0, s>>>(
      X, dY, v.st->seg, v.st->n_tiles, v.st->in_rows, v.st->out_rows, v.K, v.mirror ? 1 : 0, cin, cout, (int)pch,
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

template <typename T>
static sscn_status launch_wgrad(const T* X, const T* dY, const View& v, int cin, int cout, float* dW,
                                hipStream_t s, int64_t max_ppo, int64_t n_pairs) {
  const int ca = wgrad_blocks(cin), cb = wgrad_blocks(cout);
#define SSCN_WG(A, B) \
  if (ca == A && cb == B) return launch_wgrad_reg<T, A, B>(X, dY, v, cin, cout, dW, s, max_ppo, n_pairs);
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
