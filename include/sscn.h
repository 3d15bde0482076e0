/*
 * sscn.h -- C ABI of the MI355X (gfx950) sparse / submanifold sparse
 * convolution library (libsscn.so).
 *
 * Method: Graham, Engelcke & van der Maaten, "3D Semantic Segmentation with
 * Submanifold Sparse Convolutional Networks" (arXiv:1711.10275).
 *   - layer state = feature matrix (one row per active site) + a dictionary
 *     (location -> row), Sec. 4.2;
 *   - rule book R = (R_o : o in F), F = {0..f-1}^3, each R_o a list of
 *     (input row, output row) pairs, Sec. 4.2;
 *   - SC(m, n, f, s) and SSC(m, n, f) active sets, Sec. 4.1;
 *   - output = 0, then out[k] += in[j] * W^o for every (j, k) in R_o,
 *     Sec. 4.2.
 *
 * Conventions shared by every call
 *   - d = 3.  Filter offsets are numbered o = i0*f*f + i1*f + i2.
 *   - The operation is a cross-correlation: an SSC output at y reads the
 *     input at y + i - (f-1)/2, an SC output at y reads the input at s*y + i.
 *   - coords: int32, n x 4 rows (b, x0, x1, x2), row-major, 16-byte aligned,
 *     row j <-> feature row j.  0 <= b < 32768, 0 <= x_d < spatial_size[d]
 *     <= 65536.  The batch index is part of the location, so samples never
 *     interact.
 *   - features: row-major n x C.  weights: [K][c_in][c_out] (K = f^3).
 *   - dtype SSCN_F32: everything fp32.  SSCN_BF16: features, weights, out
 *     and dgrad are bfloat16; products are accumulated in fp32 and rounded
 *     once (nearest-even) when written; wgrad is always fp32.
 *   - Pointers are DEVICE pointers unless marked (host).  The caller owns
 *     every feature / weight / coordinate / output buffer.  Outputs are fully
 *     overwritten and must not alias inputs.
 *   - Work is enqueued on `stream` (may be NULL = the default stream).  A
 *     rule book may be used on its build stream at once; on another stream
 *     only after the caller has ordered that stream after the build stream.
 *   - Errors are returned as codes, never thrown across the ABI; on failure
 *     *out is left untouched and sscn_last_error() (thread-local) describes
 *     the failure.  A device fault surfaces at the next synchronising call as
 *     SSCN_ERR_DEVICE.
 *   - Sizes: n * f^3 must stay below 2^31 (positions are 32-bit).
 */
#ifndef SSCN_H
#define SSCN_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SSCN_OK = 0,
  SSCN_ERR_INVALID_ARG = 1,  /* null pointer with n > 0, n < 0, bad f / s / C / dtype, misaligned coords */
  SSCN_ERR_SHAPE = 2,        /* SC: L < f or (L - f) % s != 0; channel count or dtype inconsistent with the rule book */
  SSCN_ERR_OUT_OF_RANGE = 3, /* a coordinate outside [0, L) or a batch index outside [0, 32768) */
  SSCN_ERR_DUPLICATE = 4,    /* two rows at one location (one row per active site, Sec. 4.2) */
  SSCN_ERR_OOM = 5,          /* device allocation failed */
  SSCN_ERR_DEVICE = 6        /* a HIP runtime error */
} sscn_status;

typedef enum { SSCN_F32 = 0, SSCN_BF16 = 1 } sscn_dtype;

/* Opaque rule book; library-owned and immutable after its build. */
typedef struct sscn_rulebook_s* sscn_rulebook;

/*
 * ssc_rulebook_build -- rule book of SSC(., ., f) (Sec. 4.1 "Submanifold
 * sparse convolution"; Sec. 4.2, last paragraph: the input dictionary is
 * re-used as the output dictionary).
 *   coords        device, n x 4 int32 (see conventions)
 *   n             number of active sites (n = 0 gives an empty rule book)
 *   spatial_size  host, 3 extents L_d
 *   filter_size   f, odd (else SSCN_ERR_INVALID_ARG)
 *   out           receives the handle; free with sscn_rulebook_free
 * The output set equals the input set and output row k is input row k.
 * Builds a GPU open-addressing dictionary, probes the f^3 neighbours of
 * every site and compacts the hits into R.  Blocks the host once to read
 * back sizes and error flags; the row-block plan that the layer kernels
 * use is queued behind that readback and may still be running on `stream`
 * when the call returns (work on other streams waits for it).
 */
sscn_status ssc_rulebook_build(const int32_t* coords, int64_t n, const int32_t* spatial_size,
                               int32_t filter_size, hipStream_t stream, sscn_rulebook* out);

/*
 * sc_rulebook_build -- rule book of SC(., ., f, s) (Sec. 4.1 "Sparse
 * convolutional operations"; Sec. 4.2 step 1).
 *   spatial_size  host, 3 extents L_d with L_d >= f and (L_d - f) % s == 0
 *                 (else SSCN_ERR_SHAPE); output extent (L_d - f + s) / s
 *   filter_size, stride  f >= 1, s >= 1
 * An output site is active iff its f^3 field holds an active input.  Output
 * rows are numbered in the order of first visit when input rows are taken
 * in row order and, per input, offsets in increasing o (the single pass of
 * Sec. 4.2 step 1 with that iteration order); read them back with
 * sscn_rulebook_out_coords.  Blocks the host once.
 */
sscn_status sc_rulebook_build(const int32_t* coords, int64_t n, const int32_t* spatial_size,
                              int32_t filter_size, int32_t stride, hipStream_t stream,
                              sscn_rulebook* out);

/*
 * sscn_rulebook_build_nd -- the rule book of SSC(., ., f) (submanifold != 0,
 * stride 1) or SC(., ., f, s) on a d-dimensional grid, d = dim in [1, 4]
 * (the layers are defined for any d, Sec. 3; 4-D data such as RGB-D video,
 * Sec. 1).  d = 3 is ssc_rulebook_build / sc_rulebook_build.
 *   coords        device, n x (d + 1) int32 rows (b, x_0, .., x_{d-1}),
 *                 4-byte aligned
 *   spatial_size  host, d extents
 * Offsets are numbered in base f with the first coordinate most
 * significant (o = ((i_0 f + i_1) f + ..) ); K = f^d <= 512 and
 * 32768 * prod(spatial_size) < 2^63 (else SSCN_ERR_INVALID_ARG); SC shape
 * rules, output numbering, errors and storage as in three dimensions, so
 * every other call takes the result unchanged.  sscn_rulebook_out_coords
 * then gives n_out x (d + 1) rows.  Blocks the host once.
 */
sscn_status sscn_rulebook_build_nd(const int32_t* coords, int64_t n, int32_t dim, const int32_t* spatial_size,
                                   int32_t filter_size, int32_t stride, int32_t submanifold, hipStream_t stream,
                                   sscn_rulebook* out);

/*
 * sscn_rulebook_transpose -- the inverted connections R^T_o = {(k, j) :
 * (j, k) in R_o}: the rule book of the deconvolution DC that inverts an SC
 * (Sec. 4.1 "Other operators"); its output set is the SC's input set, in
 * the SC's input row order.  For an SSC rule book R^T_o = R_{K-1-o}.  The
 * view shares storage with (and keeps alive) its parent; free it with
 * sscn_rulebook_free.  Transposing a transposed view gives a view of the
 * parent.  No device work, no synchronisation.
 */
sscn_status sscn_rulebook_transpose(sscn_rulebook rb, sscn_rulebook* out);

typedef struct {
  int64_t n_in, n_out, n_pairs;
  int32_t filter_size, stride, submanifold, transposed, n_offsets;
  int32_t dim;                      /* spatial dimensions d (3 unless built by sscn_rulebook_build_nd) */
  int32_t in_size[4], out_size[4];  /* grid extents; the first d entries are used */
} sscn_rulebook_info;

/*
 * sscn_rulebook_query -- sizes of a rule book (host only, no device work).
 *   info              host, filled in
 *   pairs_per_offset  host, n_offsets entries |R_o| (nullable)
 * sum_o |R_o| * c_in * c_out is the layer's multiply-add count (Table 2:
 * a*m*n summed over active output sites).
 */
sscn_status sscn_rulebook_query(sscn_rulebook rb, sscn_rulebook_info* info,
                                int64_t* pairs_per_offset);

/*
 * sscn_rulebook_out_coords -- device n_out x (d + 1) int32 coordinates of
 * the output sites (n_out x 4 for d = 3), in output row order, grid of
 * extent info.out_size.
 */
sscn_status sscn_rulebook_out_coords(sscn_rulebook rb, int32_t* out_coords, hipStream_t stream);

/*
 * sscn_rulebook_export -- every pair as (in_rows[p], out_rows[p],
 * offsets[p]), p < n_pairs, sorted by (offset, out row, in row).  Device
 * int32 arrays of n_pairs entries each.
 */
sscn_status sscn_rulebook_export(sscn_rulebook rb, int32_t* in_rows, int32_t* out_rows,
                                 int32_t* offsets, hipStream_t stream);

/* Release a rule book or view (storage goes when its last view goes). NULL is a no-op.
 * The storage returns to the library's device-memory cache, ordered on the
 * build stream: before it can be handed out again, the build stream is made
 * to wait (an event per stream) for all work that this library queued on
 * other streams reading the rule book.  The build stream must therefore
 * still exist when the last view is freed.  Cached memory goes back to the
 * device when an allocation would fail. */
void sscn_rulebook_free(sscn_rulebook rb);

/*
 * sparse_conv_forward -- out = 0; out[k] += features[j] * W^o for every
 * (j, k) in R_o (Sec. 4.2 step 2).  With a transposed rule book this is
 * the deconvolution DC with its own weights [K][c_in][c_out].
 *   features  device n_in x c_in     weights  device K x c_in x c_out
 *   out       device n_out x c_out, overwritten
 * Asynchronous on `stream`.
 */
sscn_status sparse_conv_forward(const void* features, const void* weights, sscn_rulebook rb,
                                int32_t c_in, int32_t c_out, sscn_dtype dtype, void* out,
                                hipStream_t stream);

/*
 * One destination of sparse_conv_forward_heads.  The layer output y (n_out x
 * c_out) is written as max(0, y[k][c] * scale[c] + shift[c]) -- the
 * inference-form batch normalisation and ReLU that pre-activate the next
 * unit of a network (Sec. 5) -- or as y itself when scale is NULL, rounded
 * once to the layer's dtype.
 *   data        device, row k at data + k * row_stride (elements of dtype),
 *               c_out consecutive elements per row
 *   row_stride  >= c_out; a wider stride writes into the columns of a
 *               concatenation buffer
 *   scale/shift device fp32, c_out entries each; both NULL or both set
 */
typedef struct {
  void* data;
  int64_t row_stride;
  const float* scale;
  const float* shift;
} sscn_conv_output;

/*
 * sparse_conv_forward_heads -- sparse_conv_forward writing the result to
 * n_heads (1 or 2) destinations (host array `heads`), each with its own
 * optional activation.  Destinations must not overlap each other or the
 * inputs.  SSCN_ERR_INVALID_ARG for a bad head (NULL data, stride < c_out,
 * only one of scale / shift).  Asynchronous on `stream`.
 */
sscn_status sparse_conv_forward_heads(const void* features, const void* weights, sscn_rulebook rb,
                                      int32_t c_in, int32_t c_out, sscn_dtype dtype, int32_t n_heads,
                                      const sscn_conv_output* heads, hipStream_t stream);

/*
 * sparse_conv_forward_ex -- sparse_conv_forward_heads with a bias and a
 * residual: every active output row becomes
 *   v[k] = y[k] + bias + residual[k]
 * before the heads map it.  The bias is a convolution's bias term (the
 * ground state at inactive sites is not stored, Sec. 3 footnote); the
 * residual is the identity shortcut of a residual block (Sec. 5: the
 * block's input, same sites and channels as its output).
 *   bias         device fp32, c_out entries, nullable
 *   residual     device n_out x c_out in dtype, row k at residual + k *
 *                residual_ld, nullable; may be one of the heads' buffers
 *                only if it is that head's own row (read before written)
 */
sscn_status sparse_conv_forward_ex(const void* features, const void* weights, sscn_rulebook rb, int32_t c_in,
                                   int32_t c_out, sscn_dtype dtype, const float* bias, const void* residual,
                                   int64_t residual_ld, int32_t n_heads, const sscn_conv_output* heads,
                                   hipStream_t stream);

/*
 * sparse_conv_forward_noalloc -- sparse_conv_forward for callers that cannot
 * allocate device memory (code under stream capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, same kernels and the
 * same (bit-identical) result; it allocates nothing:
 *   - the forward's one temporary, a transposed copy of the weights, goes to
 *     a fixed 8 MiB region of the library's code object (one per device,
 *     held until the process ends): K * c_in * c_out elements of dtype must
 *     fit in 8 MiB, else SSCN_ERR_INVALID_ARG (nothing is queued);
 *   - the rule book's kernel tables must already exist: a 3-d SSC rule
 *     book of filter size 1 or 3 has them from its build, any other gets them
 *     from one sparse_conv_forward / sparse_conv_backward on it (same
 *     direction); otherwise SSCN_ERR_INVALID_ARG, `out` untouched.
 * Every call on a device shares that device's region, which keeps the last
 * call's contents: calls that overlap on one device (concurrent streams or
 * host threads) race on it and must be serialised by the caller.
 * Asynchronous on `stream`.
 */
sscn_status sparse_conv_forward_noalloc(const void* features, const void* weights, sscn_rulebook rb,
                                        int32_t c_in, int32_t c_out, sscn_dtype dtype, void* out,
                                        hipStream_t stream);

/*
 * sparse_conv_backward -- gradients of sparse_conv_forward (its adjoint):
 *   dgrad[j] = sum_o sum_{(j,k) in R_o} dout[k] * (W^o)^T   (n_in x c_in)
 *   wgrad[o] = sum_{(j,k) in R_o} features[j]^T dout[k]    (K x c_in x c_out, fp32)
 * dgrad runs the forward machinery over the transposed rule book; wgrad is
 * a per-offset gathered (c_in x pairs) x (pairs x c_out) contraction.
 *   features  device n_in x c_in (needed only for wgrad; nullable if wgrad is NULL)
 *   dout      device n_out x c_out
 *   dgrad     device n_in x c_in, overwritten (nullable: skipped)
 *   wgrad     device fp32 K x c_in x c_out, overwritten (nullable: skipped)
 * Asynchronous on `stream`.
 */
sscn_status sparse_conv_backward(const void* features, const void* weights, const void* dout,
                                 sscn_rulebook rb, int32_t c_in, int32_t c_out, sscn_dtype dtype,
                                 void* dgrad, float* wgrad, hipStream_t stream);

/*
 * Pooling (Sec. 4.1 "Other operators"): MP(f, s) and AP(f, s) are variants of
 * SC(., ., f, s) -- same active output sites, same connections -- that
 * reduce instead of multiply:
 *   MP: out[k][c] = max(0, max over (j, k) in R_o of features[j][c])
 *       (the maximum of the zero vector and the active inputs of the field);
 *   AP: out[k][c] = f^-3 * sum over (j, k) in R_o of features[j][c]
 *       (inactive sites contribute zero).
 *   rb        an SC(f, s) rule book (not an SSC one, not a transposed view;
 *             else SSCN_ERR_INVALID_ARG); rows as in sparse_conv_forward
 *   features  device n_in x c, out device n_out x c (overwritten), in dtype;
 *             bf16: the maximum is exact, the AP sum is taken in fp32 and
 *             rounded once
 *   argmax    MP only (else ignored, nullable): device uint8 n_out x c, the
 *             offset o of the input that attains each maximum (the smallest
 *             such o when several tie), 255 where the zero vector does;
 *             K = f^3 must be at most 254
 * Output rows are written once (no atomics): the result is deterministic.
 */
typedef enum { SSCN_POOL_MAX = 0, SSCN_POOL_AVG = 1 } sscn_pool_mode;
sscn_status sscn_pool_forward(const void* features, sscn_rulebook rb, int32_t c, sscn_dtype dtype,
                              sscn_pool_mode mode, void* out, uint8_t* argmax, hipStream_t stream);

/*
 * sscn_pool_backward -- gradient of sscn_pool_forward with respect to its
 * features: MP routes dout[k][c] to the input at offset argmax[k][c] (none
 * for 255); AP gives every input of the field f^-3 * dout[k][c], summed over
 * the outputs it belongs to.
 *   dout    device n_out x c;  argmax  MP: the forward's argmax (nullable for AP)
 *   dgrad   device n_in x c, overwritten
 */
sscn_status sscn_pool_backward(const void* dout, const uint8_t* argmax, sscn_rulebook rb, int32_t c,
                               sscn_dtype dtype, sscn_pool_mode mode, void* dgrad, hipStream_t stream);

/*
 * sscn_upsample_forward -- nearest-neighbour upsampling of the FCN (Sec. 5):
 * undoes the downsampling of an SC(s, s) rule book rb (filter size equal to
 * the stride, else SSCN_ERR_INVALID_ARG) by copying each of its output
 * sites' features to every input site in that site's s^3 block.
 *   features  device rb.n_out x c;  out  device rb.n_in x c (overwritten),
 *   in the rule book's input row order
 */
sscn_status sscn_upsample_forward(const void* features, sscn_rulebook rb, int32_t c, sscn_dtype dtype,
                                  void* out, hipStream_t stream);

/*
 * sscn_upsample_backward -- its gradient: dgrad[k] = sum of dout[j] over the
 * input sites j of output site k's block.
 *   dout  device rb.n_in x c;  dgrad  device rb.n_out x c (overwritten)
 */
sscn_status sscn_upsample_backward(const void* dout, sscn_rulebook rb, int32_t c, sscn_dtype dtype,
                                   void* dgrad, hipStream_t stream);

/*
 * sscn_affine_relu -- y[r][c] = max(0, x[r][c] * scale[c] + shift[c]) over the
 * n active rows: batch normalisation in inference form followed by ReLU,
 * both restricted to active sites (Sec. 4.1 "Other operators"; the
 * pre-activated blocks of Sec. 5).  x, y: n x c in `dtype` (may alias);
 * scale, shift: device fp32, c entries each.
 */
sscn_status sscn_affine_relu(const void* x, const float* scale, const float* shift, int64_t n,
                             int32_t c, sscn_dtype dtype, void* y, hipStream_t stream);

/*
 * sscn_concat_cols -- y = [a | b] row by row: a is n x ca, b is n x cb, y is
 * n x (ca + cb), all in `dtype` (the skip-connection merge of the U-Net of
 * Sec. 5).  y must not alias a or b.
 */
sscn_status sscn_concat_cols(const void* a, int32_t ca, const void* b, int32_t cb, int64_t n,
                             sscn_dtype dtype, void* y, hipStream_t stream);

/*
 * sscn_time_next_launch -- measurement aid: the next launch of a row-block
 * (forward / dgrad) or wgrad kernel made by a call on this host thread
 * records `before` at that kernel's start and `after` at its end (with the
 * dispatch itself, hipExtLaunchKernelGGL: no separate event packets), so
 * hipEventElapsedTime(before, after) is that one kernel's time even when
 * the call queues other small kernels around it.  The events belong to the
 * caller (created with timing enabled); the request is used once.  NULL,
 * NULL cancels it.  Not a paper operation.
 */
sscn_status sscn_time_next_launch(hipEvent_t before, hipEvent_t after);

/*
 * sscn_release_cached -- give the library's idle device blocks on the
 * current device back to the device (after a device-wide synchronisation),
 * e.g. when another allocator in the process runs out of memory.  Storage
 * of live rule books is not touched.  Not a paper operation: memory
 * management of the rule-book storage of Sec. 4.2.
 */
sscn_status sscn_release_cached(void);

/*
 * sscn_set_device_memory_cap -- cap the device memory the library holds per
 * device (rule-book storage, build temporaries and its cache of idle
 * blocks) at `bytes`; 0 removes the cap.  A new block that would exceed
 * it first releases the idle blocks, then fails with SSCN_ERR_OOM as a real
 * out-of-memory would, so that this path can be exercised (a request that
 * an idle block of the cache serves allocates nothing and always succeeds).  Read from the
 * environment variable SSCN_DEVICE_MEMORY_CAP (bytes) at the first
 * allocation unless set here.  Not a paper operation.
 */
sscn_status sscn_set_device_memory_cap(uint64_t bytes);

/*
 * sscn_set_deterministic -- on != 0: sparse_conv_backward's wgrad adds the
 * partial sums of its work items in a fixed order instead of with atomic
 * additions, so dW is bit-reproducible from run to run (for filters of at
 * most 128 offsets; the bf16 kernel of 32 x 32, 64 x 32, 64 x 64 and
 * 128 x 64 channels always is).  It costs a buffer of the partial blocks
 * and one more pass.  Process-wide; off by default.  Not a paper
 * operation: the reduction order of the sums of Sec. 4.1.
 */
sscn_status sscn_set_deterministic(int32_t on);

/*
 * ------------------------------------------------------------------ training
 * Batch normalisation "applied over the set of active sites" and activation
 * functions restricted to them (Sec. 4.1 "Other operators"); the final
 * per-site linear layer and softmax (Sec. 5); negative log-likelihood and
 * SGD with Nesterov momentum and L2 weight decay (Sec. 6.2).
 *
 * Matrices are n x c row-major with a row stride (`ld*`, elements, >= c), so
 * that a column range of a wider buffer (a concatenation) can be passed by
 * offsetting the pointer.  Per-channel vectors are device fp32, c entries.
 * Column reductions are deterministic: fixed per-workgroup fp64 partial sums
 * added in a fixed order (no atomics).
 */

/*
 * sscn_batchnorm_forward -- batch statistics of x over its n active rows:
 * mean, invstd = 1/sqrt(var + eps) (biased variance), scale = gamma * invstd
 * and shift = beta - mean * scale (the inference-form affine map, as
 * sscn_affine_relu and conv output heads take it).  Training applies the
 * normalisation with sscn_batchnorm_relu_apply.  running_mean / running_var
 * (both or neither) are updated as (1 - momentum) r + momentum stat, with the
 * unbiased variance.  n >= 1 (else SSCN_ERR_INVALID_ARG).
 */
sscn_status sscn_batchnorm_forward(const void* x, int64_t ldx, int64_t n, int32_t c, sscn_dtype dtype,
                                   const float* gamma, const float* beta, float eps, float momentum,
                                   float* running_mean, float* running_var, float* mean, float* invstd,
                                   float* scale, float* shift, hipStream_t stream);

/*
 * sscn_batchnorm_relu_apply -- y = relu((x - mean) * scale + beta), the
 * normalisation with batch statistics followed by ReLU (x, y may be equal
 * but must not otherwise overlap).  The mean is subtracted first, so the
 * result stays accurate when a channel's variance is tiny next to its mean.
 */
sscn_status sscn_batchnorm_relu_apply(const void* x, int64_t ldx, int64_t n, int32_t c, sscn_dtype dtype,
                                      const float* mean, const float* scale, const float* beta, void* y,
                                      int64_t ldy, hipStream_t stream);

/*
 * sscn_batchnorm_relu_backward_params -- first half of the gradient of
 * a = sscn_batchnorm_relu_apply(x): with dz = dA where the forward's ReLU
 * passed ((x - mean) * scale + beta > 0, evaluated exactly as the forward
 * does) and 0 elsewhere, and xhat = (x - mean) * invstd,
 *   dbeta = sum over rows of dz,  dgamma = sum over rows of dz * xhat.
 */
sscn_status sscn_batchnorm_relu_backward_params(const void* dA, int64_t ldd, const void* x, int64_t ldx,
                                                int64_t n, int32_t c, sscn_dtype dtype, const float* mean,
                                                const float* invstd, const float* scale, const float* beta,
                                                float* dgamma, float* dbeta, hipStream_t stream);

/*
 * sscn_batchnorm_relu_backward_input -- second half: the gradient at x,
 *   dx = gamma * invstd * (dz - dbeta / n - xhat * dgamma / n)  (+ add),
 * for any column range of the layer (offset every pointer and vector by the
 * range's first column; n stays the layer's row count).  `add` (nullable,
 * row stride ld_add) is a gradient from another consumer of x, summed in.
 */
sscn_status sscn_batchnorm_relu_backward_input(const void* dA, int64_t ldd, const void* x, int64_t ldx,
                                               int64_t n, int32_t c, sscn_dtype dtype, const float* gamma,
                                               const float* beta, const float* mean, const float* invstd,
                                               const float* scale, const float* dgamma, const float* dbeta,
                                               const void* add, int64_t ld_add, void* dx, int64_t ldx_out,
                                               hipStream_t stream);

/* sscn_column_sum -- out[col] = sum over the n rows of x[row][col] (a bias gradient), fp32 out. */
sscn_status sscn_column_sum(const void* x, int64_t ldx, int64_t n, int32_t c, sscn_dtype dtype, float* out,
                            hipStream_t stream);

/* sscn_add -- y = a + b elementwise (identity residual connections, Sec. 5; gradient sums). */
sscn_status sscn_add(const void* a, int64_t lda, const void* b, int64_t ldb, int64_t n, int32_t c,
                     sscn_dtype dtype, void* y, int64_t ldy, hipStream_t stream);

/*
 * sscn_softmax_nll -- per active site, softmax over `classes` logits and the
 * negative log-likelihood of its label (Sec. 5, Sec. 6.2):
 *   loss (device, 1 float) = mean over the n sites of
 *                            logsumexp(logits[r]) - logits[r][labels[r]]
 *   dlogits[r][k] = (softmax(logits[r])[k] - [k == labels[r]]) / n
 * logits and dlogits: contiguous n x classes in dtype; labels int32 in
 * [0, classes) (a label outside gives a NaN loss).  n >= 1.
 */
sscn_status sscn_softmax_nll(const void* logits, int64_t n, int32_t classes, sscn_dtype dtype,
                             const int32_t* labels, float* loss, void* dlogits, hipStream_t stream);

/*
 * sscn_sgd_nesterov -- one step of SGD with Nesterov momentum and L2 weight
 * decay (Sec. 6.2), elementwise over `count` fp32 parameters:
 *   g' = g + weight_decay * p;  buf = momentum * buf + g';
 *   p = p - lr * (g' + momentum * buf)
 * (buf starts at zero).  params_bf16 (nullable) receives p rounded to
 * bfloat16 (the copy a bf16 network convolves with).
 */
sscn_status sscn_sgd_nesterov(float* params, const float* grads, float* momentum_buf, int64_t count, float lr,
                              float momentum, float weight_decay, void* params_bf16, hipStream_t stream);

/* Thread-local message describing the last failure on this thread ("" if none). */
const char* sscn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SSCN_H */
