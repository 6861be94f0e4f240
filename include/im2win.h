/*
 * im2win.h -- im2win convolution on AMD Instinct MI355X (gfx950).
 *
 * Plain C interface: no HIP or framework types cross it, only host scalars
 * and device pointers.  The operation follows the paper's definitions:
 *
 *   convolution (Sec. III-A, Eq. 1), with the stride written in, 0-based:
 *     O[i][m][n][j] = sum_{u<K_h} sum_{v<K_w} sum_{r<C_i}
 *                       I[i][m*s+u][n*s+v][r] * F[u][v][r][j]
 *   window tensor (Sec. III-B, Eq. 2), NHWC element order:
 *     W[i][m][k*K_h+u][r] = I[i][m*s+u][k][r]
 *   windowed convolution (Sec. III-C, Eq. 3): the window of output (i,m,n) is
 *     the contiguous span of strip (i,m) that starts at element n*s*K_h*C_i and
 *     holds K = K_h*K_w*C_i elements in (filter column, filter row, channel)
 *     order.
 *
 * Layouts (all dense, row-major, no padding):
 *   input  I  NHWC [N][H_i][W_i][C_i]
 *   filter F  [K_h][K_w][C_i][C_o]     (filter height, width, in, out channel)
 *   output O  NHWC [N][H_o][W_o][C_o], H_o = (H_i-K_h)/s + 1, W_o = (W_i-K_w)/s + 1
 *   workspace (caller-allocated device memory, see conv_workspace_bytes):
 *     [0, win)        window tensor W [N][H_o][W_i*K_h][C_i], win = N*H_o*W_i*K_h*C_i*elt
 *     [win, pad_end)  zero bytes, pad_end = round_up(win, 256) + 256; they let
 *                     the kernels read past the last window without leaving
 *                     the buffer
 *     [pad_end, ...)  the filter repacked in window order (tap k = (v*K_h+u)*C_i+r)
 *                     and zero-padded, written by the conv call:
 *                       fp16 / bf16: C_o_pad*K_w*T_pad 16-bit values, C_o_pad = round_up(C_o, 256),
 *                             T_pad = round_up(K_h*C_i, 64): tiles of TB taps, each
 *                             holding C_o_pad rows per slice, either one slice of
 *                             K_pad = round_up(K, 64) taps or one slice of T_pad taps
 *                             per filter column; TB depends on the kernel the layer
 *                             runs (an internal layout, rewritten by every conv call)
 *                       fp32: the larger of [K_pad32][C_o_pad32] fp32, K_pad32 =
 *                             round_up(K, 16), C_o_pad32 = round_up(C_o, 32) (vector-ALU
 *                             kernels; channels 2i and 2i+1 swapped in each row for the
 *                             LDS-staged kernel) and round_up(C_o, 128)*round_up(K, 32)
 *                             fp32 (conv_im2win_fp32_mfma)
 *
 * Scope: one stride and one dilation for both axes; zero padding and dilation
 * through the *_padded / *_dilated calls below; no groups or bias.
 *
 * Ownership and threading: the caller allocates and frees every buffer; the
 * library allocates nothing and keeps no state except a once-filled per-device
 * record of whether the device is a gfx950.  Calls are reentrant.
 *
 * Streams: every device call only enqueues work on `hip_stream` (a
 * hipStream_t; NULL is the null stream) and returns without synchronising.
 * A conv call reads the window tensor, so it must be ordered after the
 * transform that wrote it (same stream, or an event).
 *
 * Errors: arguments are checked before anything is enqueued, in this order:
 * null pointers -> dimensions -> index ranges -> alignment -> buffer extents
 * (each pointer must lie in one device allocation that holds the whole
 * buffer) -> overlap -> workspace size -> device -> launch.  The first failing
 * check's status is returned; nothing is printed and no exception leaves the
 * library.  Kernel choice: each conv call picks its kernel from the layer's
 * shape (conv_im2win_kernel_name reports which).  Tuning variables in the
 * environment can force another, to measure kernels against each other:
 * IM2WIN_FP16_KERNEL (pipe | regs), IM2WIN_FP16_COL, IM2WIN_FP16_TILE,
 * IM2WIN_FP16_SEG, IM2WIN_FP32_KERNEL (a variant name | regs),
 * IM2WIN_FP32_TILE, IM2WIN_FP32_MFMA_TILE (variant names),
 * IM2WIN_TRANSFORM_ORDER and IM2WIN_TILE_ORDER (xcd | linear),
 * IM2WIN_TRANSFORM_KERNEL (pieces | gather: the 3-channel transform),
 * IM2WIN_FP16_PERSIST (on | off: the column-staged kernel's persistent launch),
 * IM2WIN_TAP_ORDER (linear | column: the filter columns' tap slices in turn,
 * the columns grouped by residue mod the stride), IM2WIN_FP16_SPLIT (1..8: the K range
 * of the row-per-pixel fp16 kernel split over that many workgroups per output
 * tile, their fp32 partial tiles added afterwards in a fixed order; a split
 * the default plan does not make needs ks * tiles * 64 KiB of workspace beyond
 * conv_workspace_bytes, else IM2WIN_EWORKSPACE).  A value
 * that names no kernel, contradictory values, or a forced kernel that cannot
 * run the layer make the call return IM2WIN_EINVAL (checked after the
 * workspace size, before the device).  Numerics: fp32 conv accumulates in fp32 (FMA); fp16 and bf16 conv
 * take 16-bit operands, accumulate in fp32 and round to nearest-even on store.
 */
#ifndef IM2WIN_H
#define IM2WIN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element types: fp32, IEEE fp16, bf16 (bfloat16: fp32's 8-bit exponent, 8-bit significand). */
typedef enum { IM2WIN_F32 = 0, IM2WIN_F16 = 1, IM2WIN_BF16 = 2 } im2win_dtype_t;

enum {
    IM2WIN_OK = 0,
    IM2WIN_EINVAL = -1,     /* null pointer, bad dtype, dims <= 0, K_h > H_i, K_w > W_i, s < 1 */
    IM2WIN_EALIGN = -2,     /* a device pointer is not 16-byte aligned */
    IM2WIN_ERANGE = -3,     /* a size overflows the library's index ranges (see below) */
    IM2WIN_ENODEV = -4,     /* the current device is not a gfx950 GPU, or none is usable */
    IM2WIN_ELAUNCH = -5,    /* a kernel launch was rejected by the runtime */
    IM2WIN_EWORKSPACE = -6, /* ws_bytes < conv_workspace_bytes(...) */
    IM2WIN_EOVERLAP = -7,   /* two buffers overlap */
    IM2WIN_EBUFFER = -8     /* a pointer is not device memory, or its allocation is too small */
};

/*
 * Output extent (no padding): *H_o = (H_i - K_h)/s + 1, *W_o = (W_i - K_w)/s + 1
 * (Table I sizes).  Host only.  Returns IM2WIN_OK or IM2WIN_EINVAL.
 */
int conv_output_dims(int64_t H_i, int64_t W_i, int64_t K_h, int64_t K_w, int64_t stride,
                     int64_t *H_o, int64_t *W_o);

/*
 * Bytes of workspace the transform and the conv of this layer need (layout
 * above): the window tensor of Eq. 2, the zero pad and the packed filter.  Host only, no device calls.  Returns a
 * negative status for invalid arguments (IM2WIN_EINVAL, IM2WIN_ERANGE).
 *
 * Index ranges the kernels support (else IM2WIN_ERANGE): one strip
 * W_i*K_h*C_i < 2^20 elements, K = K_h*K_w*C_i < 2^24, C_o < 2^19,
 * N*H_o*W_o < 2^31 output pixels, N*H_o < 2^31 strips, for IM2WIN_F16/BF16 a packed
 * filter (above) below 2^31 bytes, and every byte count below 2^62.
 */
int64_t conv_workspace_bytes(int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o,
                             int64_t K_h, int64_t K_w, int64_t stride, im2win_dtype_t dt);

/*
 * Bytes of the full-batch im2col matrix of the same layer,
 * N*H_o*W_o * K_h*K_w*C_i * elt (one row per output pixel, one column per
 * filter tap and channel; Sec. III-B and Fig. 1).  The comparator for the
 * workspace figure; the library never builds it.  Host only.
 */
int64_t conv_im2col_bytes(int64_t N, int64_t C_i, int64_t H_i, int64_t W_i,
                          int64_t K_h, int64_t K_w, int64_t stride, im2win_dtype_t dt);

/*
 * The im2win transform (Sec. III-B, Eq. 2).
 *   in_nhwc  device, input I (fp32, fp16 or bf16 bits, per `dt`), read only
 *   ws       device, workspace of ws_bytes >= conv_workspace_bytes(..., dt);
 *            the window tensor and the zero pad are written, the rest of the
 *            workspace is left alone
 * The copy is bit-exact and does not depend on the element type beyond its
 * size.  C_o and K_w only size the workspace check.  Besides the ranges of
 * conv_workspace_bytes, the window tensor must hold fewer than 2^32 16-byte
 * granules when C_i*elt is a multiple of 16 bytes, else fewer than 2^32
 * elements (IM2WIN_ERANGE).
 */
int conv_im2win_transform(const void *in_nhwc, void *ws, int64_t ws_bytes,
                          int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o,
                          int64_t K_h, int64_t K_w, int64_t stride, im2win_dtype_t dt,
                          void *hip_stream);

/*
 * The im2win transform of a zero-padded input (Eq. 2 applied to the input
 * surrounded by pad_h zero rows above and below and pad_w zero columns left
 * and right; the paper's layers have no padding, real CNN layers do).  The
 * padded input is never built: window-tensor positions outside the stored
 * input are written as zeros.
 *   in_nhwc  device, the stored input I [N][H_i][W_i][C_i], read only
 *   ws       device, workspace of ws_bytes >= conv_workspace_bytes(N, C_i,
 *            H_i + 2*pad_h, W_i + 2*pad_w, ..., dt); layout as above for the
 *            padded extents
 *   pad_h, pad_w  >= 0; pad 0 gives exactly conv_im2win_transform's result
 * The convolution of the padded layer is then conv_im2win_fp32/fp16 called
 * with H_i + 2*pad_h and W_i + 2*pad_w as the input extents (their output is
 * H_o = floor((H_i + 2*pad_h - K_h)/s) + 1 by W_o likewise).  Errors as for
 * conv_im2win_transform, with the padded extents checked as the layer
 * (IM2WIN_EINVAL for a negative pad, IM2WIN_ERANGE for pads above 2^29).
 */
int conv_im2win_transform_padded(const void *in_nhwc, void *ws, int64_t ws_bytes, int64_t N,
                                 int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h,
                                 int64_t K_w, int64_t stride, int64_t pad_h, int64_t pad_w,
                                 im2win_dtype_t dt, void *hip_stream);

/*
 * fp32 windowed convolution on the vector ALUs (Sec. III-C, Eq. 3; the
 * paper's CUDA-core variant, Sec. IV-A).
 *   ws              device, workspace holding the fp32 window tensor written
 *                   by conv_im2win_transform(..., IM2WIN_F32); the window
 *                   tensor is read, the packed-filter region is overwritten
 *   filt_khkwcico   device, fp32 filter F [K_h][K_w][C_i][C_o]; read only
 *   out_nhwc        device, fp32 output O [N][H_o][W_o][C_o]; every element
 *                   is written exactly once
 * Each output is one fp32 fused multiply-add chain over the window's taps in
 * (filter column, filter row, channel) order.
 */
int conv_im2win_fp32(void *ws, int64_t ws_bytes, const float *filt_khkwcico,
                     float *out_nhwc, int64_t N, int64_t C_i, int64_t H_i, int64_t W_i,
                     int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride, void *hip_stream);

/*
 * fp32 windowed convolution on the matrix cores: the sums of
 * conv_im2win_fp32 computed as the product of Alg. 1 (M = C_o by N =
 * N*H_o*W_o over K = C_i*K_h*K_w) with v_mfma_f32_32x32x2_f32, fp32 operands
 * and fp32 accumulation.  An alternate fp32 path (the paper's fp32 variant
 * runs on the vector units, Sec. III-F).  Arguments, workspace, buffer rules
 * and errors as for conv_im2win_fp32.  Results meet the same bound; the
 * order of the fp32 additions differs from the vector-ALU kernel's, so the
 * bits may differ.  Layers whose C_i is not a multiple of 4 (windows not made
 * of whole 16-byte chunks) run the vector-ALU kernel instead.
 */
int conv_im2win_fp32_mfma(void *ws, int64_t ws_bytes, const float *filt_khkwcico, float *out_nhwc, int64_t N,
                          int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w,
                          int64_t stride, void *hip_stream);

/*
 * fp16 windowed convolution on the matrix cores (Sec. III-D, Alg. 1: the
 * output as an M = C_o by N = N*H_o*W_o product over K = C_i*K_h*K_w).
 *   ws              device, workspace holding the fp16 window tensor written
 *                   by conv_im2win_transform(..., IM2WIN_F16); the window
 *                   tensor is read, the packed-filter region is overwritten
 *   filt_khkwcico   device, fp16 bits of F [K_h][K_w][C_i][C_o]; read only
 *   out_nhwc        device, fp16 bits of O [N][H_o][W_o][C_o]; every element
 *                   is written exactly once
 * Products of fp16 operands are accumulated in fp32; each output is rounded
 * to fp16 (nearest-even) once.
 */
int conv_im2win_fp16(void *ws, int64_t ws_bytes, const uint16_t *filt_khkwcico,
                     uint16_t *out_nhwc, int64_t N, int64_t C_i, int64_t H_i, int64_t W_i,
                     int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride, void *hip_stream);

/*
 * bf16 windowed convolution on the matrix cores: the same product as
 * conv_im2win_fp16 (Sec. III-D, Alg. 1) with bf16 operands.  An extension:
 * the paper's multi-precision support (Sec. III-F) has two variants, fp32 on
 * the vector units and fp16 on the matrix units; bf16 is a third operand type
 * for the same kernels, with fp32's exponent range.
 *   ws              device, workspace holding the bf16 window tensor written
 *                   by conv_im2win_transform(..., IM2WIN_BF16); the window
 *                   tensor is read, the packed-filter region is overwritten
 *   filt_khkwcico   device, bf16 bits of F [K_h][K_w][C_i][C_o]; read only
 *   out_nhwc        device, bf16 bits of O [N][H_o][W_o][C_o]; every element
 *                   is written exactly once
 * Products of bf16 operands are accumulated in fp32; each output is rounded
 * to bf16 (nearest-even) once.  Workspace, index ranges and errors as for
 * conv_im2win_fp16 (the workspace of IM2WIN_BF16 equals that of IM2WIN_F16).
 */
int conv_im2win_bf16(void *ws, int64_t ws_bytes, const uint16_t *filt_khkwcico,
                     uint16_t *out_nhwc, int64_t N, int64_t C_i, int64_t H_i, int64_t W_i,
                     int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride, void *hip_stream);

/*
 * Filter dilation (an extension; the paper's layers have none): tap (u, v) of
 * output (m, n) reads input row m*s + u*d and column n*s + v*d, so
 *   O[i][m][n][j] = sum_u sum_v sum_r I[i][m*s+u*d][n*s+v*d][r] * F[u][v][r][j],
 * the dilated filter spans E_h = (K_h-1)*d + 1 rows and E_w columns, and
 * H_o = (H_i - E_h)/s + 1, W_o likewise.  d = 1 is the plain convolution.
 *
 * Window tensor with dilation: each strip (i, m) holds rows m*s + u*d of the
 * input, and its columns are grouped by residue mod d: with Wq = ceil(W_i/d)
 * columns per group, strip column P holds input column (P mod Wq)*d +
 * floor(P/Wq) (zero filler where that is >= W_i), element (P*K_h + u)*C_i + r.
 * The window of output column n is then one contiguous span of K elements
 * starting at column ((n*s) mod d)*Wq + floor(n*s/d), in (filter column,
 * filter row, channel) order as in Eq. 3.  Workspace layout as above with
 * strips of d*Wq*K_h*C_i elements (at most (d-1)*K_h*C_i more than W_i*K_h*C_i).
 */

/* Output extent with dilation (no padding).  Host only.  IM2WIN_EINVAL when
 * the dilated filter does not fit or an argument is out of range. */
int conv_output_dims_dilated(int64_t H_i, int64_t W_i, int64_t K_h, int64_t K_w, int64_t stride,
                             int64_t dilation, int64_t *H_o, int64_t *W_o);

/* Workspace bytes of a dilated layer (H_i, W_i: the padded extents when the
 * transform pads).  Index ranges as for conv_workspace_bytes, with the strip
 * d*ceil(W_i/d)*K_h*C_i below 2^20 elements.  Host only. */
int64_t conv_workspace_bytes_dilated(int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o,
                                     int64_t K_h, int64_t K_w, int64_t stride, int64_t dilation,
                                     im2win_dtype_t dt);

/*
 * The dilated window tensor of the input zero-padded by pad_h rows and pad_w
 * columns on each side (pads >= 0; dilation >= 1; dilation 1 is
 * conv_im2win_transform_padded).
 *   in_nhwc  device, the stored input [N][H_i][W_i][C_i], read only
 *   ws       device, ws_bytes >= conv_workspace_bytes_dilated(N, C_i,
 *            H_i + 2*pad_h, W_i + 2*pad_w, C_o, K_h, K_w, stride, dilation, dt)
 * Errors as for conv_im2win_transform_padded.
 */
int conv_im2win_transform_dilated(const void *in_nhwc, void *ws, int64_t ws_bytes, int64_t N, int64_t C_i,
                                  int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w,
                                  int64_t stride, int64_t pad_h, int64_t pad_w, int64_t dilation,
                                  im2win_dtype_t dt, void *hip_stream);

/*
 * Dilated windowed convolution from the dilated window tensor in `ws`
 * (written by conv_im2win_transform_dilated with the same dt and dilation),
 * in the precision `dt` names: IM2WIN_F32 on the vector ALUs (filter and
 * output fp32), IM2WIN_F16 / IM2WIN_BF16 on the matrix cores (16-bit filter
 * and output bits, fp32 accumulation, one rounding on store).  H_i, W_i are
 * the (padded) extents the window tensor was built for.  Numerics, buffer
 * rules and errors as for conv_im2win_fp32/fp16/bf16; dilation 1 gives their
 * results bit for bit.
 */
int conv_im2win_dilated(void *ws, int64_t ws_bytes, const void *filt_khkwcico, void *out_nhwc, int64_t N,
                        int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w,
                        int64_t stride, int64_t dilation, im2win_dtype_t dt, void *hip_stream);

/*
 * Mini-batch im2win: bytes of workspace conv_im2win_chunked needs for chunks
 * of n_chunk images (n_chunk is clamped to N), with one window-tensor slot, or
 * two when two_streams is non-zero:
 *   nslots * round_up(pad_end(n_chunk), 256) + packed filter bytes,
 * where pad_end(n) is the pad end of an n-image window tensor (layout above).
 * Host only.  Returns a negative status for invalid arguments.
 */
int64_t conv_chunked_workspace_bytes(int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o,
                                     int64_t K_h, int64_t K_w, int64_t stride, int64_t n_chunk,
                                     int two_streams, im2win_dtype_t dt);

/*
 * Transform + windowed convolution of the whole batch in chunks of n_chunk
 * images (the mini-batch strategy of Sec. IV-C, against the full-batch
 * conv_im2win_transform + conv_im2win_fp32/fp16/bf16 pair): the workspace holds the
 * window tensor of one chunk, or of two when a second stream is given.
 *   in_nhwc         device, input I (fp32, fp16 or bf16 bits per `dt`), read only
 *   filt_khkwcico   device, filter F, read only
 *   out_nhwc        device, output O, written once per element
 *   ws              device, ws_bytes >= conv_chunked_workspace_bytes(...,
 *                   hip_stream_aux != NULL, dt); slot layout as above, the
 *                   packed filter after the slots
 *   hip_stream      the filter pack and the chunks (transform, then conv) are
 *                   enqueued here
 *   hip_stream_aux  NULL, or a second stream: chunks then alternate between
 *                   the two streams (chunk c on hip_stream_aux when c is odd),
 *                   each stream using its own workspace slot, so two chunks
 *                   are in flight and one's transform overlaps the other's
 *                   conv.  The aux stream first waits for the work already on
 *                   hip_stream and hip_stream finally waits for the aux
 *                   stream, so all of the call is ordered before later work on
 *                   hip_stream.  The ordering uses two HIP events created and
 *                   destroyed within the call (no device memory is allocated).
 * The kernel is chosen once, for a full chunk of n_chunk images (see
 * conv_im2win_kernel_name), and runs every chunk, the last one included, so
 * every output is bit-identical to what conv_im2win_fp32/fp16/bf16 give for it
 * in a batch of n_chunk images.  Against a full-batch call (whose kernel,
 * picked for N images, may sum in another order) it agrees within the error
 * bound of the exact result.  Errors as for the other calls; input, filter, output and workspace must not
 * overlap, and the two streams must differ.
 */
int conv_im2win_chunked(const void *in_nhwc, const void *filt_khkwcico, void *out_nhwc, void *ws,
                        int64_t ws_bytes, int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o,
                        int64_t K_h, int64_t K_w, int64_t stride, int64_t n_chunk, im2win_dtype_t dt,
                        void *hip_stream, void *hip_stream_aux);

/*
 * Allocation-free mini-batch call, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid it): conv_im2win_chunked on one stream and one workspace slot, with
 * the workspace in a static device buffer of IM2WIN_STATIC_SCRATCH_BYTES that
 * the library holds on every GPU it runs on until the process ends.
 *   in_nhwc, filt_khkwcico, out_nhwc, N .. n_chunk, dt, hip_stream
 *           as for conv_im2win_chunked (the caller still allocates the input,
 *           filter and output)
 * Returns IM2WIN_EWORKSPACE, before anything is enqueued, when
 * conv_chunked_workspace_bytes(..., n_chunk, 0, dt) exceeds
 * IM2WIN_STATIC_SCRATCH_BYTES (choose a smaller n_chunk).  The call makes no
 * device allocation and creates no events; its first call on a device looks
 * up that device's buffer once.  All calls on one GPU share its buffer and
 * the buffer keeps the last call's contents: calls that overlap on one GPU
 * (on different streams, or from several host threads without ordering)
 * race.  Output, numerics and other errors as for conv_im2win_chunked.
 */
#define IM2WIN_STATIC_SCRATCH_BYTES ((int64_t)128 << 20)
int conv_im2win_chunked_noalloc(const void *in_nhwc, const void *filt_khkwcico, void *out_nhwc, int64_t N,
                                int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w,
                                int64_t stride, int64_t n_chunk, im2win_dtype_t dt, void *hip_stream);

/*
 * Names the kernel the conv call of this layer runs, e.g.
 * "conv_fp16_col k3c64p128t32s2" (kernel family, then variant): the choice
 * the call makes from the shape and the tuning variables above.
 *   dt                 IM2WIN_F32 (vector ALUs, or the matrix cores when
 *                      fp32_matrix_cores is non-zero: conv_im2win_fp32_mfma),
 *                      IM2WIN_F16 or IM2WIN_BF16 (same kernels)
 *   dilation           1 for the plain layer (conv_im2win_dilated otherwise)
 *   buf, buf_len       host buffer receiving a NUL-terminated name (64 bytes
 *                      always suffice)
 * For the mini-batch call, pass N = n_chunk: every chunk runs the kernel of a
 * full chunk.  Host only.  Returns IM2WIN_OK, the status the conv call would
 * return for bad dims or tuning variables, or IM2WIN_ERANGE when buf_len is
 * too short.
 */
int conv_im2win_kernel_name(int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h,
                            int64_t K_w, int64_t stride, int64_t dilation, im2win_dtype_t dt,
                            int fp32_matrix_cores, char *buf, int64_t buf_len);

/* A static, human-readable name for a status code. */
const char *conv_im2win_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* IM2WIN_H */
