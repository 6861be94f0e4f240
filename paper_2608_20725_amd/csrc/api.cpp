// Host side of the C interface: argument checks, workspace accounting,
// device check and kernel dispatch.  The operations themselves run in the
// gfx950 kernels of transform.hip, conv_fp32*.hip and conv_fp16*.hip; the
// mini-batch entry points are in chunked.cpp.
#include "../../include/im2win.h"
#include "common.hpp"

#include <atomic>
#include <stdlib.h>
#include <string.h>

using namespace im2win;

namespace {

constexpr int64_t kMaxStrip = int64_t(1) << 20;
constexpr int64_t kMaxK = int64_t(1) << 24;
constexpr int64_t kMaxCo = int64_t(1) << 19;
constexpr int64_t kMaxBytes = int64_t(1) << 62;
constexpr int64_t kPad = 256;

bool mul_ok(int64_t a, int64_t b, int64_t lim, int64_t *out)
{
    if (a < 0 || b < 0)
        return false;
    if (a != 0 && b > lim / a)
        return false;
    *out = a * b;
    return true;
}

}  // namespace

// Shared with the chunked entry points (chunked.cpp).
namespace im2win {

// Fills `sh` from the user's arguments (filter dilation d, 1 for none);
// returns a status.
int make_shape_dil(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi, int64_t Co, int64_t Kh,
                   int64_t Kw, int64_t s, int64_t d, int dt, Shape *sh)
{
    if (dt != IM2WIN_F32 && dt != IM2WIN_F16 && dt != IM2WIN_BF16)
        return IM2WIN_EINVAL;
    if (N <= 0 || Ci <= 0 || Hi <= 0 || Wi <= 0 || Co <= 0 || Kh <= 0 || Kw <= 0 || s <= 0 || d <= 0)
        return IM2WIN_EINVAL;
    if (Hi > INT32_MAX || Wi > INT32_MAX || d > INT32_MAX)  // 32-bit row and column indices in the kernels
        return IM2WIN_ERANGE;
    // the dilated filter spans (K-1)*d + 1 rows and columns
    const int64_t Eh = (Kh - 1) * d + 1, Ew = (Kw - 1) * d + 1;
    if (Kh > Hi || Kw > Wi || Eh > Hi || Ew > Wi)
        return IM2WIN_EINVAL;
    Shape r;
    memset(&r, 0, sizeof r);
    r.N = N; r.Ci = Ci; r.Hi = Hi; r.Wi = Wi; r.Co = Co; r.Kh = Kh; r.Kw = Kw; r.s = s;
    r.d = d;
    r.Ho = (Hi - Eh) / s + 1;
    r.Wo = (Wi - Ew) / s + 1;
    // strip columns grouped by residue mod d, Wq per group
    r.Wq = (Wi + d - 1) / d;
    r.cols = d * r.Wq;  // < W_i + d <= 2^32
    r.elt = dt == IM2WIN_F32 ? 4 : 2;
    int64_t t;
    if (!mul_ok(r.cols, Kh, kMaxStrip, &t) || !mul_ok(t, Ci, kMaxStrip - 1, &r.L))
        return IM2WIN_ERANGE;
    if (!mul_ok(Kh, Kw, kMaxK, &t) || !mul_ok(t, Ci, kMaxK - 1, &r.K))
        return IM2WIN_ERANGE;
    if (Co >= kMaxCo)
        return IM2WIN_ERANGE;
    r.S = s * Kh * Ci;  // s <= W_i and Kh*Ci <= L: below 2^46
    if (!mul_ok(N, r.Ho, INT32_MAX, &r.strips))
        return IM2WIN_ERANGE;
    if (!mul_ok(r.strips, r.Wo, INT32_MAX, &r.P))
        return IM2WIN_ERANGE;
    if (!mul_ok(r.strips, r.L, kMaxBytes, &r.win_elems) ||
        !mul_ok(r.win_elems, r.elt, kMaxBytes, &r.win_bytes))
        return IM2WIN_ERANGE;
    r.pad_end = round_up(r.win_bytes, kPad) + kPad;
    r.Co_pad = round_up(Co, 256);
    r.K_pad = round_up(r.K, 64);
    r.K_pad32 = round_up(r.K, 16);
    r.Co_pad32 = round_up(Co, 32);
    r.Tp = round_up(Kh * Ci, 64);
    // the 16-bit kernels address the packed filter with 31-bit offsets
    if (dt != IM2WIN_F32 && r.Co_pad * r.Kw * r.Tp * 2 >= (int64_t)kMaxRecords)
        return IM2WIN_ERANGE;
    *sh = r;
    return IM2WIN_OK;
}

int make_shape(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi, int64_t Co, int64_t Kh, int64_t Kw,
               int64_t s, int dt, Shape *sh)
{
    return make_shape_dil(N, Ci, Hi, Wi, Co, Kh, Kw, s, 1, dt, sh);
}

TileGrid make_tilegrid(int64_t gx, int64_t gy, bool linear)
{
    // XCD order against launch order on MI355X (128 images): fp16 3x3 C=128
    // at 28x28 487 -> 583 TFLOP/s, 3x3 C=512 at 7x7 276 -> 309, 1x1 C=1024
    // at 14x14 632 -> 655; fp32 5x5 C_o=256 at 24x24 81.9 -> 86.5.  With one
    // channel tile there is nothing to share and launch order measured
    // slightly ahead (56x56 C=64: 457 vs 449 fp16, 78.5 vs 76.6 fp32).
    return TileGrid{(uint32_t)gx, (uint32_t)gy, (linear || gy <= 1) ? 0u : 1u};
}

int64_t packed_filter_bytes(const Shape &sh, int dt)
{
    // fp16 / bf16: room for every packed layout (C_o_pad*K_pad <= C_o_pad*K_w*Tp);
    // fp32: the vector-ALU layout [K_pad32][C_o_pad32] or the matrix-core one
    // [K/32][C_o_pad][32], whichever is larger
    if (dt != IM2WIN_F32)
        return sh.Co_pad * sh.Kw * sh.Tp * 2;
    const int64_t valu = sh.K_pad32 * sh.Co_pad32 * 4, mfma = fp32_mfma_packed_bytes(sh);
    return valu > mfma ? valu : mfma;
}

int64_t workspace_bytes(const Shape &sh, int dt)
{
    const int64_t base = sh.pad_end + packed_filter_bytes(sh, dt);
    if (dt == IM2WIN_F32)
        return base;
    // the split-K region of the plan a call makes without tuning variables
    Plan16 p;
    if (plan_fp16(sh, default_tuning(), &p) != IM2WIN_OK)
        return base;
    return base + split_bytes(sh, p);
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// The buffer [p, p+bytes) must lie inside one device allocation.
int check_extent(const void *p, int64_t bytes)
{
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    hipError_t e = hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)p);
    if (e != hipSuccess) {
        (void)hipGetLastError();  // leave no sticky error behind for the caller
        return IM2WIN_EBUFFER;
    }
    uintptr_t b = (uintptr_t)base, q = (uintptr_t)p;
    if (q < b || (uint64_t)(q - b) + (uint64_t)bytes > (uint64_t)size)
        return IM2WIN_EBUFFER;
    return IM2WIN_OK;
}

bool overlaps(const void *a, int64_t na, const void *b, int64_t nb)
{
    uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + (uint64_t)nb && y < x + (uint64_t)na;
}

// Per-device record: 0 unknown, 1 gfx950, -1 something else.
std::atomic<int> g_arch[64];

int check_device()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
        (void)hipGetLastError();
        return IM2WIN_ENODEV;
    }
    int known = g_arch[dev].load(std::memory_order_acquire);
    if (known == 0) {
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
            (void)hipGetLastError();
            return IM2WIN_ENODEV;
        }
        known = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : -1;
        g_arch[dev].store(known, std::memory_order_release);
    }
    return known == 1 ? IM2WIN_OK : IM2WIN_ENODEV;
}

int launch_status(hipError_t e)
{
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return IM2WIN_ELAUNCH;
    }
    return IM2WIN_OK;
}

}  // namespace im2win

namespace {

// The transform of the input zero-padded by pad_h / pad_w, for a filter
// dilated by d (1: none).
int transform_pad_dil(const void *in_nhwc, void *ws, int64_t ws_bytes, int64_t N, int64_t C_i, int64_t H_i,
                      int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride, int64_t pad_h,
                      int64_t pad_w, int64_t d, int dt, void *hip_stream)
{
    if (!in_nhwc || !ws)
        return IM2WIN_EINVAL;
    if (pad_h < 0 || pad_w < 0 || H_i <= 0 || W_i <= 0)
        return IM2WIN_EINVAL;
    if (pad_h > INT32_MAX / 4 || pad_w > INT32_MAX / 4 || H_i > INT32_MAX || W_i > INT32_MAX)
        return IM2WIN_ERANGE;
    Shape sh;  // the padded layer
    int rc = make_shape_dil(N, C_i, H_i + 2 * pad_h, W_i + 2 * pad_w, C_o, K_h, K_w, stride, d, dt, &sh);
    if (rc != IM2WIN_OK)
        return rc;
    if (!transform_range_ok(sh))
        return IM2WIN_ERANGE;
    if (!aligned16(in_nhwc) || !aligned16(ws))
        return IM2WIN_EALIGN;
    int64_t in_bytes;  // the stored input, without the padding
    if (!mul_ok(N * H_i, W_i * C_i, kMaxBytes / 4, &in_bytes))
        return IM2WIN_ERANGE;
    in_bytes *= sh.elt;
    if (ws_bytes < 0)
        return IM2WIN_EWORKSPACE;
    if ((rc = check_extent(in_nhwc, in_bytes)) != IM2WIN_OK)
        return rc;
    if ((rc = check_extent(ws, ws_bytes)) != IM2WIN_OK)
        return rc;
    if (overlaps(in_nhwc, in_bytes, ws, ws_bytes))
        return IM2WIN_EOVERLAP;
    if (ws_bytes < workspace_bytes(sh, dt))
        return IM2WIN_EWORKSPACE;
    Tuning tu;
    if ((rc = read_tuning(&tu)) != IM2WIN_OK)
        return rc;
    if ((rc = check_device()) != IM2WIN_OK)
        return rc;
    const Pad pad{H_i, W_i, pad_h, pad_w};
    return launch_status(launch_transform(sh, in_nhwc, ws, (hipStream_t)hip_stream, tu, &pad));
}

// The fp32 convolution, filter dilated by d (1: none): on the vector ALUs,
// or on the matrix cores when `mfma` is set and the layer allows it.
int conv32(void *ws, int64_t ws_bytes, const float *filt_khkwcico, float *out_nhwc, int64_t N, int64_t C_i,
           int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride, int64_t d,
           void *hip_stream, bool mfma = false)
{
    if (!ws || !filt_khkwcico || !out_nhwc)
        return IM2WIN_EINVAL;
    Shape sh;
    int rc = make_shape_dil(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, d, IM2WIN_F32, &sh);
    if (rc != IM2WIN_OK)
        return rc;
    if (!aligned16(ws) || !aligned16(filt_khkwcico) || !aligned16(out_nhwc))
        return IM2WIN_EALIGN;
    const int64_t f_bytes = sh.K * C_o * 4, o_bytes = sh.P * C_o * 4;
    if (ws_bytes < 0)
        return IM2WIN_EWORKSPACE;
    if ((rc = check_extent(ws, ws_bytes)) != IM2WIN_OK ||
        (rc = check_extent(filt_khkwcico, f_bytes)) != IM2WIN_OK ||
        (rc = check_extent(out_nhwc, o_bytes)) != IM2WIN_OK)
        return rc;
    if (overlaps(ws, ws_bytes, out_nhwc, o_bytes) || overlaps(filt_khkwcico, f_bytes, out_nhwc, o_bytes) ||
        overlaps(ws, ws_bytes, filt_khkwcico, f_bytes))
        return IM2WIN_EOVERLAP;
    if (ws_bytes < workspace_bytes(sh, IM2WIN_F32))
        return IM2WIN_EWORKSPACE;
    Tuning tu;
    Plan32 plan;
    if ((rc = read_tuning(&tu)) != IM2WIN_OK || (rc = plan_fp32(sh, tu, mfma, &plan)) != IM2WIN_OK)
        return rc;
    if ((rc = check_device()) != IM2WIN_OK)
        return rc;
    void *packed = (char *)ws + sh.pad_end;
    const hipStream_t st = (hipStream_t)hip_stream;
    if (plan.fam == Fam32::Mfma)
        return launch_status(launch_conv_fp32_mfma(sh, plan, tu, filt_khkwcico, packed, out_nhwc, ws, st));
    if ((rc = launch_status(launch_pack_fp32(sh, plan, filt_khkwcico, packed, st))) != IM2WIN_OK)
        return rc;
    return launch_status(launch_conv_fp32(sh, plan, tu, ws, packed, out_nhwc, st));
}

}  // namespace

extern "C" {

int conv_output_dims(int64_t H_i, int64_t W_i, int64_t K_h, int64_t K_w, int64_t stride,
                     int64_t *H_o, int64_t *W_o)
{
    if (!H_o || !W_o)
        return IM2WIN_EINVAL;
    if (H_i <= 0 || W_i <= 0 || K_h <= 0 || K_w <= 0 || stride <= 0 || K_h > H_i || K_w > W_i)
        return IM2WIN_EINVAL;
    *H_o = (H_i - K_h) / stride + 1;
    *W_o = (W_i - K_w) / stride + 1;
    return IM2WIN_OK;
}

int conv_output_dims_dilated(int64_t H_i, int64_t W_i, int64_t K_h, int64_t K_w, int64_t stride,
                             int64_t dilation, int64_t *H_o, int64_t *W_o)
{
    if (!H_o || !W_o)
        return IM2WIN_EINVAL;
    if (H_i <= 0 || W_i <= 0 || K_h <= 0 || K_w <= 0 || stride <= 0 || dilation <= 0 ||
        dilation > INT32_MAX || K_h > H_i || K_w > W_i)
        return IM2WIN_EINVAL;
    const int64_t Eh = (K_h - 1) * dilation + 1, Ew = (K_w - 1) * dilation + 1;
    if (Eh > H_i || Ew > W_i)
        return IM2WIN_EINVAL;
    *H_o = (H_i - Eh) / stride + 1;
    *W_o = (W_i - Ew) / stride + 1;
    return IM2WIN_OK;
}

int64_t conv_workspace_bytes_dilated(int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o,
                                     int64_t K_h, int64_t K_w, int64_t stride, int64_t dilation,
                                     im2win_dtype_t dt)
{
    Shape sh;
    int rc = make_shape_dil(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dilation, (int)dt, &sh);
    if (rc != IM2WIN_OK)
        return rc;
    return workspace_bytes(sh, (int)dt);
}

int64_t conv_workspace_bytes(int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o,
                             int64_t K_h, int64_t K_w, int64_t stride, im2win_dtype_t dt)
{
    Shape sh;
    int rc = make_shape(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, (int)dt, &sh);
    if (rc != IM2WIN_OK)
        return rc;
    return workspace_bytes(sh, (int)dt);
}

int64_t conv_im2col_bytes(int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t K_h,
                          int64_t K_w, int64_t stride, im2win_dtype_t dt)
{
    Shape sh;
    int rc = make_shape(N, C_i, H_i, W_i, 1, K_h, K_w, stride, (int)dt, &sh);
    if (rc != IM2WIN_OK)
        return rc;
    int64_t e, b;
    if (!mul_ok(sh.P, sh.K, kMaxBytes, &e) || !mul_ok(e, sh.elt, kMaxBytes, &b))
        return IM2WIN_ERANGE;
    return b;
}

int conv_im2win_transform(const void *in_nhwc, void *ws, int64_t ws_bytes, int64_t N,
                          int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h,
                          int64_t K_w, int64_t stride, im2win_dtype_t dt, void *hip_stream)
{
    if (!in_nhwc || !ws)
        return IM2WIN_EINVAL;
    Shape sh;
    int rc = make_shape(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, (int)dt, &sh);
    if (rc != IM2WIN_OK)
        return rc;
    if (!transform_range_ok(sh))
        return IM2WIN_ERANGE;
    if (!aligned16(in_nhwc) || !aligned16(ws))
        return IM2WIN_EALIGN;
    const int64_t in_bytes = N * H_i * W_i * C_i * sh.elt;
    if (ws_bytes < 0)
        return IM2WIN_EWORKSPACE;
    if ((rc = check_extent(in_nhwc, in_bytes)) != IM2WIN_OK)
        return rc;
    if ((rc = check_extent(ws, ws_bytes)) != IM2WIN_OK)
        return rc;
    if (overlaps(in_nhwc, in_bytes, ws, ws_bytes))
        return IM2WIN_EOVERLAP;
    if (ws_bytes < workspace_bytes(sh, (int)dt))
        return IM2WIN_EWORKSPACE;
    Tuning tu;
    if ((rc = read_tuning(&tu)) != IM2WIN_OK)
        return rc;
    if ((rc = check_device()) != IM2WIN_OK)
        return rc;
    return launch_status(launch_transform(sh, in_nhwc, ws, (hipStream_t)hip_stream, tu));
}

int conv_im2win_transform_padded(const void *in_nhwc, void *ws, int64_t ws_bytes, int64_t N,
                                 int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h,
                                 int64_t K_w, int64_t stride, int64_t pad_h, int64_t pad_w,
                                 im2win_dtype_t dt, void *hip_stream)
{
    return transform_pad_dil(in_nhwc, ws, ws_bytes, N, C_i, H_i, W_i, C_o, K_h, K_w, stride, pad_h, pad_w, 1,
                             (int)dt, hip_stream);
}

int conv_im2win_transform_dilated(const void *in_nhwc, void *ws, int64_t ws_bytes, int64_t N, int64_t C_i,
                                  int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w,
                                  int64_t stride, int64_t pad_h, int64_t pad_w, int64_t dilation,
                                  im2win_dtype_t dt, void *hip_stream)
{
    return transform_pad_dil(in_nhwc, ws, ws_bytes, N, C_i, H_i, W_i, C_o, K_h, K_w, stride, pad_h, pad_w,
                             dilation, (int)dt, hip_stream);
}

int conv_im2win_fp32(void *ws, int64_t ws_bytes, const float *filt_khkwcico,
                     float *out_nhwc, int64_t N, int64_t C_i, int64_t H_i, int64_t W_i,
                     int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride, void *hip_stream)
{
    return conv32(ws, ws_bytes, filt_khkwcico, out_nhwc, N, C_i, H_i, W_i, C_o, K_h, K_w, stride, 1, hip_stream);
}

int conv_im2win_fp32_mfma(void *ws, int64_t ws_bytes, const float *filt_khkwcico, float *out_nhwc, int64_t N,
                          int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w,
                          int64_t stride, void *hip_stream)
{
    return conv32(ws, ws_bytes, filt_khkwcico, out_nhwc, N, C_i, H_i, W_i, C_o, K_h, K_w, stride, 1, hip_stream,
                  true);
}

}  // extern "C"

namespace {

// The 16-bit matrix-core convolution, fp16 or bf16 operands (`dt`, `op`).
int conv16(void *ws, int64_t ws_bytes, const uint16_t *filt_khkwcico, uint16_t *out_nhwc, int64_t N,
           int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride,
           int64_t d, void *hip_stream, int dt, Op16 op)
{
    if (!ws || !filt_khkwcico || !out_nhwc)
        return IM2WIN_EINVAL;
    Shape sh;
    int rc = make_shape_dil(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, d, dt, &sh);
    if (rc != IM2WIN_OK)
        return rc;
    if (!aligned16(ws) || !aligned16(filt_khkwcico) || !aligned16(out_nhwc))
        return IM2WIN_EALIGN;
    const int64_t f_bytes = sh.K * C_o * 2, o_bytes = sh.P * C_o * 2;
    if (ws_bytes < 0)
        return IM2WIN_EWORKSPACE;
    if ((rc = check_extent(ws, ws_bytes)) != IM2WIN_OK ||
        (rc = check_extent(filt_khkwcico, f_bytes)) != IM2WIN_OK ||
        (rc = check_extent(out_nhwc, o_bytes)) != IM2WIN_OK)
        return rc;
    if (overlaps(ws, ws_bytes, out_nhwc, o_bytes) || overlaps(filt_khkwcico, f_bytes, out_nhwc, o_bytes) ||
        overlaps(ws, ws_bytes, filt_khkwcico, f_bytes))
        return IM2WIN_EOVERLAP;
    if (ws_bytes < workspace_bytes(sh, dt))
        return IM2WIN_EWORKSPACE;
    Tuning tu;
    Plan16 plan;
    if ((rc = read_tuning(&tu)) != IM2WIN_OK || (rc = plan_fp16(sh, tu, &plan)) != IM2WIN_OK)
        return rc;
    // a K split forced through the tuning may need more than the default plan
    const int64_t pf = packed_filter_bytes(sh, dt);
    if (ws_bytes < sh.pad_end + pf + split_bytes(sh, plan))
        return IM2WIN_EWORKSPACE;
    if ((rc = check_device()) != IM2WIN_OK)
        return rc;
    void *packed = (char *)ws + sh.pad_end;
    void *split = plan.ks > 1 ? (char *)packed + pf : nullptr;
    const hipStream_t st = (hipStream_t)hip_stream;
    if ((rc = launch_status(launch_pack_fp16(sh, plan, filt_khkwcico, packed, st, split))) != IM2WIN_OK)
        return rc;
    return launch_status(launch_conv_fp16(sh, plan, tu, ws, packed, out_nhwc, st, op, split));
}

}  // namespace

extern "C" {

int conv_im2win_fp16(void *ws, int64_t ws_bytes, const uint16_t *filt_khkwcico,
                     uint16_t *out_nhwc, int64_t N, int64_t C_i, int64_t H_i, int64_t W_i,
                     int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride, void *hip_stream)
{
    return conv16(ws, ws_bytes, filt_khkwcico, out_nhwc, N, C_i, H_i, W_i, C_o, K_h, K_w, stride, 1, hip_stream,
                  IM2WIN_F16, Op16::F16);
}

int conv_im2win_bf16(void *ws, int64_t ws_bytes, const uint16_t *filt_khkwcico,
                     uint16_t *out_nhwc, int64_t N, int64_t C_i, int64_t H_i, int64_t W_i,
                     int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride, void *hip_stream)
{
    return conv16(ws, ws_bytes, filt_khkwcico, out_nhwc, N, C_i, H_i, W_i, C_o, K_h, K_w, stride, 1, hip_stream,
                  IM2WIN_BF16, Op16::BF16);
}

int conv_im2win_dilated(void *ws, int64_t ws_bytes, const void *filt_khkwcico, void *out_nhwc, int64_t N,
                        int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w,
                        int64_t stride, int64_t dilation, im2win_dtype_t dt, void *hip_stream)
{
    switch (dt) {
    case IM2WIN_F32:
        return conv32(ws, ws_bytes, static_cast<const float *>(filt_khkwcico), static_cast<float *>(out_nhwc), N,
                      C_i, H_i, W_i, C_o, K_h, K_w, stride, dilation, hip_stream);
    case IM2WIN_F16:
    case IM2WIN_BF16:
        return conv16(ws, ws_bytes, static_cast<const uint16_t *>(filt_khkwcico),
                      static_cast<uint16_t *>(out_nhwc), N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dilation,
                      hip_stream, (int)dt, dt == IM2WIN_BF16 ? Op16::BF16 : Op16::F16);
    default:
        return IM2WIN_EINVAL;
    }
}

int conv_im2win_kernel_name(int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h,
                            int64_t K_w, int64_t stride, int64_t dilation, im2win_dtype_t dt, int fp32_matrix_cores,
                            char *buf, int64_t buf_len)
{
    if (!buf || buf_len < 1)
        return IM2WIN_EINVAL;
    buf[0] = 0;
    Shape sh;
    int rc = make_shape_dil(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dilation, (int)dt, &sh);
    if (rc != IM2WIN_OK)
        return rc;
    Tuning tu;
    if ((rc = read_tuning(&tu)) != IM2WIN_OK)
        return rc;
    char name[64];
    if (dt == IM2WIN_F32) {
        Plan32 p;
        if ((rc = plan_fp32(sh, tu, fp32_matrix_cores != 0, &p)) != IM2WIN_OK)
            return rc;
        plan32_name(sh, p, name, (int)sizeof name);
    } else {
        Plan16 p;
        if ((rc = plan_fp16(sh, tu, &p)) != IM2WIN_OK)
            return rc;
        plan16_name(sh, p, name, (int)sizeof name);
    }
    if ((int64_t)strlen(name) >= buf_len)
        return IM2WIN_ERANGE;
    strcpy(buf, name);
    return IM2WIN_OK;
}

const char *conv_im2win_strerror(int status)
{
    switch (status) {
    case IM2WIN_OK: return "ok";
    case IM2WIN_EINVAL: return "invalid argument";
    case IM2WIN_EALIGN: return "pointer not 16-byte aligned";
    case IM2WIN_ERANGE: return "size outside the supported index range";
    case IM2WIN_ENODEV: return "no gfx950 device";
    case IM2WIN_ELAUNCH: return "kernel launch failed";
    case IM2WIN_EWORKSPACE: return "workspace too small";
    case IM2WIN_EOVERLAP: return "buffers overlap";
    case IM2WIN_EBUFFER: return "not device memory, or the allocation is too small";
    default: return "unknown status";
    }
}

}  // extern "C"
