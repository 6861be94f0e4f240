// im2win transform (Sec. III-B, Eq. 2) for gfx950.
//
//   W[i][m][k*K_h + u][r] = I[i][m*s + u][k][r]
//
// Pure copy, HBM-bound: every byte of the window tensor is written once; the
// K_h/s-fold re-reads of input rows are served by L2 and the Infinity Cache.
// Three kernels:
//   * vec:    C_i*elt is a multiple of 16 bytes.  A thread copies whole
//             16-byte granules; a workgroup covers a contiguous run of the
//             window tensor (possibly across strips), so the stores of a wave
//             are one contiguous 1 KiB run, in an XCD-aware block order.
//   * gather: any other C_i.  A thread assembles one 16-byte granule of the
//             flat window tensor element by element; granules may straddle
//             strips.
//   * pieces3: the gather for C_i = 3 (the stem layers), undilated and
//             unpadded (fp32; fp16 with K_h <= 3), reading each 3-channel
//             pixel it needs with one load.
// All zero the pad bytes that follow the window tensor.
//
// Zero padding of the input (not in the paper's layers) is folded in: the
// window tensor is that of the input surrounded by ph zero rows and pw zero
// columns on each side, and positions outside the stored input are written
// as zeros; the padded input itself is never built.
#include "common.hpp"

#include <stdlib.h>
#include <string.h>

namespace im2win {
namespace {

constexpr int kThreads = 256;
constexpr int kGranPerThread = 4;

struct TArgs {
    const char *in;
    char *ws;
    uint32_t Ci, Hi, Wi, Kh, s, Ho;  // Hi x Wi: the stored (unpadded) input
    uint32_t Wp, ph, pw;             // padded width Wi + 2*pw; zero rows / columns per side
    uint32_t d, Wq, cols;            // dilation; strip columns per residue group; d*Wq columns
    uint32_t L;              // strip length (elements)
    uint32_t strips;
    uint32_t gran_per_strip; // vec: 16-byte granules per strip
    uint64_t win_elems;
    uint64_t win_bytes, pad_end;
    uint64_t grans;          // gather: 16-byte granules of the window tensor
    uint64_t in_pixels;      // pieces3: pixels of the input (N * H_i * W_i)
    uint32_t xcd_order;      // vec: 1 = XCD-aware block order, 0 = linear (ablation)
    FastDiv div_Ci, div_Kh, div_Wi, div_Ho, div_L, div_gps, div_Wq;
};

// Padded-input column held by strip column position k: k itself, or with
// dilation d (columns grouped by residue mod d, Wq per group) column
// (k mod Wq)*d + floor(k/Wq); positions past the padded width are filler and
// map to columns >= Wp, outside the stored input like the right-hand padding.
__device__ inline uint32_t strip_col(uint32_t k, const TArgs &a)
{
    if (a.d == 1)
        return k;
    const uint32_t g = fdiv(k, a.div_Wq);
    return (k - g * a.Wq) * a.d + g;
}

__device__ inline void zero_pad(const TArgs &a)
{
    // [win_bytes, pad_end) holds at most 256 + 255 + 15 bytes
    for (uint64_t b = a.win_bytes + threadIdx.x; b < a.pad_end; b += blockDim.x)
        a.ws[b] = 0;
}

// XCD-aware block order: the hardware deals the blocks of a launch to the 8
// XCDs round-robin (block b to XCD b % 8), and each XCD has its own L2.  Block
// b works on logical block xcd_block(b), so that every XCD walks one
// contiguous run of the window tensor: strips that share input rows are then
// copied by the same XCD at about the same time and the re-reads hit its L2.
// A bijection on [0, nb).
__device__ inline uint32_t xcd_block(uint32_t b, uint32_t nb)
{
    const uint32_t x = b % 8, j = b / 8;
    const uint32_t per = nb / 8, rem = nb % 8;
    return x * per + (x < rem ? x : rem) + j;
}

template <int ELT>
__global__ __launch_bounds__(kThreads) void transform_vec(TArgs a)
{
    constexpr uint32_t V = 16 / ELT;  // elements per granule
    if (blockIdx.x == 0)
        zero_pad(a);
    // granules of the whole window tensor, numbered strip by strip
    // (granule counts fit 32 bits: transform_range_ok)
    const uint32_t lb = a.xcd_order ? xcd_block(blockIdx.x, gridDim.x) : blockIdx.x;
    const uint32_t gb = lb * (kThreads * kGranPerThread);
#pragma unroll
    for (int t = 0; t < kGranPerThread; ++t) {
        const uint32_t g = gb + t * kThreads + threadIdx.x;
        if (g < a.grans) {
            const uint32_t q = fdiv(g, a.div_gps);  // strip
            const uint32_t pos = (g - q * a.gran_per_strip) * V;
            const uint32_t i = fdiv(q, a.div_Ho);
            const uint32_t m = q - i * a.Ho;
            const uint32_t seg = fdiv(pos, a.div_Ci);  // k*K_h + u
            const uint32_t r = pos - seg * a.Ci;
            const uint32_t k = fdiv(seg, a.div_Kh);
            const uint32_t u = seg - k * a.Kh;
            // a granule lies inside one (column, row) piece of C_i elements:
            // all of it is padding or none
            const int32_t h = (int32_t)(m * a.s + u * a.d) - (int32_t)a.ph;
            const int32_t w = (int32_t)strip_col(k, a) - (int32_t)a.pw;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (h >= 0 && h < (int32_t)a.Hi && w >= 0 && w < (int32_t)a.Wi) {
                const uint64_t src = (((uint64_t)i * a.Hi + (uint32_t)h) * a.Wi + (uint32_t)w) * a.Ci + r;
                v = *reinterpret_cast<const uint4 *>(a.in + src * ELT);
            }
            *reinterpret_cast<uint4 *>(a.ws + (uint64_t)g * 16) = v;
        }
    }
}

template <int ELT>
__device__ inline void store_elem_t(uint32_t *w, int e, uint32_t bits)
{
    if (ELT == 4) {
        w[e] = bits;
    } else {
        const int d = e >> 1;
        w[d] = (e & 1) ? (w[d] & 0xffffu) | (bits << 16) : (w[d] & 0xffff0000u) | (bits & 0xffffu);
    }
}

// The gather of the 3-channel layers with one load per piece: a 16-byte
// granule of the window tensor (8 fp16 or 4 fp32 elements) spans at most 4
// (fp16) or 2 (fp32) pieces, a piece being the 3 channels of one input pixel
// (one column of one filter row of one strip).  Each piece is read with one
// load, 8 bytes for fp16 (6 used) and 12 for fp32, instead of one load per
// element; the granule is assembled in registers and stored whole, so a
// wave's stores stay one contiguous 1 KiB run.  An 8-byte fp16 read would
// reach 2 bytes past the last pixel of the input: that piece is read as 4 + 2
// bytes.
template <int ELT>
__global__ __launch_bounds__(kThreads) void transform_pieces3(TArgs a)
{
    constexpr uint32_t V = 16 / ELT;                // elements per granule
    constexpr int NP = ELT == 2 ? 4 : 2;            // pieces a granule can touch
    const uint64_t g = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
    if (blockIdx.x == 0)
        zero_pad(a);
    if (g >= a.grans)
        return;
    // first element of this granule (win_elems < 2^32, checked on the host)
    const uint32_t e0 = (uint32_t)(g * V);
    uint32_t q = fdiv(e0, a.div_L);
    const uint32_t pos = e0 - q * a.L;
    uint32_t seg = fdiv(pos, a.div_Ci);              // k*K_h + u of the first piece
    const uint32_t r0 = pos - seg * 3;               // its first channel used
    const uint32_t segs = a.L / 3;                   // pieces per strip (W_i * K_h)
    uint32_t el[NP * 3];                             // the pieces' elements (ELT bytes each)
#pragma unroll
    for (int j = 0; j < NP; ++j) {
        el[3 * j] = el[3 * j + 1] = el[3 * j + 2] = 0u;
        // piece j holds granule elements 3j - r0 .. 3j - r0 + 2
        if (3 * j >= (int)(r0 + V) || (uint64_t)e0 + 3 * j - r0 >= a.win_elems)
            continue;
        if (seg == segs) {  // into the next strip
            seg = 0;
            ++q;
        }
        const uint32_t k = fdiv(seg, a.div_Kh), u = seg - k * a.Kh;
        const uint32_t i = fdiv(q, a.div_Ho), m = q - i * a.Ho;
        const uint64_t px = ((uint64_t)i * a.Hi + m * a.s + u) * a.Wi + k;  // input pixel
        const char *src = a.in + px * (3 * ELT);
        if (ELT == 4) {
            uint32_t v[3];
            __builtin_memcpy(v, src, 12);
            el[3 * j] = v[0]; el[3 * j + 1] = v[1]; el[3 * j + 2] = v[2];
        } else {
            uint64_t v;  // one 8-byte load (the last pixel: 4 + 2 bytes)
            if (px + 1 < a.in_pixels) {
                __builtin_memcpy(&v, src, 8);
            } else {
                uint32_t lo;
                uint16_t hi;
                __builtin_memcpy(&lo, src, 4);
                __builtin_memcpy(&hi, src + 4, 2);
                v = lo | ((uint64_t)hi << 32);
            }
            el[3 * j] = (uint32_t)v & 0xffffu;
            el[3 * j + 1] = (uint32_t)(v >> 16) & 0xffffu;
            el[3 * j + 2] = (uint32_t)(v >> 32) & 0xffffu;
        }
        ++seg;
    }
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (uint32_t t = 0; t < V; ++t) {
        // element t of the granule is element r0 + t of the pieces' run
        // (r0 < 3)
        const uint32_t bits = r0 == 0 ? el[t] : r0 == 1 ? el[t + 1] : el[t + 2];
        store_elem_t<ELT>(w, (int)t, bits);
    }
    // bytes past the window tensor are inside the zero pad: zeros are written
    *reinterpret_cast<uint4 *>(a.ws + g * 16) = make_uint4(w[0], w[1], w[2], w[3]);
}

template <int ELT>
__device__ inline void store_elem(uint32_t *w, int e, uint32_t bits)
{
    if (ELT == 4) {
        w[e] = bits;
    } else {
        const int d = e >> 1;
        w[d] = (e & 1) ? (w[d] & 0xffffu) | (bits << 16) : (w[d] & 0xffff0000u) | (bits & 0xffffu);
    }
}

template <int ELT>
__global__ __launch_bounds__(kThreads) void transform_gather(TArgs a)
{
    constexpr uint32_t V = 16 / ELT;
    const uint64_t g = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
    if (blockIdx.x == 0)
        zero_pad(a);
    if (g >= a.grans)
        return;
    // first element of this granule; win_elems < 2^32 is checked on the host
    uint32_t e = (uint32_t)(g * V);
    uint32_t q = fdiv(e, a.div_L);
    uint32_t pos = e - q * a.L;
    uint32_t seg = fdiv(pos, a.div_Ci);
    uint32_t r = pos - seg * a.Ci;
    uint32_t k = fdiv(seg, a.div_Kh);
    uint32_t u = seg - k * a.Kh;
    uint32_t i = fdiv(q, a.div_Ho);
    uint32_t m = q - i * a.Ho;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (uint32_t t = 0; t < V; ++t) {
        if ((uint64_t)e + t < a.win_elems) {
            const int32_t hh = (int32_t)(m * a.s + u * a.d) - (int32_t)a.ph;
            const int32_t ww = (int32_t)strip_col(k, a) - (int32_t)a.pw;
            uint32_t bits = 0;
            if (hh >= 0 && hh < (int32_t)a.Hi && ww >= 0 && ww < (int32_t)a.Wi) {
                const uint64_t src = (((uint64_t)i * a.Hi + (uint32_t)hh) * a.Wi + (uint32_t)ww) * a.Ci + r;
                if (ELT == 4)
                    bits = reinterpret_cast<const uint32_t *>(a.in)[src];
                else
                    bits = reinterpret_cast<const uint16_t *>(a.in)[src];
            }
            store_elem<ELT>(w, (int)t, bits);
            // advance (r, u, k, m, i) to the next window-tensor element
            if (++r == a.Ci) {
                r = 0;
                if (++u == a.Kh) {
                    u = 0;
                    if (++k == a.cols) {
                        k = 0;
                        if (++m == a.Ho) {
                            m = 0;
                            ++i;
                        }
                    }
                }
            }
        }
    }
    // bytes past the window tensor are inside the zero pad: zeros are written
    *reinterpret_cast<uint4 *>(a.ws + g * 16) = make_uint4(w[0], w[1], w[2], w[3]);
}

}  // namespace

bool transform_range_ok(const Shape &sh)
{
    if ((sh.Ci * sh.elt) % 16 == 0)  // granule indices fit 32 bits
        return (uint64_t)sh.win_bytes / 16 + kThreads * kGranPerThread < (1ull << 32);
    return (uint64_t)sh.win_elems + 16 < (1ull << 32);
}

hipError_t launch_transform(const Shape &sh, const void *in, void *ws, hipStream_t st, const Tuning &t,
                            const Pad *pad)
{
    TArgs a;
    a.in = static_cast<const char *>(in);
    a.ws = static_cast<char *>(ws);
    a.Ci = (uint32_t)sh.Ci;
    a.Wp = (uint32_t)sh.Wi;
    if (pad) {
        a.Hi = (uint32_t)pad->Hi; a.Wi = (uint32_t)pad->Wi;
        a.ph = (uint32_t)pad->ph; a.pw = (uint32_t)pad->pw;
    } else {
        a.Hi = (uint32_t)sh.Hi; a.Wi = (uint32_t)sh.Wi;
        a.ph = 0; a.pw = 0;
    }
    a.Kh = (uint32_t)sh.Kh; a.s = (uint32_t)sh.s; a.Ho = (uint32_t)sh.Ho;
    a.L = (uint32_t)sh.L;
    a.strips = (uint32_t)sh.strips;
    a.win_elems = (uint64_t)sh.win_elems;
    a.win_bytes = (uint64_t)sh.win_bytes;
    a.pad_end = (uint64_t)sh.pad_end;
    a.div_Ci = make_fastdiv((uint32_t)sh.Ci);
    a.div_Kh = make_fastdiv((uint32_t)sh.Kh);
    a.div_Wi = make_fastdiv((uint32_t)sh.Wi);
    a.div_Ho = make_fastdiv((uint32_t)sh.Ho);
    a.div_L = make_fastdiv((uint32_t)sh.L);
    a.d = (uint32_t)sh.d;
    a.Wq = (uint32_t)sh.Wq;
    a.cols = (uint32_t)sh.cols;
    a.div_Wq = make_fastdiv((uint32_t)sh.Wq);
    // IM2WIN_TRANSFORM_ORDER=linear deals blocks in launch order (to measure
    // what the XCD-aware order gains)
    a.xcd_order = t.transform_linear ? 0u : 1u;
    void *args[] = {&a};
    const bool vec = (sh.Ci * sh.elt) % 16 == 0;
    if (vec) {
        a.gran_per_strip = (uint32_t)(sh.L * sh.elt / 16);
        a.div_gps = make_fastdiv(a.gran_per_strip);
        a.grans = (uint64_t)sh.win_bytes / 16;
        const uint64_t per_block = kThreads * kGranPerThread;
        const uint64_t blocks = (a.grans + per_block - 1) / per_block;
        if (blocks > 0x7fffffffull)
            return hipErrorInvalidValue;
        const void *f = sh.elt == 4 ? (const void *)&transform_vec<4> : (const void *)&transform_vec<2>;
        return hipLaunchKernel(f, dim3((uint32_t)blocks), dim3(kThreads), args, 0, st);
    }
    a.gran_per_strip = 0;
    a.grans = ((uint64_t)sh.win_bytes + 15) / 16;
    const uint64_t blocks = (a.grans + kThreads - 1) / kThreads;
    if (blocks > 0x7fffffffull)
        return hipErrorInvalidValue;
    // pieces3: 3-channel layers, undilated and unpadded; in fp16 only with
    // filters of up to 3 rows.  Measured against the element gather (GB/s of
    // algorithmic traffic, 128 images): fp32 11x11 stride 4 at 227x227 4512
    // against 4059, 7x7 stride 2 3925 / 3180, 3x3 at 224x224 4277 / 3996;
    // fp16 3x3 2613 / 2376, 7x7 even, 11x11 2135 / 2298 (a granule's pieces
    // then come from up to four input rows).  IM2WIN_TRANSFORM_KERNEL=gather
    // keeps every layer on the element gather.
    const bool unpadded = !pad || (pad->ph == 0 && pad->pw == 0);
    if (sh.Ci == 3 && sh.d == 1 && unpadded && !t.transform_gather && (sh.elt == 4 || sh.Kh <= 3)) {
        a.in_pixels = (uint64_t)sh.N * a.Hi * a.Wi;
        const void *f = sh.elt == 4 ? (const void *)&transform_pieces3<4> : (const void *)&transform_pieces3<2>;
        return hipLaunchKernel(f, dim3((uint32_t)blocks), dim3(kThreads), args, 0, st);
    }
    // gather: element indices fit 32 bits (transform_range_ok)
    const void *f = sh.elt == 4 ? (const void *)&transform_gather<4> : (const void *)&transform_gather<2>;
    return hipLaunchKernel(f, dim3((uint32_t)blocks), dim3(kThreads), args, 0, st);
}

}  // namespace im2win
