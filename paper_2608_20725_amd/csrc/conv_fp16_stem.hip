// fp16 windowed convolution on the matrix cores for short windows that are
// not 16-byte aligned: the 3-channel stem layers with K = K_h*K_w*C_i of at
// most 160 taps (Sec. III-B..D, Eq. 3, Table I cv3 and cv7).
//
// With C_i = 3 a window is K_w input columns of K_h*3 taps, and consecutive
// windows of a strip are S = s*K_h*3 elements apart, so they start on 2-byte
// boundaries only.  Such a layer has few taps per output and many outputs
// (3x3 over 224x224: 27 taps, 64 channels): it moves far more output bytes
// than window bytes and filter bytes together, and its speed is set by how
// the outputs are written, not by the matrix cores.  The kernel is shaped by
// that:
//   * the whole filter is an MFMA operand held in registers: each wave loads
//     its C_o x K slice once (the packed filter, 64-tap tiles of C_o_pad
//     rows; taps past K are zero there) and keeps it for all its pixels;
//   * a wave computes 32 consecutive pixels x all C_o channels at a time
//     (v_mfma_f32_32x32x16, fp32 accumulation); lane l reads the 8 taps
//     16*ks + 8*(l/32) .. of pixel l%32's window with one 16-byte load from
//     its 2-byte-aligned start in the window tensor; taps past K are cleared
//     in registers (they belong to the next window, or to the zero pad after
//     the tensor), so a non-finite neighbour cannot leak in;
//   * the 32 pixels' output rows are contiguous in the NHWC output, so the
//     wave turns its sums (rounded to 16 bits once, nearest-even) into rows
//     in a private LDS area and copies the 32*C_o*2 bytes out with 16-byte
//     stores, 1 KiB per store instruction (with the nontemporal policy when
//     the whole output is large; see kStreamOutBytes);
//   * waves stride over the 32-pixel blocks of the layer; the window loads of
//     the next block are issued before the current block's multiplies and
//     stores.
// No workgroup-wide synchronisation: each wave owns its LDS area.
#include "common.hpp"
#include "mfma16.hpp"

#include <string.h>

namespace im2win {
namespace {

struct StemArgs {
    const uint16_t *ws;      // window tensor (16-bit elements), zero pad after it
    const uint16_t *packed;  // F' in 64-tap tiles: [K_pad/64][Co_pad][64]
    uint16_t *out;
    uint32_t P, K, Co, Co_pad, Wo, nblk;
    uint32_t streamed;       // 1: output stores streamed (nontemporal)
    uint64_t L, S;           // strip length and window step (elements)
    FastDiv div_Wo;
};

constexpr int kStemWaves = 4;

template <class E, int WM, int KS>
struct Stem {
    typedef typename E::v8 v8;

    // Window taps of k-step ks for this lane's pixel of block blk.
    __device__ static inline void load(const StemArgs &a, uint32_t blk, uint32_t lane, v8 (&b)[KS])
    {
        const uint32_t p = blk * 32 + (lane & 31);
        const bool live = p < a.P;
        const uint32_t q = live ? fdiv(p, a.div_Wo) : 0u;
        const uint64_t w0 = (uint64_t)q * a.L + (uint64_t)(p - q * a.Wo) * a.S;
        const char *src = reinterpret_cast<const char *>(a.ws + w0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const uint32_t k = 16 * ks + 8 * (lane >> 5);
            uint32_t v[4] = {0u, 0u, 0u, 0u};
            if (live && k < a.K) {
                // unaligned 16-byte load; at most 7 elements past the last
                // window, inside the zero pad that follows the tensor
                __builtin_memcpy(v, src + 2 * k, 16);
                const uint32_t nv = a.K - k;  // taps of these 8 inside the window
                if (nv < 8) {
#pragma unroll
                    for (int d = 0; d < 4; ++d)
                        v[d] &= ((uint32_t)(2 * d) < nv ? 0xffffu : 0u) |
                                ((uint32_t)(2 * d + 1) < nv ? 0xffff0000u : 0u);
                }
            }
            __builtin_memcpy(&b[ks], v, 16);
        }
    }
};

template <class E, int WM, int KS>
struct StemBlock {
    typedef typename E::v8 v8;
    // LDS rows of the output: NCHP 16-byte chunks (a power of two >= the
    // C_o/8 chunks of an output row), chunk c of row n at chunk c ^ (n % NCHP)
    static constexpr int NCHP = WM == 1 ? 4 : WM == 2 ? 8 : 16;
    static constexpr int PITCH = 16 * NCHP;
    static constexpr int RP = 64 / NCHP;  // rows one copy instruction covers

    // Multiplies block blk (its windows in b) and stores its 32 output rows.
    __device__ static inline void run(const StemArgs &a, const v8 (&af)[WM][KS], const v8 (&b)[KS], uint32_t blk,
                                      uint32_t lane, char *lds)
    {
        f32x16_acc acc[WM];
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                acc[i][e] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int i = 0; i < WM; ++i)
                acc[i] = E::mfma(af[i][ks], b[ks], acc[i]);
        // lane holds pixel n = lane%32, channels 32*i + 8*g + 4*(lane/32) + 0..3
        const uint32_t n = lane & 31;
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const uint32_t c0 = 32 * i + 8 * g + 4 * (lane >> 5);
                if (c0 < a.Co) {
                    uint32_t h[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        h[e] = E::bits(acc[i][4 * g + e]);
                    const uint32_t pc = (c0 / 8) ^ (n % NCHP);
                    *reinterpret_cast<uint2 *>(lds + n * PITCH + 16 * pc + 2 * (c0 % 8)) =
                        make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
                }
            }
        // the wave's own LDS writes, read back below by other lanes
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
        __builtin_amdgcn_wave_barrier();
        const uint32_t live = a.P - blk * 32 < 32 ? a.P - blk * 32 : 32;
        const uint32_t nch = a.Co / 8;  // 16-byte chunks per output row
        const uint32_t c = lane % NCHP, r0 = lane / NCHP;
        char *dst = reinterpret_cast<char *>(a.out + (uint64_t)blk * 32 * a.Co);
        const __amdgpu_buffer_rsrc_t ro = make_rsrc(dst, live * a.Co * 2u);
#pragma unroll
        for (int k = 0; k < 32 / RP; ++k) {
            const uint32_t r = r0 + RP * k;
            if (r < live && c < nch) {
                const u32x4 v = *reinterpret_cast<const u32x4 *>(lds + r * PITCH + 16 * (c ^ (r % NCHP)));
                if (a.streamed)
                    store16_nt(v, ro, r * 2 * a.Co + 16 * c);
                else
                    *reinterpret_cast<u32x4 *>(dst + r * 2 * a.Co + 16 * c) = v;
            }
        }
        // every lane has read its chunks before the next block's rows land
        __builtin_amdgcn_s_waitcnt(0xC07F);
        __builtin_amdgcn_wave_barrier();
    }
};

template <class E, int WM, int KS>
__global__ __launch_bounds__(64 * kStemWaves) void conv_fp16_stem(StemArgs a)
{
    using T = Stem<E, WM, KS>;
    using B = StemBlock<E, WM, KS>;
    typedef typename E::v8 v8;
    __shared__ __attribute__((aligned(16))) char rows[kStemWaves][32 * B::PITCH];

    const uint32_t lane = threadIdx.x & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    char *lds = rows[wave];

    // the filter operand: channel 32*i + lane%32, taps 16*ks + 8*(lane/32) ..
    v8 af[WM][KS];
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const uint32_t j = 32 * i + (lane & 31), k = 16 * ks + 8 * (lane >> 5);
            af[i][ks] = *reinterpret_cast<const v8 *>(a.packed + ((uint64_t)(k / 64) * a.Co_pad + j) * 64 + k % 64);
        }

    // blocks blk, blk + nw, blk + 2*nw, ... of this wave; the windows of the
    // two blocks after the current one are in flight while it is multiplied
    // and stored (three register buffers, rotated by unrolling)
    const uint32_t nw = gridDim.x * kStemWaves;
    uint32_t blk = blockIdx.x * kStemWaves + wave;
    v8 b0[KS], b1[KS], b2[KS];
    if (blk < a.nblk)
        T::load(a, blk, lane, b0);
    if (blk + nw < a.nblk)
        T::load(a, blk + nw, lane, b1);
    while (blk < a.nblk) {
        if (blk + 2 * nw < a.nblk)
            T::load(a, blk + 2 * nw, lane, b2);
        B::run(a, af, b0, blk, lane, lds);
        blk += nw;
        if (blk >= a.nblk)
            break;
        if (blk + 2 * nw < a.nblk)
            T::load(a, blk + 2 * nw, lane, b0);
        B::run(a, af, b1, blk, lane, lds);
        blk += nw;
        if (blk >= a.nblk)
            break;
        if (blk + 2 * nw < a.nblk)
            T::load(a, blk + 2 * nw, lane, b1);
        B::run(a, af, b2, blk, lane, lds);
        blk += nw;
    }
}

struct StemVariant {
    const void *f[2];  // fp16 and bf16 operands
    int wm, ks;
};

template <int WM, int KS>
StemVariant stem_variant()
{
    return StemVariant{{(const void *)&conv_fp16_stem<F16Op, WM, KS>, (const void *)&conv_fp16_stem<BF16Op, WM, KS>},
                       WM, KS};
}

// Channel blocks of 32 (1..4) x k-steps of 16 taps (2, 4, 6, 8, 10).
const StemVariant *stem_variants(int *n)
{
    static const StemVariant v[] = {
        stem_variant<1, 2>(), stem_variant<1, 4>(), stem_variant<1, 6>(), stem_variant<1, 8>(), stem_variant<1, 10>(),
        stem_variant<2, 2>(), stem_variant<2, 4>(), stem_variant<2, 6>(), stem_variant<2, 8>(), stem_variant<2, 10>(),
        stem_variant<3, 2>(), stem_variant<3, 4>(), stem_variant<3, 6>(), stem_variant<3, 8>(), stem_variant<3, 10>(),
        stem_variant<4, 2>(), stem_variant<4, 4>(), stem_variant<4, 6>(), stem_variant<4, 8>(), stem_variant<4, 10>(),
    };
    *n = (int)(sizeof v / sizeof v[0]);
    return v;
}

}  // namespace

// The variant for the layer, or -1 when it cannot run it: windows not
// 16-byte aligned, undilated, K <= 160, C_o <= 128 and a multiple of 8
// (16-byte output rows).
int stem_plan(const Shape &sh)
{
    if (sh.Ci % 8 == 0 || sh.d != 1 || sh.K > 160 || sh.Co > 128 || sh.Co % 8 != 0 || sh.P >= ((int64_t)1 << 32) - 32)
        return -1;
    const int wm = (int)((sh.Co + 31) / 32);
    int ks = (int)((sh.K + 15) / 16);
    ks = (ks + 1) / 2 * 2;
    return (wm - 1) * 5 + ks / 2 - 1;
}

// The planner's choice: windows of up to 64 taps.  Measured against the
// segment-staged kernel (fp16, 128 images, TFLOP/s): 3x3 C_i = 3 over
// 224x224 with C_o = 32 / 64 / 128: 74 / 104 / 117 against 47 / 82 / 80;
// 4x4 C_i = 3: 193 against 144; 3x3 C_i = 5: 165 against 128; 7x3 and 5x5
// C_i = 3 (63, 75 taps): even; the 7x7 stride-2 stem (147 taps): 206
// against 287, since holding ten k-steps of filter and windows in registers
// leaves one wave per SIMD.
int stem_default(const Shape &sh)
{
    return sh.K <= 64 ? stem_plan(sh) : -1;
}

const char *stem_name(int v)
{
    static const char *names[] = {"m1k2", "m1k4", "m1k6", "m1k8", "m1k10", "m2k2", "m2k4", "m2k6", "m2k8", "m2k10",
                                  "m3k2", "m3k4", "m3k6", "m3k8", "m3k10", "m4k2", "m4k4", "m4k6", "m4k8", "m4k10"};
    return v >= 0 && v < 20 ? names[v] : "?";
}

hipError_t launch_conv_fp16_stem(const Shape &sh, int plan, const void *ws, const void *packed, uint16_t *out,
                                 hipStream_t st, Op16 op)
{
    int n;
    const StemVariant &v = stem_variants(&n)[plan];
    StemArgs a;
    a.ws = static_cast<const uint16_t *>(ws);
    a.packed = static_cast<const uint16_t *>(packed);
    a.out = out;
    a.P = (uint32_t)sh.P; a.K = (uint32_t)sh.K; a.Co = (uint32_t)sh.Co; a.Co_pad = (uint32_t)sh.Co_pad;
    a.Wo = (uint32_t)sh.Wo;
    a.nblk = (uint32_t)((sh.P + 31) / 32);
    a.streamed = stream_out(sh.P * sh.Co * 2) ? 1u : 0u;
    a.L = (uint64_t)sh.L; a.S = (uint64_t)sh.S;
    a.div_Wo = make_fastdiv((uint32_t)sh.Wo);
    // One round of resident workgroups (as many per CU as registers and LDS
    // allow), each wave striding over the blocks: on 3x3 C_i = 3 over
    // 224x224 this ran at 105 TFLOP/s against 87-93 with two to five times
    // as many workgroups queued behind the first round, and 68 with one
    // workgroup per CU.  Fewer when the layer has fewer blocks.
    const void *f = v.f[op == Op16::BF16];
    int dev = 0, cus = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, f, 64 * kStemWaves, 0);
    if (e != hipSuccess)
        return e;
    int64_t wgs = (int64_t)(cus > 0 ? cus : 1) * (per_cu > 0 ? per_cu : 1);
    const int64_t need = (a.nblk + kStemWaves - 1) / kStemWaves;
    if (wgs > need)
        wgs = need;
    void *args[] = {&a};
    return hipLaunchKernel(f, dim3((uint32_t)wgs), dim3(64 * kStemWaves), args, 0, st);
}

}  // namespace im2win
