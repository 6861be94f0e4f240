// fp32 windowed convolution on the vector ALUs for short windows that are
// not 16-byte aligned: the 3-channel stem layers with K = K_h*K_w*C_i of at
// most 32 taps (Sec. III-C, Eq. 3, Table I cv7).
//
// 3x3 over 224x224 with C_i = 3 does 27 multiply-adds per output element and
// writes 256 bytes per pixel (64 fp32 channels) from a 108-byte window: the
// output, not the window tensor, is the traffic that matters.  The kernel:
//   * lane l of a wave owns pixel 64*blk + l and holds its whole window (K
//     values, one 4-byte-aligned span of the window tensor) in registers;
//   * the filter is wave-uniform: tap t's C_o values come through the scalar
//     cache as SGPR operands of the FMAs (packed fp32 filter, F'[t][j] at
//     t*C_o_pad32 + j), 32 channels at a time, so each lane accumulates 32
//     output channels of its pixel with one FMA per (tap, channel), taps in
//     window order;
//   * a wave's 64 pixels x 32 channels go through a private LDS area so that
//     each store instruction writes eight whole 128-byte lines (a plain store
//     from the FMA layout would write 16 bytes into 64 different lines);
//   * waves stride over the 64-pixel blocks, one resident round of
//     workgroups.
// No workgroup-wide synchronisation: each wave owns its LDS area.
#include "common.hpp"

namespace im2win {
namespace {

struct S32Args {
    const float *ws;      // window tensor
    const float *packed;  // F' [K_pad32][C_o_pad32]
    float *out;
    uint32_t P, K, Co, Co_pad, Wo, nblk;
    uint64_t L, S;        // strip length and window step (elements)
    FastDiv div_Wo;
};

constexpr int kS32Waves = 4;
typedef const float __attribute__((address_space(4))) *cfloat_ptr;

// The window of this lane's pixel in block blk, as 16-byte loads from its
// 4-byte-aligned start, issued without branches (raw: values past K belong
// to the next window or to the zero pad after the tensor, at most 60 bytes
// past the last window; a pixel past P reads the tensor's first bytes).
// They are masked where they are used, so that the compiler's memory-counter
// waits do not make these prefetch loads wait for the previous block's
// stores.
template <int KMAX>
__device__ inline void load_window(const S32Args &a, uint32_t blk, uint32_t lane, u32x4 (&x)[(KMAX + 3) / 4])
{
    const uint32_t p = blk * 64 + lane;
    const bool live = p < a.P;
    const uint32_t q = live ? fdiv(p, a.div_Wo) : 0u;
    const uint64_t w0 = live ? (uint64_t)q * a.L + (uint64_t)(p - q * a.Wo) * a.S : 0u;
    const char *win = reinterpret_cast<const char *>(a.ws + w0);
#pragma unroll
    for (int g = 0; g < (KMAX + 3) / 4; ++g)
        __builtin_memcpy(&x[g], win + 16 * g, 16);
}

template <int KMAX>
__global__ __launch_bounds__(64 * kS32Waves) void conv_fp32_stem(S32Args a)
{
    constexpr int KW4 = (KMAX + 3) / 4;
    // per wave: 64 rows (pixels) of 32 floats; 16-byte chunk k of row r at
    // chunk k ^ (r % 8), so the 16 lanes of one LDS cycle hit 64 banks once
    __shared__ __attribute__((aligned(16))) float rows[kS32Waves][64 * 32];
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    float *lds = rows[wave];
    const uint32_t nw = gridDim.x * kS32Waves;
    const cfloat_ptr filt = (cfloat_ptr)a.packed;

    uint32_t blk = blockIdx.x * kS32Waves + wave;
    u32x4 xn[KW4];
    load_window<KMAX>(a, blk, lane, xn);
    for (; blk < a.nblk; blk += nw) {
        // this block's taps: zero past K and for pixels past P
        const bool live = blk * 64 + lane < a.P;
        float x[KW4 * 4];
#pragma unroll
        for (int g = 0; g < KW4; ++g)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                x[4 * g + e] = live && (uint32_t)(4 * g + e) < a.K ? __uint_as_float(xn[g][e]) : 0.f;
        // the next block's window loads run under this block's FMAs and
        // stores (past the last block they are issued too and never used)
        load_window<KMAX>(a, blk + nw, lane, xn);
        // the block's rows are one contiguous run of the output; rows past
        // the last pixel fall outside the resource and are dropped
        const uint32_t live_rows = a.P - blk * 64 < 64 ? a.P - blk * 64 : 64;
        const __amdgpu_buffer_rsrc_t ro = make_rsrc(a.out + (uint64_t)blk * 64 * a.Co, live_rows * a.Co * 4u);
        for (uint32_t c0 = 0; c0 < a.Co; c0 += 32) {
            float acc[32];
#pragma unroll
            for (int j = 0; j < 32; ++j)
                acc[j] = 0.f;
            // all KMAX taps: past K the window value is 0 and the packed
            // filter row is zero (K_pad32 >= KMAX), which adds exactly 0
#pragma unroll
            for (int t = 0; t < KMAX; ++t) {
                const cfloat_ptr w = filt + (uint64_t)t * a.Co_pad + c0;
#pragma unroll
                for (int j = 0; j < 32; ++j)
                    acc[j] = __builtin_fmaf(x[t], w[j], acc[j]);
            }
            // row `lane` of the LDS tile: chunks of 4 channels, swizzled
#pragma unroll
            for (int k = 0; k < 8; ++k)
                *reinterpret_cast<float4 *>(lds + lane * 32 + 4 * (k ^ (lane & 7))) =
                    make_float4(acc[4 * k], acc[4 * k + 1], acc[4 * k + 2], acc[4 * k + 3]);
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's rows are in LDS
            __builtin_amdgcn_wave_barrier();
            // instruction i: rows 8*i + lane/8, chunk lane%8 (channels
            // c0 + 4*(lane%8) ..): eight 128-byte line pieces of the output;
            // chunks past C_o read nothing (their offset is out of range)
            const uint32_t k = lane & 7;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const uint32_t r = 8 * i + (lane >> 3);
                const u32x4 v = *reinterpret_cast<const u32x4 *>(lds + r * 32 + 4 * (k ^ (r & 7)));
                __builtin_amdgcn_raw_buffer_store_b128(v, ro, c0 + 4 * k < a.Co ? (r * a.Co + c0 + 4 * k) * 4u : kOOB,
                                                       0, 0);
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);  // reads done before the next rows land
            __builtin_amdgcn_wave_barrier();
        }
    }
}

}  // namespace

// Windows not 16-byte aligned (C_i % 4 != 0), undilated, K <= 32, C_o a
// multiple of 4 (16-byte output chunks): 0 (up to 16 taps), 1 (27 taps) or
// 2 (up to 32); -1 when the kernel cannot run the layer.
int stem32_plan(const Shape &sh)
{
    if (sh.Ci % 4 == 0 || sh.d != 1 || sh.K > 32 || sh.Co % 4 != 0)
        return -1;
    return sh.K <= 16 ? 0 : sh.K == 27 ? 1 : 2;
}

// The planner's choice: windows of up to 27 taps.  Measured against the
// DMA-staged kernel (fp32, 128 images, TFLOP/s): 3x3 C_i = 3 over 224x224
// with C_o = 32 / 64 / 128: 43.3 / 49.0 / 53.4 against 24.8 / 38.0 / 39.4;
// stride 2: 36.1 against 33.0; 2x2 C_i = 3: 25.9 against 19.0; at 30 taps
// (2x3 over 5 channels) even.  The FMAs take the filter as an SGPR operand,
// which the two VALU pipes do not issue together, so the kernel tops out near
// half the vector peak; its gain is in loads and stores.
int stem32_default(const Shape &sh)
{
    return sh.K <= 27 ? stem32_plan(sh) : -1;
}

const char *stem32_name(int v) { return v == 0 ? "k16" : v == 1 ? "k27" : "k32"; }

hipError_t launch_conv_fp32_stem(const Shape &sh, int v, const void *ws, const void *packed, float *out,
                                 hipStream_t st)
{
    S32Args a;
    a.ws = static_cast<const float *>(ws);
    a.packed = static_cast<const float *>(packed);
    a.out = out;
    a.P = (uint32_t)sh.P; a.K = (uint32_t)sh.K; a.Co = (uint32_t)sh.Co; a.Co_pad = (uint32_t)sh.Co_pad32;
    a.Wo = (uint32_t)sh.Wo;
    a.nblk = (uint32_t)((sh.P + 63) / 64);
    a.L = (uint64_t)sh.L; a.S = (uint64_t)sh.S;
    a.div_Wo = make_fastdiv((uint32_t)sh.Wo);
    // taps per window as a compile-time count: 16 (K <= 16), 27 (3x3 over 3
    // channels) or 32 (K <= 32; the packed filter's zero rows pad K)
    const void *f = v == 0   ? (const void *)&conv_fp32_stem<16>
                    : v == 1 ? (const void *)&conv_fp32_stem<27>
                             : (const void *)&conv_fp32_stem<32>;
    // one round of resident workgroups (as many per CU as registers and LDS
    // allow); fewer when the layer has fewer blocks
    int dev = 0, cus = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, f, 64 * kS32Waves, 0);
    if (e != hipSuccess)
        return e;
    int64_t wgs = (int64_t)(cus > 0 ? cus : 1) * (per_cu > 0 ? per_cu : 1);
    const int64_t need = (a.nblk + kS32Waves - 1) / kS32Waves;
    if (wgs > need)
        wgs = need;
    void *args[] = {&a};
    return hipLaunchKernel(f, dim3((uint32_t)wgs), dim3(64 * kS32Waves), args, 0, st);
}

}  // namespace im2win
