// fp16 windowed convolution on the gfx950 matrix cores (Sec. III-D, Alg. 1).
//
// The output is the product D[j][p] = sum_k F'[j][k] * Wn[p][k] with
// M = C_o (filter rows), N = N*H_o*W_o (output pixels) and K = K_h*K_w*C_i:
//   * F' is the filter repacked into window order (pack_filter_fp16 below):
//     F'[j][(v*K_h + u)*C_i + r] = F[u][v][r][j], zero-padded to
//     [C_o_pad][K_pad];
//   * Wn[p][.] is the window of pixel p: a contiguous span of its strip in the
//     window tensor (Eq. 3), so a tile of windows is loaded row by row with
//     16-byte loads, exactly like a matrix with one row pointer per pixel.
//
// Workgroup: WGM x WGN waves; a wave computes a (32*WM) x (32*WN) block of D
// with v_mfma_f32_32x32x16_f16 (fp16 operands, fp32 accumulators).  K is
// walked 64 at a time; each stage of filter rows and window rows goes
// global -> registers -> LDS, double-buffered so that the loads of stage t+1
// overlap the matrix operations of stage t (Alg. 1's double buffering; the
// paper's asynchronous copy maps to loads that are issued before the MFMAs
// and only waited for after them).  The epilogue rounds each fp32 sum to fp16
// once (nearest-even) and stores NHWC.
#include "common.hpp"

namespace im2win {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BK = 64;       // taps per stage
constexpr int LDK = BK + 8;  // halves per LDS row: 144 bytes, offsets rows across banks

struct C16Args {
    const uint16_t *ws;      // window tensor (fp16 bits)
    const uint16_t *packed;  // F' [Co_pad][K_pad]
    uint16_t *out;
    uint64_t win_bytes;
    uint32_t P, K, K_pad, Co, Wo, L, S;
    FastDiv div_Wo;
};

// ---------------------------------------------------------------------------
// Filter repack (window order, zero-padded).  One thread per 16-byte granule
// of F'.
struct PackArgs {
    const uint16_t *filt;
    uint16_t *packed;
    uint64_t grans;
    uint32_t K, K_pad, Co, Ci, Kh, Kw;
};

__global__ __launch_bounds__(256) void pack_filter_fp16(PackArgs a)
{
    const uint32_t gpr = a.K_pad / 8;  // granules per packed row
    for (uint64_t g = (uint64_t)blockIdx.x * 256 + threadIdx.x; g < a.grans;
         g += (uint64_t)gridDim.x * 256) {
        const uint32_t j = (uint32_t)(g / gpr);
        const uint32_t k0 = (uint32_t)(g % gpr) * 8;
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
            uint32_t lo = 0, hi = 0;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const uint32_t k = k0 + e + h;
                uint32_t bits = 0;
                if (j < a.Co && k < a.K) {
                    const uint32_t khci = a.Kh * a.Ci;
                    const uint32_t v = k / khci, rem = k % khci;
                    const uint32_t u = rem / a.Ci, r = rem % a.Ci;
                    const uint64_t frow = ((uint64_t)u * a.Kw + v) * a.Ci + r;
                    bits = a.filt[frow * a.Co + j];
                }
                if (h == 0)
                    lo = bits;
                else
                    hi = bits;
            }
            w[e / 2] = lo | (hi << 16);
        }
        *reinterpret_cast<uint4 *>(a.packed + g * 8) = make_uint4(w[0], w[1], w[2], w[3]);
    }
}

// ---------------------------------------------------------------------------
template <int WM, int WN, int WGM, int WGN, bool ALIGNED>
struct Cfg {
    static constexpr int NT = 64 * WGM * WGN;
    static constexpr int BMc = 32 * WM * WGM;  // channels per workgroup
    static constexpr int BNp = 32 * WN * WGN;  // pixels per workgroup
    static constexpr int FG = BMc * (BK / 8);  // filter granules per stage
    static constexpr int WG = BNp * (BK / 8);  // window granules per stage
    static constexpr int FPT = FG / NT;
    static constexpr int WPT = WG / NT;
    static_assert(FG % NT == 0 && WG % NT == 0, "stage granules must split evenly over threads");
};

// One K stage in flight: global -> registers (load), registers -> LDS (store).
template <int WM, int WN, int WGM, int WGN, bool ALIGNED>
struct Stage16 {
    using C = Cfg<WM, WN, WGM, WGN, ALIGNED>;
    u32x4 fr[C::FPT], wr[C::WPT];

    __device__ inline void load(__amdgpu_buffer_rsrc_t rs, const uint32_t *rowoff, const uint16_t *fb,
                                uint32_t p0, uint32_t k0, const C16Args &a)
    {
        const uint32_t tid = threadIdx.x;
        // filter rows: always inside the zero-padded packed filter
#pragma unroll
        for (int j = 0; j < C::FPT; ++j) {
            const uint32_t g = tid + j * C::NT;
            const uint32_t row = g >> 3, c8 = g & 7;
            fr[j] = *reinterpret_cast<const u32x4 *>(fb + (uint64_t)row * a.K_pad + k0 + 8 * c8);
        }
        // window rows: masked-off loads (pixel past P, tap past K) use an
        // out-of-range offset and read zero
#pragma unroll
        for (int j = 0; j < C::WPT; ++j) {
            const uint32_t g = tid + j * C::NT;
            const uint32_t row = g >> 3, c8 = g & 7;
            const uint32_t k = k0 + 8 * c8;
            const bool ok = p0 + row < a.P;
            const uint32_t base = (rowoff[row] + k) * 2u;
            if (ALIGNED) {
                wr[j] = ld_b128(rs, (ok && k < a.K) ? base : kOOB);
            } else {
                uint32_t h[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    h[e] = ld_b16(rs, (ok && k + e < a.K) ? base + 2u * e : kOOB);
                wr[j] = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                              h[6] | (h[7] << 16)};
            }
        }
    }

    __device__ inline void store(_Float16 (*Fs)[LDK], _Float16 (*Ws)[LDK])
    {
        const uint32_t tid = threadIdx.x;
#pragma unroll
        for (int j = 0; j < C::FPT; ++j) {
            const uint32_t g = tid + j * C::NT;
            *reinterpret_cast<u32x4 *>(&Fs[g >> 3][8 * (g & 7)]) = fr[j];
        }
#pragma unroll
        for (int j = 0; j < C::WPT; ++j) {
            const uint32_t g = tid + j * C::NT;
            *reinterpret_cast<u32x4 *>(&Ws[g >> 3][8 * (g & 7)]) = wr[j];
        }
    }
};

template <int WM, int WN, int WGM, int WGN, bool ALIGNED>
__global__ __launch_bounds__(64 * WGM * WGN) void conv_fp16_kernel(C16Args a)
{
    using C = Cfg<WM, WN, WGM, WGN, ALIGNED>;
    __shared__ __attribute__((aligned(16))) _Float16 Fs[2][C::BMc][LDK];
    __shared__ __attribute__((aligned(16))) _Float16 Ws[2][C::BNp][LDK];
    __shared__ uint32_t rowoff[C::BNp];

    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63;
    const uint32_t wave = tid >> 6;
    const uint32_t wm = wave / WGN, wn = wave % WGN;
    const uint32_t p0 = blockIdx.x * C::BNp;
    const uint32_t ch0 = blockIdx.y * C::BMc;

    const uint32_t q0 = fdiv(p0, a.div_Wo);
    const uint64_t tb_elem = (uint64_t)q0 * a.L;
    const uint64_t left = a.win_bytes - tb_elem * 2;
    const __amdgpu_buffer_rsrc_t rs =
        make_rsrc(a.ws + tb_elem, (uint32_t)(left < kMaxRecords ? left : kMaxRecords));
    for (uint32_t t = tid; t < C::BNp; t += C::NT) {
        const uint32_t p = p0 + t;
        uint32_t off = 0;
        if (p < a.P) {
            const uint32_t q = fdiv(p, a.div_Wo);
            off = (q - q0) * a.L + (p - q * a.Wo) * a.S;
        }
        rowoff[t] = off;
    }
    __syncthreads();

    const uint16_t *fb = a.packed + (uint64_t)ch0 * a.K_pad;
    Stage16<WM, WN, WGM, WGN, ALIGNED> stg;

    floatx16 acc[WM][WN];
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                acc[i][j][e] = 0.f;

    const uint32_t nst = a.K_pad / BK;
    stg.load(rs, rowoff, fb, p0, 0, a);
    stg.store(Fs[0], Ws[0]);
    __syncthreads();

    const uint32_t arow = wm * 32 * WM + (lane & 31);
    const uint32_t brow = wn * 32 * WN + (lane & 31);
    const uint32_t kl = 8 * (lane >> 5);
    for (uint32_t st = 0; st < nst; ++st) {
        const int buf = st & 1;
        if (st + 1 < nst)
            stg.load(rs, rowoff, fb, p0, (st + 1) * BK, a);
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            half8 af[WM], bf[WN];
#pragma unroll
            for (int i = 0; i < WM; ++i)
                af[i] = *reinterpret_cast<const half8 *>(&Fs[buf][arow + 32 * i][16 * ks + kl]);
#pragma unroll
            for (int j = 0; j < WN; ++j)
                bf[j] = *reinterpret_cast<const half8 *>(&Ws[buf][brow + 32 * j][16 * ks + kl]);
#pragma unroll
            for (int i = 0; i < WM; ++i)
#pragma unroll
                for (int j = 0; j < WN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[i], bf[j], acc[i][j], 0, 0, 0);
        }
        if (st + 1 < nst)
            stg.store(Fs[buf ^ 1], Ws[buf ^ 1]);
        __syncthreads();
    }

    // D[ch][px]: lane holds px = lane & 31 of its block and, for accumulator
    // element e, channel 8*(e/4) + 4*(lane/32) + e%4.
#pragma unroll
    for (int j = 0; j < WN; ++j) {
        const uint32_t p = p0 + wn * 32 * WN + 32 * j + (lane & 31);
        if (p >= a.P)
            continue;
        uint16_t *o = a.out + (uint64_t)p * a.Co;
#pragma unroll
        for (int i = 0; i < WM; ++i) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const uint32_t c = ch0 + wm * 32 * WM + 32 * i + 8 * g + 4 * (lane >> 5);
                _Float16 h[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    h[e] = (_Float16)acc[i][j][4 * g + e];
                if (c + 3 < a.Co && (a.Co & 3) == 0) {
                    uint2 v;
                    v.x = (uint32_t)__builtin_bit_cast(uint16_t, h[0]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, h[1]) << 16);
                    v.y = (uint32_t)__builtin_bit_cast(uint16_t, h[2]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, h[3]) << 16);
                    *reinterpret_cast<uint2 *>(o + c) = v;
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (c + e < a.Co)
                            o[c + e] = __builtin_bit_cast(uint16_t, h[e]);
                }
            }
        }
    }
}

template <int WM, int WN, int WGM, int WGN>
void pick(bool aligned, const void **f, int *nt, int *bm, int *bn)
{
    *f = aligned ? (const void *)&conv_fp16_kernel<WM, WN, WGM, WGN, true>
                 : (const void *)&conv_fp16_kernel<WM, WN, WGM, WGN, false>;
    *nt = 64 * WGM * WGN;
    *bm = 32 * WM * WGM;
    *bn = 32 * WN * WGN;
}

}  // namespace

hipError_t launch_pack_fp16(const Shape &sh, const uint16_t *filt, void *packed, hipStream_t st)
{
    PackArgs a;
    a.filt = filt;
    a.packed = static_cast<uint16_t *>(packed);
    a.grans = (uint64_t)sh.Co_pad * sh.K_pad / 8;
    a.K = (uint32_t)sh.K; a.K_pad = (uint32_t)sh.K_pad; a.Co = (uint32_t)sh.Co;
    a.Ci = (uint32_t)sh.Ci; a.Kh = (uint32_t)sh.Kh; a.Kw = (uint32_t)sh.Kw;
    uint64_t blocks = (a.grans + 255) / 256;
    if (blocks > 65536)
        blocks = 65536;
    void *args[] = {&a};
    return hipLaunchKernel((const void *)&pack_filter_fp16, dim3((uint32_t)blocks), dim3(256), args, 0, st);
}

hipError_t launch_conv_fp16(const Shape &sh, const void *ws, const void *packed, uint16_t *out,
                            hipStream_t st)
{
    C16Args a;
    a.ws = static_cast<const uint16_t *>(ws);
    a.packed = static_cast<const uint16_t *>(packed);
    a.out = out;
    a.win_bytes = (uint64_t)sh.win_bytes;
    a.P = (uint32_t)sh.P; a.K = (uint32_t)sh.K; a.K_pad = (uint32_t)sh.K_pad;
    a.Co = (uint32_t)sh.Co; a.Wo = (uint32_t)sh.Wo; a.L = (uint32_t)sh.L; a.S = (uint32_t)sh.S;
    a.div_Wo = make_fastdiv((uint32_t)sh.Wo);
    const bool aligned = (sh.Ci % 8) == 0;  // every window starts on a 16-byte boundary
    const void *f;
    int nt, bm, bn;
    if (sh.Co <= 32)
        pick<1, 2, 1, 4>(aligned, &f, &nt, &bm, &bn);
    else if (sh.Co <= 64)
        pick<2, 2, 1, 4>(aligned, &f, &nt, &bm, &bn);
    else
        pick<2, 2, 2, 2>(aligned, &f, &nt, &bm, &bn);
    dim3 grid((uint32_t)((sh.P + bn - 1) / bn), (uint32_t)((sh.Co + bm - 1) / bm));
    void *args[] = {&a};
    return hipLaunchKernel(f, grid, dim3(nt), args, 0, st);
}

}  // namespace im2win
