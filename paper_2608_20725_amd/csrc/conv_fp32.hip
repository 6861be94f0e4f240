// fp32 windowed convolution on the gfx950 vector ALUs (Sec. III-C, Eq. 3).
//
//   O[p][j] = sum_{k<K} Wn[p][k] * F'[k][j]
//
// Wn[p][.] is the window of output pixel p = (i, m, n): the contiguous span of
// strip (i, m) starting at n*s*K_h*C_i, in (filter column v, filter row u,
// channel r) order.  F' is the filter repacked into the same tap order,
// F'[(v*K_h + u)*C_i + r][j] = F[u][v][r][j] (the filter laid out height
// before width, Sec. III-C), zero-padded to [K_pad32][C_o_pad32]: a tap's
// filter row is one row of F' and consecutive taps are consecutive rows.
//
// Work split (wave64):
//   * a workgroup owns 64*TM consecutive output pixels and WAVES*TN output
//     channels; each wave owns TN channels and each lane TM consecutive
//     pixels, so a lane keeps a TM x TN block of fp32 accumulators;
//   * windows are staged through LDS KC taps at a time, transposed to
//     [tap][pixel] so that a lane fetches its TM pixels with 16-byte LDS
//     reads; stages are double-buffered: the global loads of stage t+1 are in
//     flight while stage t is multiplied;
//   * filter values are the same for every lane of a wave: the stage's slab
//     of the packed filter (KC rows, the workgroup's channels) is staged into
//     LDS with the windows, and each wave reads its TN values of a tap with
//     broadcast LDS reads; per tap a lane does TM*TN FMAs for TM/4 + TN/4
//     16-byte LDS reads.  (A variant reads the filter rows with scalar loads
//     into SGPRs instead; it loses on this part because the scalar cache
//     misses most rows, and remains only for filters too large for the LDS
//     variant's 31-bit offsets.)
// The row offset of every pixel's window is computed once per workgroup (the
// index precomputation of Sec. III-E).  Taps past K read zero window values
// (masked loads) against zero filter rows (padding): they add exactly 0.
#include "common.hpp"

#include <stdlib.h>
#include <string.h>

namespace im2win {
namespace {

struct C32Args {
    const float *ws;
    const float *packed;  // F' [K_pad32][Co_pad32]
    float *out;
    uint64_t win_bytes;
    uint32_t P, K, K_pad, Co, Co_pad, Wo, L;
    WinCols wc;              // window start of an output column in its strip
    FastDiv div_Wo;
    TapOrder to;             // order of the tap blocks (the DMA-staged kernel's)
};

// ---------------------------------------------------------------------------
// Filter repack: one thread per 4 consecutive channels of one tap row of F'
// (32-bit indices, the host checks the count; divisions by multiplication).
struct Pack32Args {
    const float *filt;
    float *packed;
    uint32_t quads;
    uint32_t K, Co, Co_pad, Ci, Kh, Kw;
    uint32_t pair_swap;  // store channels 2i and 2i+1 swapped (the DMA-staged kernel's order)
    FastDiv div_qpr, div_khci, div_ci;  // C_o_pad/4, K_h*C_i, C_i
};

__global__ __launch_bounds__(256) void pack_filter_fp32(Pack32Args a)
{
    const uint32_t qpr = a.Co_pad / 4;  // quads per packed row
    for (uint32_t g = blockIdx.x * 256 + threadIdx.x; g < a.quads; g += gridDim.x * 256) {
        const uint32_t k = fdiv(g, a.div_qpr);
        const uint32_t j0 = (g - k * qpr) * 4;
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        if (k < a.K) {
            const uint32_t vv = fdiv(k, a.div_khci), rem = k - vv * a.Kh * a.Ci;
            const uint32_t u = fdiv(rem, a.div_ci), r = rem - u * a.Ci;
            const float *src = a.filt + (((uint64_t)u * a.Kw + vv) * a.Ci + r) * a.Co;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (j0 + e < a.Co)
                    v[e] = src[j0 + e];
        }
        *reinterpret_cast<float4 *>(a.packed + g * 4) =
            a.pair_swap ? make_float4(v[1], v[0], v[3], v[2]) : make_float4(v[0], v[1], v[2], v[3]);
    }
}

// ---------------------------------------------------------------------------
template <int TM, int TN, int KC, int WAVES, bool V4>
struct Geo {
    static constexpr int BM = 64 * TM;      // pixels per workgroup
    static constexpr int LDA = BM + 4;      // floats per staged tap row
    static constexpr int NT = 64 * WAVES;
    // V4: float4 granules of the [BM][KC] stage; else single floats
    static constexpr int ITEMS = V4 ? (BM * KC / 4 + NT - 1) / NT : (BM * KC + NT - 1) / NT;
    static_assert(KC == 8 || KC == 16, "stage depth (the packed filter has 16-tap padding)");
    static_assert(TM % 4 == 0, "pixels per lane in 16-byte LDS reads");
    static_assert(TN % 16 == 0 && TN <= 32, "channels per wave (32-channel padding)");
};

template <int TM, int TN, int KC, int WAVES, bool V4>
struct Stage {
    using G = Geo<TM, TN, KC, WAVES, V4>;
    u32x4 v4[V4 ? G::ITEMS : 1];
    uint32_t v1[V4 ? 1 : G::ITEMS];

    // Masked-off loads (pixel past P, tap past K) use an out-of-range offset
    // and read zero: no branches, and no access leaves the window tensor.
    __device__ inline void load(__amdgpu_buffer_rsrc_t rs, const uint32_t *rowoff, uint32_t p0,
                                uint32_t k0, const C32Args &a)
    {
        const uint32_t tid = threadIdx.x;
        constexpr int Q = KC / 4;  // granules per row
        if (V4) {
#pragma unroll
            for (int j = 0; j < G::ITEMS; ++j) {
                const uint32_t f = tid + j * G::NT;
                const uint32_t row = (f / Q) % G::BM, kq = f % Q;
                const uint32_t k = k0 + 4 * kq;
                const bool ok = f < G::BM * Q && p0 + row < a.P && k < a.K;
                v4[j] = ld_b128(rs, ok ? (rowoff[row] + k) * 4u : kOOB);
            }
        } else {
#pragma unroll
            for (int j = 0; j < G::ITEMS; ++j) {
                const uint32_t f = tid + j * G::NT;
                const uint32_t row = (f / KC) % G::BM, kk = f % KC;
                const uint32_t k = k0 + kk;
                const bool ok = f < G::BM * KC && p0 + row < a.P && k < a.K;
                v1[j] = ld_b32(rs, ok ? (rowoff[row] + k) * 4u : kOOB);
            }
        }
    }

    __device__ inline void store(float (*As)[G::LDA])
    {
        const uint32_t tid = threadIdx.x;
        constexpr int Q = KC / 4;
        if (V4) {
#pragma unroll
            for (int j = 0; j < G::ITEMS; ++j) {
                const uint32_t f = tid + j * G::NT;
                if (f < G::BM * Q) {
                    // element by value: taking the bits of a vector element
                    // through its address is not reliable with this compiler
                    const uint32_t row = f / Q, kq = f % Q;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        As[4 * kq + e][row] = __uint_as_float(v4[j][e]);
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < G::ITEMS; ++j) {
                const uint32_t f = tid + j * G::NT;
                if (f < G::BM * KC)
                    As[f % KC][f / KC] = __uint_as_float(v1[j]);
            }
        }
    }
};

// Filter slab of one stage for the LDS-filter variant: KC packed rows times
// the workgroup's TN*WAVES channels, staged through LDS next to the windows
// with coalesced 16-byte loads issued a stage ahead.  Columns past the
// packed filter read zero.
template <int TN, int KC, int WAVES>
struct FStage {
    static constexpr int NT = 64 * WAVES;
    static constexpr int CW = TN * WAVES;  // channels of the workgroup
    static constexpr int Q = KC * CW / 4;  // 16-byte granules per stage
    static constexpr int ITEMS = (Q + NT - 1) / NT;
    u32x4 v[ITEMS];

    __device__ inline void load(__amdgpu_buffer_rsrc_t rf, uint32_t k0, uint32_t jb, uint32_t co_pad)
    {
#pragma unroll
        for (int j = 0; j < ITEMS; ++j) {
            const uint32_t g = threadIdx.x + j * NT;
            const uint32_t row = (g / (CW / 4)) % KC, c4 = g % (CW / 4);
            const uint32_t col = jb + 4 * c4;
            const bool ok = g < (uint32_t)Q && col < co_pad;
            v[j] = ld_b128(rf, ok ? ((k0 + row) * co_pad + col) * 4u : kOOB);
        }
    }

    __device__ inline void store(float (*Fs)[CW])
    {
#pragma unroll
        for (int j = 0; j < ITEMS; ++j) {
            const uint32_t g = threadIdx.x + j * NT;
            if (g < (uint32_t)Q) {
                const uint32_t row = g / (CW / 4), c4 = g % (CW / 4);
                *reinterpret_cast<float4 *>(&Fs[row][4 * c4]) =
                    make_float4(__uint_as_float(v[j][0]), __uint_as_float(v[j][1]),
                                __uint_as_float(v[j][2]), __uint_as_float(v[j][3]));
            }
        }
    }
};

// The packed filter is read through the constant address space: the kernel
// never writes it, and loads from that space with a uniform address become
// s_load.
typedef const __attribute__((address_space(4))) float cfloat;
typedef float f32x16 __attribute__((ext_vector_type(16), aligned(4)));
typedef const __attribute__((address_space(4))) f32x16 cf32x16;

// TN filter values of one packed row: identical for every lane, so they land
// in SGPRs (one s_load_dwordx16 per 16 channels).
template <int TN>
__device__ inline void load_filter(float (&f)[TN], cfloat *fp)
{
#pragma unroll
    for (int h = 0; h < TN / 16; ++h) {
        const f32x16 v = *(cf32x16 *)(fp + 16 * h);
#pragma unroll
        for (int c = 0; c < 16; ++c)
            f[16 * h + c] = v[c];
    }
}

template <int TM, int TN>
__device__ inline void tap_fma(float (&acc)[TM][TN], const float (&x)[TM], const float (&f)[TN])
{
#pragma unroll
    for (int t = 0; t < TM; ++t)
#pragma unroll
        for (int c = 0; c < TN; ++c)
            acc[t][c] = __builtin_fmaf(x[t], f[c], acc[t][c]);
}

template <int TM, int LDA>
__device__ inline void read_pixels(float (&x)[TM], const float (*As)[LDA], int kk, uint32_t lane)
{
#pragma unroll
    for (int q = 0; q < TM / 4; ++q) {
        const float4 v = *reinterpret_cast<const float4 *>(&As[kk][TM * lane + 4 * q]);
        x[4 * q + 0] = v.x;
        x[4 * q + 1] = v.y;
        x[4 * q + 2] = v.z;
        x[4 * q + 3] = v.w;
    }
}

// Waits for every outstanding LDS and scalar load (lgkmcnt = 0), leaving
// vector-memory loads in flight.
__device__ inline void wait_lgkm() { __builtin_amdgcn_s_waitcnt(0xc07f); }

// Multiplies one LDS stage of KC taps whose first packed filter row is `fp`,
// TP taps per group.  The LDS reads and the filter loads of group g+1 are
// issued before the FMAs of group g and waited for after them: scalar loads
// can return out of order, so the only safe wait is for all of them, and the
// group size sets how much work covers each wait (the filter rows mostly
// come from L2, since every wave streams its own column block of F').  The
// scheduling fence keeps the compiler from hoisting further loads, which
// would exhaust the SGPRs.
template <int TM, int TN, int KC, int TP, int LDA>
__device__ inline void stage_fma(float (&acc)[TM][TN], const float (*As)[LDA], cfloat *fp,
                                 uint32_t row_stride, uint32_t lane)
{
    static_assert(KC % TP == 0, "taps per group");
    float fc[TP][TN], fn[TP][TN], xc[TP][TM], xn[TP][TM];
#pragma unroll
    for (int q = 0; q < TP; ++q) {
        load_filter<TN>(fc[q], fp + q * row_stride);
        read_pixels<TM, LDA>(xc[q], As, q, lane);
    }
    wait_lgkm();
#pragma unroll
    for (int kk = 0; kk < KC; kk += TP) {
        if (kk + TP < KC) {
            fp += TP * row_stride;
#pragma unroll
            for (int q = 0; q < TP; ++q) {
                load_filter<TN>(fn[q], fp + q * row_stride);
                read_pixels<TM, LDA>(xn[q], As, kk + TP + q, lane);
            }
        }
#pragma unroll
        for (int q = 0; q < TP; ++q)
            tap_fma<TM, TN>(acc, xc[q], fc[q]);
        wait_lgkm();
        __builtin_amdgcn_sched_barrier(0);
        if (kk + TP < KC) {
#pragma unroll
            for (int q = 0; q < TP; ++q) {
#pragma unroll
                for (int c = 0; c < TN; ++c)
                    fc[q][c] = fn[q][c];
#pragma unroll
                for (int t = 0; t < TM; ++t)
                    xc[q][t] = xn[q][t];
            }
        }
    }
}

// LDS-filter variant of stage_fma: the wave's TN filter values of a tap are
// one LDS row segment at a wave-uniform address (a broadcast read); LDS
// returns in order, so the compiler's own waits pipeline tap kk+1's reads
// behind tap kk's FMAs.
template <int TM, int TN, int KC, int LDA, int CW>
__device__ inline void stage_fma_lds(float (&acc)[TM][TN], const float (*As)[LDA],
                                     const float (*Fs)[CW], uint32_t wave, uint32_t lane)
{
    float fc[TN], fn[TN], xc[TM], xn[TM];
    auto read_filter = [&](float (&f)[TN], int kk) {
#pragma unroll
        for (int q = 0; q < TN / 4; ++q) {
            const float4 v = *reinterpret_cast<const float4 *>(&Fs[kk][wave * TN + 4 * q]);
            f[4 * q + 0] = v.x;
            f[4 * q + 1] = v.y;
            f[4 * q + 2] = v.z;
            f[4 * q + 3] = v.w;
        }
    };
    read_filter(fc, 0);
    read_pixels<TM, LDA>(xc, As, 0, lane);
#pragma unroll
    for (int kk = 0; kk < KC; ++kk) {
        if (kk + 1 < KC) {
            read_filter(fn, kk + 1);
            read_pixels<TM, LDA>(xn, As, kk + 1, lane);
        }
        tap_fma<TM, TN>(acc, xc, fc);
        if (kk + 1 < KC) {
#pragma unroll
            for (int c = 0; c < TN; ++c)
                fc[c] = fn[c];
#pragma unroll
            for (int t = 0; t < TM; ++t)
                xc[t] = xn[t];
        }
    }
}

// TP = 0 selects the LDS-filter variant; TP >= 1 reads filter rows with
// scalar loads, TP taps per wait.
template <int TM, int TN, int KC, int TP, int WAVES, bool V4>
__global__ __launch_bounds__(64 * WAVES) void conv_fp32_kernel(C32Args a)
{
    using G = Geo<TM, TN, KC, WAVES, V4>;
    constexpr bool FL = TP == 0;
    constexpr int CW = TN * WAVES;
    __shared__ __attribute__((aligned(16))) float As[2][KC][G::LDA];
    __shared__ __attribute__((aligned(16))) float Fs[FL ? 2 : 1][FL ? KC : 1][CW];
    __shared__ uint32_t rowoff[G::BM];

    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t p0 = blockIdx.x * G::BM;
    const uint32_t jw = blockIdx.y * (TN * WAVES) + wave * TN;  // first channel of this wave

    // window offsets of the workgroup's pixels, relative to the strip of p0
    const uint32_t q0 = fdiv(p0, a.div_Wo);
    const uint64_t tb_elem = (uint64_t)q0 * a.L;
    const uint64_t left = a.win_bytes - tb_elem * 4;
    const __amdgpu_buffer_rsrc_t rs =
        make_rsrc(a.ws + tb_elem, (uint32_t)(left < kMaxRecords ? left : kMaxRecords));
    for (uint32_t t = tid; t < G::BM; t += G::NT) {
        const uint32_t p = p0 + t;
        uint32_t off = 0;
        if (p < a.P) {
            const uint32_t q = fdiv(p, a.div_Wo);
            off = (q - q0) * a.L + a.wc.start(p - q * a.Wo);
        }
        rowoff[t] = off;
    }
    __syncthreads();

    float acc[TM][TN];
#pragma unroll
    for (int t = 0; t < TM; ++t)
#pragma unroll
        for (int c = 0; c < TN; ++c)
            acc[t][c] = 0.f;

    const uint32_t nst = a.K_pad / KC;
    const uint32_t jb = blockIdx.y * CW;  // first channel of the workgroup
    const uint64_t fbytes = (uint64_t)a.K_pad * a.Co_pad * 4;
    const __amdgpu_buffer_rsrc_t rf =
        make_rsrc(a.packed, (uint32_t)(fbytes < kMaxRecords ? fbytes : kMaxRecords));
    Stage<TM, TN, KC, WAVES, V4> stg;
    FStage<TN, KC, WAVES> fst;
    stg.load(rs, rowoff, p0, 0, a);
    if (FL)
        fst.load(rf, 0, jb, a.Co_pad);
    stg.store(As[0]);
    if (FL)
        fst.store(Fs[0]);
    __syncthreads();

    // a wave whose channels all lie past C_o (a ragged last channel block)
    // only helps with the loads
    const bool active = jw < a.Co;
    cfloat *fp = (cfloat *)a.packed + jw;
    for (uint32_t st = 0; st < nst; ++st) {
        if (st + 1 < nst) {
            // first tap of stage st+1 (KC divides the tap blocks of the order)
            const uint32_t k1 = a.to.map((st + 1) * KC);
            stg.load(rs, rowoff, p0, k1, a);
            if (FL)
                fst.load(rf, k1, jb, a.Co_pad);
        }
        if (active) {
            if constexpr (FL)
                stage_fma_lds<TM, TN, KC, G::LDA, CW>(acc, As[st & 1], Fs[st & 1], wave, lane);
            else
                stage_fma<TM, TN, KC, TP, G::LDA>(acc, As[st & 1],
                                                  fp + (uint64_t)a.to.map(st * KC) * a.Co_pad, a.Co_pad, lane);
        }
        if (st + 1 < nst) {
            stg.store(As[(st + 1) & 1]);
            if (FL)
                fst.store(Fs[(st + 1) & 1]);
        }
        __syncthreads();
    }

    if (!active)
        return;
#pragma unroll
    for (int t = 0; t < TM; ++t) {
        const uint32_t p = p0 + TM * lane + t;
        if (p >= a.P)
            continue;
        float *o = a.out + (uint64_t)p * a.Co + jw;
        if (jw + TN <= a.Co && (a.Co & 3) == 0) {
#pragma unroll
            for (int c = 0; c < TN; c += 4)
                *reinterpret_cast<float4 *>(o + c) =
                    make_float4(acc[t][c], acc[t][c + 1], acc[t][c + 2], acc[t][c + 3]);
        } else {
#pragma unroll
            for (int c = 0; c < TN; ++c)
                if (jw + c < a.Co)
                    o[c] = acc[t][c];
        }
    }
}

// ---------------------------------------------------------------------------
// Kernel selection.  A tile is (pixels per lane TM, channels per wave TN,
// taps per stage KC, taps per filter-load group TP); the number of waves per
// workgroup is chosen per layer.
struct Tile {
    const char *name;
    int tm, tn, kc, tp;
};

// Measured on MI355X: the LDS-filter tiles beat the scalar-load tiles on
// every layer tried (the scalar cache hits ~25 % of filter rows, so
// scalar-load waits dominate); the scalar-load tile remains for filters too
// large for 31-bit LDS-stage offsets.
const Tile kTiles[] = {
    {"m4n16f", 4, 16, 16, 0},
    {"m8n16f", 8, 16, 8, 0},
    {"m4n16p2", 4, 16, 16, 2},
};
constexpr int kScalarTile = 2;

template <int TM, int TN, int KC, int TP, int W>
const void *kernel_for(bool v4)
{
    return v4 ? (const void *)&conv_fp32_kernel<TM, TN, KC, TP, W, true>
              : (const void *)&conv_fp32_kernel<TM, TN, KC, TP, W, false>;
}

template <int TM, int TN, int KC, int TP>
const void *kernel_for(int waves, bool v4)
{
    switch (waves) {
    case 8: return kernel_for<TM, TN, KC, TP, 8>(v4);
    case 4: return kernel_for<TM, TN, KC, TP, 4>(v4);
    case 2: return kernel_for<TM, TN, KC, TP, 2>(v4);
    default: return kernel_for<TM, TN, KC, TP, 1>(v4);
    }
}

const void *kernel_for(const Tile &t, int waves, bool v4)
{
    if (t.tm == 8)
        return kernel_for<8, 16, 8, 0>(waves, v4);
    return t.tp == 2 ? kernel_for<4, 16, 16, 2>(waves, v4) : kernel_for<4, 16, 16, 0>(waves, v4);
}

}  // namespace

int regs32_find(const char *name)
{
    const int ntiles = (int)(sizeof kTiles / sizeof kTiles[0]);
    for (int t = 0; t < ntiles; ++t)
        if (strcmp(name, kTiles[t].name) == 0)
            return t;
    return -1;
}

const char *regs32_name(int v) { return kTiles[v].name; }

bool regs32_fits(const Shape &sh, int v)
{
    const int ntiles = (int)(sizeof kTiles / sizeof kTiles[0]);
    if (v < 0 || v >= ntiles)
        return false;
    // the LDS-filter tiles address the packed filter with 31-bit offsets
    return kTiles[v].tp != 0 || sh.K_pad32 * sh.Co_pad32 * 4 <= (int64_t)kMaxRecords;
}

hipError_t launch_pack_fp32(const Shape &sh, const Plan32 &p, const float *filt, void *packed, hipStream_t st)
{
    Pack32Args a;
    a.filt = filt;
    a.packed = static_cast<float *>(packed);
    const uint64_t quads = (uint64_t)sh.K_pad32 * sh.Co_pad32 / 4;
    if (quads >= (1ull << 31))
        return hipErrorInvalidValue;
    a.quads = (uint32_t)quads;
    a.K = (uint32_t)sh.K; a.Co = (uint32_t)sh.Co; a.Co_pad = (uint32_t)sh.Co_pad32;
    a.Ci = (uint32_t)sh.Ci; a.Kh = (uint32_t)sh.Kh; a.Kw = (uint32_t)sh.Kw;
    a.div_qpr = make_fastdiv(a.Co_pad / 4);
    a.div_khci = make_fastdiv(a.Kh * a.Ci);
    a.div_ci = make_fastdiv(a.Ci);
    // the DMA- and column-staged kernels read channel pairs swapped
    a.pair_swap = p.fam == Fam32::Dma || p.fam == Fam32::Cols;
    uint64_t blocks = (quads + 255) / 256;
    if (blocks > 65536)
        blocks = 65536;
    void *args[] = {&a};
    return hipLaunchKernel((const void *)&pack_filter_fp32, dim3((uint32_t)blocks), dim3(256), args, 0, st);
}

hipError_t launch_conv_fp32(const Shape &sh, const Plan32 &p, const Tuning &t, const void *ws,
                            const void *packed, float *out, hipStream_t st)
{
    if (p.fam == Fam32::Dma)
        return launch_conv_fp32_dma(sh, p.v, t, ws, packed, out, st);
    if (p.fam == Fam32::Stem)
        return launch_conv_fp32_stem(sh, p.v, ws, packed, out, st);
    if (p.fam == Fam32::Cols)
        return launch_conv_fp32_cols(sh, p.v, t, ws, packed, out, st);
    C32Args a;
    a.ws = static_cast<const float *>(ws);
    a.packed = static_cast<const float *>(packed);
    a.out = out;
    a.win_bytes = (uint64_t)sh.win_bytes;
    a.P = (uint32_t)sh.P; a.K = (uint32_t)sh.K; a.K_pad = (uint32_t)sh.K_pad32;
    a.Co = (uint32_t)sh.Co; a.Co_pad = (uint32_t)sh.Co_pad32;
    a.Wo = (uint32_t)sh.Wo; a.L = (uint32_t)sh.L; a.wc = make_wincols(sh);
    a.div_Wo = make_fastdiv((uint32_t)sh.Wo);
    // the DMA-staged kernel's tap order (16-tap blocks), so both sum every
    // output in the same order
    a.to = make_taporder(sh.Kw, sh.Kh, sh.Ci, kTapBlock32, t.tap_order == Tuning::kLinear, sh.s);

    const Tile &tile = kTiles[p.v];
    // Channel groups per workgroup: the largest of 8, 4, 2, 1 waves (TN
    // channels each) that leaves no more idle channels than any smaller one.
    int waves = 1;
    int64_t best = -1;
    for (int w : {8, 4, 2, 1}) {
        const int64_t span = (int64_t)tile.tn * w, tiles = (sh.Co + span - 1) / span;
        const int64_t idle = tiles * span - sh.Co;
        if (best < 0 || idle < best) {
            best = idle;
            waves = w;
        }
    }
    const bool v4 = (sh.Ci % 4) == 0;  // every window starts on a 16-byte boundary
    const void *f = kernel_for(tile, waves, v4);
    const int64_t span = (int64_t)tile.tn * waves;
    const int64_t bm = 64 * tile.tm;
    dim3 grid((uint32_t)((sh.P + bm - 1) / bm), (uint32_t)((sh.Co + span - 1) / span));
    void *args[] = {&a};
    return hipLaunchKernel(f, grid, dim3(64 * waves), args, 0, st);
}

}  // namespace im2win
