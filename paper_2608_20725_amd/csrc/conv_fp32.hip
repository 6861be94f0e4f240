// fp32 windowed convolution on the gfx950 vector ALUs (Sec. III-C, Eq. 3).
//
//   O[p][j] = sum_{k<K} Wn[p][k] * F[frow(k)][j]
//
// Wn[p][.] is the window of output pixel p = (i, m, n): the contiguous span of
// strip (i, m) starting at n*s*K_h*C_i, in (filter column v, filter row u,
// channel r) order; frow(k) = (u*K_w + v)*C_i + r is the matching row of the
// [K_h][K_w][C_i][C_o] filter, so no repacked filter is needed.
//
// Work split (wave64):
//   * a workgroup owns 256 consecutive output pixels and WAVES*16 output
//     channels; each wave owns 16 channels, each lane 4 consecutive pixels,
//     so a lane keeps a 4 x 16 block of fp32 accumulators;
//   * windows are staged through LDS 16 taps at a time, transposed to
//     [tap][pixel] so that a lane fetches its 4 pixels with one 16-byte LDS
//     read; stages are double-buffered: the global loads of stage t+1 are in
//     flight while stage t is multiplied;
//   * filter values are the same for every lane of a wave, so they are read
//     with scalar loads into SGPRs and each multiply-add takes one operand from
//     an SGPR: per tap a lane does 64 FMAs for one LDS read.
// The row offset of every pixel's window is computed once per workgroup (the
// index precomputation of Sec. III-E).
#include "common.hpp"

namespace im2win {
namespace {

constexpr int TM = 4;        // pixels per lane
constexpr int TN = 16;       // channels per wave
constexpr int KC = 16;       // taps per LDS stage
constexpr int BM = 64 * TM;  // pixels per workgroup
constexpr int LDA = BM + 4;  // floats per staged tap row

struct C32Args {
    const float *ws;
    const float *filt;
    float *out;
    uint64_t win_bytes;
    uint32_t P, K, Co, Ci, Kh, Kw, Wo, L, S, KhCi;
    FastDiv div_Wo, div_Ci, div_KhCi;
};

// Filter row of window tap k = (v*K_h + u)*C_i + r, i.e. (u*K_w + v)*C_i + r.
// k is wave-uniform, so this runs on the scalar unit, branch-free.
__device__ inline uint32_t filter_row(uint32_t k, const C32Args &a)
{
    const uint32_t v = fdiv(k, a.div_KhCi);
    const uint32_t rem = k - v * a.KhCi;
    const uint32_t u = fdiv(rem, a.div_Ci);
    const uint32_t r = rem - u * a.Ci;
    return (u * a.Kw + v) * a.Ci + r;
}

template <bool VEC, int WAVES>
struct Stage {
    static constexpr int NT = 64 * WAVES;
    // VEC: float4 granules of the [BM][KC] stage; else single floats
    static constexpr int ITEMS = VEC ? (BM * KC / 4 + NT - 1) / NT : (BM * KC + NT - 1) / NT;
    u32x4 v4[VEC ? ITEMS : 1];
    uint32_t v1[VEC ? 1 : ITEMS];

    // Masked-off loads (pixel past P, tap past K) use an out-of-range offset
    // and read zero: no branches, and no access leaves the window tensor.
    __device__ inline void load(__amdgpu_buffer_rsrc_t rs, const uint32_t *rowoff, uint32_t p0,
                                uint32_t k0, const C32Args &a)
    {
        const uint32_t tid = threadIdx.x;
        if (VEC) {
#pragma unroll
            for (int j = 0; j < ITEMS; ++j) {
                const uint32_t f = tid + j * NT;
                const uint32_t row = (f >> 2) & (BM - 1), kq = f & 3;
                const uint32_t k = k0 + 4 * kq;
                const bool ok = f < BM * KC / 4 && p0 + row < a.P && k < a.K;
                v4[j] = ld_b128(rs, ok ? (rowoff[row] + k) * 4u : kOOB);
            }
        } else {
#pragma unroll
            for (int j = 0; j < ITEMS; ++j) {
                const uint32_t f = tid + j * NT;
                const uint32_t row = (f >> 4) & (BM - 1), kk = f & 15;
                const uint32_t k = k0 + kk;
                const bool ok = f < BM * KC && p0 + row < a.P && k < a.K;
                v1[j] = ld_b32(rs, ok ? (rowoff[row] + k) * 4u : kOOB);
            }
        }
    }

    __device__ inline void store(float (*As)[LDA])
    {
        const uint32_t tid = threadIdx.x;
        if (VEC) {
#pragma unroll
            for (int j = 0; j < ITEMS; ++j) {
                const uint32_t f = tid + j * NT;
                if (f < BM * KC / 4) {
                    // element by value: taking the bits of a vector element
                    // through its address is not reliable with this compiler
                    const uint32_t row = f >> 2, kq = f & 3;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        As[4 * kq + e][row] = __uint_as_float(v4[j][e]);
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < ITEMS; ++j) {
                const uint32_t f = tid + j * NT;
                if (f < BM * KC)
                    As[f & 15][f >> 4] = __uint_as_float(v1[j]);
            }
        }
    }
};

// The 16 filter values of channels jw..jw+15 at one filter row: identical
// for every lane, so they land in SGPRs (one s_load_dwordx16 when the wave's
// channels are all valid).
// The filter is read through the constant address space: the kernel never
// writes it, and loads from that space with a uniform address become s_load.
typedef const __attribute__((address_space(4))) float cfloat;
typedef float f32x16 __attribute__((ext_vector_type(16), aligned(4)));
typedef const __attribute__((address_space(4))) f32x16 cf32x16;

template <bool FULLCH>
__device__ inline void load_filter(float (&f)[TN], uint32_t frow, const C32Args &a, uint32_t jw)
{
    cfloat *fp = (cfloat *)a.filt + (uint64_t)frow * a.Co + jw;
    if (FULLCH) {
        const f32x16 v = *(cf32x16 *)fp;
#pragma unroll
        for (int c = 0; c < TN; ++c)
            f[c] = v[c];
    } else {
#pragma unroll
        for (int c = 0; c < TN; ++c)
            f[c] = fp[(jw + c < a.Co) ? c : 0];
    }
}

__device__ inline void tap_fma(float (&acc)[TM][TN], const float4 x, const float (&f)[TN])
{
    const float xs[TM] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int t = 0; t < TM; ++t)
#pragma unroll
        for (int c = 0; c < TN; ++c)
            acc[t][c] = __builtin_fmaf(xs[t], f[c], acc[t][c]);
}

// Waits for every outstanding LDS and scalar load (lgkmcnt = 0), leaving
// vector-memory loads in flight.
__device__ inline void wait_lgkm() { __builtin_amdgcn_s_waitcnt(0xc07f); }

// Multiplies one LDS stage of `ntaps` (<= KC) taps starting at tap k0.  The
// LDS read and the filter loads of tap kk+1 are issued before the 64 FMAs of
// tap kk and waited for after them; the scheduling fence keeps the compiler
// from hoisting further loads (which would exhaust the SGPRs).  The tap
// guards are wave-uniform branches; full and partial stages share one body so
// the accumulators stay in one set of registers.
template <bool FULLCH>
__device__ inline void stage_fma(float (&acc)[TM][TN], float (*As)[LDA], uint32_t k0,
                                 uint32_t ntaps, const C32Args &a, uint32_t jc, uint32_t lane)
{
    float fc[TN], fn[TN];
    float4 xc, xn;
    load_filter<FULLCH>(fc, filter_row(k0, a), a, jc);
    xc = *reinterpret_cast<const float4 *>(&As[0][TM * lane]);
    wait_lgkm();
#pragma unroll
    for (int kk = 0; kk < KC; ++kk) {
        const bool more = kk + 1 < KC && (uint32_t)kk + 1 < ntaps;
        if (more) {
            load_filter<FULLCH>(fn, filter_row(k0 + kk + 1, a), a, jc);
            xn = *reinterpret_cast<const float4 *>(&As[kk + 1][TM * lane]);
        }
        if ((uint32_t)kk < ntaps)
            tap_fma(acc, xc, fc);
        wait_lgkm();
        __builtin_amdgcn_sched_barrier(0);
        if (more) {
#pragma unroll
            for (int c = 0; c < TN; ++c)
                fc[c] = fn[c];
            xc = xn;
        }
    }
}

// FULLCH (C_o >= 16): every wave multiplies 16 existing channels; a wave
// whose 16 channels would run past C_o computes channels C_o-16..C_o-1
// instead and stores only the ones no other wave owns.  Otherwise (C_o < 16)
// filter reads are clamped channel by channel.
template <bool VEC, int WAVES, bool FULLCH>
__global__ __launch_bounds__(64 * WAVES) void conv_fp32_kernel(C32Args a)
{
    __shared__ float As[2][KC][LDA];
    __shared__ uint32_t rowoff[BM];

    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t p0 = blockIdx.x * BM;
    const uint32_t jw = blockIdx.y * (TN * WAVES) + wave * TN;  // first channel this wave owns
    const uint32_t jc = (!FULLCH || jw + TN <= a.Co) ? jw : a.Co - TN;  // first channel it computes

    // window offsets of the workgroup's pixels, relative to the strip of p0
    const uint32_t q0 = fdiv(p0, a.div_Wo);
    const uint64_t tb_elem = (uint64_t)q0 * a.L;
    const uint64_t left = a.win_bytes - tb_elem * 4;
    const __amdgpu_buffer_rsrc_t rs =
        make_rsrc(a.ws + tb_elem, (uint32_t)(left < kMaxRecords ? left : kMaxRecords));
    for (uint32_t t = tid; t < BM; t += 64 * WAVES) {
        const uint32_t p = p0 + t;
        uint32_t off = 0;
        if (p < a.P) {
            const uint32_t q = fdiv(p, a.div_Wo);
            off = (q - q0) * a.L + (p - q * a.Wo) * a.S;
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

    const uint32_t nst = (a.K + KC - 1) / KC;
    Stage<VEC, WAVES> stg;
    stg.load(rs, rowoff, p0, 0, a);
    stg.store(As[0]);
    __syncthreads();

    const bool active = jw < a.Co;
    for (uint32_t st = 0; st < nst; ++st) {
        const uint32_t k0 = st * KC;
        if (st + 1 < nst)
            stg.load(rs, rowoff, p0, k0 + KC, a);
        const uint32_t ntaps = min((uint32_t)KC, a.K - k0);
        if (active)
            stage_fma<FULLCH>(acc, As[st & 1], k0, ntaps, a, jc, lane);
        if (st + 1 < nst)
            stg.store(As[(st + 1) & 1]);
        __syncthreads();
    }

    if (!active)
        return;
#pragma unroll
    for (int t = 0; t < TM; ++t) {
        const uint32_t p = p0 + TM * lane + t;
        if (p >= a.P)
            continue;
        float *o = a.out + (uint64_t)p * a.Co + jc;
        if (jc == jw && jw + TN <= a.Co && (a.Co & 3) == 0) {
#pragma unroll
            for (int c = 0; c < TN; c += 4)
                *reinterpret_cast<float4 *>(o + c) =
                    make_float4(acc[t][c], acc[t][c + 1], acc[t][c + 2], acc[t][c + 3]);
        } else {
#pragma unroll
            for (int c = 0; c < TN; ++c)
                if (jc + c >= jw && jc + c < a.Co)
                    o[c] = acc[t][c];
        }
    }
}

template <int WAVES>
const void *pick(bool vec, bool fullch)
{
    if (fullch)
        return vec ? (const void *)&conv_fp32_kernel<true, WAVES, true>
                   : (const void *)&conv_fp32_kernel<false, WAVES, true>;
    return vec ? (const void *)&conv_fp32_kernel<true, WAVES, false>
               : (const void *)&conv_fp32_kernel<false, WAVES, false>;
}

}  // namespace

hipError_t launch_conv_fp32(const Shape &sh, const void *ws, const float *filt, float *out,
                            hipStream_t st)
{
    C32Args a;
    a.ws = static_cast<const float *>(ws);
    a.filt = filt;
    a.out = out;
    a.win_bytes = (uint64_t)sh.win_bytes;
    a.P = (uint32_t)sh.P; a.K = (uint32_t)sh.K; a.Co = (uint32_t)sh.Co; a.Ci = (uint32_t)sh.Ci;
    a.Kh = (uint32_t)sh.Kh; a.Kw = (uint32_t)sh.Kw; a.Wo = (uint32_t)sh.Wo;
    a.L = (uint32_t)sh.L; a.S = (uint32_t)sh.S; a.KhCi = (uint32_t)(sh.Kh * sh.Ci);
    a.div_Wo = make_fastdiv((uint32_t)sh.Wo);
    a.div_Ci = make_fastdiv((uint32_t)sh.Ci);
    a.div_KhCi = make_fastdiv(a.KhCi);
    // Channel groups per workgroup: the largest of 8, 4, 2, 1 waves (16
    // channels each) that leaves no more idle channels than any smaller one.
    int waves = 1;
    int64_t best = -1;
    for (int w : {8, 4, 2, 1}) {
        const int64_t span = 16 * w, tiles = (sh.Co + span - 1) / span;
        const int64_t idle = tiles * span - sh.Co;
        if (best < 0 || idle < best) {
            best = idle;
            waves = w;
        }
    }
    const bool vec = (sh.Ci % 4) == 0;  // every window starts on a 16-byte boundary
    const bool fullch = sh.Co >= TN;
    const void *f = waves == 8   ? pick<8>(vec, fullch)
                    : waves == 4 ? pick<4>(vec, fullch)
                    : waves == 2 ? pick<2>(vec, fullch)
                                 : pick<1>(vec, fullch);
    const int64_t span = 16 * waves;
    dim3 grid((uint32_t)((sh.P + BM - 1) / BM), (uint32_t)((sh.Co + span - 1) / span));
    void *args[] = {&a};
    return hipLaunchKernel(f, grid, dim3(64 * waves), args, 0, st);
}

}  // namespace im2win
