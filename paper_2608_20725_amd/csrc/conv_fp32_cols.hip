// fp32 windowed convolution on the vector ALUs, staged by input column
// (Sec. III-B, III-C, Eq. 3).
//
// A strip of the window tensor is W_i input columns of T = K_h*C_i elements,
// and the window of output column n is columns n*s .. n*s+K_w-1 (Eq. 3), so
// neighbouring windows share K_w - s columns.  The DMA-staged kernel loads
// each pixel's window slice per stage, i.e. every column about K_w/s times;
// this kernel loads each distinct column of its tile once per tap block and
// lets the K_w windows that use it read it from LDS:
//
//   O[p][j] = sum_tb sum_v sum_{t in block tb} X[col(p, v)][t] * F'[v*T + t][j]
//
// A stage is one block of KT consecutive t (KT = 16 or 8) of
//   * every distinct column the tile's windows touch: row R(p) + v holds
//     column col(p, v) (R as in the column-staged fp16 kernel: consecutive
//     pixels of a strip run share K_w - min(s, K_w) rows), KT*4 bytes each;
//   * the K_w filter slices [v][KT taps][64 channels] of that block;
// fetched with buffer_load ... lds into a two-slot ring.  The lane tile and
// the inner loop are those of the DMA-staged kernel (8 or 4 pixels x 8
// channels per lane, 16-byte LDS reads, filter channel pairs swapped against
// VGPR bank conflicts); only the row a pixel reads for filter column v moves.
// Each output adds its taps in the order (tb, v, t): column order with
// blocks of KT taps.  Taps past T (in the last block) read zero against
// masked filter rows.
#include "common.hpp"

#include <type_traits>

#include <string.h>

namespace im2win {
namespace {

typedef __attribute__((address_space(3))) void *lds_ptr;

struct C32cArgs {
    const float *ws;
    const float *packed;  // F' [K_pad32][Co_pad32], channel pairs swapped
    float *out;
    uint64_t win_bytes;
    uint32_t P, Co, Co_pad, Wo, L, T, s, ms, nst, fbytes;
    TileGrid tg;
    FastDiv div_Wo;
};

constexpr uint32_t kNoColumn = 0xffffffffu;

template <int KW_, int KT_, int NRMAX_, int TM_>
struct CCfg {
    static constexpr int KW = KW_, KT = KT_, NRMAX = NRMAX_, TM = TM_;
    static constexpr bool SERIAL = false;
    static constexpr int TN = 8, LC = 8, NW = 4, NT = 64 * NW;
    static constexpr int LP = 64 / LC;           // lane groups along pixels
    static constexpr int WBM = LP * TM;          // pixels per wave
    static constexpr int BM = NW * WBM;          // pixels per workgroup (waves along pixels)
    static constexpr int CW = LC * TN;           // 64 channels per workgroup
    static constexpr int QPR = KT / 4;           // 16-byte quads per row
    static constexpr int RB = KT * 4;            // bytes per LDS row
    static constexpr int RPI = 1024 / RB;        // rows per 1 KiB load
    static constexpr int LPR = RB / 16;          // lanes per row in a load
    static constexpr int WBYTES = NRMAX * RB;
    static constexpr int FBYTES = KW * KT * CW * 4;
    static constexpr int IW = NRMAX / RPI / NW;  // window loads per wave per stage
    // filter loads per wave per stage; loads past the slices read nothing
    // into spare LDS, so every wave issues the same count
    static constexpr int IF = (FBYTES / 1024 + NW - 1) / NW;
    static constexpr int IB = IW + IF;
    static constexpr int SLOT = WBYTES + NW * IF * 1024;
    static_assert(NRMAX % (RPI * NW) == 0, "window rows split evenly over the waves");
    static_assert(FBYTES % 1024 == 0, "whole 1 KiB filter loads");
    static_assert(KT == 8 || KT == 16, "tap block");
};

// The same tile with its ring serialized (check variant: its output must
// match the ring's bit for bit).
template <class Base>
struct Serialized : Base {
    static constexpr bool SERIAL = true;
};

template <int VM>
__device__ inline void wait_vmcnt()
{
    __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <class C>
struct CTile {
    __amdgpu_buffer_rsrc_t rw, rf;
    uint32_t woff[C::IW];  // window byte offset of this lane's quad at t = 0 (kOOB: no column)
    uint32_t wk;           // first tap of the lane's quad within a block
    uint32_t foff[C::IF];  // filter byte offset at block 0 (kOOB: past the pad)
    uint32_t ftr[C::IF];   // tap row of the lane's filter quad within a block
    uint32_t Rj[C::TM];    // LDS row of each of this lane's pixels
    uint32_t lane, wave, T, nst, bpitch;
    float acc[C::TM][C::TN];


    __device__ inline void issue(uint32_t st, char *slot)
    {
        const uint32_t t0 = st * C::KT;
        const bool past = st >= nst;
#pragma unroll
        for (int i = 0; i < C::IW; ++i) {
            const uint32_t b = wave + C::NW * i;
            const uint32_t off = (!past && woff[i] != kOOB && t0 + wk < T) ? woff[i] + 4u * t0 : kOOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr)(slot + 1024 * b), 16, off, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < C::IF; ++i) {
            const uint32_t b = wave + C::NW * i;
            const uint32_t off = (!past && foff[i] != kOOB && t0 + ftr[i] < T) ? foff[i] + t0 * bpitch : kOOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rf, (lds_ptr)(slot + C::WBYTES + 1024 * b), 16, off, 0, 0, 0);
        }
    }

    __device__ inline void compute(const char *slot)
    {
        const char *fs = slot + C::WBYTES + (lane % C::LC) * C::TN * 4;
        // one filter column at a time (unrolled, the scheduler would keep the
        // addresses and operands of all K_w columns live at once)
#pragma unroll 1
        for (int v = 0; v < C::KW; ++v) {
#pragma unroll
            for (int q = 0; q < C::QPR; ++q) {
                float f[4][C::TN];
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int c = 0; c < C::TN; c += 4) {
                        const float4 fv = *reinterpret_cast<const float4 *>(
                            fs + ((v * C::KT + 4 * q + e) * C::CW) * 4 + 4 * c);
                        f[e][c] = fv.y;  // channel pairs stored swapped
                        f[e][c + 1] = fv.x;
                        f[e][c + 2] = fv.w;
                        f[e][c + 3] = fv.z;
                    }
#pragma unroll
                for (int t = 0; t < C::TM; ++t) {
                    // row Rj[t] + v, quad q: a constant offset from the pixel's row
                    const float4 xv = *reinterpret_cast<const float4 *>(slot + Rj[t] * C::RB + v * C::RB + 16 * q);
                    const float x[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e)
#pragma unroll
                        for (int c = 0; c < C::TN; ++c)
                            acc[t][c] = __builtin_fmaf(x[e], f[e][c], acc[t][c]);
                }
            }
        }
    }

    template <int N>
    __device__ inline void step(uint32_t st, char (&cur)[N], char (&next)[N])
    {
        if constexpr (C::SERIAL) {
            wait_vmcnt<0>();
            ring_barrier();
            if (st < nst)
                compute(cur);
            ring_barrier();
            issue(st + 1, next);
            return;
        }
        wait_vmcnt<0>();
        ring_barrier();
        issue(st + 1, next);
        if (st < nst)
            compute(cur);
    }
};

template <class C>
__global__ __launch_bounds__(C::NT) void conv_fp32_cols(C32cArgs a)
{
    __shared__ __attribute__((aligned(1024))) char r0[C::SLOT];
    __shared__ __attribute__((aligned(1024))) char r1[C::SLOT];
    __shared__ uint32_t tbl[C::NRMAX];

    CTile<C> w;
    const uint32_t tid = threadIdx.x;
    w.lane = tid & 63;
    w.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    __builtin_assume(w.wave < (uint32_t)C::NW);
    w.T = a.T;
    w.nst = a.nst;
    w.bpitch = a.Co_pad * 4u;
    uint32_t tx, ty;
    a.tg.tile(tx, ty);
    const uint32_t p0 = tx * C::BM;
    const uint32_t jb = ty * C::CW;
    const uint32_t q0 = fdiv(p0, a.div_Wo);

    const uint64_t tb = (uint64_t)q0 * a.L;
    const uint64_t left = a.win_bytes - tb * 4;
    w.rw = make_rsrc(a.ws + tb, (uint32_t)(left < kMaxRecords ? left : kMaxRecords));
    w.rf = make_rsrc(a.packed, a.fbytes);
    // row addresses in bytes from here on (see below)

    // column table: element offset (from strip q0) of the column each row holds
    for (uint32_t r = tid; r < (uint32_t)C::NRMAX; r += C::NT)
        tbl[r] = kNoColumn;
    __syncthreads();
    const uint32_t kwm = C::KW - a.ms;
    for (uint32_t n = tid; n < (uint32_t)C::BM; n += C::NT) {
        const uint32_t p = p0 + n;
        if (p < a.P) {
            const uint32_t q = fdiv(p, a.div_Wo);
            const uint32_t c = p - q * a.Wo;
            const uint32_t k = q - q0;
            const uint32_t R = n * a.ms + k * kwm;
            const bool last = n == (uint32_t)C::BM - 1 || p + 1 == a.P || c + 1 == a.Wo;
            const uint32_t nv = last ? (uint32_t)C::KW : a.ms;
            for (uint32_t v = 0; v < nv; ++v)
                tbl[R + v] = k * a.L + (c * a.s + v) * a.T;
        }
    }
    __syncthreads();

    // window loads: instruction i fills rows RPI*b .. of the stage (b = wave
    // + NW*i); lane -> row RPI*b + lane/LPR, quad lane%LPR.  Rows are not
    // swizzled: the lanes of one read that differ hold consecutive pixels
    // whose rows are 64 or 32 bytes apart, and every quad keeps a constant
    // offset from its pixel's row, so the inner loop addresses all its
    // operands from TM row registers.
    w.wk = 4 * (w.lane % C::LPR);
#pragma unroll
    for (int i = 0; i < C::IW; ++i) {
        const uint32_t b = w.wave + C::NW * i;
        const uint32_t r = C::RPI * b + w.lane / C::LPR;
        const uint32_t e = tbl[r];
        w.woff[i] = e == kNoColumn ? kOOB : (e + w.wk) * 4u;
    }
    // filter loads: instruction i fills bytes 1024*b .. of the [K_w][KT][64]
    // slices (b = wave + NW*i): lane -> element 256*b + 4*lane = filter
    // column v, tap row tr, channels jb + col .. +3
#pragma unroll
    for (int i = 0; i < C::IF; ++i) {
        const uint32_t b = w.wave + C::NW * i;
        const uint32_t e = 256 * b + 4 * w.lane;
        const uint32_t v = e / (C::KT * C::CW), rem = e % (C::KT * C::CW);
        const uint32_t tr = rem / C::CW, col = jb + rem % C::CW;
        w.ftr[i] = tr;
        w.foff[i] = (v < (uint32_t)C::KW && col < a.Co_pad) ? ((v * a.T + tr) * a.Co_pad + col) * 4u : kOOB;
    }
    // this lane's pixels and their rows
    const uint32_t pl0 = w.wave * C::WBM + w.lane / C::LC;
#pragma unroll
    for (int t = 0; t < C::TM; ++t) {
        const uint32_t n = pl0 + C::LP * t;
        const uint32_t p = p0 + n;
        // a pixel past P reads row 0 (its sums are never stored)
        w.Rj[t] = p < a.P ? n * a.ms + (fdiv(p, a.div_Wo) - q0) * kwm : 0u;
    }
#pragma unroll
    for (int t = 0; t < C::TM; ++t)
#pragma unroll
        for (int c = 0; c < C::TN; ++c)
            w.acc[t][c] = 0.f;

    w.issue(0, r0);
    for (uint32_t st = 0; st < w.nst; st += 2) {
        w.step(st, r0, r1);
        w.step(st + 1, r1, r0);
    }
    // no load may still be writing LDS when the workgroup ends
    wait_vmcnt<0>();

    const uint32_t jw = jb + (w.lane % C::LC) * C::TN;
    if (jw >= a.Co)
        return;
#pragma unroll
    for (int t = 0; t < C::TM; ++t) {
        const uint32_t p = p0 + pl0 + C::LP * t;
        if (p >= a.P)
            continue;
        float *o = a.out + (uint64_t)p * a.Co + jw;
        if (jw + C::TN <= a.Co && (a.Co & 3) == 0) {
#pragma unroll
            for (int c = 0; c < C::TN; c += 4)
                *reinterpret_cast<float4 *>(o + c) =
                    make_float4(w.acc[t][c], w.acc[t][c + 1], w.acc[t][c + 2], w.acc[t][c + 3]);
        } else {
#pragma unroll
            for (int c = 0; c < C::TN; ++c)
                if (jw + c < a.Co)
                    o[c] = w.acc[t][c];
        }
    }
}

struct CVariant {
    const char *name;
    const void *f;
    int kw, kt, nrmax, bm;
};

template <int KW, int KT, int NRMAX, int TM, bool SERIAL = false>
CVariant c_variant(const char *name)
{
    using B = CCfg<KW, KT, NRMAX, TM>;
    using C = typename std::conditional<SERIAL, Serialized<B>, B>::type;
    return CVariant{name, (const void *)&conv_fp32_cols<C>, KW, KT, NRMAX, C::BM};
}

// name: filter width, pixels per tile, taps per block
const CVariant *c_variants(int *n)
{
    static const CVariant v[] = {
        c_variant<3, 16, 320, 8>("k3p256t16"),
        c_variant<3, 16, 192, 4>("k3p128t16"),
        c_variant<3, 8, 384, 8>("k3p256t8"),
        c_variant<7, 8, 640, 8>("k7p256t8"),
        c_variant<7, 8, 384, 4>("k7p128t8"),
        c_variant<5, 8, 384, 8>("k5p256t8"),
        // serialized ring (check variant)
        c_variant<3, 16, 320, 8, true>("k3p256t16-serial"),
    };
    *n = (int)(sizeof v / sizeof v[0]);
    return v;
}

// Rows a tile of bn consecutive pixels needs at most (as for the fp16
// column-staged kernel).
int64_t cols_rows_needed(const Shape &sh, int64_t bn)
{
    const int64_t ms = sh.s < sh.Kw ? sh.s : sh.Kw;
    int64_t runs = (bn - 1 + sh.Wo - 1) / sh.Wo + 1;
    if (runs > bn)
        runs = bn;
    return (bn - runs) * ms + runs * sh.Kw;
}

}  // namespace

int cols32_find(const char *name)
{
    int n;
    const CVariant *v = c_variants(&n);
    for (int t = 0; t < n; ++t)
        if (strcmp(name, v[t].name) == 0)
            return t;
    return -1;
}

const char *cols32_name(int v)
{
    int n;
    return c_variants(&n)[v].name;
}

bool cols32_fits(const Shape &sh, int pick)
{
    int n;
    const CVariant *v = c_variants(&n);
    if (pick < 0 || pick >= n)
        return false;
    if (sh.Ci % 4 != 0 || sh.d != 1 || sh.Kw != v[pick].kw)
        return false;  // 16-byte columns, consecutive strip columns, the variant's filter width
    if (cols_rows_needed(sh, v[pick].bm) > v[pick].nrmax)
        return false;
    // filter offsets (rows up to K, one block past the last) and the window
    // offsets inside a tile (its strips plus one column) need 31 bits
    if ((sh.K + 16) * sh.Co_pad32 * 4 >= (int64_t)kMaxRecords)
        return false;
    const int64_t strips_per_tile = (v[pick].bm - 1) / sh.Wo + 2;
    if ((strips_per_tile * sh.L + sh.Kh * sh.Ci) * 4 >= (int64_t)kOOB)
        return false;
    return true;
}

// Not the default anywhere: same-process runs inside the benchmark step
// (transform, then conv) against the DMA-staged kernel, fp32 TFLOP/s, 128
// images: 3x3 C=64 at 56x56 72.9 vs 73.3 (HBM-side fetch 309 vs 512 MB, for
// 297 MB of window tensor), 3x3 C=512 at 14x14 82.5-83.2 vs 82.0-83.2, 3x3
// 64 -> 128 at 112x112 89.4 vs 93.2; standalone 7x7 stride 2 84.1 vs 87.4,
// 5x5 C_o=256 70.6 vs 81.3.  The vector-ALU conv is bound by FMA issue, not
// by the window bytes it fetches, and the column tile holds two or three
// workgroups per CU against the DMA-staged tile's four.
int cols32_default(const Shape &sh)
{
    (void)sh;
    return -1;
}

hipError_t launch_conv_fp32_cols(const Shape &sh, int plan, const Tuning &t, const void *ws, const void *packed,
                                 float *out, hipStream_t st)
{
    int n;
    const CVariant &v = c_variants(&n)[plan];
    C32cArgs a;
    a.ws = static_cast<const float *>(ws);
    a.packed = static_cast<const float *>(packed);
    a.out = out;
    a.win_bytes = (uint64_t)sh.win_bytes;
    a.P = (uint32_t)sh.P; a.Co = (uint32_t)sh.Co; a.Co_pad = (uint32_t)sh.Co_pad32;
    a.Wo = (uint32_t)sh.Wo; a.L = (uint32_t)sh.L; a.T = (uint32_t)(sh.Kh * sh.Ci);
    a.s = (uint32_t)sh.s; a.ms = (uint32_t)(sh.s < sh.Kw ? sh.s : sh.Kw);
    a.nst = (a.T + v.kt - 1) / v.kt;
    const uint64_t fb = (uint64_t)sh.K_pad32 * sh.Co_pad32 * 4;
    a.fbytes = (uint32_t)(fb < kMaxRecords ? fb : kMaxRecords);
    a.div_Wo = make_fastdiv((uint32_t)sh.Wo);
    const int64_t gx = (sh.P + v.bm - 1) / v.bm, gy = (sh.Co + 63) / 64;
    if (gx * gy > 0x7fffffff)
        return hipErrorInvalidValue;
    a.tg = make_tilegrid(gx, gy, t.tile_linear);
    void *args[] = {&a};
    return hipLaunchKernel(v.f, dim3((uint32_t)(gx * gy)), dim3(256), args, 0, st);
}

}  // namespace im2win
