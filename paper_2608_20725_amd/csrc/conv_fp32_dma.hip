// fp32 windowed convolution on the gfx950 vector ALUs, stages loaded straight
// into LDS (Sec. III-C, Eq. 3).
//
//   O[p][j] = sum_{k<K} Wn[p][k] * F'[k][j]
//
// Wn[p][.] is the window of output pixel p (a contiguous span of its strip,
// Eq. 3) and F' the filter repacked into window tap order, [K_pad32][C_o_pad32]
// with channels 2i and 2i+1 swapped (pack_filter_fp32; see DTile::compute).
//
// Work split (wave64, four waves):
//   * a lane keeps a TM x TN block of fp32 accumulators (TM pixels, TN
//     channels); LC lanes of a wave share pixels and split channels, so a
//     wave covers (64/LC)*TM pixels x LC*TN channels, and the four waves lie
//     along channels or pixels so that a workgroup covers 64 channels; lane
//     group g of a wave owns pixels g, g + 64/LC, g + 2*64/LC, ...;
//   * a stage is 16 taps.  The windows of the workgroup's pixels for those
//     taps (64 bytes per pixel) and the stage's 16 x 64 filter slab are
//     fetched with buffer_load ... lds, which writes each lane's 16 bytes
//     straight to LDS: no staging registers and no transposing stores, and
//     the ring of NS slots keeps NS-1 stages in flight;
//   * per group of 4 taps a lane reads its TM pixels' 4-tap quads (TM 16-byte
//     reads) and, per tap, its TN filter values (TN/4 16-byte reads), then
//     does 4*TM*TN FMAs with every operand in VGPRs: (TM + TN) LDS reads per
//     4*TM*TN FMAs.  LDS read instructions, not FMAs, bound the simpler
//     tilings on this part, so the tile trades them against registers.
// Window rows in LDS are [pixel][16 taps] = 64 bytes; quad q of pixel p sits
// at slot q ^ (p & 3), so the 16 lanes that read quad q of 16 consecutive
// pixels hit all 64 banks.  Taps past K read zero (masked loads) against zero
// filter rows (padding), so they add exactly 0.
#include "common.hpp"

#include <type_traits>

#include <stdlib.h>
#include <string.h>

namespace im2win {
namespace {

typedef __attribute__((address_space(3))) void *lds_ptr;

struct D32Args {
    const float *ws;
    const float *packed;  // F' [K_pad32][Co_pad32]
    float *out;
    uint64_t win_bytes;
    uint32_t P, K, K_pad, Co, Co_pad, Wo, L;
    WinCols wc;              // window start of an output column in its strip
    TileGrid tg;             // pixel x channel tiles of the 1-D launch
    FastDiv div_Wo;
    TapOrder to;             // order of the stages' tap blocks (blocks of KT taps)
};

// Lane tile TM pixels x TN channels; LC lanes of a wave share pixels and
// split channels, so a wave covers (64/LC)*TM pixels x LC*TN channels; of the
// four waves, KS split the taps of a stage (each takes KC of them, and their
// sums are added at the end), WCH lie along channels and the rest along
// pixels.
template <int TM_, int TN_, int LC_, int WCH_, int NS_, int KC_ = 16, int GR_ = 16, int KS_ = 1, int NW_ = 4>
struct DCfg {
    static constexpr int TM = TM_, TN = TN_, LC = LC_, WCH = WCH_, NS = NS_, KC = KC_;
    static constexpr bool SERIAL = false;  // see Serialized
    // bytes one lane moves per window load: 16 when every window starts on a
    // 16-byte boundary (C_i a multiple of 4), else 4 (any fp32 window)
    static constexpr int GR = GR_;
    static constexpr int KS = KS_;                // waves along the taps
    static constexpr int KT = KS * KC;            // taps per stage
    static constexpr int QPR = KC / 4;            // 16-byte quads per wave per stage
    static constexpr int LPR = KT * 4 / GR;       // lanes per window row in a load
    static constexpr int PPI = 64 / LPR;          // pixels per window load
    static constexpr int NW = NW_, NT = 64 * NW;  // waves, threads
    static constexpr int WPX = NW / (WCH * KS);   // waves along pixels
    static constexpr int LP = 64 / LC;            // lane groups along pixels
    static constexpr int WBM = LP * TM;           // pixels per wave
    static constexpr int BM = WPX * WBM;          // pixels per workgroup
    static constexpr int CW = WCH * LC * TN;      // channels per workgroup
    static_assert(TN % 4 == 0 && NW % (WCH * KS) == 0, "tile");
    static_assert(CW % 16 == 0, "whole 1 KiB filter loads per stage");
    static_assert(KS == 1 || (KC == 16 && GR == 16), "tap split: 16-tap quads groups, 16-byte loads");
    static constexpr int WBYTES = BM * KT * 4;    // window part of a stage
    static constexpr int FBYTES = KT * CW * 4;    // filter part of a stage
    static constexpr int IW = WBYTES / (64 * GR) / NW;  // window loads per wave per stage
    // filter loads per wave per stage; loads past the slab read nothing into
    // a spare 1 KiB block, so every wave issues the same count
    static constexpr int IF = (FBYTES / 1024 + NW - 1) / NW;
    static constexpr int IB = IW + IF;
    static constexpr int STAGE_ALLOC = WBYTES + NW * IF * 1024;
    // every wave's sums, for the final add of the tap slices: NW parts of
    // WAVE_PART bytes laid over the ring slots, none straddling two slots
    static constexpr int WAVE_PART = KS > 1 ? TM * TN * 64 * 4 : 1024;
    static constexpr int PART_BYTES = KS > 1 ? NW * WAVE_PART : 0;
    static constexpr int SLOT_MIN = (STAGE_ALLOC + WAVE_PART - 1) / WAVE_PART * WAVE_PART;
    static constexpr int SLOT_PART = ((PART_BYTES + NS - 1) / NS + WAVE_PART - 1) / WAVE_PART * WAVE_PART;
    // bytes of one ring slot (each slot is an LDS array of its own)
    static constexpr int SLOT = SLOT_MIN > SLOT_PART ? SLOT_MIN : SLOT_PART;
    static_assert(WBYTES % (64 * GR * NW) == 0, "even split over waves");
    static_assert(GR == 16 || GR == 4, "window load granule");
    static_assert(KC == 8 || KC == 16, "stage depth");
    static_assert(NS >= 2 && NS <= 3, "ring depth");
    static_assert((NS - 2) * IB <= 63, "vmcnt range");
};

// The same tile with its ring serialized: a stage's loads are issued only
// after every wave has finished with the previous stage, and waited for in
// full, so no load is in flight while LDS is read.  Same sums in the same
// order; a check variant for the ring's waits and barriers.
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
struct DTile {
    __amdgpu_buffer_rsrc_t rw, rf;
    uint32_t woff[C::IW];  // window byte offset at tap 0 (kOOB: no pixel)
    uint32_t wk;           // first tap of the lane's granule within the stage
    uint32_t foff[C::IF];  // filter byte offset at tap 0 (kOOB: column past the pad)
    uint32_t wave, lane, K, Co_pad, nst;
    TapOrder to;
    float acc[C::TM][C::TN];

    __device__ inline void issue(uint32_t st, char *slot)
    {
        // first tap of the stage; in column order every stage is whole
        // (K_h*C_i a multiple of KT), so the masks below see the true taps
        const uint32_t k0 = to.map(st * C::KT);
        const bool past = st >= nst;
#pragma unroll
        for (int i = 0; i < C::IW; ++i) {
            const uint32_t b = wave + C::NW * i;
            const uint32_t off = (!past && k0 + wk < K) ? woff[i] + 4u * k0 : kOOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr)(slot + 64 * C::GR * b), C::GR, off, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < C::IF; ++i) {
            const uint32_t b = wave + C::NW * i;
            const uint32_t off = past ? kOOB : foff[i] + 4u * k0 * Co_pad;  // foff is kOOB past the slab
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rf, (lds_ptr)(slot + C::WBYTES + 1024 * b), 16, off,
                                                     0, 0, 0);
        }
    }

    // Window quad q of local pixel p sits at slot q ^ swz(p) of its row (the
    // swizzle stays inside each group of 4 quads).
    __device__ static inline uint32_t wslot(uint32_t p, uint32_t q)
    {
        return C::QPR == 4 ? q ^ (p & 3) : q ^ ((p >> 3) & 1);
    }

    // this wave's place: tap slice, pixel group, channel group
    __device__ inline uint32_t wks() const { return wave / (C::WCH * C::WPX); }
    __device__ inline uint32_t wpx() const { return (wave / C::WCH) % C::WPX; }
    __device__ inline uint32_t wch() const { return wave % C::WCH; }

    // VGPR banks of the FMAs.  On gfx950 two waves of a SIMD issue fp32 FMAs
    // together at full rate unless an FMA's first source stays in one VGPR
    // bank from one FMA to the next while its accumulator and second source
    // share a bank (probe at four waves per SIMD: 110 vs 131 TFLOP/s; 128
    // with the filter value first, whose bank then matches the
    // accumulator's).  Here the pixel value is the first source and repeats
    // over TN FMAs, and the filter value of channel j comes from element
    // j % 4 of a ds_read_b128 tuple while the sum of channel j is stored from
    // element j % 4 of a 16-byte store tuple: with filter rows in channel
    // order both share a bank whatever names the registers get.  So the
    // filter pack stores channels 2i and 2i+1 swapped, the reads below swap
    // them back, and the filter value of channel j sits in element j ^ 1,
    // another bank than its accumulator.  Sums and their order are unchanged.
    __device__ inline void compute(const char *slot)
    {
        // this lane's channels of the slice's first tap, and its first pixel
        const uint32_t q0 = wks() * C::QPR;
        const char *fs = slot + C::WBYTES + q0 * 4 * C::CW * 4 + (wch() * C::LC + lane % C::LC) * C::TN * 4;
        const uint32_t pl0 = wpx() * C::WBM + lane / C::LC;
#pragma unroll
        for (int q = 0; q < C::QPR; ++q) {
            // filter values of the quad's 4 taps
            float f[4][C::TN];
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int c = 0; c < C::TN; c += 4) {
                    const float4 v =
                        *reinterpret_cast<const float4 *>(fs + (4 * q + e) * C::CW * 4 + 4 * c);
                    f[e][c] = v.y;  // pairs stored swapped (see above)
                    f[e][c + 1] = v.x;
                    f[e][c + 2] = v.w;
                    f[e][c + 3] = v.z;
                }
#pragma unroll
            for (int t = 0; t < C::TM; ++t) {
                const uint32_t p = pl0 + C::LP * t;
                // q0 is a multiple of 4 and the swizzle stays inside groups of
                // 4 quads: quad q0 + q of the row sits at slot q0 + wslot(p, q)
                const float4 v =
                    *reinterpret_cast<const float4 *>(slot + 16 * q0 + p * (C::KT * 4) + 16 * wslot(p, q));
                const float x[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int c = 0; c < C::TN; ++c)
                        acc[t][c] = __builtin_fmaf(x[e], f[e][c], acc[t][c]);
            }
        }
    }

    // The slots are passed as the LDS arrays themselves: once inlined, every
    // access names its array, so the compiler can tell that reading the
    // current slot does not depend on the loads just issued into the next
    // one and does not wait for them.
    template <int N>
    __device__ inline void step(uint32_t st, char (&cur)[N], char (&next)[N])
    {
        if constexpr (C::SERIAL) {
            wait_vmcnt<0>();
            ring_barrier();
            if (st < nst)
                compute(cur);
            ring_barrier();
            issue(st + C::NS - 1, next);
            return;
        }
        wait_vmcnt<(C::NS - 2) * C::IB>();
        ring_barrier();
        issue(st + C::NS - 1, next);
        if (st < nst)
            compute(cur);
    }
};

template <class C>
__global__ __launch_bounds__(C::NT) void conv_fp32_dma(D32Args a)
{
    // ring slots: separate arrays (see DTile::step)
    constexpr int S2 = C::NS > 2 ? C::SLOT : 1024;
    __shared__ __attribute__((aligned(1024))) char r0[C::SLOT];
    __shared__ __attribute__((aligned(1024))) char r1[C::SLOT];
    __shared__ __attribute__((aligned(1024))) char r2[S2];

    DTile<C> w;
    const uint32_t tid = threadIdx.x;
    w.lane = tid & 63;
    w.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    __builtin_assume(w.wave < (uint32_t)C::NW);
    w.K = a.K;
    w.Co_pad = a.Co_pad;
    w.to = a.to;
    w.nst = (a.K_pad + C::KT - 1) / C::KT;  // taps past K_pad read zero (masked, or past the filter)
    uint32_t tx, ty;
    a.tg.tile(tx, ty);
    const uint32_t p0 = tx * C::BM;
    const uint32_t jb = ty * C::CW;  // first channel of the workgroup

    // windows are addressed from the strip of p0 on
    const uint32_t q0 = fdiv(p0, a.div_Wo);
    const uint64_t tb = (uint64_t)q0 * a.L;
    const uint64_t left = a.win_bytes - tb * 4;
    w.rw = make_rsrc(a.ws + tb, (uint32_t)(left < kMaxRecords ? left : kMaxRecords));
    const uint64_t fbytes = (uint64_t)a.K_pad * a.Co_pad * 4;
    w.rf = make_rsrc(a.packed, (uint32_t)(fbytes < kMaxRecords ? fbytes : kMaxRecords));

    // Window load i of this wave fills pixels PPI*b .. PPI*b+PPI-1 (b = wave
    // + 4i): lane -> pixel PPI*b + lane/LPR and granule g = lane%LPR of its
    // LDS row, in LDS quad g*GR/16; that quad holds quad wslot(pixel, .) of
    // the pixel's stage taps (with 4-byte granules, element g%4 of it).  The
    // tap depends on the pixel only through the swizzle bits of pl, which
    // are the same for every load of a lane (PPI*b is a multiple of 16 when
    // the swizzle uses pl & 3 and of 32 when it uses bit 3), so it is kept
    // once per lane.
    {
        const uint32_t pl = w.lane / C::LPR;
        const uint32_t g = w.lane % C::LPR;
        w.wk = C::GR == 16 ? 4 * DTile<C>::wslot(pl, g) : 4 * DTile<C>::wslot(pl, g / 4) + g % 4;
    }
    static_assert(C::PPI % (C::QPR == 4 ? 4 : 16) == 0, "swizzle bits of pl fixed per lane");
#pragma unroll
    for (int i = 0; i < C::IW; ++i) {
        const uint32_t b = w.wave + C::NW * i;
        const uint32_t pl = C::PPI * b + w.lane / C::LPR;
        const uint32_t p = p0 + pl;
        w.woff[i] = kOOB;
        if (p < a.P) {
            const uint32_t q = fdiv(p, a.div_Wo);
            w.woff[i] = ((q - q0) * a.L + a.wc.start(p - q * a.Wo) + w.wk) * 4u;
        }
    }
    // Filter load i fills bytes 1024*b .. 1024*b+1023 of the stage's [KT][CW]
    // slab (b = wave + NW*i): lane -> element e = 256*b + 4*lane, tap e / CW,
    // channels jb + e % CW .. +3.
#pragma unroll
    for (int i = 0; i < C::IF; ++i) {
        const uint32_t b = w.wave + C::NW * i;
        const uint32_t e = 256 * b + 4 * w.lane;
        const uint32_t row = e / C::CW, col = jb + e % C::CW;
        w.foff[i] = (row < (uint32_t)C::KT && col < a.Co_pad) ? (row * a.Co_pad + col) * 4u : kOOB;
    }
#pragma unroll
    for (int t = 0; t < C::TM; ++t)
#pragma unroll
        for (int c = 0; c < C::TN; ++c)
            w.acc[t][c] = 0.f;

    w.issue(0, r0);
    if constexpr (C::NS == 2) {
        for (uint32_t st = 0; st < w.nst; st += 2) {
            w.step(st, r0, r1);
            w.step(st + 1, r1, r0);
        }
    } else {
        w.issue(1, r1);
        for (uint32_t st = 0; st < w.nst; st += 3) {
            w.step(st, r0, r2);
            w.step(st + 1, r1, r0);
            w.step(st + 2, r2, r1);
        }
    }
    // no load may still be writing LDS when the workgroup ends
    wait_vmcnt<0>();

    // first channel of this lane, and its first pixel
    const uint32_t jw = jb + (w.wch() * C::LC + w.lane % C::LC) * C::TN;
    const uint32_t pl0 = w.wpx() * C::WBM + w.lane / C::LC;
    if constexpr (C::KS > 1) {
        // Every wave stores its sums in LDS; then the KS waves with the same
        // pixels and channels each finish TM/KS of the lane's pixel rows,
        // adding the tap slices' sums in slice order (a fixed order: the
        // result does not depend on timing).
        constexpr int PPS = C::SLOT / C::WAVE_PART;  // parts per slot
        static_assert(C::NS * PPS >= C::NW, "the parts fit in the ring");
        const uint32_t ks = w.wks(), grp = w.wpx() * C::WCH + w.wch();
        auto part = [&](uint32_t k) {
            const uint32_t idx = k * (C::NW / C::KS) + grp;
            char *slot = idx < (uint32_t)PPS ? r0 : r1;
            if constexpr (C::NS > 2)
                slot = idx < 2u * PPS ? slot : r2;
            return reinterpret_cast<float4 *>(slot + (idx % PPS) * C::WAVE_PART);
        };
        __syncthreads();  // every wave is done with the ring
        float4 *mine = part(ks);
#pragma unroll
        for (int t = 0; t < C::TM; ++t)
#pragma unroll
            for (int c = 0; c < C::TN; c += 4)
                mine[(t * (C::TN / 4) + c / 4) * 64 + w.lane] =
                    make_float4(w.acc[t][c], w.acc[t][c + 1], w.acc[t][c + 2], w.acc[t][c + 3]);
        __syncthreads();
        if (jw >= a.Co)
            return;
        for (int r = 0; r < C::TM / C::KS; ++r) {
            const uint32_t t = r * C::KS + ks;
            const uint32_t p = p0 + pl0 + C::LP * t;
            if (p >= a.P)
                continue;
            float v[C::TN];
#pragma unroll
            for (int c = 0; c < C::TN; c += 4) {
                float4 sum = part(0)[(t * (C::TN / 4) + c / 4) * 64 + w.lane];
#pragma unroll
                for (int k = 1; k < C::KS; ++k) {
                    const float4 u = part(k)[(t * (C::TN / 4) + c / 4) * 64 + w.lane];
                    sum.x += u.x;
                    sum.y += u.y;
                    sum.z += u.z;
                    sum.w += u.w;
                }
                v[c] = sum.x;
                v[c + 1] = sum.y;
                v[c + 2] = sum.z;
                v[c + 3] = sum.w;
            }
            float *o = a.out + (uint64_t)p * a.Co + jw;
            if (jw + C::TN <= a.Co && (a.Co & 3) == 0) {
#pragma unroll
                for (int c = 0; c < C::TN; c += 4)
                    *reinterpret_cast<float4 *>(o + c) = make_float4(v[c], v[c + 1], v[c + 2], v[c + 3]);
            } else {
#pragma unroll
                for (int c = 0; c < C::TN; ++c)
                    if (jw + c < a.Co)
                        o[c] = v[c];
            }
        }
        return;
    }

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

struct DVariant {
    const char *name;
    const void *f;
    int bm, cw, gr, nt, kt;
};

template <int TM, int TN, int LC, int WCH, int NS, int KC, int GR = 16, int KS = 1, int NW = 4, bool SERIAL = false>
DVariant d_variant(const char *name)
{
    using B = DCfg<TM, TN, LC, WCH, NS, KC, GR, KS, NW>;
    using C = typename std::conditional<SERIAL, Serialized<B>, B>::type;
    return DVariant{name, (const void *)&conv_fp32_dma<C>, C::BM, C::CW, GR, C::NT, C::KT};
}

const DVariant *d_variants(int *n)
{
    // name: pixels x channels per lane, lanes along channels, ring slots,
    // taps per wave per stage, then g4 (4-byte window loads) or tN (the
    // waves split a stage's taps N ways).
    // Measured on MI355X over the benchmark layers, each conv right after
    // its transform: 8 x 8 lane tiles with 16-tap stages beat 4 x 16,
    // 8 x 16, 12 x 8 and 16 x 8 tiles and 8-tap stages (larger tiles lose
    // occupancy, 8-tap stages add barriers).  With the taps split four ways
    // (a 32- or 64-pixel tile, 64 taps per stage, 2 workgroups per CU)
    // layers whose 256-pixel grid is small gain: 3x3 C=512 at 7x7 (104
    // tiles) 18.5 -> 54.1 TFLOP/s with 64-pixel tiles, 3x3 C=256 at 14x14
    // (288) 46.9 -> 62.8, 3x3 C=512 at 14x14 (576) 62.7 -> 73.3, 5x5 C_o=256
    // at 24x24 (800) 65.9 -> 69.3 with 32-pixel tiles; from about 1500 tiles
    // on (the 56x56 C=64 and 1x1 C=1024 layers) the 256-pixel tile is ahead
    // again (69.8 vs 63.9, 70.7 vs 67.5).  Two-way splits, a 3-slot ring, the
    // 256-pixel tile held to 2 workgroups per CU, and 128- or 64-pixel tiles
    // of two or one waves (more, smaller workgroups: 68.1 vs 64.9 and 60.8
    // on the 56x56 layer) measured lower.  6- and 8-pixel lane tiles of four
    // waves (192- and 128-pixel tiles, 4 and 5 waves per SIMD) come within
    // about 3 % of the 256-pixel tile either way (1x1 C=1024: 84.9 and 85.6
    // vs 83.1; 112x112 C_o=128: 90.3 and 88.9 vs 90.8), inside run-to-run
    // spread, so the default stays; a tap-major inner loop that reads every
    // operand a tap ahead measured no faster.  The 32-pixel tap-split tile
    // doubled to 64 pixels with eight waves (two pixel groups, same sums in
    // the same order) runs four waves per SIMD instead of two: 3x3 C=512 at
    // 14x14 91.9 vs 86.0, 3x3 C=128 at 28x28 85.8 vs 80.9, 5x5 C_o=256 at
    // 24x24 88.9 vs 86.1, 3x3 C=256 at 12x12 and 14x14 +1 %; on 3x3 C=512 at
    // 7x7 (104 tiles) the 64-pixel four-wave tile stays ahead (74.0 vs
    // 73.3), and an eight-wave 128-pixel tile or a two-way split of eight
    // waves measured lower.
    static const DVariant v[] = {
        d_variant<8, 8, 8, 1, 2, 16>("p8c8l8s2k16"),
        d_variant<6, 8, 8, 1, 2, 16>("p6c8l8s2k16"),
        d_variant<4, 8, 8, 1, 2, 16>("p4c8l8s2k16"),
        d_variant<4, 16, 1, 4, 2, 16>("p4c16l1s2k16"),
        // 96-channel tiles (12 channels per lane) for C_o = 96, 288, ...
        d_variant<8, 12, 8, 1, 2, 16>("p8c12l8s2k16"),
        d_variant<4, 12, 8, 1, 2, 16>("p4c12l8s2k16"),
        d_variant<8, 12, 8, 1, 2, 16, 4>("p8c12l8s2k16g4"),
        d_variant<4, 12, 8, 1, 2, 16, 4>("p4c12l8s2k16g4"),
        // 4-byte window loads: windows that start anywhere (C_i % 4 != 0)
        d_variant<8, 8, 8, 1, 2, 16, 4>("p8c8l8s2k16g4"),
        d_variant<6, 8, 8, 1, 2, 16, 4>("p6c8l8s2k16g4"),
        d_variant<4, 8, 8, 1, 2, 16, 4>("p4c8l8s2k16g4"),
        d_variant<8, 8, 8, 1, 2, 16, 16, 4>("p8c8l8s2k16t4"),
        d_variant<4, 8, 8, 1, 2, 16, 16, 4>("p4c8l8s2k16t4"),
        // eight waves: two 32-pixel groups, each splitting the taps four ways
        d_variant<4, 8, 8, 1, 2, 16, 16, 4, 8>("p4c8l8s2k16t4w8"),
        // serialized rings of three of the above (check variants)
        d_variant<8, 8, 8, 1, 2, 16, 16, 1, 4, true>("p8c8l8s2k16-serial"),
        d_variant<6, 8, 8, 1, 2, 16, 4, 1, 4, true>("p6c8l8s2k16g4-serial"),
        d_variant<4, 8, 8, 1, 2, 16, 16, 4, 4, true>("p4c8l8s2k16t4-serial"),
        d_variant<4, 8, 8, 1, 2, 16, 16, 4, 8, true>("p4c8l8s2k16t4w8-serial"),
    };
    *n = (int)(sizeof v / sizeof v[0]);
    return v;
}

}  // namespace

int dma32_find(const char *name)
{
    int n;
    const DVariant *v = d_variants(&n);
    for (int t = 0; t < n; ++t)
        if (strcmp(name, v[t].name) == 0)
            return t;
    return -1;
}

const char *dma32_name(int v)
{
    int n;
    return d_variants(&n)[v].name;
}

bool dma32_fits(const Shape &sh, int pick)
{
    int n;
    const DVariant *v = d_variants(&n);
    if (pick < 0 || pick >= n)
        return false;
    // filter offsets, up to one 64-tap stage past K_pad32, need 31 bits
    if ((sh.K_pad32 + 64) * sh.Co_pad32 * 4 > (int64_t)kMaxRecords)
        return false;
    // 16-byte window loads need every window on a 16-byte boundary
    return v[pick].gr == 4 || sh.Ci % 4 == 0;
}

int dma32_default(const Shape &sh)
{
    const bool aligned = sh.Ci % 4 == 0;
    const int64_t tiles256 = ((sh.P + 255) / 256) * ((sh.Co + 63) / 64);
    // unaligned windows (C_i % 4 != 0, the 3-channel stems): the 6-pixel
    // lane tile, 7x7 C_i=3 stride 2 67.2 vs 64.1 TFLOP/s (8-pixel) and 3x3
    // C_i=3 36.6 vs 34.4, same machine
    // strided overlapping windows (K_w > s > 1) re-read more of their
    // columns from L2 and run better with the 6-pixel tile's five workgroups
    // per CU: 7x7 C=64 stride 2 at 224x224, 95.0 vs 92.7 TFLOP/s in the
    // benchmark step (3x3 C=64 -> 128 stride 1 at 112x112: 94.8 vs 97.7)
    const bool strided = sh.s > 1 && sh.Kw > sh.s;
    const char *name = !aligned          ? "p6c8l8s2k16g4"
                       : tiles256 <= 128  ? "p8c8l8s2k16t4"
                       : tiles256 <= 1024 ? "p4c8l8s2k16t4w8"
                       : strided          ? "p6c8l8s2k16"
                                          : "p8c8l8s2k16";
    // 96-channel tiles where they pad fewer channels than 64-channel ones
    // (C_o = 96: 0 against 32 of 128) and still give four workgroups per CU:
    // 11x11 C_i=3 C_o=96 stride 4, 60.7 -> 74.8 TFLOP/s; 3x3 C=64 -> 96 at
    // 56x56, 70.0 -> 84.0.  The 8 x 12 lane tile (2 waves per SIMD) measured
    // 68.7 and 80.2.
    const int64_t pad64 = (sh.Co + 63) / 64 * 64 - sh.Co, pad96 = (sh.Co + 95) / 96 * 96 - sh.Co;
    if (pad96 < pad64 && ((sh.P + 127) / 128) * ((sh.Co + 95) / 96) >= 1024)
        name = aligned ? "p4c12l8s2k16" : "p4c12l8s2k16g4";
    const int pick = dma32_find(name);
    return dma32_fits(sh, pick) ? pick : -1;
}

hipError_t launch_conv_fp32_dma(const Shape &sh, int plan, const Tuning &t, const void *ws, const void *packed,
                                float *out, hipStream_t st)
{
    int n;
    const DVariant &v = d_variants(&n)[plan];
    D32Args a;
    a.ws = static_cast<const float *>(ws);
    a.packed = static_cast<const float *>(packed);
    a.out = out;
    a.win_bytes = (uint64_t)sh.win_bytes;
    a.P = (uint32_t)sh.P; a.K = (uint32_t)sh.K; a.K_pad = (uint32_t)sh.K_pad32;
    a.Co = (uint32_t)sh.Co; a.Co_pad = (uint32_t)sh.Co_pad32;
    a.Wo = (uint32_t)sh.Wo; a.L = (uint32_t)sh.L; a.wc = make_wincols(sh);
    a.div_Wo = make_fastdiv((uint32_t)sh.Wo);
    // column tap order unless IM2WIN_TAP_ORDER=linear (7x7 stride 2 C=64 at
    // 224x224: 87.2 vs 84.6 TFLOP/s; 3x3 C=64 at 56x56: 76.4 vs 72.1; other
    // layers within +-2 %), its columns grouped by residue mod the stride
    // (7x7 stride 2: 87.3 vs 83.9 with the columns in plain order)
    a.to = make_taporder(sh.Kw, sh.Kh, sh.Ci, kTapBlock32 > (uint32_t)v.kt ? kTapBlock32 : (uint32_t)v.kt,
                         t.tap_order == Tuning::kLinear, sh.s);
    const int64_t gx = (sh.P + v.bm - 1) / v.bm, gy = (sh.Co + v.cw - 1) / v.cw;
    if (gx * gy > 0x7fffffff)
        return hipErrorInvalidValue;
    a.tg = make_tilegrid(gx, gy, t.tile_linear);
    void *args[] = {&a};
    return hipLaunchKernel(v.f, dim3((uint32_t)(gx * gy)), dim3(v.nt), args, 0, st);
}

}  // namespace im2win
