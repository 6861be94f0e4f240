// fp16 windowed convolution on the matrix cores for windows that are not
// 16-byte aligned (C_i*2 not a multiple of 16, e.g. the 3-channel stem
// layers), staged by strip segment (Sec. III-B..D, Eq. 3, Alg. 1).
//
// The windows of consecutive output columns of one strip are overlapping
// spans of that strip, S = s*K_h*C_i elements apart.  A tile of BN
// consecutive pixels touches at most RMAX strips; for each strip it needs one
// contiguous segment, from the first pixel's window start to the last
// pixel's window start + K_pad.  The kernel loads each segment once, as
// 16-byte granules from the granule that holds its first element
// (buffer_load ... lds: aligned loads, no element loads), keeps all of them in
// LDS for the whole K loop, and reads every pixel's MFMA operand from there at
// its own (2-byte aligned) offset.  The filter, packed stage-major (64-tap
// tiles of C_o_pad contiguous rows), streams through a two-slot ring.
//
// Taps past K: the filter rows are zero there, and the window values past a
// pixel's K taps (which belong to the next pixel) are cleared in registers,
// so they add exactly 0 and a non-finite neighbour cannot leak in.
#include "common.hpp"
#include "epilogue16.hpp"

#include <type_traits>

#include <stdlib.h>
#include <string.h>

namespace im2win {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void *lds_ptr;

constexpr int BK = 64;  // taps per filter stage

struct SegArgs {
    const uint16_t *ws;
    const uint16_t *packed;
    uint16_t *out;
    uint64_t pad_end;  // window tensor bytes plus the transform's zero pad
    uint32_t pk_bytes;
    uint32_t P, K, K_pad, Co, Co_pad, Wo, L, S;
    FastDiv div_Wo;
};

template <int WM_, int WN_, int WGM_, int WGN_, int GMAX_, int RMAX_>
struct SegCfg {
    static constexpr int WM = WM_, WN = WN_, WGM = WGM_, WGN = WGN_;
    static constexpr int NW = WGM * WGN, NT = 64 * NW;
    static constexpr int BM = 32 * WM * WGM, BN = 32 * WN * WGN;
    static constexpr int GMAX = GMAX_;  // 16-byte granules of window segments a tile may need
    static constexpr int RMAX = RMAX_;  // strips a tile may touch
    static constexpr bool SERIAL = false;  // see Serialized
    static constexpr int ASTAGE = BM * 128;        // filter rows of one stage
    static constexpr int IA = BM / 8 / NW;         // filter loads per wave per stage
    static constexpr int IBMAX = GMAX / 64 / NW;   // segment loads per wave, at most
    static_assert(BM % (8 * NW) == 0, "filter blocks split evenly over the waves");
    static_assert(GMAX % (64 * NW) == 0, "segment blocks split evenly over the waves");
    static_assert(GMAX * 16 >= BM * BN * 2, "the epilogue tile fits the segment area");
    static_assert(RMAX >= 2 && RMAX <= 64 && (RMAX & (RMAX - 1)) == 0, "one lane per strip, scanned in log2 steps");
};

// The same tile with the filter ring serialized: a stage's filter loads are
// issued only after every wave has finished with the previous stage, so no
// load is in flight while LDS is read.  Same sums in the same order; a check
// variant for the ring's waits and barriers.
template <class Base>
struct Serialized : Base {
    static constexpr bool SERIAL = true;
};

__device__ inline uint32_t rsw(uint32_t r) { return (r ^ (r >> 3)) & 7u; }

template <int VM>
__device__ inline void wait_vmcnt()
{
    __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4) | (15 << 8));
}

// E: the operand type (F16Op or BF16Op).
template <class C, class E>
struct SegTile {
    typedef typename E::v8 v8;
    __amdgpu_buffer_rsrc_t rf;
    uint32_t aoff[C::IA];  // filter byte offset at stage 0
    uint32_t bb[C::WN];    // LDS byte offset of each of this lane's pixels' window
    uint32_t wave, lane, wm, wn, K, nst, apitch;
    floatx16 acc[C::WM][C::WN];

    __device__ inline void issue_a(uint32_t st, char *slot)
    {
#pragma unroll
        for (int i = 0; i < C::IA; ++i) {
            const uint32_t b = wave + C::NW * i;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rf, (lds_ptr)(slot + 1024 * b), 16, aoff[i] + st * apitch,
                                                     0, 0, 0);
        }
    }

    // 16 bytes of LDS from a 2-byte-aligned offset.  An unaligned ds_read_b128
    // stalls the LDS pipe (~11 cycles per read measured on the 3-channel
    // stem); three aligned 8-byte reads of the span and a byte-align of each
    // dword in registers give the same bytes.
    __device__ static inline void read16(const char *lds, uint32_t o, v8 &dst)
    {
        const uint32_t base = o & ~7u, sh = o & 7u;
        const uint2 a0 = *reinterpret_cast<const uint2 *>(lds + base);
        const uint2 a1 = *reinterpret_cast<const uint2 *>(lds + base + 8);
        const uint2 a2 = *reinterpret_cast<const uint2 *>(lds + base + 16);
        const uint32_t w[6] = {a0.x, a0.y, a1.x, a1.y, a2.x, a2.y};
        const bool hi4 = sh >= 4;
        const uint32_t b = sh & 3u;
        uint32_t out[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t lo = hi4 ? w[i + 1] : w[i], hi = hi4 ? w[i + 2] : w[i + 1];
            out[i] = __builtin_amdgcn_alignbyte(hi, lo, b);
        }
        __builtin_memcpy(&dst, out, 16);
    }

    __device__ inline void compute(uint32_t st, const char *aslot, const char *seg)
    {
        const bool tail = st * BK + BK > K;
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            const uint32_t ch = 2 * ks + (lane >> 5);
            const uint32_t k = st * BK + 8 * ch;  // first of this lane's 8 taps
            v8 af[C::WM], bf[C::WN];
#pragma unroll
            for (int i = 0; i < C::WM; ++i) {
                const uint32_t r = wm * 32 * C::WM + 32 * i + (lane & 31);
                af[i] = *reinterpret_cast<const v8 *>(aslot + r * 128 + 16u * (ch ^ rsw(r)));
            }
#pragma unroll
            for (int j = 0; j < C::WN; ++j) {
                read16(seg, bb[j] + 2 * k, bf[j]);  // a window starts at any element
                if (tail) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (k + e >= K)
                            bf[j][e] = (typename E::elem)0.f;
                }
            }
#pragma unroll
            for (int i = 0; i < C::WM; ++i)
#pragma unroll
                for (int j = 0; j < C::WN; ++j)
                    acc[i][j] = E::mfma(af[i], bf[j], acc[i][j]);
        }
    }
};

template <class C, class E>
__global__ __launch_bounds__(C::NT) void conv_fp16_seg(SegArgs a)
{
    __shared__ __attribute__((aligned(1024))) char r0[C::ASTAGE];
    __shared__ __attribute__((aligned(1024))) char r1[C::ASTAGE];
    // 16 bytes of slack: a fragment read spans up to 8 bytes past its 16
    __shared__ __attribute__((aligned(1024))) char seg[C::GMAX * 16 + 16];

    SegTile<C, E> w;
    const uint32_t tid = threadIdx.x;
    w.lane = tid & 63;
    w.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    __builtin_assume(w.wave < (uint32_t)C::NW);
    w.wm = w.wave / C::WGN;
    w.wn = w.wave % C::WGN;
    w.K = a.K;
    w.nst = a.K_pad / BK;
    const uint32_t p0 = blockIdx.x * C::BN;
    const uint32_t ch0 = blockIdx.y * C::BM;
    const uint32_t q0 = fdiv(p0, a.div_Wo);
    const uint32_t plast = (p0 + C::BN < a.P ? p0 + C::BN : a.P) - 1;

    // Segments: one per strip q0 + t the tile touches (t < RMAX), measured in
    // elements from the start of strip q0 and begun at the granule holding
    // the first pixel's window start; their granules are laid out one after
    // another in `seg`.  Every wave builds the table itself, lane t holding
    // strip t: cnt = its granules, gb = granules of the strips before it, and
    // rel = (first element of its segment) - 8*gb, so that element e of strip
    // run t sits at LDS element e - rel.
    uint32_t cnt = 0, rel = 0;
    if (w.lane < (uint32_t)C::RMAX) {
        const uint32_t q = q0 + w.lane;
        const uint32_t pf = q * a.Wo > p0 ? q * a.Wo : p0;  // first pixel of the tile in strip q
        const uint32_t pe = (q + 1) * a.Wo - 1 < plast ? (q + 1) * a.Wo - 1 : plast;
        if (pf <= pe) {
            const uint32_t s0 = w.lane * a.L + (pf - q * a.Wo) * a.S;
            const uint32_t s1 = w.lane * a.L + (pe - q * a.Wo) * a.S + a.K_pad;
            rel = s0 & ~7u;
            cnt = (s1 - rel + 7) / 8;
        }
    }
    uint32_t inc = cnt;  // inclusive prefix sum over the lanes
#pragma unroll
    for (int d = 1; d < C::RMAX; d <<= 1) {
        const uint32_t v = __shfl_up(inc, d, 64);
        if (w.lane >= (uint32_t)d)
            inc += v;
    }
    rel -= 8 * (inc - cnt);  // unsigned wrap-around is intended
    const uint32_t G = __builtin_amdgcn_readlane(inc, C::RMAX - 1);
    uint32_t gb[C::RMAX];  // first granule of each strip run (wave-uniform)
#pragma unroll
    for (int t = 0; t < C::RMAX; ++t)
        gb[t] = __builtin_amdgcn_readlane(inc - cnt, t);

    const uint64_t tb = (uint64_t)q0 * a.L;
    // granules reach up to 7 elements past a window's end: the zero pad
    // after the window tensor keeps them inside the workspace
    const uint64_t left = a.pad_end - tb * 2;
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.ws + tb, (uint32_t)(left < kMaxRecords ? left : kMaxRecords));
    w.rf = make_rsrc(a.packed + (uint64_t)ch0 * BK, a.pk_bytes - ch0 * (uint32_t)BK * 2u);
    w.apitch = a.Co_pad * (uint32_t)BK * 2u;

    // Segment loads: instruction i of this wave fills granules
    // 64*(wave + NW*i) .. +63; those past G read nothing (zero fill).
#pragma unroll
    for (int i = 0; i < C::IBMAX; ++i) {
        const uint32_t blk = w.wave + C::NW * i;
        if (blk * 64 >= G)
            break;  // uniform: the wave's remaining blocks are all past G
        const uint32_t g = blk * 64 + w.lane;
        uint32_t r = 0;
#pragma unroll
        for (int t = 1; t < C::RMAX; ++t)
            r += g >= gb[t] ? 1u : 0u;
        const uint32_t rl = __shfl(rel, (int)r, 64);
        const uint32_t off = g < G ? (rl + 8 * g) * 2u : kOOB;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr)(seg + 1024 * blk), 16, off, 0, 0, 0);
    }
    // filter loads: lane -> row 8*blk + lane/8, 16-byte chunk (lane%8)^rsw(row)
#pragma unroll
    for (int i = 0; i < C::IA; ++i) {
        const uint32_t blk = w.wave + C::NW * i;
        const uint32_t row = 8 * blk + w.lane / 8;
        const uint32_t c = (w.lane % 8) ^ rsw(row);
        w.aoff[i] = (row * (uint32_t)BK + 8 * c) * 2u;
    }
    // this lane's pixels: LDS offset of the window start
#pragma unroll
    for (int j = 0; j < C::WN; ++j) {
        const uint32_t p = p0 + w.wn * 32 * C::WN + 32 * j + (w.lane & 31);
        // a pixel past P reads from granule 0 (its result is never stored)
        const bool live = p < a.P;
        const uint32_t q = live ? fdiv(p, a.div_Wo) : q0;
        const uint32_t r = q - q0;
        const uint32_t rl = __shfl(rel, (int)r, 64);
        const uint32_t el = r * a.L + (p - q * a.Wo) * a.S;
        w.bb[j] = live ? (el - rl) * 2u : 0u;
    }
#pragma unroll
    for (int i = 0; i < C::WM; ++i)
#pragma unroll
        for (int j = 0; j < C::WN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                w.acc[i][j][e] = 0.f;

    w.issue_a(0, r0);
    // two-slot filter ring: wait for stage st (and, at st = 0, the
    // segments), then load stage st+1 into the other slot, then multiply
    if constexpr (C::SERIAL) {
        for (uint32_t st = 0; st < w.nst; st += 2) {
            wait_vmcnt<0>();
            ring_barrier();
            w.compute(st, r0, seg);
            ring_barrier();
            if (st + 1 < w.nst) {
                w.issue_a(st + 1, r1);
                wait_vmcnt<0>();
                ring_barrier();
                w.compute(st + 1, r1, seg);
                ring_barrier();
                if (st + 2 < w.nst)
                    w.issue_a(st + 2, r0);
            }
        }
    } else {
        for (uint32_t st = 0; st < w.nst; st += 2) {
            wait_vmcnt<0>();
            ring_barrier();
            if (st + 1 < w.nst)
                w.issue_a(st + 1, r1);
            w.compute(st, r0, seg);
            if (st + 1 < w.nst) {
                wait_vmcnt<0>();
                ring_barrier();
                if (st + 2 < w.nst)
                    w.issue_a(st + 2, r0);
                w.compute(st + 1, r1, seg);
            }
        }
    }
    wait_vmcnt<0>();

    store_tile_lds<E, C::WM, C::WN, C::WGM, C::WGN>(w.acc, seg, a.out, a.P, a.Co, p0, ch0, w.wm, w.wn, w.lane,
                                                 tid);
}

struct SegVariant {
    const char *name;
    const void *f[2];  // fp16 and bf16 operands
    int bm, bn, gmax, rmax, nt;
};

template <int WM, int WN, int WGM, int WGN, int GMAX, int RMAX, bool SERIAL = false>
SegVariant seg_variant(const char *name)
{
    using B = SegCfg<WM, WN, WGM, WGN, GMAX, RMAX>;
    using C = typename std::conditional<SERIAL, Serialized<B>, B>::type;
    return SegVariant{name, {(const void *)&conv_fp16_seg<C, F16Op>, (const void *)&conv_fp16_seg<C, BF16Op>}, C::BM,
                      C::BN, GMAX, RMAX, C::NT};
}

const SegVariant *seg_variants(int *n)
{
    // name: channels x pixels per tile
    static const SegVariant v[] = {
        seg_variant<2, 2, 1, 4, 2560, 16>("s64p256"),
        seg_variant<3, 1, 1, 4, 2560, 16>("s96p128"),
        seg_variant<2, 2, 2, 2, 2560, 16>("s128p128"),
        // a 16 KiB segment area (more workgroups per CU) for short windows
        seg_variant<2, 1, 1, 4, 1024, 16>("s64p128g1024"),
        // serialized filter ring (check variant)
        seg_variant<2, 2, 1, 4, 2560, 16, true>("s64p256-serial"),
    };
    *n = (int)(sizeof v / sizeof v[0]);
    return v;
}

// Granules a tile of bn consecutive pixels needs at most.  A tile split into
// `runs` strip runs of c_1 + ... + c_runs = bn pixels needs, per run,
// (c - 1)*S + K_pad elements from a start rounded down by at most 7, i.e. at
// most ((c - 1)*S + K_pad + 14) / 8 granules; summed over the runs that is at
// most ((bn - runs)*S + runs*(K_pad + 14)) / 8.  The number of runs can be
// anything from 1 to runs_max, so the bound takes the largest.
int64_t seg_granules_needed(const Shape &sh, int bn, int64_t runs_max)
{
    int64_t worst = 0;
    for (int64_t runs = 1; runs <= runs_max && runs <= bn; ++runs) {
        const int64_t g = ((bn - runs) * sh.S + runs * (sh.K_pad + 14)) / 8;
        worst = g > worst ? g : worst;
    }
    return worst;
}

}  // namespace

int seg_find(const char *name)
{
    int n;
    const SegVariant *v = seg_variants(&n);
    for (int t = 0; t < n; ++t)
        if (strcmp(name, v[t].name) == 0)
            return t;
    return -1;
}

const char *seg_name(int v)
{
    int n;
    return seg_variants(&n)[v].name;
}

bool seg_fits(const Shape &sh, int pick)
{
    int n;
    const SegVariant *v = seg_variants(&n);
    if (pick < 0 || pick >= n)
        return false;
    if (sh.d != 1)
        return false;  // strip segments assume windows s*K_h*C_i apart
    // strips a tile of bn pixels can touch, wherever it starts in a strip
    const int64_t runs = (v[pick].bn - 1 + sh.Wo - 1) / sh.Wo + 1;
    if (runs > v[pick].rmax || seg_granules_needed(sh, v[pick].bn, runs) > v[pick].gmax)
        return false;
    // byte offsets inside the tile's strips stay below the buffer limit, and
    // pixel indices of the strips after the tile's last one fit 32 bits
    if ((runs * sh.L + sh.K_pad + 8) * 2 >= (int64_t)kMaxRecords)
        return false;
    if (sh.P + (int64_t)v[pick].rmax * sh.Wo >= (int64_t)1 << 32)
        return false;
    return true;
}

int seg_default(const Shape &sh)
{
    if (sh.Ci % 8 == 0)
        return -1;  // 16-byte-aligned windows have their own kernels
    // C_o <= 64: 64 x 128 tiles with a 16 KiB segment area when the
    // segments fit it (five workgroups per CU instead of two: 7x7 s2 C_i=3
    // at 227x227 284 vs 245 TFLOP/s, 3x3 C_i=3 at 224x224 83 vs 79)
    if (sh.Co <= 64 && seg_fits(sh, seg_find("s64p128g1024")))
        return seg_find("s64p128g1024");
    const int pick = sh.Co <= 64 ? 0 : sh.Co <= 96 ? 1 : 2;
    return seg_fits(sh, pick) ? pick : -1;
}

hipError_t launch_conv_fp16_seg(const Shape &sh, int plan, const void *ws, const void *packed,
                                uint16_t *out, hipStream_t st, Op16 op)
{
    int n;
    const SegVariant &v = seg_variants(&n)[plan];
    SegArgs a;
    a.ws = static_cast<const uint16_t *>(ws);
    a.packed = static_cast<const uint16_t *>(packed);
    a.out = out;
    a.pad_end = (uint64_t)sh.pad_end;
    a.pk_bytes = (uint32_t)(sh.Co_pad * sh.K_pad * 2);
    a.P = (uint32_t)sh.P; a.K = (uint32_t)sh.K; a.K_pad = (uint32_t)sh.K_pad;
    a.Co = (uint32_t)sh.Co; a.Co_pad = (uint32_t)sh.Co_pad;
    a.Wo = (uint32_t)sh.Wo; a.L = (uint32_t)sh.L; a.S = (uint32_t)sh.S;
    a.div_Wo = make_fastdiv((uint32_t)sh.Wo);
    void *args[] = {&a};
    dim3 grid((uint32_t)((sh.P + v.bn - 1) / v.bn), (uint32_t)((sh.Co + v.bm - 1) / v.bm));
    return hipLaunchKernel(v.f[op == Op16::BF16], grid, dim3(v.nt), args, 0, st);
}

}  // namespace im2win
