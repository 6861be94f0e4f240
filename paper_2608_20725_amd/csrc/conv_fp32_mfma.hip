// fp32 windowed convolution on the gfx950 matrix cores (an alternate fp32
// path beside the vector-ALU one; Sec. III-C, Eq. 3 computed as the product
// of Alg. 1).
//
// The output is D[j][p] = sum_k F'[j][k] * Wn[p][k] (M = C_o, N = pixels,
// K = K_h*K_w*C_i) in fp32 with v_mfma_f32_32x32x2_f32: fp32 operands, fp32
// accumulation.  Everything around the multiply follows the row-per-pixel
// fp16 kernel: a stage is 32 taps (128 bytes) of the workgroup's BM filter
// rows and BN window rows, fetched with buffer_load ... lds into a ring of
// NS slots, rows XOR-swizzled in 16-byte chunks.
//
// Operands: one 16-byte LDS read gives a lane four consecutive taps of its
// row.  For the 8 taps of chunk pair (2g, 2g+1), lanes 0-31 read chunk 2g and
// lanes 32-63 chunk 2g+1, and MFMA t (t < 4) takes element t of each: it sums
// taps 8g+t and 8g+4+t.  A and B use the same assignment, so the four MFMAs
// cover the eight taps exactly once; only the order of the fp32 additions
// differs from a tap-by-tap sum.
//
// Windows must start on 16-byte boundaries and hold whole 16-byte chunks
// (C_i a multiple of 4); the launcher sends other layers to the vector-ALU
// kernels.
#include "common.hpp"

#include <stdlib.h>
#include <string.h>

namespace im2win {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void *lds_ptr;

constexpr int BK = 32;  // taps per stage (128-byte rows)

struct M32Args {
    const float *ws;      // window tensor
    const float *packed;  // [K_pad/32][C_o_pad][32]
    float *out;
    uint64_t win_bytes;
    uint32_t pk_bytes;
    uint32_t P, K, K_pad, Co, Co_pad, Wo, L;
    WinCols wc;
    TileGrid tg;          // pixel x channel tiles of the 1-D launch
    FastDiv div_Wo;
};

// Filter repack: element (tile, j, t) = F'[j][tile*32 + t] with
// F'[j][(v*K_h + u)*C_i + r] = F[u][v][r][j] (window tap order), zero for
// j >= C_o or a tap past K.  One thread per 16-byte granule.
struct P32Args {
    const float *filt;
    float *packed;
    uint64_t grans;
    uint32_t K, Co, Co_pad, Ci, Kh, Kw;
};

__global__ __launch_bounds__(256) void pack_filter_fp32_mfma(P32Args a)
{
    for (uint64_t g = (uint64_t)blockIdx.x * 256 + threadIdx.x; g < a.grans; g += (uint64_t)gridDim.x * 256) {
        const uint64_t e0 = g * 4;
        const uint32_t t0 = (uint32_t)(e0 % BK);
        const uint64_t q = e0 / BK;
        const uint32_t j = (uint32_t)(q % a.Co_pad);
        const uint32_t tile = (uint32_t)(q / a.Co_pad);
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t k = tile * BK + t0 + e;
            float x = 0.f;
            if (j < a.Co && k < a.K) {
                const uint32_t khci = a.Kh * a.Ci;
                const uint32_t fv = k / khci, rem = k % khci;
                const uint32_t u = rem / a.Ci, r = rem % a.Ci;
                x = a.filt[(((uint64_t)u * a.Kw + fv) * a.Ci + r) * a.Co + j];
            }
            v[e] = x;
        }
        *reinterpret_cast<float4 *>(a.packed + g * 4) = make_float4(v[0], v[1], v[2], v[3]);
    }
}

template <int WM_, int WN_, int WGM_, int WGN_, int NS_>
struct MCfg {
    static constexpr int WM = WM_, WN = WN_, WGM = WGM_, WGN = WGN_, NS = NS_;
    static constexpr int NW = WGM * WGN, NT = 64 * NW;
    static constexpr int BM = 32 * WM * WGM;     // channels per workgroup
    static constexpr int BN = 32 * WN * WGN;     // pixels per workgroup
    static constexpr int ROWS = BM + BN;
    static constexpr int STAGE = ROWS * 128;     // bytes per stage
    static constexpr int BLOCKS = ROWS / 8;      // 1 KiB (8-row) blocks per stage
    static_assert(BLOCKS % NW == 0, "blocks split evenly over the waves");
    static constexpr int I = BLOCKS / NW;        // loads per wave per stage
    static_assert(NS >= 2 && NS <= 3, "ring depth");
    static_assert((NS - 2) * I <= 63, "vmcnt range");
};

template <int VM>
__device__ inline void wait_vmcnt()
{
    __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4) | (15 << 8));
}

// 16-byte chunk c of row r sits in slot c ^ rsw(r): the 16 lanes that read
// one chunk of 16 consecutive rows touch 16 different slots of the 64 banks.
__device__ inline uint32_t rsw(uint32_t r) { return (r ^ (r >> 3)) & 7u; }

template <class C>
struct MTile {
    __amdgpu_buffer_rsrc_t rf, rw;
    uint32_t voff[C::I];    // byte offset of this lane's chunk at tap 0 (kOOB: no pixel)
    uint32_t vtap[C::I];    // first tap of this lane's chunk within a stage
    uint32_t wave, lane, K, nst, apitch, arow, brow;
    floatx16 acc[C::WM][C::WN];

    // Stage s >= nst loads nothing (zero-filled).
    __device__ inline void issue(uint32_t st, char *slot)
    {
        const uint32_t k0 = st * BK;
        const bool past = st >= nst;
#pragma unroll
        for (int j = 0; j < C::I; ++j) {
            const uint32_t b = wave + C::NW * j;
            const bool filt = b < (uint32_t)C::BM / 8;
            uint32_t off = voff[j] + (filt ? st * apitch : 4u * k0);
            if (past || (!filt && k0 + vtap[j] >= K))
                off = kOOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(filt ? rf : rw, (lds_ptr)(slot + 1024 * b), 16, off, 0, 0, 0);
        }
    }

    __device__ inline void frags(const char *slot, int g, floatx4 (&af)[C::WM], floatx4 (&bf)[C::WN])
    {
        const uint32_t ch = 2 * g + (lane >> 5);
#pragma unroll
        for (int i = 0; i < C::WM; ++i) {
            const uint32_t r = arow + 32 * i;
            af[i] = *reinterpret_cast<const floatx4 *>(slot + r * 128 + 16u * (ch ^ rsw(r)));
        }
#pragma unroll
        for (int j = 0; j < C::WN; ++j) {
            const uint32_t r = brow + 32 * j;
            bf[j] = *reinterpret_cast<const floatx4 *>(slot + r * 128 + 16u * (ch ^ rsw(r)));
        }
    }

    // The four chunk pairs of a stage; the next pair's operands are read
    // before the current pair's 4*WM*WN matrix operations.
    __device__ inline void compute(const char *slot)
    {
        floatx4 af[2][C::WM], bf[2][C::WN];
        frags(slot, 0, af[0], bf[0]);
#pragma unroll
        for (int g = 0; g < BK / 8; ++g) {
            if (g + 1 < BK / 8)
                frags(slot, g + 1, af[(g + 1) & 1], bf[(g + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int i = 0; i < C::WM; ++i)
#pragma unroll
                    for (int j = 0; j < C::WN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[g & 1][i][t], bf[g & 1][j][t],
                                                                         acc[i][j], 0, 0, 0);
        }
    }

    // Ring slots are separate LDS arrays named at compile time, so reading
    // the current slot does not wait for the loads landing in the next.
    template <int N>
    __device__ inline void step(uint32_t st, char (&cur)[N], char (&next)[N])
    {
        wait_vmcnt<(C::NS - 2) * C::I>();
        ring_barrier();
        issue(st + C::NS - 1, next);
        if (st < nst)
            compute(cur);
    }
};

template <class C>
__global__ __launch_bounds__(C::NT) void conv_fp32_mfma(M32Args a)
{
    constexpr int S2 = C::NS > 2 ? C::STAGE : 1024;
    __shared__ __attribute__((aligned(1024))) char r0[C::STAGE];
    __shared__ __attribute__((aligned(1024))) char r1[C::STAGE];
    __shared__ __attribute__((aligned(1024))) char r2[S2];
    __shared__ uint32_t rowoff[C::BN];

    MTile<C> w;
    const uint32_t tid = threadIdx.x;
    w.lane = tid & 63;
    w.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    __builtin_assume(w.wave < (uint32_t)C::NW);
    w.K = a.K;
    w.nst = a.K_pad / BK;
    const uint32_t wm = w.wave / C::WGN, wn = w.wave % C::WGN;
    uint32_t tx, ty;
    a.tg.tile(tx, ty);
    const uint32_t p0 = tx * C::BN;
    const uint32_t ch0 = ty * C::BM;

    // windows from the strip of p0 on; the packed filter from row ch0 of tile 0
    const uint32_t q0 = fdiv(p0, a.div_Wo);
    const uint64_t tb = (uint64_t)q0 * a.L;
    const uint64_t left = a.win_bytes - tb * 4;
    w.rw = make_rsrc(a.ws + tb, (uint32_t)(left < kMaxRecords ? left : kMaxRecords));
    w.rf = make_rsrc(a.packed + (uint64_t)ch0 * BK, a.pk_bytes - ch0 * (uint32_t)BK * 4u);
    w.apitch = a.Co_pad * (uint32_t)BK * 4u;
    for (uint32_t t = tid; t < (uint32_t)C::BN; t += C::NT) {
        const uint32_t p = p0 + t;
        uint32_t off = 0;
        if (p < a.P) {
            const uint32_t q = fdiv(p, a.div_Wo);
            off = (q - q0) * a.L + a.wc.start(p - q * a.Wo);
        }
        rowoff[t] = off;
    }
    __syncthreads();

    // Lane L of a load fills LDS slot L & 7 of row 8*block + L/8 with chunk
    // (L & 7) ^ rsw(row) of that row (rows counted from the first filter row).
    const uint32_t rib = w.lane >> 3, slot = w.lane & 7;
#pragma unroll
    for (int j = 0; j < C::I; ++j) {
        const uint32_t b = w.wave + C::NW * j;
        if (b < (uint32_t)C::BM / 8) {
            const uint32_t row = 8 * b + rib;
            const uint32_t c = slot ^ rsw(row);
            w.voff[j] = row * (uint32_t)BK * 4u + 16u * c;
            w.vtap[j] = 4 * c;
        } else {
            const uint32_t row = 8 * (b - C::BM / 8) + rib;
            const uint32_t c = slot ^ rsw(C::BM + row);
            w.voff[j] = (p0 + row < a.P) ? rowoff[row] * 4u + 16u * c : kOOB;
            w.vtap[j] = 4 * c;
        }
    }
    w.arow = wm * 32 * C::WM + (w.lane & 31);
    w.brow = C::BM + wn * 32 * C::WN + (w.lane & 31);
#pragma unroll
    for (int i = 0; i < C::WM; ++i)
#pragma unroll
        for (int j = 0; j < C::WN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                w.acc[i][j][e] = 0.f;

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
    wait_vmcnt<0>();  // no load may still be writing LDS when the workgroup ends

    // Lane holds pixel pb + 32*j + (lane & 31) and, for accumulator element e
    // of block (i, j), channel cb + 32*i + 8*(e/4) + 4*(lane/32) + e%4: four
    // consecutive channels per 16-byte store.
    const uint32_t pb = p0 + wn * 32 * C::WN, cb = ch0 + wm * 32 * C::WM;
#pragma unroll
    for (int j = 0; j < C::WN; ++j) {
        const uint32_t p = pb + 32 * j + (w.lane & 31);
        if (p >= a.P)
            continue;
        float *o = a.out + (uint64_t)p * a.Co;
#pragma unroll
        for (int i = 0; i < C::WM; ++i) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const uint32_t c = cb + 32 * i + 8 * g + 4 * (w.lane >> 5);
                const floatx16 &v = w.acc[i][j];
                if (c + 3 < a.Co && (a.Co & 3) == 0) {
                    *reinterpret_cast<float4 *>(o + c) =
                        make_float4(v[4 * g], v[4 * g + 1], v[4 * g + 2], v[4 * g + 3]);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (c + e < a.Co)
                            o[c + e] = v[4 * g + e];
                }
            }
        }
    }
}

struct MVariant {
    const char *name;
    const void *f;
    int bm, bn, nt;
};

template <int WM, int WN, int WGM, int WGN, int NS>
MVariant m_variant(const char *name)
{
    using C = MCfg<WM, WN, WGM, WGN, NS>;
    return MVariant{name, (const void *)&conv_fp32_mfma<C>, C::BM, C::BN, C::NT};
}

const MVariant *m_variants(int *n)
{
    // channels x pixels per workgroup, ring slots
    static const MVariant v[] = {
        m_variant<2, 2, 2, 2, 2>("c128p128s2"),
        m_variant<2, 2, 1, 4, 2>("c64p256s2"),
        m_variant<1, 2, 1, 4, 2>("c32p256s2"),
        // smaller tiles for layers with few output pixels
        m_variant<1, 2, 2, 2, 2>("c64p128s2"),
        m_variant<1, 1, 1, 4, 2>("c32p128s2"),
    };
    *n = (int)(sizeof v / sizeof v[0]);
    return v;
}

int64_t co_pad_mfma(int64_t Co) { return round_up(Co, 128); }
int64_t k_pad_mfma(int64_t K) { return round_up(K, BK); }

}  // namespace

bool fp32_mfma_ok(const Shape &sh)
{
    // whole 16-byte chunks per window, 31-bit offsets into the packed filter,
    // and every window byte offset of a 256-pixel tile (its strips plus one
    // window) below the out-of-range marker
    const int64_t strips_per_tile = (256 - 1) / sh.Wo + 2;
    return sh.Ci % 4 == 0 && co_pad_mfma(sh.Co) * k_pad_mfma(sh.K) * 4 < (int64_t)kMaxRecords &&
           (strips_per_tile * sh.L + k_pad_mfma(sh.K)) * 4 < (int64_t)kOOB;
}

int64_t fp32_mfma_packed_bytes(const Shape &sh) { return co_pad_mfma(sh.Co) * k_pad_mfma(sh.K) * 4; }

int mfma32_find(const char *name)
{
    int n;
    const MVariant *v = m_variants(&n);
    for (int t = 0; t < n; ++t)
        if (strcmp(name, v[t].name) == 0)
            return t;
    return -1;
}

const char *mfma32_name(int v)
{
    int n;
    return m_variants(&n)[v].name;
}

int mfma32_default(const Shape &sh)
{
    int n;
    const MVariant *v = m_variants(&n);
    // The largest tile whose grid gives every CU two workgroups (512), else
    // the one with the most workgroups: on few-pixel layers the matrix cores
    // otherwise sit idle (3x3 C=512 at 7x7: 100 tiles of 128 x 128).
    auto tiles = [&](const MVariant &t) { return ((sh.P + t.bn - 1) / t.bn) * ((sh.Co + t.bm - 1) / t.bm); };
    if (sh.Co <= 32)
        return 2;
    if (sh.Co <= 64)
        return tiles(v[1]) >= 512 ? 1 : 3;
    return tiles(v[0]) >= 512 ? 0 : tiles(v[3]) >= 512 ? 3 : 4;
}

hipError_t launch_conv_fp32_mfma(const Shape &sh, const Plan32 &plan, const Tuning &t, const float *filt,
                                 void *packed, float *out, const void *ws, hipStream_t st)
{
    P32Args p;
    p.filt = filt;
    p.packed = static_cast<float *>(packed);
    p.K = (uint32_t)sh.K;
    p.Co = (uint32_t)sh.Co;
    p.Co_pad = (uint32_t)co_pad_mfma(sh.Co);
    p.Ci = (uint32_t)sh.Ci; p.Kh = (uint32_t)sh.Kh; p.Kw = (uint32_t)sh.Kw;
    p.grans = (uint64_t)p.Co_pad * k_pad_mfma(sh.K) / 4;
    uint64_t blocks = (p.grans + 255) / 256;
    if (blocks > 65536)
        blocks = 65536;
    void *pargs[] = {&p};
    hipError_t e = hipLaunchKernel((const void *)&pack_filter_fp32_mfma, dim3((uint32_t)blocks), dim3(256), pargs,
                                   0, st);
    if (e != hipSuccess)
        return e;

    int n;
    const MVariant *v = m_variants(&n);
    const int pick = plan.v;
    M32Args a;
    a.ws = static_cast<const float *>(ws);
    a.packed = p.packed;
    a.out = out;
    a.win_bytes = (uint64_t)sh.win_bytes;
    a.pk_bytes = (uint32_t)fp32_mfma_packed_bytes(sh);
    a.P = (uint32_t)sh.P; a.K = (uint32_t)sh.K; a.K_pad = (uint32_t)k_pad_mfma(sh.K);
    a.Co = (uint32_t)sh.Co; a.Co_pad = p.Co_pad;
    a.Wo = (uint32_t)sh.Wo; a.L = (uint32_t)sh.L;
    a.wc = make_wincols(sh);
    a.div_Wo = make_fastdiv((uint32_t)sh.Wo);
    const int64_t gx = (sh.P + v[pick].bn - 1) / v[pick].bn, gy = (sh.Co + v[pick].bm - 1) / v[pick].bm;
    if (gx * gy > 0x7fffffff)
        return hipErrorInvalidValue;
    a.tg = make_tilegrid(gx, gy, t.tile_linear);
    void *args[] = {&a};
    return hipLaunchKernel(v[pick].f, dim3((uint32_t)(gx * gy)), dim3(v[pick].nt), args, 0, st);
}

}  // namespace im2win
