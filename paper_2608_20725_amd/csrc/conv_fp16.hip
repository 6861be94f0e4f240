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
#include "epilogue16.hpp"

#include <stdlib.h>
#include <string.h>

namespace im2win {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BK = 64;       // taps per stage
constexpr int LDK = BK + 8;  // halves per LDS row: 144 bytes, offsets rows across banks

// How the row-per-pixel register-staged kernel (the one for windows that are
// not 16-byte aligned) loads a 16-byte granule of window taps: one unaligned
// load or eight element loads.  The unaligned load measured faster for long
// windows (K = 363: 248 vs 195 TFLOP/s) and slower for short ones (K = 27:
// 32 vs 41), so the element loads stay for K < 128.
constexpr int kLoadUnaligned = 1, kLoadElems = 2;

struct C16Args {
    const uint16_t *ws;      // window tensor (16-bit elements)
    const uint16_t *packed;  // F' [Co_pad][K_pad]
    uint16_t *out;
    uint64_t win_bytes;
    uint32_t P, K, K_pad, Co, Co_pad, Wo, L;
    WinCols wc;              // window start of an output column in its strip
    uint32_t pk_bytes;       // bytes of the packed filter
    TileGrid tg;             // pixel x channel tiles of the 1-D launch
    FastDiv div_Wo;
    TapOrder to;             // order of the row kernel's 64-tap stages
    // K split (row kernel): block b works on tile b % ntiles over stages
    // z*spl .. z*spl+spl-1, z = b / ntiles; with ks > 1 each block stores its
    // fp32 partial tile in `part` and split_sum adds the ks partials of every
    // output afterwards.
    float *part;
    uint32_t ks, spl, ntiles;
};

// ---------------------------------------------------------------------------
// Filter repack (window order, zero-padded).  Element (j, c, t) of the packed
// filter is F'[j][c*tlen + t] (tap k = (v*K_h + u)*C_i + r of filter column
// j) for t < tlen and j < C_o, else 0, stored at
//     ((t / TB * nv + c) * C_o_pad + j) * TB + t % TB:
// tiles of TB taps, and within a tile all C_o_pad rows of slice c one after
// the other.  A stage of a kernel that consumes TB taps at a time then finds
// its filter rows as one contiguous run, which buffer_load ... lds streams
// about twice as fast as rows scattered K_pad apart.  Layouts in use:
//   row-per-pixel pipelined kernel: nv = 1, tlen = K, tpad = K_pad, TB = 64;
//   column-staged kernel: nv = K_w, tlen = K_h*C_i, tpad = T_pad, TB = its
//     stage depth;
//   register-staged kernel: nv = 1, tlen = K, TB = tpad = K_pad, i.e. plain
//     [C_o_pad][K_pad].
// A lane packs one 8 x 8 block: channels j0 .. j0+7 of 8 consecutive taps
// t0 .. t0+7 of slice c.  It reads the 8 taps' filter rows 16 bytes at a
// time (8 channels), the 8 lanes of a tap reading one 128-byte run of C_o,
// transposes the block in registers, and writes 8 granules (one per
// channel), the 8 lanes of a channel block writing one run of packed row.
// Filters whose rows are not whole 16-byte pieces (C_o % 8; the entry points
// take only 16-byte aligned bases) are read element by element.  TB and tpad
// are multiples of 64, so a block never straddles a tile.
struct PackArgs {
    const uint16_t *filt;
    uint16_t *packed;
    uint32_t nv, tlen, tpad, tb, Co, Co_pad, Ci, Kh, Kw;
    uint32_t ntg, njb;    // 8-tap groups per slice (tpad/8), 8-channel blocks (Co_pad/8)
    uint32_t ntgw, njbw;  // waves along tap groups and channel blocks (8 of each per wave)
    uint32_t units;       // nv * ntgw * njbw waves
    uint32_t vec;         // rows are whole 16-byte pieces (C_o % 8 == 0)
    FastDiv div_khci, div_ci, div_tb;
};

__global__ __launch_bounds__(256) void pack_filter_fp16(PackArgs a)
{
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t unit = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (unit >= a.units)
        return;
    const uint32_t jh = unit % a.njbw, rest = unit / a.njbw;
    const uint32_t th = rest % a.ntgw, c = rest / a.ntgw;
    const uint32_t tg = th * 8 + (lane & 7), jb = jh * 8 + (lane >> 3);
    if (tg >= a.ntg || jb >= a.njb)
        return;
    const uint32_t t0 = tg * 8, j0 = jb * 8;
    const uint32_t khci = a.Kh * a.Ci;
    u32x4 x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const uint32_t t = t0 + e;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (t < a.tlen && j0 < a.Co) {
            // tap k of window order -> filter row (u, v, r) of [K_h][K_w][C_i]
            const uint32_t k = c * a.tlen + t;
            const uint32_t col = fdiv(k, a.div_khci), rem = k - col * khci;
            const uint32_t u = fdiv(rem, a.div_ci), r = rem - u * a.Ci;
            const uint16_t *src = a.filt + (((uint64_t)u * a.Kw + col) * a.Ci + r) * a.Co + j0;
            if (a.vec && j0 + 8 <= a.Co) {
                v = *reinterpret_cast<const u32x4 *>(src);
            } else {
                uint32_t h[8];
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    h[q] = j0 + q < a.Co ? src[q] : 0u;
#pragma unroll
                for (int d = 0; d < 4; ++d)
                    v[d] = h[2 * d] | (h[2 * d + 1] << 16);
            }
        }
        x[e] = v;
    }
    const uint32_t tt = fdiv(t0, a.div_tb), tr = t0 - tt * a.tb;
    uint16_t *dst = a.packed + ((uint64_t)(tt * a.nv + c) * a.Co_pad + j0) * a.tb + tr;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        // channel j0+q: half q%2 of dword q/2 of each tap's piece
        u32x4 o;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            const uint32_t lo = (x[2 * d][q / 2] >> (16 * (q % 2))) & 0xffffu;
            const uint32_t hi = (x[2 * d + 1][q / 2] >> (16 * (q % 2))) & 0xffffu;
            o[d] = lo | (hi << 16);
        }
        *reinterpret_cast<u32x4 *>(dst + (uint64_t)q * a.tb) = o;
    }
}

// Epilogue shared by both kernels.  D[ch][px] of one wave: lane holds pixel
// pbase + 32*j + (lane & 31) and, for accumulator element e of block (i, j),
// channel chbase + 32*i + 8*(e/4) + 4*(lane/32) + e%4.  Each sum is rounded to
// fp16 once (nearest-even) and four consecutive channels go out as 8 bytes.
template <class E, int WM, int WN>
__device__ inline void store_tile(const floatx16 (&acc)[WM][WN], const C16Args &a, uint32_t pbase,
                                  uint32_t chbase, uint32_t lane)
{
#pragma unroll
    for (int j = 0; j < WN; ++j) {
        const uint32_t p = pbase + 32 * j + (lane & 31);
        if (p >= a.P)
            continue;
        uint16_t *o = a.out + (uint64_t)p * a.Co;
#pragma unroll
        for (int i = 0; i < WM; ++i) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const uint32_t c = chbase + 32 * i + 8 * g + 4 * (lane >> 5);
                uint32_t h[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    h[e] = E::bits(acc[i][j][4 * g + e]);
                if (c + 3 < a.Co && (a.Co & 3) == 0) {
                    *reinterpret_cast<uint2 *>(o + c) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (c + e < a.Co)
                            o[c + e] = (uint16_t)h[e];
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
template <int WM, int WN, int WGM, int WGN, int LM>
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
template <int WM, int WN, int WGM, int WGN, int LM>
struct Stage16 {
    using C = Cfg<WM, WN, WGM, WGN, LM>;
    u32x4 fr[C::FPT], wr[C::WPT];

    __device__ inline void load(__amdgpu_buffer_rsrc_t rs, const uint16_t *wsb, const uint32_t *rowoff,
                                const uint16_t *fb, uint32_t p0, uint32_t k0, const C16Args &a)
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
            if (LM == kLoadElems) {
                uint32_t h[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    h[e] = ld_b16(rs, (ok && k + e < a.K) ? base + 2u * e : kOOB);
                wr[j] = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                              h[6] | (h[7] << 16)};
            } else {
                // One unaligned 16-byte load (gfx950 runs with unaligned
                // global access enabled; the zero pad after the window tensor
                // keeps the last load inside the workspace), then the taps
                // past K are cleared.
                u32x4 v = {0u, 0u, 0u, 0u};
                if (ok && k < a.K) {
                    __builtin_memcpy(&v, reinterpret_cast<const char *>(wsb) + base, 16);
                    const uint32_t nv = a.K - k;  // taps of this granule inside K
#pragma unroll
                    for (int d = 0; d < 4; ++d)
                        v[d] &= ((uint32_t)(2 * d) < nv ? 0xffffu : 0u) |
                                ((uint32_t)(2 * d + 1) < nv ? 0xffff0000u : 0u);
                }
                wr[j] = v;
            }
        }
    }

    __device__ inline void store(uint16_t (*Fs)[LDK], uint16_t (*Ws)[LDK])
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

template <class E, int WM, int WN, int WGM, int WGN, int LM>
__global__ __launch_bounds__(64 * WGM * WGN) void conv_fp16_kernel(C16Args a)
{
    typedef typename E::v8 v8;
    using C = Cfg<WM, WN, WGM, WGN, LM>;
    // raw 16-bit operand bits
    __shared__ __attribute__((aligned(16))) uint16_t Fs[2][C::BMc][LDK];
    __shared__ __attribute__((aligned(16))) uint16_t Ws[2][C::BNp][LDK];
    __shared__ uint32_t rowoff[C::BNp];

    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63;
    const uint32_t wave = tid >> 6;
    const uint32_t wm = wave / WGN, wn = wave % WGN;
    uint32_t tx, ty;
    a.tg.tile(tx, ty);
    const uint32_t p0 = tx * C::BNp;
    const uint32_t ch0 = ty * C::BMc;

    const uint32_t q0 = fdiv(p0, a.div_Wo);
    const uint64_t tb_elem = (uint64_t)q0 * a.L;
    const uint64_t left = a.win_bytes - tb_elem * 2;
    const uint16_t *wsb = a.ws + tb_elem;
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(wsb, (uint32_t)(left < kMaxRecords ? left : kMaxRecords));
    for (uint32_t t = tid; t < C::BNp; t += C::NT) {
        const uint32_t p = p0 + t;
        uint32_t off = 0;
        if (p < a.P) {
            const uint32_t q = fdiv(p, a.div_Wo);
            off = (q - q0) * a.L + a.wc.start(p - q * a.Wo);
        }
        rowoff[t] = off;
    }
    __syncthreads();

    const uint16_t *fb = a.packed + (uint64_t)ch0 * a.K_pad;
    Stage16<WM, WN, WGM, WGN, LM> stg;

    floatx16 acc[WM][WN];
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                acc[i][j][e] = 0.f;

    const uint32_t nst = a.K_pad / BK;
    stg.load(rs, wsb, rowoff, fb, p0, 0, a);
    stg.store(Fs[0], Ws[0]);
    __syncthreads();

    const uint32_t arow = wm * 32 * WM + (lane & 31);
    const uint32_t brow = wn * 32 * WN + (lane & 31);
    const uint32_t kl = 8 * (lane >> 5);
    for (uint32_t st = 0; st < nst; ++st) {
        const int buf = st & 1;
        if (st + 1 < nst)
            stg.load(rs, wsb, rowoff, fb, p0, (st + 1) * BK, a);
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            v8 af[WM], bf[WN];
#pragma unroll
            for (int i = 0; i < WM; ++i)
                af[i] = *reinterpret_cast<const v8 *>(&Fs[buf][arow + 32 * i][16 * ks + kl]);
#pragma unroll
            for (int j = 0; j < WN; ++j)
                bf[j] = *reinterpret_cast<const v8 *>(&Ws[buf][brow + 32 * j][16 * ks + kl]);
#pragma unroll
            for (int i = 0; i < WM; ++i)
#pragma unroll
                for (int j = 0; j < WN; ++j)
                    acc[i][j] = E::mfma(af[i], bf[j], acc[i][j]);
        }
        if (st + 1 < nst)
            stg.store(Fs[buf ^ 1], Ws[buf ^ 1]);
        __syncthreads();
    }

    if constexpr (epilogue16_bytes<C::BMc, C::BNp>() <= (int)sizeof(Ws)) {
        store_tile_lds<E, WM, WN, WGM, WGN>(acc, reinterpret_cast<char *>(&Ws[0][0][0]), a.out, a.P, a.Co, p0, ch0,
                                         wm, wn, lane, tid);
        return;
    }
    store_tile<E, WM, WN>(acc, a, p0 + wn * 32 * WN, ch0 + wm * 32 * WM, lane);
}

// ---------------------------------------------------------------------------
// Pipelined kernel for 16-byte-aligned windows (C_i a multiple of 8).
//
// A stage holds 64 taps of the workgroup's BMc filter rows and BNp window
// rows, 128 bytes per row, in LDS.  Stages are fetched with
// buffer_load_dwordx4 ... lds, which writes each lane's 16 bytes straight to
// LDS at base + 16 * lane: one wave instruction fills 8 consecutive rows.  An
// NSTAGE-deep ring keeps NSTAGE-1 stages in flight while the matrix cores
// work on the current one (the double buffering and asynchronous copy of
// Alg. 1, with a deeper ring because HBM latency on this part is long
// compared with one stage of MFMA work).  Rows past the last pixel and taps
// past K use an out-of-range offset, for which the load writes zeros.
//
// LDS rows are XOR-swizzled: 16-byte chunk c of row r sits in slot
// c ^ rsw(r), rsw(r) = (r ^ (r >> 3)) & 7, so the 16 lanes that read one
// chunk of 16 consecutive rows for an MFMA operand touch 16 different 16-byte
// slots of the 64 banks.  (With c ^ (r & 7), rows r and r+8 collided: bank
// conflicts measured at 3.8x the LDS instruction cycles.)
template <int WM, int WN, int WGM, int WGN, int NSTAGE>
struct PipeCfg {
    static constexpr int NW = WGM * WGN;      // waves per workgroup
    static constexpr int NT = 64 * NW;
    static_assert(NW == 4 || NW == 8, "four or eight waves per workgroup");
    static constexpr int BMc = 32 * WM * WGM;
    static constexpr int BNp = 32 * WN * WGN;
    static constexpr int ROWS = BMc + BNp;
    static constexpr int STAGE = ROWS * 128;  // bytes per stage
    static constexpr int BLOCKS = ROWS / 8;   // 8-row (1 KiB) blocks per stage
    static_assert(BLOCKS % NW == 0, "blocks split evenly over the waves");
    static constexpr int I = BLOCKS / NW;     // load instructions per wave per stage
    static_assert((BMc / 8) % NW == 0, "filter blocks split evenly over the waves");
    static constexpr int IF = BMc / 8 / NW;   // of which filter blocks
    static_assert(NSTAGE == 1 || (NSTAGE - 2) * I <= 63, "vmcnt range");
    static constexpr int LDS = NSTAGE * STAGE;
};

template <int VM>
__device__ inline void wait_vmcnt()
{
    // s_waitcnt with vmcnt = VM, expcnt and lgkmcnt left alone
    __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4) | (15 << 8));
}

typedef __attribute__((address_space(3))) void *lds_ptr;

__device__ inline uint32_t rsw(uint32_t r) { return (r ^ (r >> 3)) & 7u; }

// State of one workgroup of the pipelined kernel.  Ring slots are separate
// LDS arrays and every step of the main loop names its slot at compile time,
// so the compiler can tell that reading one slot does not depend on the
// loads still landing in the others (and inserts no wait for them).
template <class E, int WM, int WN, int WGM, int WGN, int NSTAGE>
struct Pipe {
    using C = PipeCfg<WM, WN, WGM, WGN, NSTAGE>;
    typedef typename E::v8 v8;
    __amdgpu_buffer_rsrc_t rf, rw;
    uint32_t voff[C::I];    // byte offset of this lane's chunk at tap 0 (kOOB: no pixel)
    uint32_t vchunk[C::I];  // first tap of this lane's chunk within a stage
    uint32_t wave, lane, K, nst, apitch;
    uint32_t sb;  // first stage of this block's K range
    TapOrder to;
    uint32_t arow, brow;
    floatx16 acc[WM][WN];

    // Stage s >= nst (past the end of K) loads nothing: every offset is out of
    // range and the slot is filled with zeros.
    // Offsets of stage s's loads.  A window chunk whose first tap (within
    // the stage) is at or past `lim` reads nothing: every chunk of a stage
    // past the end, the chunks past K in the last stage.  Filter rows: taps
    // k0 .. k0+63 are tile k0/64 of the packed filter (apitch bytes each);
    // window rows: taps k0 .. k0+63.
    struct StageLoads {
        uint32_t lim, fadd, wadd;
        bool past;
    };
    __device__ inline StageLoads stage_loads(uint32_t s) const
    {
        // first tap of the stage (column order only when every stage is
        // whole: K_h*C_i a multiple of 64)
        const uint32_t k0 = to.map((s + sb) * BK);
        const bool past = s >= nst;
        return StageLoads{past ? 0u : k0 + BK <= K ? 0xffffffffu : k0 < K ? K - k0 : 0u, (k0 / BK) * apitch,
                          2u * k0, past};
    }

    // Load j of a stage (j < I): block wave + NW*j.  The first IF loads of
    // every wave fill filter blocks, so which buffer a load reads is known
    // at compile time and the offsets are plain selects.
    __device__ inline void issue_one(int j, const StageLoads &sl, char *stage)
    {
        const uint32_t b = wave + C::NW * j;
        if (j < C::IF) {
            const uint32_t off = sl.past ? kOOB : voff[j] + sl.fadd;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rf, (lds_ptr)(stage + 1024 * b), 16, off, 0, 0, 0);
        } else {
            const uint32_t off = vchunk[j] >= sl.lim ? kOOB : voff[j] + sl.wadd;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr)(stage + 1024 * b), 16, off, 0, 0, 0);
        }
    }

    __device__ inline void issue(uint32_t s, char *stage)
    {
        const StageLoads sl = stage_loads(s);
#pragma unroll
        for (int j = 0; j < C::I; ++j)
            issue_one(j, sl, stage);
    }

    // Fragments of k-step ks of the stage.
    __device__ inline void frags(const char *stage, int ks, v8 (&af)[WM], v8 (&bf)[WN])
    {
        const uint32_t ch = 2 * ks + (lane >> 5);
#pragma unroll
        for (int i = 0; i < WM; ++i) {
            const uint32_t r = arow + 32 * i;
            af[i] = *reinterpret_cast<const v8 *>(stage + r * 128 + 16u * (ch ^ rsw(r)));
        }
#pragma unroll
        for (int j = 0; j < WN; ++j) {
            const uint32_t r = brow + 32 * j;
            bf[j] = *reinterpret_cast<const v8 *>(stage + r * 128 + 16u * (ch ^ rsw(r)));
        }
    }

    // All k-steps of one stage; the fragments of step ks+1 are read before
    // the matrix operations of step ks, so their LDS latency runs under them
    // (with about one wave per SIMD nothing else would hide it).  With
    // `nslot` set, the loads of stage `ns` into it are issued a few at a time
    // after the matrix operations of the first k-steps, so that their issue
    // runs while the matrix cores work instead of before the first multiply.
    __device__ inline void compute(const char *stage, uint32_t ns = 0, char *nslot = nullptr)
    {
        constexpr int KS = BK / 16;
        // loads per k-step: spread over all k-steps (measured against the
        // same loads packed into the first two k-steps or the first one: 3x3
        // C = 512 at 7x7, 424 against 422 / 424 TFLOP/s; 3x3 C = 256 at
        // 12x12, 685 against 676 / 661; all of them issued before the first
        // multiply gave 390 and 668)
        constexpr int LPS = (C::I + KS - 1) / KS;
        StageLoads sl{};
        if (nslot)
            sl = stage_loads(ns);
        v8 af[2][WM], bf[2][WN];
        frags(stage, 0, af[0], bf[0]);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (ks + 1 < KS)
                frags(stage, ks + 1, af[(ks + 1) & 1], bf[(ks + 1) & 1]);
            // keep the reads above the matrix operations (the scheduler would
            // otherwise sink them below to reuse the same registers)
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < WM; ++i)
#pragma unroll
                for (int j = 0; j < WN; ++j)
                    acc[i][j] = E::mfma(af[ks & 1][i], bf[ks & 1][j], acc[i][j]);
            if (nslot && ks * LPS < C::I) {
#pragma unroll
                for (int j = ks * LPS; j < (ks + 1) * LPS && j < C::I; ++j)
                    issue_one(j, sl, nslot);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }

    // Stage st sits in slot `cur`: wait for it, then refill the slot freed by
    // stage st-1 (`next`) with stage st+NSTAGE-1, then multiply.  Every step
    // waits for the same count and issues one stage, so the wait is exact
    // without branches; only the multiply is skipped past the last stage.
    // The slots are passed as the LDS arrays themselves so that, once
    // inlined, every access names its array.
    template <int N>
    __device__ inline void step(uint32_t st, char (&cur)[N], char (&next)[N])
    {
        // st < nst: the loops of the kernel run real stages only
        wait_vmcnt<(NSTAGE - 2) * C::I>();
        ring_barrier();
        compute(cur, st + NSTAGE - 1, next);
    }

    // One slot, no double buffering (the ablation of Alg. 1's double
    // buffer): wait for stage st, multiply, and only when every wave is done
    // reading load stage st+1 into the same slot.
    template <int N>
    __device__ inline void step_single(uint32_t st, char (&cur)[N])
    {
        wait_vmcnt<0>();
        ring_barrier();
        compute(cur);
        ring_barrier();
        issue(st + 1, cur);
    }
};

// Partial tile of a block of a K-split launch (K range z of tile `tile`),
// stored in accumulator order: wave w, block (i, j), accumulator quad q, lane
// l at float offset ((w*WM + i)*WN + j)*4 + q)*256 + 4*l of the tile's slot, so
// each store instruction writes 1 KiB contiguously.  split_sum reads them back
// with the same numbering.
template <int WM, int WN>
__device__ inline void split_store(const floatx16 (&acc)[WM][WN], const C16Args &a, uint32_t z, uint32_t tile,
                                   uint32_t wave, uint32_t lane, uint32_t nwaves)
{
    constexpr int WE = WM * WN * 16 * 64;  // floats per wave
    float *dst = a.part + ((uint64_t)z * a.ntiles + tile) * ((uint64_t)nwaves * WE) + (uint64_t)wave * WE;
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                *reinterpret_cast<float4 *>(dst + ((i * WN + j) * 4 + q) * 256 + 4 * lane) =
                    make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
}

// Second kernel of a K-split launch: every output is the sum of its ks
// partials, added in the fixed order z = 0, 1, ..., ks-1 (reproducible run to
// run), rounded to 16 bits once.  One thread per accumulator quad of a tile
// (4 consecutive channels of one pixel).
struct SumArgs {
    const float *part;
    uint16_t *out;
    uint64_t quads;           // ntiles * tile_elems / 4
    uint32_t ks, ntiles, P, Co;
    uint32_t WM, WN, WGN, BMc, BNp, tile_quads;
    TileGrid tg;
};

template <class E>
__global__ __launch_bounds__(256) void split_sum(SumArgs a)
{
    const uint64_t u = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= a.quads)
        return;
    const uint32_t tile = (uint32_t)(u / a.tile_quads), r = (uint32_t)(u - (uint64_t)tile * a.tile_quads);
    const uint32_t wq = a.WM * a.WN * 4 * 64;  // quads per wave
    const uint32_t wave = r / wq, r2 = r - wave * wq;
    const uint32_t lane = r2 & 63, r3 = r2 >> 6, q = r3 & 3, ij = r3 >> 2;
    const uint32_t j = ij % a.WN, i = ij / a.WN;
    const uint32_t wm = wave / a.WGN, wn = wave - wm * a.WGN;
    uint32_t tx, ty;
    a.tg.tile_of(tile, tx, ty);
    const uint32_t p = tx * a.BNp + wn * 32 * a.WN + 32 * j + (lane & 31);
    const uint32_t c = ty * a.BMc + wm * 32 * a.WM + 32 * i + 8 * q + 4 * (lane >> 5);
    if (p >= a.P || c >= a.Co)
        return;
    const uint64_t stride = (uint64_t)a.ntiles * a.tile_quads;
    const float4 *src = reinterpret_cast<const float4 *>(a.part) + u;
    float4 sum = src[0];
    for (uint32_t z = 1; z < a.ks; ++z) {
        const float4 v = src[z * stride];
        sum.x += v.x; sum.y += v.y; sum.z += v.z; sum.w += v.w;
    }
    const uint32_t h[4] = {E::bits(sum.x), E::bits(sum.y), E::bits(sum.z), E::bits(sum.w)};
    uint16_t *o = a.out + (uint64_t)p * a.Co + c;
    if (c + 3 < a.Co && (a.Co & 3) == 0) {
        *reinterpret_cast<uint2 *>(o) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
    } else {
        for (int e = 0; e < 4; ++e)
            if (c + e < a.Co)
                o[e] = (uint16_t)h[e];
    }
}

// Workgroups per CU the compiler is to leave registers for: the one-slot
// four-wave tile (32 KiB of LDS) fits in 128 registers, four workgroups per
// CU, without spilling (72 + 64 accumulation registers unhinted, three per
// CU): 1x1 C=1024 at 14x14, 767 against 700 TFLOP/s.  The other tiles are
// held to fewer workgroups by their LDS.
template <int NW, int NSTAGE>
constexpr int pipe_min_blocks()
{
    return NW == 4 && NSTAGE == 1 ? 4 : 1;
}

template <class E, int WM, int WN, int WGM, int WGN, int NSTAGE>
__global__ __launch_bounds__(64 * WGM * WGN, (pipe_min_blocks<WGM * WGN, NSTAGE>())) void conv_fp16_pipe(C16Args a)
{
    using C = PipeCfg<WM, WN, WGM, WGN, NSTAGE>;
    static_assert(NSTAGE >= 1 && NSTAGE <= 4, "ring depth");
    constexpr int S1 = NSTAGE > 1 ? C::STAGE : 1024;
    constexpr int S2 = NSTAGE > 2 ? C::STAGE : 1024, S3 = NSTAGE > 3 ? C::STAGE : 1024;
    __shared__ __attribute__((aligned(1024))) char r0[C::STAGE];
    __shared__ __attribute__((aligned(1024))) char r1[S1];
    __shared__ __attribute__((aligned(1024))) char r2[S2];
    __shared__ __attribute__((aligned(1024))) char r3[S3];
    __shared__ uint32_t rowoff[C::BNp];

    Pipe<E, WM, WN, WGM, WGN, NSTAGE> w;
    const uint32_t tid = threadIdx.x;
    w.lane = tid & 63;
    w.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    w.K = a.K;
    // this block's tile and K range
    const uint32_t z = blockIdx.x / a.ntiles, tile = blockIdx.x - z * a.ntiles;
    const uint32_t nst_all = a.K_pad / BK;
    w.sb = z * a.spl;
    w.nst = w.sb >= nst_all ? 0u : nst_all - w.sb < a.spl ? nst_all - w.sb : a.spl;
    const uint32_t wm = w.wave / WGN, wn = w.wave % WGN;
    uint32_t tx, ty;
    a.tg.tile_of(tile, tx, ty);
    const uint32_t p0 = tx * C::BNp;
    const uint32_t ch0 = ty * C::BMc;

    const uint32_t q0 = fdiv(p0, a.div_Wo);
    const uint64_t tb_elem = (uint64_t)q0 * a.L;
    const uint64_t left = a.win_bytes - tb_elem * 2;
    w.rw = make_rsrc(a.ws + tb_elem, (uint32_t)(left < kMaxRecords ? left : kMaxRecords));
    // the packed filter in 64-tap tiles of C_o_pad rows: row ch0 of tile 0 on
    w.rf = make_rsrc(a.packed + (uint64_t)ch0 * BK, a.pk_bytes - ch0 * (uint32_t)BK * 2u);
    w.apitch = a.Co_pad * (uint32_t)BK * 2u;
    w.to = a.to;
    for (uint32_t t = tid; t < C::BNp; t += C::NT) {
        const uint32_t p = p0 + t;
        uint32_t off = 0;
        if (p < a.P) {
            const uint32_t q = fdiv(p, a.div_Wo);
            off = (q - q0) * a.L + a.wc.start(p - q * a.Wo);
        }
        rowoff[t] = off;
    }
    __syncthreads();

    // Lane L of a load instruction fills LDS slot L & 7 of row 8*block + L/8
    // with 16-byte chunk (L & 7) ^ rsw(row) of that row (row counted from the
    // first filter row of the stage).
    const uint32_t rib = w.lane >> 3, slot = w.lane & 7;
#pragma unroll
    for (int j = 0; j < C::I; ++j) {
        const uint32_t b = w.wave + C::NW * j;
        if (b < (uint32_t)C::BMc / 8) {
            const uint32_t row = 8 * b + rib;
            const uint32_t c = slot ^ rsw(row);
            w.voff[j] = row * (uint32_t)BK * 2u + 16u * c;
            w.vchunk[j] = 8 * c;
        } else {
            const uint32_t row = 8 * (b - C::BMc / 8) + rib;
            const uint32_t c = slot ^ rsw(C::BMc + row);
            w.voff[j] = (p0 + row < a.P) ? rowoff[row] * 2u + 16u * c : kOOB;
            w.vchunk[j] = 8 * c;
        }
    }
    w.arow = wm * 32 * WM + (w.lane & 31);
    w.brow = C::BMc + wn * 32 * WN + (w.lane & 31);
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                w.acc[i][j][e] = 0.f;

    // prologue: stages 0 .. NSTAGE-2 into slots 0 .. NSTAGE-2, then stage st
    // in slot st % NSTAGE
    // (whole rounds of the ring, then the last nst % NSTAGE stages; each
    // step multiplies a real stage and issues the one NSTAGE-1 ahead, which
    // past the end loads zeros)
    w.issue(0, r0);
    uint32_t st = 0;
    if constexpr (NSTAGE == 1) {
        for (; st < w.nst; ++st)
            w.step_single(st, r0);
    } else if constexpr (NSTAGE == 2) {
        for (; st + 2 <= w.nst; st += 2) {
            w.step(st, r0, r1);
            w.step(st + 1, r1, r0);
        }
        if (st < w.nst)
            w.step(st, r0, r1);
    } else if constexpr (NSTAGE == 3) {
        w.issue(1, r1);
        for (; st + 3 <= w.nst; st += 3) {
            w.step(st, r0, r2);
            w.step(st + 1, r1, r0);
            w.step(st + 2, r2, r1);
        }
        if (st < w.nst)
            w.step(st, r0, r2);
        if (st + 1 < w.nst)
            w.step(st + 1, r1, r0);
    } else {
        w.issue(1, r1);
        w.issue(2, r2);
        for (; st + 4 <= w.nst; st += 4) {
            w.step(st, r0, r3);
            w.step(st + 1, r1, r0);
            w.step(st + 2, r2, r1);
            w.step(st + 3, r3, r2);
        }
        if (st < w.nst)
            w.step(st, r0, r3);
        if (st + 1 < w.nst)
            w.step(st + 1, r1, r0);
        if (st + 2 < w.nst)
            w.step(st + 2, r2, r1);
    }
    // no load may still be writing LDS when the workgroup ends
    wait_vmcnt<0>();

    if (a.ks > 1) {
        split_store<WM, WN>(w.acc, a, z, tile, w.wave, w.lane, C::NW);
        return;
    }
    if constexpr (epilogue16_bytes<C::BMc, C::BNp>() <= C::STAGE) {
        store_tile_lds<E, WM, WN, WGM, WGN>(w.acc, r0, a.out, a.P, a.Co, p0, ch0, wm, wn, w.lane, tid);
        return;
    }
    store_tile<E, WM, WN>(w.acc, a, p0 + wn * 32 * WN, ch0 + wm * 32 * WM, w.lane);
}

template <class E, int WM, int WN, int WGM, int WGN>
void pick_regs(bool unaligned_loads, const void **f, int *bm, int *bn)
{
    *f = unaligned_loads ? (const void *)&conv_fp16_kernel<E, WM, WN, WGM, WGN, kLoadUnaligned>
                         : (const void *)&conv_fp16_kernel<E, WM, WN, WGM, WGN, kLoadElems>;
    *bm = 32 * WM * WGM;
    *bn = 32 * WN * WGN;
}

struct PipeVariant {
    const char *name;
    const void *f[2];  // fp16 and bf16 operands
    int bm, bn, nt;
    int wm, wn, wgn;   // wave tile (MFMA blocks) and waves along pixels
};

template <int WM, int WN, int WGM, int WGN, int NS>
PipeVariant pipe_variant(const char *name)
{
    return PipeVariant{name,
                       {(const void *)&conv_fp16_pipe<F16Op, WM, WN, WGM, WGN, NS>,
                        (const void *)&conv_fp16_pipe<BF16Op, WM, WN, WGM, WGN, NS>},
                       32 * WM * WGM, 32 * WN * WGN, 64 * WGM * WGN, WM, WN, WGN};
}

// Tile shapes of the pipelined kernel: channels x pixels per workgroup,
// ring depth.
const PipeVariant *pipe_variants(int *n)
{
    static const PipeVariant v[] = {
        pipe_variant<1, 1, 1, 4, 3>("c32p128s3"),
        pipe_variant<1, 2, 2, 2, 3>("c64p128s3"),
        pipe_variant<2, 2, 2, 2, 2>("c128p128s2"),
        // eight waves, 128 x 64 wave tiles: half the L2 -> LDS traffic per
        // FLOP of the 128 x 128 tiles
        pipe_variant<4, 2, 2, 4, 2>("c256p256s2w8"),
        pipe_variant<2, 2, 2, 4, 2>("c128p256s2w8"),
        // one ring slot: no double buffering (ablation)
        pipe_variant<2, 2, 2, 2, 1>("c128p128s1"),
    };
    *n = (int)(sizeof v / sizeof v[0]);
    return v;
}

}  // namespace

// Layers with C_o >= 128 and at least four 128 x 128 tiles per CU run the
// row-per-pixel kernel with a one-slot ring.  Registers (about 200 per wave)
// hold both ring depths to two workgroups per CU; with one slot each
// workgroup alternates whole stages of loading and multiplying, and the two
// on a CU interleave.  Measured faster there (alternating runs: S7 639 vs
// 601 TFLOP/s with the column-staged kernel, S12 591 vs 547); with fewer
// tiles the two-slot ring wins (S5, S10).
bool fp16_single_slot_rows(const Shape &sh)
{
    const int64_t tiles = ((sh.P + 127) / 128) * ((sh.Co + 127) / 128);
    return sh.Ci % 8 == 0 && sh.Co >= 128 && tiles >= 1024;
}

int pipe_find(const char *name)
{
    int n;
    const PipeVariant *v = pipe_variants(&n);
    for (int t = 0; t < n; ++t)
        if (strcmp(name, v[t].name) == 0)
            return t;
    return -1;
}

const char *pipe_name(int v)
{
    int n;
    return pipe_variants(&n)[v].name;
}

int64_t pipe_tiles(const Shape &sh, int v)
{
    int n;
    const PipeVariant &pv = pipe_variants(&n)[v];
    return ((sh.P + pv.bn - 1) / pv.bn) * ((sh.Co + pv.bm - 1) / pv.bm);
}

int64_t pipe_tile_elems(int v)
{
    int n;
    const PipeVariant &pv = pipe_variants(&n)[v];
    return (int64_t)pv.bm * pv.bn;
}

namespace {

// K split of the 128 x 128 two-slot tile on a layer with at most 128 such
// tiles (fewer than one per CU) and at least 32 stages: the largest ks <= 4
// whose partial tiles keep the whole workspace within the size of the
// layer's im2col matrix; 1 when none does.  Measured on 3x3 C = 512 at 7x7
// (128 images, 100 tiles, 72 stages): unsplit 64 x 128 tiles 331 TFLOP/s,
// 128 x 128 tiles split 2 / 3 / 4 ways 350 / 376 / 408 (split 3 and 4 need
// more workspace than im2col); with more tiles or fewer stages the split's
// second kernel and partial-tile traffic cost more than it gains.
int split128(const Shape &sh)
{
    const int v = pipe_find("c128p128s2");
    const int64_t tiles = pipe_tiles(sh, v), nst = sh.K_pad / BK;
    if (sh.Ci % 8 != 0 || sh.Co < 128 || tiles > 128 || nst < 32)
        return 1;
    const int64_t base = sh.pad_end + sh.Co_pad * sh.Kw * sh.Tp * 2;  // window tensor, pad, packed filter
    const int64_t im2col = sh.P * sh.K * 2;
    for (int ks = 4; ks >= 2; --ks) {
        const int64_t spl = (nst + ks - 1) / ks;
        if ((ks - 1) * spl < nst && base + ks * tiles * pipe_tile_elems(v) * 4 <= im2col)
            return ks;
    }
    return 1;
}

}  // namespace

int pipe_default(const Shape &sh)
{
    // Defaults, measured per layer on MI355X: shapes that leave LDS for
    // two workgroups per CU (32x128, 64x128, 128x128); 64x128 also when a
    // 128x128 grid would give fewer workgroups than CUs (S11: 280 vs 220
    // TFLOP/s); 256x256 over eight waves when its grid fills 128 to 256
    // CUs (cfg4 616 vs 575, S4 670 vs 646; with fewer tiles it starves
    // the chip, with more the second round runs partly empty).
    auto tiles = [&](int64_t bm, int64_t bn) { return ((sh.P + bn - 1) / bn) * ((sh.Co + bm - 1) / bm); };
    if (sh.Co <= 32)
        return pipe_find("c32p128s3");
    if (fp16_single_slot_rows(sh))
        return pipe_find("c128p128s1");
    // too few 128 x 128 tiles to fill the chip: split K over them where the
    // workspace allows, else 64 x 128 tiles
    if (split128(sh) > 1)
        return pipe_find("c128p128s2");
    if (sh.Co <= 64 || tiles(128, 128) < 256)
        return pipe_find("c64p128s3");
    if (tiles(256, 256) >= 128 && tiles(256, 256) <= 256 && sh.Co >= 256)
        return pipe_find("c256p256s2w8");
    return pipe_find("c128p128s2");
}

int pipe_split_default(const Shape &sh, int v)
{
    return v == pipe_find("c128p128s2") ? split128(sh) : 1;
}

hipError_t launch_pack_fp16(const Shape &sh, const Plan16 &p, const uint16_t *filt, void *packed, hipStream_t st,
                            void *split)
{
    (void)split;
    PackArgs a;
    a.filt = filt;
    a.packed = static_cast<uint16_t *>(packed);
    if (p.fam == Fam16::Col) {
        a.nv = (uint32_t)sh.Kw; a.tlen = (uint32_t)(sh.Kh * sh.Ci); a.tpad = (uint32_t)sh.Tp;
        a.tb = (uint32_t)col_stage_taps(p.v);
    } else {
        a.nv = 1; a.tlen = (uint32_t)sh.K; a.tpad = (uint32_t)sh.K_pad;
        // pipelined and segment-staged kernels: 64-tap tiles; register-staged
        // kernel: one tile of K_pad taps
        a.tb = p.fam == Fam16::Regs ? a.tpad : (uint32_t)BK;
    }
    // the column-staged kernel's slices hold C_o rounded up to its tile's
    // channel count (a stage's filter rows are then one contiguous run);
    // the other kernels' tiles use C_o_pad = C_o rounded up to 256
    const int64_t rows = p.fam == Fam16::Col ? col_packed_rows(sh, p.v) : sh.Co_pad;
    a.Co = (uint32_t)sh.Co; a.Co_pad = (uint32_t)rows;
    a.Ci = (uint32_t)sh.Ci; a.Kh = (uint32_t)sh.Kh; a.Kw = (uint32_t)sh.Kw;
    if (a.tb % 8 != 0 || a.tpad % a.tb != 0 || rows % 8 != 0)
        return hipErrorInvalidValue;
    a.ntg = a.tpad / 8; a.njb = (uint32_t)(rows / 8);
    a.ntgw = (a.ntg + 7) / 8; a.njbw = (a.njb + 7) / 8;
    const uint64_t units = (uint64_t)a.nv * a.ntgw * a.njbw;
    if (units > 0xffffffffull - 3)
        return hipErrorInvalidValue;
    a.units = (uint32_t)units;
    a.vec = sh.Co % 8 == 0 ? 1u : 0u;
    a.div_khci = make_fastdiv((uint32_t)(sh.Kh * sh.Ci));
    a.div_ci = make_fastdiv((uint32_t)sh.Ci);
    a.div_tb = make_fastdiv(a.tb);
    const uint64_t blocks = (units + 3) / 4;
    void *args[] = {&a};
    return hipLaunchKernel((const void *)&pack_filter_fp16, dim3((uint32_t)blocks), dim3(256), args, 0, st);
}

hipError_t launch_conv_fp16(const Shape &sh, const Plan16 &p, const Tuning &t, const void *ws,
                            const void *packed, uint16_t *out, hipStream_t st, Op16 op, void *split)
{
    if (p.fam == Fam16::Col)
        return launch_conv_fp16_col(sh, p.v, t, ws, packed, out, st, op);
    if (p.fam == Fam16::Seg)
        return launch_conv_fp16_seg(sh, p.v, ws, packed, out, st, op);
    if (p.fam == Fam16::Stem)
        return launch_conv_fp16_stem(sh, p.v, ws, packed, out, st, op);
    C16Args a;
    a.ws = static_cast<const uint16_t *>(ws);
    a.packed = static_cast<const uint16_t *>(packed);
    a.out = out;
    a.win_bytes = (uint64_t)sh.win_bytes;
    a.P = (uint32_t)sh.P; a.K = (uint32_t)sh.K; a.K_pad = (uint32_t)sh.K_pad;
    a.Co_pad = (uint32_t)sh.Co_pad;
    a.pk_bytes = (uint32_t)(sh.Co_pad * sh.K_pad * 2);  // < 2^31 (checked with the shape)
    a.Co = (uint32_t)sh.Co; a.Wo = (uint32_t)sh.Wo; a.L = (uint32_t)sh.L; a.wc = make_wincols(sh);
    a.div_Wo = make_fastdiv((uint32_t)sh.Wo);
    // Linear tap order unless IM2WIN_TAP_ORDER=column asks for the row
    // kernel's stages in column order: on the row kernel's layers column
    // order measured from +3 % (3x3 64 -> 128 at 112x112) to -10 % (3x3
    // 256 -> 512 at 12x12), where the filter tiles' L2 reuse suffers.  The
    // register-staged kernel always walks its taps in linear order.
    a.to = make_taporder(sh.Kw, sh.Kh, sh.Ci, (uint32_t)BK, t.tap_order != Tuning::kColumn || p.fam != Fam16::Pipe,
                         sh.s);
    void *args[] = {&a};
    const uint32_t nst = (uint32_t)(sh.K_pad / BK);
    a.ks = 1; a.spl = nst; a.part = nullptr;
    if (p.fam == Fam16::Pipe) {
        int n;
        const PipeVariant &v = pipe_variants(&n)[p.v];
        const int64_t gx = (sh.P + v.bn - 1) / v.bn, gy = (sh.Co + v.bm - 1) / v.bm;
        if (gx * gy * p.ks > 0x7fffffff)
            return hipErrorInvalidValue;
        a.tg = make_tilegrid(gx, gy, t.tile_linear);
        a.ntiles = (uint32_t)(gx * gy);
        if (p.ks <= 1)
            return hipLaunchKernel(v.f[op == Op16::BF16], dim3((uint32_t)(gx * gy)), dim3(v.nt), args, 0, st);
        if (split == nullptr)
            return hipErrorInvalidValue;
        a.ks = (uint32_t)p.ks;
        a.spl = (nst + a.ks - 1) / a.ks;
        a.part = static_cast<float *>(split);
        hipError_t e =
            hipLaunchKernel(v.f[op == Op16::BF16], dim3((uint32_t)(gx * gy * a.ks)), dim3(v.nt), args, 0, st);
        if (e != hipSuccess)
            return e;
        SumArgs sa;
        sa.part = a.part;
        sa.out = out;
        sa.ks = a.ks; sa.ntiles = a.ntiles; sa.P = a.P; sa.Co = a.Co;
        sa.WM = v.wm; sa.WN = v.wn; sa.WGN = v.wgn; sa.BMc = v.bm; sa.BNp = v.bn;
        sa.tile_quads = (uint32_t)(v.bm * v.bn / 4);
        sa.quads = (uint64_t)a.ntiles * sa.tile_quads;
        sa.tg = a.tg;
        void *sargs[] = {&sa};
        const void *fs = op == Op16::BF16 ? (const void *)&split_sum<BF16Op> : (const void *)&split_sum<F16Op>;
        return hipLaunchKernel(fs, dim3((uint32_t)((sa.quads + 255) / 256)), dim3(256), sargs, 0, st);
    }
    const void *f;
    int bm, bn;
    const bool unal = sh.K >= 128;
    if (op == Op16::BF16) {
        if (p.v == 0)
            pick_regs<BF16Op, 1, 2, 1, 4>(unal, &f, &bm, &bn);
        else if (p.v == 1)
            pick_regs<BF16Op, 2, 2, 1, 4>(unal, &f, &bm, &bn);
        else
            pick_regs<BF16Op, 2, 2, 2, 2>(unal, &f, &bm, &bn);
    } else {
        if (p.v == 0)
            pick_regs<F16Op, 1, 2, 1, 4>(unal, &f, &bm, &bn);
        else if (p.v == 1)
            pick_regs<F16Op, 2, 2, 1, 4>(unal, &f, &bm, &bn);
        else
            pick_regs<F16Op, 2, 2, 2, 2>(unal, &f, &bm, &bn);
    }
    const int64_t gx = (sh.P + bn - 1) / bn, gy = (sh.Co + bm - 1) / bm;
    if (gx * gy > 0x7fffffff)
        return hipErrorInvalidValue;
    a.tg = make_tilegrid(gx, gy, t.tile_linear);
    a.ntiles = (uint32_t)(gx * gy);
    return hipLaunchKernel(f, dim3((uint32_t)(gx * gy)), dim3(256), args, 0, st);
}

}  // namespace im2win
