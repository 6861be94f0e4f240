// fp16 windowed convolution on the gfx950 matrix cores, staged by input
// column (Sec. III-B..D, Eq. 3, Alg. 1).
//
// A strip of the window tensor is a sequence of W_i input columns, each
// T = K_h*C_i elements long in (u, r) order, and the window of output column
// n is the run of columns n*s .. n*s+K_w-1.  Tap k = v*T + t of that window
// is element t of column n*s + v.  Neighbouring windows share K_w - s
// columns, so a tile of BN consecutive pixels needs far fewer distinct
// columns than BN*K_w: this kernel loads every distinct column of its tile
// once per stage and lets the K_w windows that use a column read it from LDS
// (the re-use the window layout is built for, applied on chip).
//
// Product:  D[j][p] = sum_v sum_t G[j][v][t] * X[col(p, v)][t]
//   G is the filter packed per filter column v: G[j][v][t] = F[u][v][r][j]
//   with t = u*C_i + r, zero for t >= T (T padded to Tp, a multiple of 64);
//   X[c][t] is element t of strip column c.
//
// A stage covers BT consecutive t of every column slice:
//   A rows  (v, j)  K_w*BM rows of BT filter values,
//   B rows  one per distinct column of the tile (at most NRMAX), BT values,
// fetched with buffer_load ... lds (each lane's 16 bytes go straight to LDS,
// one wave instruction fills 1 KiB = 1024/(2*BT) rows) into a two-slot ring:
// the loads of stage t+1 are in flight while the matrix cores multiply
// stage t (Alg. 1's double buffering with asynchronous copies).  Every stage
// does K_w*BT/16 MFMA k-steps; pixel p's B fragment for filter column v is
// row R(p) + v.
//
// Row numbering of the B rows: with ms = min(s, K_w), pixel slot n of the
// tile gets R(n) = n*ms + k(n)*(K_w - ms), k(n) = strips crossed since the
// tile's first pixel.  Consecutive pixels of one strip then share K_w - ms
// rows, and each strip run of the tile starts K_w rows after the previous
// run's last pixel.
//
// LDS rows are XOR-swizzled at 16-byte granularity, chunk c of row r at slot
// c ^ sw(r), so that the 32 rows one MFMA operand read touches spread over
// all banks.  The epilogue rounds each fp32 sum to fp16 once (nearest-even).
#include "common.hpp"
#include "epilogue16.hpp"

#include <stdlib.h>
#include <string.h>
#include <type_traits>

namespace im2win {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void *lds_ptr;

struct ColArgs {
    const uint16_t *ws;      // window tensor (16-bit elements)
    const uint16_t *packed;  // G in BT-tap tiles: [Tp/BT][KW][Co_pad][BT]
    uint16_t *out;
    uint64_t win_bytes;
    uint64_t pk_bytes;       // bytes of G
    uint32_t P, Co, Co_pad, Wo, L, T, Tp, s, ms, nst;
    uint32_t ntiles;         // gx * gy
    uint32_t persist;        // 1: each workgroup walks tiles blockIdx.x, + gridDim.x, ...
    TileGrid tg;             // pixel x channel tiles of the 1-D launch
    FastDiv div_Wo;
};

constexpr uint32_t kNoCol = 0xffffffffu;  // B row with no column (past the last pixel)
// Next-stage loads issued after each k-step's matrix operations (two per
// step measured best: 7x7 C = 64 stride 2 at 224x224, 759 TFLOP/s against
// 747 / 731 / 719 with 4 / 8 / 16 per step and 709 with all of them issued
// before the stage's first multiply)
constexpr int kLoadsPerStep = 2;

template <int KW_, int BT_, int WM_, int WN_, int WGM_, int WGN_, int NRMAX_, int NS_, bool PERSIST_ = true>
struct ColCfg {
    static constexpr int KW = KW_, BT = BT_, WM = WM_, WN = WN_, WGM = WGM_, WGN = WGN_;
    static constexpr int NS = NS_;              // ring slots
    static constexpr bool SERIAL = false;       // see Serialized
    static constexpr bool PERSIST = PERSIST_;   // the persistent tile loop is compiled in
    static constexpr int NW = WGM * WGN;        // waves
    static constexpr int NT = 64 * NW;
    static constexpr int BM = 32 * WM * WGM;    // channels per tile
    static constexpr int BN = 32 * WN * WGN;    // pixels per tile
    static constexpr int NRMAX = NRMAX_;        // B rows a tile may need
    static constexpr int RB = 2 * BT;           // bytes per LDS row
    static constexpr int CH = RB / 16;          // 16-byte chunks per row
    static constexpr int RPI = 1024 / RB;       // rows filled by one wave load
    static constexpr int AROWS = KW * BM;
    static constexpr int ROWS = AROWS + NRMAX;
    static constexpr int NBLK = (ROWS + RPI - 1) / RPI;  // 1 KiB blocks per stage
    static constexpr int IB = (NBLK + NW - 1) / NW;      // loads per wave per stage
    static constexpr int IA = (AROWS / RPI) % NW == 0 ? AROWS / RPI / NW : -1;  // A loads per wave
    // Every wave issues IB loads per stage (those past the stage's rows read
    // nothing and fill spare LDS with zeros), so outstanding-load counts are
    // the same for all stages and the ring waits are exact.
    static constexpr int STAGE = NW * IB * 1024;
    static_assert(NS >= 2 && NS <= 4, "ring depth");
    static_assert((NS - 2) * IB <= 63, "vmcnt range");
    static constexpr int SWS = CH == 4 ? 2 : 3;          // swizzle shift
    // LDS per workgroup (ring slots, the two-slot kernels' unused slot
    // stand-ins, the column table) and the waves per SIMD it leaves room for:
    // the register budget the compiler is held to, so that a persistent
    // tile loop does not cost occupancy
    static constexpr int LDSB = NS * STAGE + (4 - NS) * 1024 + 4 * NRMAX;
    static constexpr int WPE = (160 * 1024 / LDSB) * NW / 4 < 1 ? 1 : (160 * 1024 / LDSB) * NW / 4;
    static_assert(BT == 16 || BT == 32 || BT == 64, "stage depth");
    static_assert(AROWS % RPI == 0, "A and B rows meet at a block boundary");
};

// The same tile with its ring serialized: a stage's loads are issued only
// after every wave has finished multiplying the previous stage, and waited
// for in full, so no load is ever in flight while LDS is read.  Same sums in
// the same order; a check variant for the ring's waits and barriers (its
// output must match the ring's bit for bit).
template <class Base>
struct Serialized : Base {
    static constexpr bool SERIAL = true;
};

template <class C>
__device__ inline uint32_t sw(uint32_t r)
{
    return (r ^ (r >> C::SWS)) & (C::CH - 1);
}

template <int VM>
__device__ inline void wait_vmcnt()
{
    __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4) | (15 << 8));
}

// E: the operand type (F16Op or BF16Op).
template <class C, class E>
struct ColTile {
    typedef typename E::v8 v8;
    __amdgpu_buffer_rsrc_t rf, rw;
    uint32_t boff[C::IB];  // byte offset of this lane's chunk at t = 0 (kOOB: none)
    uint32_t bcm[C::IB];   // B rows: first t of the chunk (t-tail mask); A rows: 0
    uint32_t Rj[C::WN];    // B row of each of this lane's pixels
    uint32_t wave, lane, wm, wn, T, nst, apitch;
    floatx16 acc[C::WM][C::WN];

    // Stage st >= nst (past the end of the slices) loads nothing.
    // Offsets of stage st's loads: a chunk whose first t is at or past `lim`
    // reads nothing (A rows have bcm = 0: only stages past the end or past T).
    struct StageLoads {
        uint32_t lim, aadd, badd;
    };
    __device__ inline StageLoads stage_loads(uint32_t st) const
    {
        const uint32_t t0 = st * C::BT;
        return StageLoads{st >= nst ? 0u : t0 < T ? T - t0 : 0u, st * apitch, 2u * t0};
    }

    // Load i of a stage (i < IB).
    __device__ inline void issue_one(int i, const StageLoads &sl, char *slot)
    {
        const uint32_t b = wave + C::NW * i;
        // where the A blocks split evenly over the waves, the first IA loads
        // of every wave are A blocks (known at compile time)
        const bool isA = C::IA >= 0 ? i < C::IA : b * C::RPI < (uint32_t)C::AROWS;
        const uint32_t off = bcm[i] < sl.lim ? boff[i] + (isA ? sl.aadd : sl.badd) : kOOB;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(isA ? rf : rw, (lds_ptr)(slot + 1024 * b), 16, off, 0, 0, 0);
    }

    __device__ inline void issue(uint32_t st, char *slot)
    {
        const StageLoads sl = stage_loads(st);
#pragma unroll
        for (int i = 0; i < C::IB; ++i)
            issue_one(i, sl, slot);
    }

    // Fragments of k-step ks (filter column v = ks / (BT/16)).
    __device__ inline void frags(const char *slot, int ks, v8 (&af)[C::WM], v8 (&bf)[C::WN])
    {
        const int v = ks / (C::BT / 16), kk = ks % (C::BT / 16);
        const uint32_t chunk = 2 * kk + (lane >> 5);
        const uint32_t arow0 = wm * 32 * C::WM + (lane & 31);
#pragma unroll
        for (int i = 0; i < C::WM; ++i) {
            const uint32_t row = v * C::BM + arow0 + 32 * i;
            af[i] = *reinterpret_cast<const v8 *>(slot + row * C::RB + 16 * (chunk ^ sw<C>(row)));
        }
#pragma unroll
        for (int j = 0; j < C::WN; ++j) {
            const uint32_t row = C::AROWS + Rj[j] + v;
            bf[j] = *reinterpret_cast<const v8 *>(slot + row * C::RB + 16 * (chunk ^ sw<C>(row)));
        }
    }

    // All k-steps of one stage; the fragments of step ks+1 are read before
    // the matrix operations of step ks.  With `nslot` set, the loads of stage
    // `nst_` into it are issued a few at a time after the matrix operations
    // of each k-step, so their issue runs while the matrix cores work instead
    // of before the stage's first multiply.
    __device__ inline void compute(const char *slot, uint32_t nst_ = 0, char *nslot = nullptr)
    {
        constexpr int KS = C::KW * C::BT / 16;
        StageLoads sl{};
        if (nslot)
            sl = stage_loads(nst_);
        v8 af[2][C::WM], bf[2][C::WN];
        frags(slot, 0, af[0], bf[0]);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (ks + 1 < KS)
                frags(slot, ks + 1, af[(ks + 1) & 1], bf[(ks + 1) & 1]);
#pragma unroll
            for (int i = 0; i < C::WM; ++i)
#pragma unroll
                for (int j = 0; j < C::WN; ++j)
                    acc[i][j] = E::mfma(af[ks & 1][i], bf[ks & 1][j], acc[i][j]);
            if (nslot && ks * kLoadsPerStep < C::IB) {
                // loads 2*ks, 2*ks+1 after step ks: early in the stage, so
                // they have most of it to land, and kept there (the
                // scheduler would otherwise sink them to its end)
#pragma unroll
                for (int i = ks * kLoadsPerStep; i < (ks + 1) * kLoadsPerStep && i < C::IB; ++i)
                    issue_one(i, sl, nslot);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }

    // Stage st sits in slot `cur`: wait for it, then refill the slot freed by
    // stage st-1 (`next`) with stage st+NS-1, then multiply.  The slots are
    // separate LDS arrays named at compile time, so the compiler can tell
    // that reading one does not depend on the loads landing in the others.
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
        // st < nst: the loops below run real stages only
        wait_vmcnt<(C::NS - 2) * C::IB>();
        ring_barrier();
        compute(cur, st + C::NS - 1, next);
    }

    // The tile's resources, column table, per-lane load offsets and B rows
    // (the table in LDS; two workgroup barriers, with nothing in flight).
    template <int N>
    __device__ inline void setup(const ColArgs &a, uint32_t tile, uint32_t (&tbl)[N], uint32_t tid, uint32_t &p0,
                                 uint32_t &ch0)
    {
        uint32_t tx, ty;
        a.tg.tile_of(tile, tx, ty);
        p0 = tx * C::BN;
        ch0 = ty * C::BM;
        const uint32_t q0 = fdiv(p0, a.div_Wo);

        // B rows address the window tensor from strip q0 on, A rows the
        // filter from row ch0 on; anything past either buffer reads zero.
        const uint64_t tb = (uint64_t)q0 * a.L;
        const uint64_t wleft = a.win_bytes - tb * 2;
        rw = make_rsrc(a.ws + tb, (uint32_t)(wleft < kMaxRecords ? wleft : kMaxRecords));
        // the packed filter in BT-tap tiles: tile st holds, for each filter
        // column v, the C_o_pad rows of slice v; addressed from row ch0 of
        // (tile 0, v 0)
        const uint64_t fb = (uint64_t)ch0 * C::BT;
        rf = make_rsrc(a.packed + fb, (uint32_t)(a.pk_bytes - fb * 2));
        apitch = (uint32_t)C::KW * a.Co_pad * C::BT * 2u;

        // Column table: element offset (from strip q0) of the column each B
        // row holds.  Pixel slot n owns rows R(n) .. R(n)+ms-1; the last pixel
        // of a strip run also owns the K_w - ms rows after them.
        for (uint32_t r = tid; r < (uint32_t)C::NRMAX; r += C::NT)
            tbl[r] = kNoCol;
        __syncthreads();
        const uint32_t kwm = C::KW - a.ms;
        for (uint32_t n = tid; n < (uint32_t)C::BN; n += C::NT) {
            const uint32_t p = p0 + n;
            if (p < a.P) {
                const uint32_t q = fdiv(p, a.div_Wo);
                const uint32_t c = p - q * a.Wo;
                const uint32_t k = q - q0;
                const uint32_t R = n * a.ms + k * kwm;
                const bool last = n == (uint32_t)C::BN - 1 || p + 1 == a.P || c + 1 == a.Wo;
                const uint32_t nv = last ? (uint32_t)C::KW : a.ms;
                for (uint32_t v = 0; v < nv; ++v)
                    tbl[R + v] = k * a.L + (c * a.s + v) * a.T;
            }
        }
        __syncthreads();

        // Per-lane load offsets, fixed for the whole tile.
#pragma unroll
        for (int i = 0; i < C::IB; ++i) {
            const uint32_t b = wave + C::NW * i;
            const uint32_t row = b * C::RPI + lane / C::CH;
            const uint32_t c = (lane % C::CH) ^ sw<C>(row);
            boff[i] = kOOB;
            bcm[i] = 0;
            if (row < (uint32_t)C::AROWS) {
                const uint32_t v = row / C::BM, jl = row % C::BM;
                boff[i] = ((v * a.Co_pad + jl) * C::BT + 8 * c) * 2u;
            } else if (row < (uint32_t)C::ROWS) {
                const uint32_t e = tbl[row - C::AROWS];
                if (e != kNoCol)
                    boff[i] = (e + 8 * c) * 2u;
                bcm[i] = 8 * c;
            }
        }
#pragma unroll
        for (int j = 0; j < C::WN; ++j) {
            const uint32_t n = wn * 32 * C::WN + 32 * j + (lane & 31);
            const uint32_t p = p0 + n;
            // a pixel past P reads row 0 (its result is never stored)
            Rj[j] = p < a.P ? n * a.ms + (fdiv(p, a.div_Wo) - q0) * kwm : 0;
        }
    }

    __device__ inline void zero_acc()
    {
#pragma unroll
        for (int i = 0; i < C::WM; ++i)
#pragma unroll
            for (int j = 0; j < C::WN; ++j)
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    acc[i][j][e] = 0.f;
    }
};

// A workgroup may walk several tiles (a persistent launch) when its ring has
// two slots and the tile's epilogue fits one: after a tile's last stage
// (which sits in slot 1, the stage count being even) it stages the finished
// tile in slot 1, sets up the next tile, stores the finished one and issues
// the next tile's first stage into slot 0, so that stage's loads and the
// stores are in flight together instead of the loads waiting behind a new
// workgroup's start.
template <class C>
constexpr bool col_persist_ok()
{
    return C::PERSIST && C::NS == 2 && !C::SERIAL && epilogue16_bytes<C::BM, C::BN>() <= C::STAGE &&
           (C::BN * (2 * C::BM / 16)) % C::NT == 0;
}

template <class C, class E>
__global__ __launch_bounds__(C::NT, C::WPE) void conv_fp16_col(ColArgs a)
{
    constexpr int S2 = C::NS > 2 ? C::STAGE : 1024, S3 = C::NS > 3 ? C::STAGE : 1024;
    __shared__ __attribute__((aligned(1024))) char r0[C::STAGE];
    __shared__ __attribute__((aligned(1024))) char r1[C::STAGE];
    __shared__ __attribute__((aligned(1024))) char r2[S2];
    __shared__ __attribute__((aligned(1024))) char r3[S3];
    __shared__ uint32_t tbl[C::NRMAX];

    ColTile<C, E> w;
    const uint32_t tid = threadIdx.x;
    w.lane = tid & 63;
    w.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    __builtin_assume(w.wave < (uint32_t)C::NW);
    w.wm = w.wave / C::WGN;
    w.wn = w.wave % C::WGN;
    w.T = a.T;
    w.nst = a.Tp / C::BT;
    uint32_t tile = blockIdx.x, p0, ch0;
    w.setup(a, tile, tbl, tid, p0, ch0);
    w.zero_acc();

    // prologue: stages 0 .. NS-2 into slots 0 .. NS-2; stage st then sits
    // in slot st % NS
    // (whole rounds of the ring, then the last nst % NS stages; each step
    // multiplies a real stage and issues the one NS-1 ahead, which past the
    // end loads zeros)
    w.issue(0, r0);
    uint32_t st = 0;
    if constexpr (C::NS == 2) {
        for (;;) {
            st = 0;
            for (; st + 2 <= w.nst; st += 2) {
                w.step(st, r0, r1);
                w.step(st + 1, r1, r0);
            }
            if (st < w.nst)
                w.step(st, r0, r1);
            if constexpr (col_persist_ok<C>()) {
                const uint32_t next = tile + gridDim.x;
                if (a.persist && next < a.ntiles) {
                    // the last stage (odd) is in r1, the zero loads of the
                    // stage past the end went to r0
                    wait_vmcnt<0>();
                    ring_barrier();
                    // the finished sums into r1 (so that they are not live
                    // beside the next tile's load offsets), the next tile's
                    // set-up, r1 out to the output, then the next tile's
                    // first stage into r0: the first wait of the next tile
                    // covers these stores and loads in flight together
                    stage_tile_lds_ring<E, C::WM, C::WN, C::WGM, C::WGN>(w.acc, r1, w.wm, w.wn, w.lane);
                    w.zero_acc();
                    const uint32_t pc = p0, cc = ch0;
                    w.setup(a, next, tbl, tid, p0, ch0);
                    copy_tile_out_ring<C::BM, C::BN, C::NT>(r1, a.out, a.P, a.Co, pc, cc, tid);
                    w.issue(0, r0);
                    tile = next;
                    continue;
                }
            }
            break;
        }
    } else if constexpr (C::NS == 3) {
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

    // Epilogue: through LDS (whole output lines per wave) when the tile fits
    // a ring slot, else directly from the accumulators.
    if constexpr (epilogue16_bytes<C::BM, C::BN>() <= C::STAGE) {
        store_tile_lds<E, C::WM, C::WN, C::WGM, C::WGN>(w.acc, r0, a.out, a.P, a.Co, p0, ch0, w.wm, w.wn, w.lane,
                                                     tid);
        return;
    }
    // Lane holds pixel pb + 32*j + (lane & 31) and, for element e of block
    // (i, j), channel cb + 32*i + 8*(e/4) + 4*(lane/32) + e%4.
    const uint32_t pb = p0 + w.wn * 32 * C::WN, cb = ch0 + w.wm * 32 * C::WM;
#pragma unroll
    for (int j = 0; j < C::WN; ++j) {
        const uint32_t p = pb + 32 * j + (w.lane & 31);
        if (p >= a.P)
            continue;
        uint16_t *o = a.out + (uint64_t)p * a.Co;
#pragma unroll
        for (int i = 0; i < C::WM; ++i) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const uint32_t c = cb + 32 * i + 8 * g + 4 * (w.lane >> 5);
                uint32_t h[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    h[e] = E::bits(w.acc[i][j][4 * g + e]);
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

struct ColVariant {
    const char *name;
    const void *f[2];  // fp16 and bf16 operands
    int kw, bm, bn, nrmax, bt, nt;
    bool persist_ok;   // may walk several tiles per workgroup
};

template <int KW, int BT, int WM, int WN, int WGM, int WGN, int NRMAX, int NS, bool SERIAL = false,
          bool PERSIST = true>
ColVariant col_variant(const char *name)
{
    using B = ColCfg<KW, BT, WM, WN, WGM, WGN, NRMAX, NS, PERSIST>;
    using C = typename std::conditional<SERIAL, Serialized<B>, B>::type;
    return ColVariant{name, {(const void *)&conv_fp16_col<C, F16Op>, (const void *)&conv_fp16_col<C, BF16Op>}, KW,
                      C::BM, C::BN, NRMAX, BT, C::NT, col_persist_ok<C>()};
}

const ColVariant *col_variants(int *n)
{
    // name: filter width, channels x pixels per tile, taps per stage, ring slots
    static const ColVariant v[] = {
        col_variant<3, 32, 2, 2, 1, 4, 288, 2>("k3c64p256t32s2"),
        col_variant<3, 32, 1, 2, 2, 2, 160, 2>("k3c64p128t32s2"),
        col_variant<3, 32, 2, 2, 2, 2, 160, 2>("k3c128p128t32s2"),
        col_variant<3, 16, 2, 4, 2, 2, 288, 3>("k3c128p256t16s3"),
        col_variant<7, 16, 2, 2, 1, 4, 544, 3>("k7c64p256t16s3"),
        // (without the persistent loop: at three waves per SIMD its
        // registers would spill)
        col_variant<7, 16, 1, 2, 2, 2, 288, 2, false, false>("k7c64p128t16s2"),
        // eight waves, 256 x 256 tiles (large C_o)
        col_variant<3, 32, 4, 2, 2, 4, 320, 2>("k3c256p256t32s2w8"),
        col_variant<3, 32, 2, 3, 4, 2, 256, 2>("k3c256p192t32s2w8"),
        // 32-tap stages for 7-wide filters (two slots, 128 KiB: one
        // workgroup per CU)
        col_variant<7, 32, 2, 2, 1, 4, 544, 2>("k7c64p256t32s2"),
        // serialized rings of three of the above (check variants)
        col_variant<3, 32, 1, 2, 2, 2, 160, 2, true>("k3c64p128t32s2-serial"),
        col_variant<7, 16, 2, 2, 1, 4, 544, 3, true>("k7c64p256t16s3-serial"),
        col_variant<3, 32, 2, 3, 4, 2, 256, 2, true>("k3c256p192t32s2w8-serial"),
    };
    *n = (int)(sizeof v / sizeof v[0]);
    return v;
}

// Rows a tile of bn consecutive pixels needs at most: each strip run of c
// pixels needs (c-1)*ms + K_w rows, and bn pixels span at most
// ceil((bn-1)/W_o) + 1 runs.
int64_t col_rows_needed(const Shape &sh, int bn)
{
    const int64_t ms = sh.s < sh.Kw ? sh.s : sh.Kw;
    int64_t runs = (bn - 1 + sh.Wo - 1) / sh.Wo + 1;
    if (runs > bn)
        runs = bn;
    return (bn - runs) * ms + runs * sh.Kw;
}

}  // namespace

int col_find(const char *name)
{
    int n;
    const ColVariant *v = col_variants(&n);
    for (int t = 0; t < n; ++t)
        if (strcmp(name, v[t].name) == 0)
            return t;
    return -1;
}

const char *col_name(int v)
{
    int n;
    return col_variants(&n)[v].name;
}

bool col_fits(const Shape &sh, int pick)
{
    int n;
    const ColVariant *v = col_variants(&n);
    if (pick < 0 || pick >= n)
        return false;
    if (sh.Ci % 8 != 0)
        return false;  // windows not 16-byte aligned
    if (sh.d != 1)
        return false;  // the column table assumes consecutive strip columns
    if (v[pick].kw != sh.Kw)
        return false;
    if (col_rows_needed(sh, v[pick].bn) > v[pick].nrmax)
        return false;
    // the packed filter is addressed with 31-bit offsets
    if (sh.Co_pad * sh.Kw * sh.Tp * 2 >= (int64_t)kMaxRecords)
        return false;
    // every offset inside a tile must fit 31 bits (checked per layer: the
    // strips of one tile plus the last column's slice)
    const int64_t strips_per_tile = (v[pick].bn - 1) / sh.Wo + 2;
    if ((strips_per_tile * sh.L + sh.Tp) * 2 >= (int64_t)kOOB)
        return false;
    return true;
}

int col_default(const Shape &sh)
{
    if (sh.Ci % 8 != 0 || sh.d != 1)
        return -1;
    // Defaults, measured per layer on MI355X: the column-staged kernel
    // wins where the window rows dominate a stage (C_o <= 128); with
    // more channels the K_w*BM filter rows of a stage dominate it and the
    // row-per-pixel kernel, whose stages hold 64 taps of BM filter rows,
    // is faster.
    // With C_o > 128 the eight-wave 256-channel variants (whose filter
    // rows arrive as one contiguous run per stage) beat the row kernel
    // when their grid fills most of the 256 CUs in one round: cfg4 (192
    // tiles of 256 x 192) 808 vs 633 TFLOP/s; with ~100-130 tiles they
    // lose (S5: 536 vs 636), so those layers keep the row kernel.
    auto tiles = [&](int64_t bn) { return ((sh.P + bn - 1) / bn) * ((sh.Co + 255) / 256); };
    const char *name = nullptr;
    // the one-slot row kernel is faster on many-tile layers with C_o >= 128,
    // except 3x3 layers with C_o <= 128 (3x3 64 -> 128 at 112x112: column
    // kernel 664 vs 636 TFLOP/s)
    if (fp16_single_slot_rows(sh) && !(sh.Kw == 3 && sh.Co <= 128))
        return -1;
    // C_o <= 64: 64 x 128 tiles, three workgroups per CU, more bytes in
    // flight for these HBM-bound layers (3x3 C=64 at 56x56: 484 vs 431
    // TFLOP/s same-process; with C_o = 128, 3x3 at 28x28, 531 vs 548)
    if (sh.Kw == 3 && sh.Co <= 64)
        name = "k3c64p128t32s2";
    // 64 < C_o <= 128: one 128 x 128 tile reads each window once where two
    // 64-channel tiles read it twice (3x3 64 -> 128 at 112x112: 771 vs 714
    // TFLOP/s; 128 -> 128 at 28x28: 646 vs 603-639)
    else if (sh.Kw == 3 && sh.Co <= 128)
        name = "k3c128p128t32s2";
    // 7x7: with stride 1 and C_o <= 64 the 64 x 128 tile (two-slot ring,
    // 49 KiB, three workgroups per CU) measured 785 vs 713 TFLOP/s
    // (7x7 C=64 at 60x60, 64 images); with stride 2 (7x7 C=64 at 224x224)
    // it lost, 668 vs 701
    else if (sh.Kw == 7 && sh.s == 1 && sh.Co <= 64)
        name = "k7c64p128t16s2";
    // with stride 2 and C_o <= 64 (7x7 C=64 at 224x224) 32-tap stages in a
    // two-slot ring beat the three-slot 16-tap ring: 705 vs 684 TFLOP/s
    else if (sh.Kw == 7 && sh.Co <= 64)
        name = "k7c64p256t32s2";
    else if (sh.Kw == 7 && sh.Co <= 128)
        name = "k7c64p256t16s3";
    else if (sh.Kw == 3 && tiles(192) >= 160 && tiles(192) <= 256)
        name = "k3c256p192t32s2w8";
    else if (sh.Kw == 3 && tiles(256) >= 160 && tiles(256) <= 256)
        name = "k3c256p256t32s2w8";
    // 3x3 C=256 at 14x14 (128 images): four 64 x 128 channel tiles per
    // pixel tile beat the 128 x 128 row kernel, 583 vs 529 TFLOP/s
    else if (sh.Kw == 3 && sh.Co <= 256)
        name = "k3c64p128t32s2";
    else
        return -1;
    const int pick = col_find(name);
    return col_fits(sh, pick) ? pick : -1;
}

int col_stage_taps(int plan)
{
    int n;
    return col_variants(&n)[plan].bt;
}

int64_t col_packed_rows(const Shape &sh, int plan)
{
    int n;
    return round_up(sh.Co, col_variants(&n)[plan].bm);
}

hipError_t launch_conv_fp16_col(const Shape &sh, int plan, const Tuning &t, const void *ws, const void *packed,
                                uint16_t *out, hipStream_t st, Op16 op)
{
    int n;
    const ColVariant &v = col_variants(&n)[plan];
    ColArgs a;
    a.ws = static_cast<const uint16_t *>(ws);
    a.packed = static_cast<const uint16_t *>(packed);
    a.out = out;
    a.win_bytes = (uint64_t)sh.win_bytes;
    const int64_t rows = col_packed_rows(sh, plan);
    a.pk_bytes = (uint64_t)rows * sh.Kw * sh.Tp * 2;
    a.Co_pad = (uint32_t)rows;
    a.P = (uint32_t)sh.P; a.Co = (uint32_t)sh.Co; a.Wo = (uint32_t)sh.Wo; a.L = (uint32_t)sh.L;
    a.T = (uint32_t)(sh.Kh * sh.Ci); a.Tp = (uint32_t)sh.Tp; a.s = (uint32_t)sh.s;
    a.ms = (uint32_t)(sh.s < sh.Kw ? sh.s : sh.Kw);
    a.nst = 0;
    a.div_Wo = make_fastdiv((uint32_t)sh.Wo);
    const int64_t gx = (sh.P + v.bn - 1) / v.bn, gy = (sh.Co + v.bm - 1) / v.bm;
    if (gx * gy > 0x7fffffff)
        return hipErrorInvalidValue;
    a.tg = make_tilegrid(gx, gy, t.tile_linear);
    a.ntiles = (uint32_t)(gx * gy);
    a.persist = 0;
    uint32_t grid = a.ntiles;
    const void *f = v.f[op == Op16::BF16];
    // Persistent launch (one round of resident workgroups walking the
    // tiles) where the variant allows it, the stage count is even (the last
    // stage then sits in slot 1), the output rows are 16-byte aligned and the
    // tile's output rows fit 31-bit offsets; unless IM2WIN_FP16_PERSIST=off.
    if (v.persist_ok && t.col_persist && (sh.Tp / v.bt) % 2 == 0 && sh.Co % 8 == 0 &&
        (int64_t)v.bn * sh.Co * 2 < (int64_t)kMaxRecords) {
        int dev = 0, cus = 0, per_cu = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e == hipSuccess)
            e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e == hipSuccess)
            e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, f, v.nt, 0);
        if (e != hipSuccess)
            return e;
        const int64_t g = (int64_t)(cus > 0 ? cus : 1) * (per_cu > 0 ? per_cu : 1);
        if (g < (int64_t)a.ntiles) {
            a.persist = 1;
            grid = (uint32_t)g;
        }
    }
    void *args[] = {&a};
    return hipLaunchKernel(f, dim3(grid), dim3(v.nt), args, 0, st);
}

}  // namespace im2win
