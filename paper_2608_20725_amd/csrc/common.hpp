// Internal definitions shared by the host API and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace im2win {

// Division of a 32-bit unsigned value by a launch-constant divisor d >= 1
// with one high multiply, one add and one shift (Granlund & Montgomery,
// "Division by invariant integers using multiplication", PLDI 1994, Fig. 4.1:
// l = ceil(log2 d), m = floor(2^32 (2^l - d) / d) + 1, q = (mulhi(m, x) + x) >> l,
// the add done in 33 bits).  Exact for every x < 2^32.
struct FastDiv {
    uint32_t d;
    uint32_t mul;
    uint32_t shift;
};

inline FastDiv make_fastdiv(uint32_t d)
{
    uint32_t l = 0;
    while ((1ull << l) < d)
        ++l;
    uint64_t m = ((1ull << 32) * ((1ull << l) - d)) / d + 1;
    return FastDiv{d, (uint32_t)m, l};
}

__host__ __device__ inline uint32_t fdiv(uint32_t x, const FastDiv &f)
{
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t hi = __umulhi(x, f.mul);
#else
    uint32_t hi = (uint32_t)(((uint64_t)x * f.mul) >> 32);
#endif
    return (uint32_t)(((uint64_t)hi + x) >> f.shift);
}

// Everything a kernel needs to know about one layer.  Built and validated on
// the host (api.cpp).
struct Shape {
    int64_t N, Ci, Hi, Wi, Co, Kh, Kw, s;
    int64_t Ho, Wo;
    int64_t P;          // output pixels N*Ho*Wo
    int64_t K;          // window length Kh*Kw*Ci
    int64_t L;          // strip length Wi*Kh*Ci (elements)
    int64_t S;          // window step along a strip s*Kh*Ci (elements)
    int64_t strips;     // N*Ho
    int64_t win_elems;  // strips*L
    int64_t elt;        // element bytes
    int64_t win_bytes;  // win_elems*elt
    int64_t pad_end;    // end of the zero pad (bytes)
    int64_t Co_pad;     // packed fp16 filter rows
    int64_t K_pad;      // packed fp16 filter columns
    int64_t K_pad32;    // packed fp32 filter rows (taps)
    int64_t Co_pad32;   // packed fp32 filter columns (channels)
    int64_t Tp;         // K_h*C_i rounded up to 64 (fp16 per-column filter slices)
    int64_t d;          // filter dilation (1: none)
    int64_t Wq;         // strip columns per residue group mod d (W_i when d = 1)
    int64_t cols;       // strip columns d*Wq (>= W_i; the extra ones are zero filler)
};

inline int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

// Where the window of output column n starts inside its strip, in elements.
// Undilated (Eq. 3): n*s columns of T = K_h*C_i elements.  With filter
// dilation d the strip holds its columns grouped by residue mod d, Wq per
// group, so the window's columns n*s + v*d are the K_w consecutive ones from
// ((n*s) mod d)*Wq + floor(n*s/d) on.
struct WinCols {
    uint32_t s, d, Wq, T;
    FastDiv div_d;

    __host__ __device__ inline uint32_t start(uint32_t n) const
    {
        const uint32_t c = n * s;
        if (d == 1)
            return c * T;
        const uint32_t g = fdiv(c, div_d);
        return ((c - g * d) * Wq + g) * T;
    }
};

// Order of a kernel's K loop.  A kernel walks its taps in blocks of G (a
// stage, or part of one); linear order takes block b as taps b*G .. b*G+G-1.
// Column order (nv filter columns of T = K_h*C_i taps each, T a multiple of
// G) takes block b as taps v*T + tb*G .. of the (b % nv)-th filter column of
// the list `cols`, with tb = b / nv: the nv column slices of one tap range
// follow each other.  Neighbouring windows share input columns (a column is
// slice v of one window and slice v + s of the previous one), so in column
// order the bytes one tile reads for slice v come back for slice v + s a
// few blocks later, while they are still in L2, instead of s*T/G blocks
// later.  The list takes the columns by residue mod s (0, s, 2s, .., then
// 1, 1 + s, ..), so slice v + s is the very next block.  Each output is
// still one fixed sequence of taps, so results stay deterministic.
struct TapOrder {
    uint32_t nv, T, G;  // nv = 1: linear
    uint64_t cols;      // column of the j-th column slice of a tap block: bits 4j .. 4j+3

    __host__ __device__ inline uint32_t map(uint32_t k) const
    {
        if (nv == 1)
            return k;
        const uint32_t b = k / G, off = k - b * G;
        const uint32_t tb = b / nv, j = b - tb * nv;
        const uint32_t v = (uint32_t)(cols >> (4 * j)) & 15u;
        return v * T + tb * G + off;
    }
};

// Tile of a workgroup in a 1-D launch of gx * gy output tiles (gx along
// pixels, gy along channels).  The hardware deals the workgroups of a launch
// to the 8 XCDs round-robin (block b to XCD b % 8), each XCD with its own L2.
// With `xcd` set, XCD k walks one contiguous run of tiles numbered
// channel-fastest, so the gy channel tiles of a pixel tile, which read the
// same windows, run on one XCD at about the same time and share those windows
// through its L2; else tiles follow launch order pixel-fastest (the order of
// a 2-D launch).
struct TileGrid {
    uint32_t gx, gy, xcd;

    __device__ inline void tile(uint32_t &x, uint32_t &y) const { tile_of(blockIdx.x, x, y); }

    // Tile of block b (b < gx * gy).
    __device__ inline void tile_of(uint32_t b, uint32_t &x, uint32_t &y) const
    {
        if (!xcd) {
            y = b / gx;
            x = b - y * gx;
            return;
        }
        const uint32_t nb = gx * gy, k = b % 8, j = b / 8, per = nb / 8, rem = nb % 8;
        const uint32_t t = k * per + (k < rem ? k : rem) + j;
        x = t / gy;
        y = t - x * gy;
    }
};

// gx * gy tiles (< 2^31, the caller's grid checks); `linear` selects the
// launch order (to measure what the XCD-aware order gains).
TileGrid make_tilegrid(int64_t gx, int64_t gy, bool linear);

// Tap block of the fp32 kernels' column order: 32 fp32 taps, one 128-byte
// line of a window column, so the two 16-tap stages that share a line stay
// adjacent (7x7 stride 2 C=64 at 224x224 fetched 1.4x more with 16-tap
// blocks than in linear order).
constexpr uint32_t kTapBlock32 = 32;

// Column order for blocks of G taps when the layer allows it (K_w > 1,
// K_h*C_i a multiple of G) and `linear` is not set; else linear order.
inline TapOrder make_taporder(int64_t Kw, int64_t Kh, int64_t Ci, uint32_t G, bool linear, int64_t s = 1)
{
    const int64_t T = Kh * Ci;
    if (linear || Kw <= 1 || Kw > 16 || T % G != 0)
        return TapOrder{1u, (uint32_t)T, G, 0};
    // columns grouped by residue mod s, ascending within a group: the slice
    // after column v is column v + s, which holds the taps the next pixel
    // read in column v (s = 1 or s >= K_w: plain column order)
    uint64_t cols = 0;
    int j = 0;
    for (int64_t r = 0; r < s && r < Kw; ++r)
        for (int64_t v = r; v < Kw; v += s)
            cols |= (uint64_t)v << (4 * j++);
    return TapOrder{(uint32_t)Kw, (uint32_t)T, G, cols};
}

inline WinCols make_wincols(const Shape &sh)
{
    return WinCols{(uint32_t)sh.s, (uint32_t)sh.d, (uint32_t)sh.Wq, (uint32_t)(sh.Kh * sh.Ci),
                   make_fastdiv((uint32_t)sh.d)};
}

// Raw buffer resource (gfx9 family): base, no swizzle, num_records bytes.
// Loads whose byte offset falls outside [0, num_records) return zero and
// stores there are dropped by the hardware.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

// Byte offset used for a masked-off load: beyond every num_records the
// kernels use (they cap num_records at kMaxRecords), so the load returns 0.
constexpr uint32_t kOOB = 0x80000000u;

// Native 4 x 32-bit vector (kept in registers; HIP's uint4 is a struct whose
// copies can end up in scratch memory).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr uint32_t kMaxRecords = 0x7fffff00u;

// Large outputs of the fp16 stem kernel are stored with the nontemporal
// cache policy: the output is written once and not read again by the
// kernel, and when it is far larger than the caches the streamed writes
// reach HBM sooner.  Measured in the benchmark step (128 images, same box,
// alternating builds): the 3x3 3-channel stem over 224x224 (807 MB of
// output, whole 4 KiB blocks per wave) 104 -> 154 TFLOP/s.  Not streamed:
// outputs under 128 MiB (convs writing 3-51 MB lost 7-17 % streamed: the
// caches absorb them), the column-staged fp16 kernel (194-396 MB: -1 to
// -1.6 %), the DMA-staged fp32 kernel (at most +2.7 %, and its 32-byte row
// pieces, streamed past L2, reached HBM as up to 2.3x the bytes), and window
// tensors (the conv reads them next; streamed, the transforms lost up to
// 11 %).  The streamed stores go through a buffer resource with the nt
// policy operand: a plain store with a nontemporal hint next to an unhinted
// one is folded into a single store by the compiler, and the hint lost.
constexpr int kStoreNT = 2;
constexpr int64_t kStreamOutBytes = (int64_t)128 << 20;
inline bool stream_out(int64_t out_bytes) { return out_bytes >= kStreamOutBytes; }

// 16 bytes at byte offset off of r, streamed (kStoreNT).
__device__ inline void store16_nt(const u32x4 &v, __amdgpu_buffer_rsrc_t r, uint32_t off)
{
    __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, kStoreNT);
}

__device__ inline u32x4 ld_b128(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
}

__device__ inline uint32_t ld_b32(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
}

// Workgroup barrier of the load rings.  It does not wait for outstanding
// global loads (__syncthreads() would, and a ring would hold only one stage
// in flight); it does wait for this wave's outstanding LDS reads
// (lgkmcnt(0)).  The barrier is what hands a slot that has just been read
// to the next stage's direct-to-LDS loads, and the compiler may sink the
// last matrix operations of a stage, with the wait for their operands,
// below it: a read still in flight there can return the next stage's bytes.
// simm16: vmcnt 63 (bits 3:0 and 15:14, no wait), expcnt 7 (no wait), lgkmcnt 0.
__device__ inline void ring_barrier()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

__device__ inline uint32_t ld_b16(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
}

} // namespace im2win

// Host helpers of the C interface (api.cpp), shared with the chunked entry
// points (chunked.cpp).
namespace im2win {
int make_shape(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi, int64_t Co, int64_t Kh, int64_t Kw,
               int64_t s, int dt, Shape *sh);
// The same with filter dilation d >= 1.
int make_shape_dil(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi, int64_t Co, int64_t Kh, int64_t Kw,
                   int64_t s, int64_t d, int dt, Shape *sh);
int64_t packed_filter_bytes(const Shape &sh, int dt);
bool aligned16(const void *p);
bool overlaps(const void *a, int64_t na, const void *b, int64_t nb);
int check_extent(const void *p, int64_t bytes);
int check_device();
int launch_status(hipError_t e);
}  // namespace im2win

// Tuning overrides, read from the environment once per call and checked:
// a value that names no kernel makes the call fail with IM2WIN_EINVAL, and
// so does a kernel forced onto a layer it cannot run.  They exist to measure
// the kernels against each other (the ablation of the paper's techniques);
// without them every layer runs the kernel its shape selects.
//   IM2WIN_FP16_KERNEL     pipe (row-per-pixel kernels) | regs (register-staged)
//                          | stem (short unaligned windows, filter in registers)
//   IM2WIN_FP16_COL        a column-staged variant name
//   IM2WIN_FP16_TILE       a row-per-pixel tile name (implies pipe)
//   IM2WIN_FP16_SEG        a segment-staged variant name
//   IM2WIN_FP32_KERNEL     a DMA-staged variant name | regs | stem (short
//                          unaligned windows, filter from the scalar cache)
//   IM2WIN_FP32_TILE       a register-staged tile name (implies regs)
//   IM2WIN_FP32_COLS       a column-staged variant name
//   IM2WIN_FP32_MFMA_TILE  a matrix-core fp32 tile name
//   IM2WIN_TRANSFORM_ORDER linear | xcd
//   IM2WIN_FP16_PERSIST    on | off: column-staged fp16 kernel in one round of
//                          workgroups that walk the tiles (on by default
//                          where it applies) or one workgroup per tile
//   IM2WIN_TRANSFORM_KERNEL pieces | gather: the 3-channel layers' transform
//                          (one load per 3-channel pixel, where it is the
//                          faster, or one per element)
//   IM2WIN_TILE_ORDER      linear | xcd
//   IM2WIN_TAP_ORDER       linear | column: the K-loop order of the DMA-staged
//                          fp32 kernel (column by default) and of the
//                          row-per-pixel fp16 kernel (linear by default)
//   IM2WIN_FP16_SPLIT      1..kMaxSplit: K split of the row-per-pixel fp16
//                          kernel (refused for other kernels, for a split
//                          that leaves a block no stage, and in the
//                          mini-batch path)
namespace im2win {

struct Tuning {
    enum { kAuto = 0, kPipe = 1, kRegs = 2, kStem = 3 };
    int fp16_kernel;                   // kAuto, kPipe, kRegs, kStem
    int fp16_col, fp16_tile, fp16_seg; // variant index, -1: not forced
    int fp32_kernel;                   // DMA variant index, -1: not forced, -2: register-staged kernel,
                                       // -3: short-window kernel
    int fp32_tile;                     // register-staged tile index, -1: not forced
    int fp32_cols;                     // column-staged variant index, -1: not forced
    int fp32_mfma_tile;                // -1: not forced
    bool transform_linear, tile_linear;
    bool transform_gather;             // 3-channel transform: element gather only
    bool col_persist;                  // column-staged fp16 kernel: persistent launch where it applies
    enum { kDefault = 0, kLinear = 1, kColumn = 2 };
    int tap_order;  // kDefault: each kernel's own (column for the DMA fp32 kernel, linear for the others)
    int fp16_split; // K split of the row-per-pixel kernel: 0 (the planner's choice) or 1..kMaxSplit
};
int read_tuning(Tuning *t);
// The tuning every call runs without tuning variables.
Tuning default_tuning();

// K split of the row-per-pixel fp16 kernel: at most this many workgroups per
// output tile.
constexpr int kMaxSplit = 8;

// Variant tables of each kernel family: index of a name, -1 if none.
int col_find(const char *name);
int pipe_find(const char *name);
int seg_find(const char *name);
int dma32_find(const char *name);
int regs32_find(const char *name);
int mfma32_find(const char *name);

// The kernel one conv call runs, chosen once on the host from the layer and
// the tuning variables, and handed to both the filter pack and the conv
// launch (the packed-filter layout follows the kernel).  A plan chosen for a
// layer of N images also runs any layer that differs only in having fewer
// images (the fit checks do not grow as N shrinks), which the mini-batch
// path relies on.
enum class Fam16 { Col, Pipe, Seg, Regs, Stem };
struct Plan16 {
    Fam16 fam;
    int v;       // variant index within the family (Regs: 0..2 tile by C_o)
    int ks = 1;  // row-per-pixel kernel: K split over ks workgroups per tile (1: none)
};
enum class Fam32 { Dma, Regs, Mfma, Stem, Cols };
struct Plan32 {
    Fam32 fam;
    int v;  // variant or tile index within the family
};
// IM2WIN_OK, or IM2WIN_EINVAL for a forced kernel that cannot run the layer.
int plan_fp16(const Shape &sh, const Tuning &t, Plan16 *p);
// Bytes of the split-K region of a plan (the fp32 partial tiles), placed
// after the packed filter; 0 when ks = 1.
int64_t split_bytes(const Shape &sh, const Plan16 &p);
int plan_fp32(const Shape &sh, const Tuning &t, bool mfma, Plan32 *p);
// "family variant", e.g. "conv_fp16_col k3c64p128t32s2"; at most 63 characters.
void plan16_name(const Shape &sh, const Plan16 &p, char *buf, int len);
void plan32_name(const Shape &sh, const Plan32 &p, char *buf, int len);

// Kernel launchers.  Each returns a hipError_t from the launch itself; the
// shape has been validated and the plan made for it.
// The gather form of the transform indexes elements with 32 bits.
bool transform_range_ok(const Shape &sh);
// Zero padding folded into the transform: the Shape describes the padded
// layer; Hi x Wi is the input actually stored, ph/pw the zero rows above and
// below / columns left and right.
struct Pad {
    int64_t Hi, Wi, ph, pw;
};
hipError_t launch_transform(const Shape &sh, const void *in, void *ws, hipStream_t st, const Tuning &t,
                            const Pad *pad = nullptr);
hipError_t launch_pack_fp32(const Shape &sh, const Plan32 &p, const float *filt, void *packed, hipStream_t st);
// Dma and Regs plans (Mfma plans pack and launch through launch_conv_fp32_mfma).
hipError_t launch_conv_fp32(const Shape &sh, const Plan32 &p, const Tuning &t, const void *ws,
                            const void *packed, float *out, hipStream_t st);
// fp32 on the matrix cores: whether the layer can run there (C_i a multiple
// of 4, offsets in range), the bytes of its packed filter, and the launch
// (filter pack, then conv).
bool fp32_mfma_ok(const Shape &sh);
int mfma32_default(const Shape &sh);
int64_t fp32_mfma_packed_bytes(const Shape &sh);
hipError_t launch_conv_fp32_mfma(const Shape &sh, const Plan32 &p, const Tuning &t, const float *filt,
                                 void *packed, float *out, const void *ws, hipStream_t st);
// DMA-staged fp32 kernel (stages loaded straight into LDS): the default
// variant for this layer, or -1 when the register-staged kernel runs; and
// whether a variant can run the layer.
int dma32_default(const Shape &sh);
bool dma32_fits(const Shape &sh, int v);
const char *dma32_name(int v);
hipError_t launch_conv_fp32_dma(const Shape &sh, int v, const Tuning &t, const void *ws, const void *packed,
                                float *out, hipStream_t st);
// Column-staged fp32 kernel (each distinct input column of a tile loaded
// once per tap block): variant index of a name, name, fit, default (-1: the
// DMA-staged kernel runs), launch.
int cols32_find(const char *name);
const char *cols32_name(int v);
bool cols32_fits(const Shape &sh, int v);
int cols32_default(const Shape &sh);
hipError_t launch_conv_fp32_cols(const Shape &sh, int v, const Tuning &t, const void *ws, const void *packed,
                                 float *out, hipStream_t st);
// Short-window fp32 kernel (windows not 16-byte aligned, K <= 32, C_o % 4 == 0):
// its variant for the layer (-1: cannot run it), name, launch.
int stem32_plan(const Shape &sh);
int stem32_default(const Shape &sh);
const char *stem32_name(int v);
hipError_t launch_conv_fp32_stem(const Shape &sh, int v, const void *ws, const void *packed, float *out,
                                 hipStream_t st);
// Register-staged fp32 kernel: whether a tile can run the layer, its name.
bool regs32_fits(const Shape &sh, int v);
const char *regs32_name(int v);
const char *mfma32_name(int v);
// Operand type of the 16-bit matrix-core kernels (every one of them is
// instantiated for both).
enum class Op16 { F16, BF16 };
// `split`: the plan's split-K region (split_bytes(sh, p) bytes), nullptr when
// ks = 1 (the pack does not use it).
hipError_t launch_pack_fp16(const Shape &sh, const Plan16 &p, const uint16_t *filt, void *packed,
                            hipStream_t st, void *split = nullptr);
hipError_t launch_conv_fp16(const Shape &sh, const Plan16 &p, const Tuning &t, const void *ws,
                            const void *packed, uint16_t *out, hipStream_t st, Op16 op, void *split = nullptr);
// Column-staged fp16 kernel: the default variant for this layer (-1: the
// row-per-pixel kernels run), whether a variant can run it, its name and
// taps per stage (the packed-filter tile).
int col_default(const Shape &sh);
bool col_fits(const Shape &sh, int v);
const char *col_name(int v);
int col_stage_taps(int v);
// Rows of each packed filter slice of the column-staged kernel: C_o rounded up
// to the variant's channels per tile (at most C_o_pad).
int64_t col_packed_rows(const Shape &sh, int v);
// The layer runs the one-slot row-per-pixel fp16 kernel (many tiles, C_o >= 128).
bool fp16_single_slot_rows(const Shape &sh);
// Segment-staged fp16 kernel for windows that are not 16-byte aligned: the
// default variant (-1: the register-staged kernel runs), fit, name.
int seg_default(const Shape &sh);
bool seg_fits(const Shape &sh, int v);
const char *seg_name(int v);
hipError_t launch_conv_fp16_seg(const Shape &sh, int v, const void *ws, const void *packed,
                                uint16_t *out, hipStream_t st, Op16 op);
// Short-window fp16 kernel (windows not 16-byte aligned, K <= 160, C_o <= 128,
// C_o % 8 == 0): its variant for the layer (-1: cannot run it), name, launch.
int stem_plan(const Shape &sh);
int stem_default(const Shape &sh);
const char *stem_name(int v);
hipError_t launch_conv_fp16_stem(const Shape &sh, int v, const void *ws, const void *packed, uint16_t *out,
                                 hipStream_t st, Op16 op);
hipError_t launch_conv_fp16_col(const Shape &sh, int v, const Tuning &t, const void *ws, const void *packed,
                                uint16_t *out, hipStream_t st, Op16 op);
// Row-per-pixel fp16 tiles: default for the layer, name, and the K split the
// planner picks for a tile (1: none).
int pipe_default(const Shape &sh);
const char *pipe_name(int v);
int pipe_split_default(const Shape &sh, int v);
// Output tiles of a row-per-pixel variant on a layer, and its 64-tap stages.
int64_t pipe_tiles(const Shape &sh, int v);
int64_t pipe_tile_elems(int v);
} // namespace im2win
