// Output epilogue of the 16-bit (fp16 / bf16) matrix-core kernels.
//
// A wave's v_mfma_f32_32x32x16_f16 sums are spread so that lane l holds pixel
// (l & 31) and, for accumulator element e, channel 8*(e/4) + 4*(l/32) + e%4 of
// each 32x32 block: stored directly, one wave instruction writes 8-byte pieces
// of 32 different pixels' rows, and the memory pipeline pays per cache line
// touched.  Here every sum is rounded to the output type once (nearest-even), the
// workgroup's tile is assembled in LDS as [pixel][channel], and the tile is
// then copied to the NHWC output in 16-byte pieces, a wave covering whole
// consecutive pixel rows (whole 128-byte lines when the tile spans 64 or more
// channels of the output row).
#pragma once

#include "common.hpp"
#include "mfma16.hpp"

namespace im2win {

// Bytes of LDS the staged epilogue needs for a BM x BN tile.
template <int BM, int BN>
constexpr int epilogue16_bytes()
{
    return BM * BN * 2;
}

// acc[i][j]: block (i, j) of the wave whose tile starts at channel
// wch = wm*32*WM and pixel wpx = wn*32*WN of the workgroup tile (p0, ch0).
// `lds` must hold epilogue16_bytes<BM, BN>() bytes that no wave still reads or
// loads into; the function synchronises the workgroup itself.
// E (F16Op or BF16Op) rounds the sums to the output type.
template <class E, int WM, int WN, int WGM, int WGN>
__device__ inline void store_tile_lds(const f32x16_acc (&acc)[WM][WN], char *lds, uint16_t *out, uint32_t P,
                                      uint32_t Co, uint32_t p0, uint32_t ch0, uint32_t wm, uint32_t wn,
                                      uint32_t lane, uint32_t tid)
{
    constexpr int BM = 32 * WM * WGM, BN = 32 * WN * WGN, NT = 64 * WGM * WGN;
    constexpr int RB = 2 * BM;          // bytes per pixel row
    constexpr int CHR = RB / 16;        // 16-byte chunks per row
    static_assert(CHR >= 4, "at least 32 channels per tile");
    // chunk k of row px sits at slot k ^ sw(px): the 16 lanes that write one
    // channel group of 16 consecutive rows, and the lanes that read one row,
    // touch 16 different 16-byte slots of the 64 banks
    auto sw = [](uint32_t px) -> uint32_t {
        return CHR >= 16 ? (px & 15u) : CHR == 8 ? ((px ^ (px >> 3)) & 7u) : ((px ^ (px >> 2)) & 3u);
    };
    __syncthreads();
#pragma unroll
    for (int j = 0; j < WN; ++j) {
        const uint32_t px = wn * 32 * WN + 32 * j + (lane & 31);
#pragma unroll
        for (int i = 0; i < WM; ++i) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const uint32_t ch = wm * 32 * WM + 32 * i + 8 * g + 4 * (lane >> 5);
                uint32_t h[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    h[e] = E::bits(acc[i][j][4 * g + e]);
                const uint32_t k = ch / 8;
                *reinterpret_cast<uint2 *>(lds + px * RB + 16 * (k ^ sw(px)) + 2 * (ch % 8)) =
                    make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
            }
        }
    }
    __syncthreads();
    const bool vec = (Co & 7) == 0;  // 16-byte aligned output rows
    for (uint32_t c = tid; c < (uint32_t)(BN * CHR); c += NT) {
        const uint32_t px = c / CHR, k = c % CHR;
        const uint32_t p = p0 + px, ch = ch0 + 8 * k;
        if (p >= P || ch >= Co)
            continue;
        const uint4 v = *reinterpret_cast<const uint4 *>(lds + px * RB + 16 * (k ^ sw(px)));
        uint16_t *o = out + (uint64_t)p * Co + ch;
        if (vec && ch + 8 <= Co) {
            *reinterpret_cast<uint4 *>(o) = v;
        } else {
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (ch + e < Co)
                    o[e] = (uint16_t)(w[e / 2] >> (16 * (e % 2)));
        }
    }
}

// The same epilogue in two halves, for a workgroup that goes on to another
// tile: C_o a multiple of 8 (16-byte output pieces) and the tile's pieces
// dealt evenly to the threads.  Its barriers wait for LDS operations only
// (__syncthreads would also wait for loads in flight), and every thread
// issues the same epilogue16_stores() buffer stores, those past the last
// pixel or channel at out-of-range offsets that store nothing.
// Slot of 16-byte chunk k of pixel row px (CHR chunks per row): the 16 lanes
// that write one channel group of 16 consecutive rows, and the lanes that
// read one row, touch 16 different 16-byte slots of the 64 banks.
template <int CHR>
__device__ inline uint32_t epilogue16_swizzle(uint32_t px)
{
    return CHR >= 16 ? (px & 15u) : CHR == 8 ? ((px ^ (px >> 3)) & 7u) : ((px ^ (px >> 2)) & 3u);
}

template <int BM, int BN, int NT>
constexpr int epilogue16_stores()
{
    return BN * (2 * BM / 16) / NT;
}

// First half: the workgroup's rounded sums into LDS as [pixel][channel].
template <class E, int WM, int WN, int WGM, int WGN>
__device__ inline void stage_tile_lds_ring(const f32x16_acc (&acc)[WM][WN], char *lds, uint32_t wm, uint32_t wn,
                                           uint32_t lane)
{
    constexpr int BM = 32 * WM * WGM;
    constexpr int RB = 2 * BM;    // bytes per pixel row
    constexpr int CHR = RB / 16;  // 16-byte chunks per row
    static_assert(CHR >= 4, "at least 32 channels per tile");
    ring_barrier();
#pragma unroll
    for (int j = 0; j < WN; ++j) {
        const uint32_t px = wn * 32 * WN + 32 * j + (lane & 31);
#pragma unroll
        for (int i = 0; i < WM; ++i) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const uint32_t ch = wm * 32 * WM + 32 * i + 8 * g + 4 * (lane >> 5);
                uint32_t h[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    h[e] = E::bits(acc[i][j][4 * g + e]);
                const uint32_t k = ch / 8;
                *reinterpret_cast<uint2 *>(lds + px * RB + 16 * (k ^ epilogue16_swizzle<CHR>(px)) + 2 * (ch % 8)) =
                    make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
            }
        }
    }
    ring_barrier();
}

// Second half: the tile from LDS to the output, exactly
// epilogue16_stores<BM, BN, NT>() buffer stores per thread.
template <int BM, int BN, int NT>
__device__ inline void copy_tile_out_ring(const char *lds, uint16_t *out, uint32_t P, uint32_t Co, uint32_t p0,
                                          uint32_t ch0, uint32_t tid)
{
    constexpr int RB = 2 * BM;
    constexpr int CHR = RB / 16;
    static_assert((BN * CHR) % NT == 0, "whole pieces per thread");
    // rows from pixel p0 on; pixels past P fall outside the resource
    const uint32_t rows = P - p0 < (uint32_t)BN ? P - p0 : (uint32_t)BN;
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + (uint64_t)p0 * Co, rows * Co * 2u);
#pragma unroll
    for (int n = 0; n < epilogue16_stores<BM, BN, NT>(); ++n) {
        const uint32_t c = tid + (uint32_t)NT * n;
        const uint32_t px = c / CHR, k = c % CHR;
        const uint32_t ch = ch0 + 8 * k;
        const u32x4 v = *reinterpret_cast<const u32x4 *>(lds + px * RB + 16 * (k ^ epilogue16_swizzle<CHR>(px)));
        __builtin_amdgcn_raw_buffer_store_b128(v, ro, ch < Co ? (px * Co + ch) * 2u : kOOB, 0, 0);
    }
}

}  // namespace im2win
