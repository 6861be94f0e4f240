// Mini-batch (N-chunked) im2win: the transform and the windowed convolution
// run on chunks of n_chunk images, so the workspace holds the window tensor of
// one chunk (or two, double-buffered) instead of the whole batch.  The paper
// processes the full batch at once and notes the memory this costs next to
// mini-batch methods (Sec. IV-C); this entry point bounds it.  With a second
// stream, alternate chunks run on the two streams, so two chunks are in flight
// and the transform of one overlaps the convolution of the other.
//
// The kernel plan is made once, from the shape of a full chunk, and used for the
// filter pack and for every chunk, the last (possibly smaller) one included, so
// the packed filter always has the layout the kernel reads.  The output equals,
// bit for bit, that of the full-batch entry points run on a chunk-sized batch;
// against a full-batch call it may differ in the last bits where the larger
// batch selects another kernel (another summation order).
#include "common.hpp"

#include "../../include/im2win.h"

#include <mutex>
#include <string.h>

namespace im2win {
namespace {

constexpr int64_t kSlotAlign = 256;

struct Plan {
    Shape chunk;        // shape of a full chunk (n_chunk images)
    int64_t n_chunk;
    int64_t nslots;
    int64_t slot_bytes;
    int64_t packed_off;
    int64_t ws_bytes;
};

int make_plan(int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w,
              int64_t stride, int64_t n_chunk, int two_streams, int dt, Plan *p)
{
    if (n_chunk <= 0 || N <= 0)
        return IM2WIN_EINVAL;
    Shape full;
    int rc = make_shape(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dt, &full);
    if (rc != IM2WIN_OK)
        return rc;
    p->n_chunk = n_chunk < N ? n_chunk : N;
    if ((rc = make_shape(p->n_chunk, C_i, H_i, W_i, C_o, K_h, K_w, stride, dt, &p->chunk)) != IM2WIN_OK)
        return rc;
    if (!transform_range_ok(p->chunk))
        return IM2WIN_ERANGE;
    p->nslots = two_streams ? 2 : 1;
    p->slot_bytes = round_up(p->chunk.pad_end, kSlotAlign);
    p->packed_off = p->nslots * p->slot_bytes;
    p->ws_bytes = p->packed_off + packed_filter_bytes(p->chunk, dt);
    return IM2WIN_OK;
}

// Enqueues the filter pack and every chunk (arguments checked by the caller).
int enqueue_chunks(const void *in, const void *filt, void *out, char *wsb, const Plan &p, const Plan16 &p16,
                   const Plan32 &p32, const Tuning &tu, int64_t N, int64_t C_i, int64_t H_i, int64_t W_i,
                   int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride, int dt, hipStream_t st, hipStream_t aux,
                   hipEvent_t ev_start, hipEvent_t ev_done)
{
    int rc;
    Shape full;
    make_shape(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dt, &full);
    const int64_t elt = full.elt;
    void *packed = wsb + p.packed_off;
    // the filter is packed once, for the plan every chunk runs
    if (dt == IM2WIN_F32)
        rc = launch_status(launch_pack_fp32(p.chunk, p32, static_cast<const float *>(filt), packed, st));
    else
        rc = launch_status(launch_pack_fp16(p.chunk, p16, static_cast<const uint16_t *>(filt), packed, st));
    if (rc != IM2WIN_OK)
        return rc;
    // With two streams, chunk c runs (transform, then conv) on stream c % 2
    // in slot c % 2: two chunks are in flight at once, the transform of one
    // overlapping the conv of the other, and a slot is reused only by later
    // work on the same stream.  The aux stream starts after everything already
    // queued on `st` (the input, the packed filter, earlier users of this
    // workspace) and `st` finally waits for the aux stream.
    if (aux != nullptr) {
        if (hipEventRecord(ev_start, st) != hipSuccess || hipStreamWaitEvent(aux, ev_start, 0) != hipSuccess)
            return IM2WIN_ELAUNCH;
    }
    const int64_t in_img = H_i * W_i * C_i * elt, out_img = full.Ho * full.Wo * C_o * elt;
    const int64_t nchunks = (N + p.n_chunk - 1) / p.n_chunk;
    for (int64_t c = 0; c < nchunks; ++c) {
        const int64_t i0 = c * p.n_chunk;
        const int64_t n = N - i0 < p.n_chunk ? N - i0 : p.n_chunk;
        Shape sh = p.chunk;
        if (n != p.n_chunk)
            make_shape(n, C_i, H_i, W_i, C_o, K_h, K_w, stride, dt, &sh);
        const int slot = (int)(c % p.nslots);
        char *wsl = wsb + slot * p.slot_bytes;
        const char *inc = static_cast<const char *>(in) + i0 * in_img;
        char *outc = static_cast<char *>(out) + i0 * out_img;
        hipStream_t cs = (aux != nullptr && slot == 1) ? aux : st;
        if ((rc = launch_status(launch_transform(sh, inc, wsl, cs, tu))) != IM2WIN_OK)
            return rc;
        if (dt == IM2WIN_F32)
            rc = launch_status(launch_conv_fp32(sh, p32, tu, wsl, packed, reinterpret_cast<float *>(outc), cs));
        else
            rc = launch_status(launch_conv_fp16(sh, p16, tu, wsl, packed, reinterpret_cast<uint16_t *>(outc), cs,
                                                dt == IM2WIN_BF16 ? Op16::BF16 : Op16::F16));
        if (rc != IM2WIN_OK)
            return rc;
    }
    if (aux != nullptr) {
        if (hipEventRecord(ev_done, aux) != hipSuccess || hipStreamWaitEvent(st, ev_done, 0) != hipSuccess)
            return IM2WIN_ELAUNCH;
    }
    return IM2WIN_OK;
}

// Checks the arguments of a mini-batch call (the workspace only when `ws` is
// given) and makes its plans.
int check_chunked(const void *in, const void *filt, void *out, void *ws, int64_t ws_bytes, int64_t N, int64_t C_i,
                  int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride,
                  int64_t n_chunk, int dt, hipStream_t st, hipStream_t aux, Plan *p, Tuning *tu, Plan16 *p16,
                  Plan32 *p32)
{
    if (!in || !filt || !out)
        return IM2WIN_EINVAL;
    int rc = make_plan(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, n_chunk, aux != nullptr, dt, p);
    if (rc != IM2WIN_OK)
        return rc;
    if (aux != nullptr && aux == st)
        return IM2WIN_EINVAL;
    if (!aligned16(in) || !aligned16(filt) || !aligned16(out) || (ws && !aligned16(ws)))
        return IM2WIN_EALIGN;
    Shape full;
    make_shape(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, dt, &full);
    const int64_t elt = full.elt;
    const int64_t in_bytes = N * H_i * W_i * C_i * elt, f_bytes = full.K * C_o * elt,
                  o_bytes = full.P * C_o * elt;
    if (ws && ws_bytes < 0)
        return IM2WIN_EWORKSPACE;
    if ((rc = check_extent(in, in_bytes)) != IM2WIN_OK || (rc = check_extent(filt, f_bytes)) != IM2WIN_OK ||
        (rc = check_extent(out, o_bytes)) != IM2WIN_OK || (ws && (rc = check_extent(ws, ws_bytes)) != IM2WIN_OK))
        return rc;
    if (overlaps(in, in_bytes, out, o_bytes) || overlaps(filt, f_bytes, out, o_bytes))
        return IM2WIN_EOVERLAP;
    if (ws && (overlaps(in, in_bytes, ws, ws_bytes) || overlaps(filt, f_bytes, ws, ws_bytes) ||
               overlaps(out, o_bytes, ws, ws_bytes)))
        return IM2WIN_EOVERLAP;
    if (ws && ws_bytes < p->ws_bytes)
        return IM2WIN_EWORKSPACE;
    if ((rc = read_tuning(tu)) != IM2WIN_OK)
        return rc;
    if (dt == IM2WIN_F32)
        return plan_fp32(p->chunk, *tu, false, p32);
    // Chunks run the row-per-pixel kernel without a K split: the split's
    // counters and partial tiles would be shared by the chunks in flight on
    // the two streams.  A split forced through the tuning is refused.
    if (tu->fp16_split > 1)
        return IM2WIN_EINVAL;
    tu->fp16_split = 1;
    return plan_fp16(p->chunk, *tu, p16);
}

int run_chunked(const void *in, const void *filt, void *out, void *ws, int64_t ws_bytes, int64_t N,
                int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w,
                int64_t stride, int64_t n_chunk, int dt, hipStream_t st, hipStream_t aux)
{
    if (!ws)
        return IM2WIN_EINVAL;
    Plan p;
    Tuning tu;
    Plan16 p16{};
    Plan32 p32{};
    int rc = check_chunked(in, filt, out, ws, ws_bytes, N, C_i, H_i, W_i, C_o, K_h, K_w, stride, n_chunk, dt, st,
                           aux, &p, &tu, &p16, &p32);
    if (rc != IM2WIN_OK)
        return rc;
    if ((rc = check_device()) != IM2WIN_OK)
        return rc;
    // Two events order the streams; they are made here and released at the
    // end of the call (a recorded event that is destroyed is released once
    // it completes, and the waits already enqueued on it stay in force).
    hipEvent_t ev_start = nullptr, ev_done = nullptr;
    if (aux != nullptr) {
        if (hipEventCreateWithFlags(&ev_start, hipEventDisableTiming) != hipSuccess)
            return launch_status(hipErrorOutOfMemory);
        if (hipEventCreateWithFlags(&ev_done, hipEventDisableTiming) != hipSuccess) {
            (void)hipEventDestroy(ev_start);
            return launch_status(hipErrorOutOfMemory);
        }
    }
    rc = enqueue_chunks(in, filt, out, static_cast<char *>(ws), p, p16, p32, tu, N, C_i, H_i, W_i, C_o, K_h, K_w,
                        stride, dt, st, aux, ev_start, ev_done);
    if (aux != nullptr) {
        (void)hipEventDestroy(ev_start);
        (void)hipEventDestroy(ev_done);
    }
    return rc;
}

// The workspace of the allocation-free mini-batch call: a static device
// array, one copy on every GPU the library runs on, held until the process
// ends.  Host code never uses the array's name as an address: each device's
// copy is found once, with that device current, through
// hipGetSymbolAddress, and that pointer is what the kernels receive.
constexpr int64_t kScratchBytes = IM2WIN_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDev = 64;
struct ScratchDev {
    std::once_flag once;
    int rc = IM2WIN_ENODEV;
    void *ptr = nullptr;
};
ScratchDev g_scratch[kMaxDev];

// This device's copy of `scratch` (set up on the first call per device).
int scratch_for_current_device(void **out)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) {
        (void)hipGetLastError();
        return IM2WIN_ENODEV;
    }
    ScratchDev &d = g_scratch[dev];
    std::call_once(d.once, [&d]() {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            d.rc = IM2WIN_ENODEV;
            return;
        }
        d.ptr = p;
        d.rc = IM2WIN_OK;
    });
    *out = d.ptr;
    return d.rc;
}

int run_chunked_noalloc(const void *in, const void *filt, void *out, int64_t N, int64_t C_i, int64_t H_i,
                        int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w, int64_t stride, int64_t n_chunk, int dt,
                        hipStream_t st)
{
    Plan p;
    Tuning tu;
    Plan16 p16{};
    Plan32 p32{};
    int rc = check_chunked(in, filt, out, nullptr, 0, N, C_i, H_i, W_i, C_o, K_h, K_w, stride, n_chunk, dt, st,
                           nullptr, &p, &tu, &p16, &p32);
    if (rc != IM2WIN_OK)
        return rc;
    if (p.ws_bytes > kScratchBytes)
        return IM2WIN_EWORKSPACE;
    if ((rc = check_device()) != IM2WIN_OK)
        return rc;
    void *ws = nullptr;
    if ((rc = scratch_for_current_device(&ws)) != IM2WIN_OK)
        return rc;
    // one stream, one slot: no events are needed
    return enqueue_chunks(in, filt, out, static_cast<char *>(ws), p, p16, p32, tu, N, C_i, H_i, W_i, C_o, K_h, K_w,
                          stride, dt, st, nullptr, nullptr, nullptr);
}

}  // namespace
}  // namespace im2win

using namespace im2win;

extern "C" {

int64_t conv_chunked_workspace_bytes(int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o,
                                     int64_t K_h, int64_t K_w, int64_t stride, int64_t n_chunk,
                                     int two_streams, im2win_dtype_t dt)
{
    if (dt != IM2WIN_F32 && dt != IM2WIN_F16 && dt != IM2WIN_BF16)
        return IM2WIN_EINVAL;
    Plan p;
    int rc = make_plan(N, C_i, H_i, W_i, C_o, K_h, K_w, stride, n_chunk, two_streams, (int)dt, &p);
    if (rc != IM2WIN_OK)
        return rc;
    return p.ws_bytes;
}

int conv_im2win_chunked(const void *in_nhwc, const void *filt_khkwcico, void *out_nhwc, void *ws,
                        int64_t ws_bytes, int64_t N, int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o,
                        int64_t K_h, int64_t K_w, int64_t stride, int64_t n_chunk, im2win_dtype_t dt,
                        void *hip_stream, void *hip_stream_aux)
{
    if (dt != IM2WIN_F32 && dt != IM2WIN_F16 && dt != IM2WIN_BF16)
        return IM2WIN_EINVAL;
    return run_chunked(in_nhwc, filt_khkwcico, out_nhwc, ws, ws_bytes, N, C_i, H_i, W_i, C_o, K_h, K_w, stride,
                       n_chunk, (int)dt, (hipStream_t)hip_stream, (hipStream_t)hip_stream_aux);
}

int conv_im2win_chunked_noalloc(const void *in_nhwc, const void *filt_khkwcico, void *out_nhwc, int64_t N,
                                int64_t C_i, int64_t H_i, int64_t W_i, int64_t C_o, int64_t K_h, int64_t K_w,
                                int64_t stride, int64_t n_chunk, im2win_dtype_t dt, void *hip_stream)
{
    if (dt != IM2WIN_F32 && dt != IM2WIN_F16 && dt != IM2WIN_BF16)
        return IM2WIN_EINVAL;
    return run_chunked_noalloc(in_nhwc, filt_khkwcico, out_nhwc, N, C_i, H_i, W_i, C_o, K_h, K_w, stride, n_chunk,
                               (int)dt, (hipStream_t)hip_stream);
}

}  // extern "C"
