// Kernel choice: the tuning variables and the plan each conv call runs.
//
// A conv call makes its plan once, on the host, from the layer's shape and
// the (checked) tuning variables, and hands the same plan to the filter pack
// and to the conv launch, so the packed-filter layout always matches the
// kernel that reads it.  conv_im2win_kernel_name reports the plan.
#include "../../include/im2win.h"
#include "common.hpp"

#include <stdio.h>
#include <stdlib.h>
#include <string.h>

namespace im2win {

namespace {

// Variable unset or empty: not forced (-1).  Otherwise the index `find`
// gives, or IM2WIN_EINVAL for a name no kernel has.
int read_name(const char *var, int (*find)(const char *), int *out)
{
    *out = -1;
    const char *e = getenv(var);
    if (!e || !*e)
        return IM2WIN_OK;
    *out = find(e);
    return *out >= 0 ? IM2WIN_OK : IM2WIN_EINVAL;
}

// linear | xcd (the default); anything else is an error.
int read_order(const char *var, const char *other, bool *linear)
{
    *linear = false;
    const char *e = getenv(var);
    if (!e || !*e || strcmp(e, other) == 0)
        return IM2WIN_OK;
    if (strcmp(e, "linear") == 0) {
        *linear = true;
        return IM2WIN_OK;
    }
    return IM2WIN_EINVAL;
}

}  // namespace

int read_tuning(Tuning *t)
{
    int rc;
    t->fp16_kernel = Tuning::kAuto;
    if (const char *e = getenv("IM2WIN_FP16_KERNEL")) {
        if (strcmp(e, "pipe") == 0)
            t->fp16_kernel = Tuning::kPipe;
        else if (strcmp(e, "regs") == 0)
            t->fp16_kernel = Tuning::kRegs;
        else if (strcmp(e, "stem") == 0)
            t->fp16_kernel = Tuning::kStem;
        else if (*e)
            return IM2WIN_EINVAL;
    }
    if ((rc = read_name("IM2WIN_FP16_COL", col_find, &t->fp16_col)) != IM2WIN_OK ||
        (rc = read_name("IM2WIN_FP16_TILE", pipe_find, &t->fp16_tile)) != IM2WIN_OK ||
        (rc = read_name("IM2WIN_FP16_SEG", seg_find, &t->fp16_seg)) != IM2WIN_OK ||
        (rc = read_name("IM2WIN_FP32_TILE", regs32_find, &t->fp32_tile)) != IM2WIN_OK ||
        (rc = read_name("IM2WIN_FP32_MFMA_TILE", mfma32_find, &t->fp32_mfma_tile)) != IM2WIN_OK ||
        (rc = read_name("IM2WIN_FP32_COLS", cols32_find, &t->fp32_cols)) != IM2WIN_OK)
        return rc;
    const char *e = getenv("IM2WIN_FP32_KERNEL");
    if (e && strcmp(e, "regs") == 0)
        t->fp32_kernel = -2;
    else if (e && strcmp(e, "stem") == 0)
        t->fp32_kernel = -3;
    else if ((rc = read_name("IM2WIN_FP32_KERNEL", dma32_find, &t->fp32_kernel)) != IM2WIN_OK)
        return rc;
    if ((rc = read_order("IM2WIN_TRANSFORM_ORDER", "xcd", &t->transform_linear)) != IM2WIN_OK ||
        (rc = read_order("IM2WIN_TILE_ORDER", "xcd", &t->tile_linear)) != IM2WIN_OK)
        return rc;
    t->col_persist = true;
    if (const char *e = getenv("IM2WIN_FP16_PERSIST")) {
        if (strcmp(e, "off") == 0)
            t->col_persist = false;
        else if (*e && strcmp(e, "on") != 0)
            return IM2WIN_EINVAL;
    }
    t->transform_gather = false;
    if (const char *e = getenv("IM2WIN_TRANSFORM_KERNEL")) {
        if (strcmp(e, "gather") == 0)
            t->transform_gather = true;
        else if (*e && strcmp(e, "pieces") != 0)
            return IM2WIN_EINVAL;
    }
    t->tap_order = Tuning::kDefault;
    if (const char *e = getenv("IM2WIN_TAP_ORDER")) {
        if (strcmp(e, "linear") == 0)
            t->tap_order = Tuning::kLinear;
        else if (strcmp(e, "column") == 0)
            t->tap_order = Tuning::kColumn;
        else if (*e)
            return IM2WIN_EINVAL;
    }
    t->fp16_split = 0;
    if (const char *e = getenv("IM2WIN_FP16_SPLIT")) {
        if (*e) {
            char *end = nullptr;
            const long v = strtol(e, &end, 10);
            if (*end != 0 || v < 1 || v > kMaxSplit)
                return IM2WIN_EINVAL;
            t->fp16_split = (int)v;
        }
    }
    // contradictory choices
    const int fam16 = (t->fp16_col >= 0) + (t->fp16_seg >= 0) + (t->fp16_tile >= 0 || t->fp16_kernel == Tuning::kPipe) +
                      (t->fp16_kernel == Tuning::kRegs) + (t->fp16_kernel == Tuning::kStem);
    if (fam16 > 1)
        return IM2WIN_EINVAL;
    if ((t->fp32_tile >= 0) + (t->fp32_kernel >= 0 || t->fp32_kernel == -3 || t->fp32_kernel == -2) +
            (t->fp32_cols >= 0) > 1)
        return IM2WIN_EINVAL;
    return IM2WIN_OK;
}

Tuning default_tuning()
{
    Tuning t;
    t.fp16_kernel = Tuning::kAuto;
    t.fp16_col = t.fp16_tile = t.fp16_seg = -1;
    t.fp32_kernel = t.fp32_tile = t.fp32_mfma_tile = t.fp32_cols = -1;
    t.transform_linear = t.tile_linear = false;
    t.transform_gather = false;
    t.col_persist = true;
    t.tap_order = Tuning::kDefault;
    t.fp16_split = 0;
    return t;
}

namespace {

// Every one of the ks K ranges of ceil(nst / ks) stages is non-empty.
bool split_ok(const Shape &sh, int ks)
{
    const int64_t nst = sh.K_pad / 64, spl = (nst + ks - 1) / ks;
    return ks >= 1 && ks <= kMaxSplit && (ks - 1) * spl < nst;
}

// The K split of a row-per-pixel plan: forced by the tuning, else the
// planner's choice for the variant.
int with_split(const Shape &sh, const Tuning &t, Plan16 *p)
{
    p->ks = 1;
    if (p->fam != Fam16::Pipe) {
        return t.fp16_split > 1 ? IM2WIN_EINVAL : IM2WIN_OK;
    }
    const int ks = t.fp16_split > 0 ? t.fp16_split : pipe_split_default(sh, p->v);
    if (!split_ok(sh, ks))
        return IM2WIN_EINVAL;
    p->ks = ks;
    return IM2WIN_OK;
}

int plan_fp16_family(const Shape &sh, const Tuning &t, Plan16 *p);

}  // namespace

int64_t split_bytes(const Shape &sh, const Plan16 &p)
{
    if (p.fam != Fam16::Pipe || p.ks <= 1)
        return 0;
    return (int64_t)p.ks * pipe_tiles(sh, p.v) * pipe_tile_elems(p.v) * 4;
}

int plan_fp16(const Shape &sh, const Tuning &t, Plan16 *p)
{
    const int rc = plan_fp16_family(sh, t, p);
    return rc != IM2WIN_OK ? rc : with_split(sh, t, p);
}

namespace {

int plan_fp16_family(const Shape &sh, const Tuning &t, Plan16 *p)
{
    const bool aligned = sh.Ci % 8 == 0;  // every window starts on a 16-byte boundary
    // register-staged tile by output channels
    const int regs_tile = sh.Co <= 32 ? 0 : sh.Co <= 64 ? 1 : 2;
    if (t.fp16_kernel == Tuning::kRegs) {
        *p = Plan16{Fam16::Regs, regs_tile};
        return IM2WIN_OK;
    }
    if (t.fp16_kernel == Tuning::kStem) {
        const int v = stem_plan(sh);
        if (v < 0)
            return IM2WIN_EINVAL;
        *p = Plan16{Fam16::Stem, v};
        return IM2WIN_OK;
    }
    if (t.fp16_col >= 0) {
        if (!col_fits(sh, t.fp16_col))
            return IM2WIN_EINVAL;
        *p = Plan16{Fam16::Col, t.fp16_col};
        return IM2WIN_OK;
    }
    if (t.fp16_seg >= 0) {
        if (aligned || !seg_fits(sh, t.fp16_seg))
            return IM2WIN_EINVAL;
        *p = Plan16{Fam16::Seg, t.fp16_seg};
        return IM2WIN_OK;
    }
    if (t.fp16_tile >= 0 || t.fp16_kernel == Tuning::kPipe) {
        if (!aligned)
            return IM2WIN_EINVAL;
        *p = Plan16{Fam16::Pipe, t.fp16_tile >= 0 ? t.fp16_tile : pipe_default(sh)};
        return IM2WIN_OK;
    }
    if (aligned) {
        const int c = col_default(sh);
        *p = c >= 0 ? Plan16{Fam16::Col, c} : Plan16{Fam16::Pipe, pipe_default(sh)};
        return IM2WIN_OK;
    }
    const int sm = stem_default(sh);
    if (sm >= 0) {
        *p = Plan16{Fam16::Stem, sm};
        return IM2WIN_OK;
    }
    const int sg = seg_default(sh);
    *p = sg >= 0 ? Plan16{Fam16::Seg, sg} : Plan16{Fam16::Regs, regs_tile};
    return IM2WIN_OK;
}

}  // namespace

int plan_fp32(const Shape &sh, const Tuning &t, bool mfma, Plan32 *p)
{
    if (mfma) {
        if (fp32_mfma_ok(sh)) {
            *p = Plan32{Fam32::Mfma, t.fp32_mfma_tile >= 0 ? t.fp32_mfma_tile : mfma32_default(sh)};
            return IM2WIN_OK;
        }
        // layers the matrix-core kernel cannot take run the vector-ALU
        // kernels (documented); a forced matrix-core tile is an error
        if (t.fp32_mfma_tile >= 0)
            return IM2WIN_EINVAL;
    }
    if (t.fp32_kernel >= 0) {
        if (!dma32_fits(sh, t.fp32_kernel))
            return IM2WIN_EINVAL;
        *p = Plan32{Fam32::Dma, t.fp32_kernel};
        return IM2WIN_OK;
    }
    if (t.fp32_cols >= 0) {
        if (!cols32_fits(sh, t.fp32_cols))
            return IM2WIN_EINVAL;
        *p = Plan32{Fam32::Cols, t.fp32_cols};
        return IM2WIN_OK;
    }
    if (t.fp32_kernel == -3) {
        const int v = stem32_plan(sh);
        if (v < 0)
            return IM2WIN_EINVAL;
        *p = Plan32{Fam32::Stem, v};
        return IM2WIN_OK;
    }
    if (t.fp32_kernel == -2 || t.fp32_tile >= 0) {
        const int v = t.fp32_tile >= 0 ? t.fp32_tile : 0;
        if (!regs32_fits(sh, v)) {
            if (t.fp32_tile >= 0)
                return IM2WIN_EINVAL;
            *p = Plan32{Fam32::Regs, regs32_find("m4n16p2")};  // filter read from global memory
            return IM2WIN_OK;
        }
        *p = Plan32{Fam32::Regs, v};
        return IM2WIN_OK;
    }
    const int sm = stem32_default(sh);
    if (sm >= 0) {
        *p = Plan32{Fam32::Stem, sm};
        return IM2WIN_OK;
    }
    const int cl = cols32_default(sh);
    if (cl >= 0) {
        *p = Plan32{Fam32::Cols, cl};
        return IM2WIN_OK;
    }
    const int d = dma32_default(sh);
    if (d >= 0) {
        *p = Plan32{Fam32::Dma, d};
        return IM2WIN_OK;
    }
    *p = Plan32{Fam32::Regs, regs32_fits(sh, 0) ? 0 : regs32_find("m4n16p2")};
    return IM2WIN_OK;
}

void plan16_name(const Shape &sh, const Plan16 &p, char *buf, int len)
{
    switch (p.fam) {
    case Fam16::Col: snprintf(buf, len, "conv_fp16_col %s", col_name(p.v)); break;
    case Fam16::Pipe:
        if (p.ks > 1)
            snprintf(buf, len, "conv_fp16_pipe %s k%d", pipe_name(p.v), p.ks);
        else
            snprintf(buf, len, "conv_fp16_pipe %s", pipe_name(p.v));
        break;
    case Fam16::Seg: snprintf(buf, len, "conv_fp16_seg %s", seg_name(p.v)); break;
    case Fam16::Stem: snprintf(buf, len, "conv_fp16_stem %s", stem_name(p.v)); break;
    case Fam16::Regs: {
        static const char *tiles[] = {"c32p256", "c64p256", "c128p128"};
        // unaligned 16-byte loads for windows of 128 taps or more, element
        // loads for shorter ones
        snprintf(buf, len, "conv_fp16_kernel %s%s", tiles[p.v], sh.K >= 128 ? "u" : "e");
        break;
    }
    }
}

void plan32_name(const Shape &sh, const Plan32 &p, char *buf, int len)
{
    (void)sh;
    switch (p.fam) {
    case Fam32::Dma: snprintf(buf, len, "conv_fp32_dma %s", dma32_name(p.v)); break;
    case Fam32::Regs: snprintf(buf, len, "conv_fp32_kernel %s", regs32_name(p.v)); break;
    case Fam32::Stem: snprintf(buf, len, "conv_fp32_stem %s", stem32_name(p.v)); break;
    case Fam32::Cols: snprintf(buf, len, "conv_fp32_cols %s", cols32_name(p.v)); break;
    case Fam32::Mfma: snprintf(buf, len, "conv_fp32_mfma %s", mfma32_name(p.v)); break;
    }
}

}  // namespace im2win
