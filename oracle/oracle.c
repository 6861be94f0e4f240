/*
 * Oracle for im2win convolution -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct CPU reference in double precision.  Only
 * the test-suite, the package smoke check and the CPU-baseline leg of the
 * benchmark may load it; the product path never calls, links or imports it.
 * It shares no source, header, table or helper with the GPU library.
 *
 * Conventions (the readings of the paper that the tests pin):
 *   - tensors are NHWC: input I[N][H_i][W_i][C_i], output O[N][H_o][W_o][C_o];
 *   - the filter is stored F[K_h][K_w][C_i][C_o] (height, width, input
 *     channel, output channel);
 *   - indices are 0-based, one stride s for both spatial axes, no padding
 *     (except in the two *_pad functions), no dilation, no groups, no bias,
 *     no filter flip (cross-correlation);
 *   - H_o = floor((H_i - K_h) / s) + 1 and W_o likewise (Table I sizes).
 *
 * Every function follows one passage of the paper:
 *   oracle_conv_f64            Sec. III-A, Eq. (1), with the stride written in
 *   oracle_conv_f64_points     Eq. (1) at selected output coordinates
 *   oracle_im2win              Sec. III-B, Eq. (2), NHWC element order
 *   oracle_windowed_conv_f64   Sec. III-C, Eq. (3): the same sums read out of
 *                              the window tensor
 *   oracle_window_elems /      element counts of the window tensor (Eq. 2
 *   oracle_im2col_elems        index ranges) and of the im2col matrix
 *                              (Sec. III-B, Fig. 1 right)
 *   oracle_conv_pad_f64 /      Eq. (1) and Eq. (2) on a zero-padded input
 *   oracle_im2win_pad          (an extension: the paper's layers have no
 *                              padding), read through an index rule, never
 *                              built
 *   oracle_conv_dil_f64 /      Eq. (1), Eq. (2) and Eq. (3) with filter
 *   oracle_im2win_dil /        dilation (an extension, with padding): taps
 *   oracle_windowed_conv_dil_f64  d apart, and a window tensor whose strip
 *                              columns are grouped by residue mod d so that
 *                              every window stays one contiguous span
 */
#include <stdint.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Output extent along one spatial axis (no padding). Returns -1 when the
 * filter does not fit or an argument is out of range. */
int64_t oracle_out_extent(int64_t in, int64_t k, int64_t s)
{
    if (in <= 0 || k <= 0 || s <= 0 || k > in)
        return -1;
    return (in - k) / s + 1;
}

int oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads the following parallel loops use (timing only; results do not
 * depend on it: each output is summed by one thread in a fixed order). */
void oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/*
 * Eq. (1), written with the stride:
 *   O[i][m][n][j] = sum_u sum_v sum_r I[i][m*s+u][n*s+v][r] * F[u][v][r][j]
 * and, as the tolerance denominator of the parity tests,
 *   A[i][m][n][j] = sum_u sum_v sum_r |I[i][m*s+u][n*s+v][r]| * |F[u][v][r][j]|.
 * Seven nested loops, one fp64 accumulator per output, fixed order
 * (i, m, n, j, u, v, r).  `absout` may be NULL.
 */
int oracle_conv_f64(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi, int64_t Co,
                    int64_t Kh, int64_t Kw, int64_t s,
                    const double *in, const double *filt,
                    double *out, double *absout)
{
    int64_t Ho = oracle_out_extent(Hi, Kh, s);
    int64_t Wo = oracle_out_extent(Wi, Kw, s);
    if (N <= 0 || Ci <= 0 || Co <= 0 || Ho < 0 || Wo < 0)
        return -1;

#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < N; ++i) {
        for (int64_t m = 0; m < Ho; ++m) {
            for (int64_t n = 0; n < Wo; ++n) {
                for (int64_t j = 0; j < Co; ++j) {
                    double acc = 0.0, aacc = 0.0;
                    for (int64_t u = 0; u < Kh; ++u) {
                        for (int64_t v = 0; v < Kw; ++v) {
                            for (int64_t r = 0; r < Ci; ++r) {
                                double x = in[((i * Hi + (m * s + u)) * Wi + (n * s + v)) * Ci + r];
                                double w = filt[((u * Kw + v) * Ci + r) * Co + j];
                                acc += x * w;
                                aacc += fabs(x) * fabs(w);
                            }
                        }
                    }
                    int64_t o = ((i * Ho + m) * Wo + n) * Co + j;
                    out[o] = acc;
                    if (absout)
                        absout[o] = aacc;
                }
            }
        }
    }
    return 0;
}

/*
 * Eq. (1) at `npts` chosen output coordinates.  `pts` holds 4 int64 per point
 * (i, m, n, j); out[p] / absout[p] receive the sum and the |x||w| sum.
 */
int oracle_conv_f64_points(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi, int64_t Co,
                           int64_t Kh, int64_t Kw, int64_t s,
                           const double *in, const double *filt,
                           int64_t npts, const int64_t *pts,
                           double *out, double *absout)
{
    int64_t Ho = oracle_out_extent(Hi, Kh, s);
    int64_t Wo = oracle_out_extent(Wi, Kw, s);
    if (N <= 0 || Ci <= 0 || Co <= 0 || Ho < 0 || Wo < 0 || npts < 0)
        return -1;
    for (int64_t p = 0; p < npts; ++p) {
        int64_t i = pts[4 * p], m = pts[4 * p + 1], n = pts[4 * p + 2], j = pts[4 * p + 3];
        if (i < 0 || i >= N || m < 0 || m >= Ho || n < 0 || n >= Wo || j < 0 || j >= Co)
            return -1;
    }

#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t p = 0; p < npts; ++p) {
        int64_t i = pts[4 * p], m = pts[4 * p + 1], n = pts[4 * p + 2], j = pts[4 * p + 3];
        double acc = 0.0, aacc = 0.0;
        for (int64_t u = 0; u < Kh; ++u) {
            for (int64_t v = 0; v < Kw; ++v) {
                for (int64_t r = 0; r < Ci; ++r) {
                    double x = in[((i * Hi + (m * s + u)) * Wi + (n * s + v)) * Ci + r];
                    double w = filt[((u * Kw + v) * Ci + r) * Co + j];
                    acc += x * w;
                    aacc += fabs(x) * fabs(w);
                }
            }
        }
        out[p] = acc;
        if (absout)
            absout[p] = aacc;
    }
    return 0;
}

/* Element count of the window tensor: Eq. (2) ranges i<N, m<H_o, k<W_i,
 * u<K_h, r<C_i. */
int64_t oracle_window_elems(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi,
                            int64_t Kh, int64_t s)
{
    int64_t Ho = oracle_out_extent(Hi, Kh, s);
    if (N <= 0 || Ci <= 0 || Ho < 0)
        return -1;
    return N * Ho * Wi * Kh * Ci;
}

/* Element count of the full-batch im2col matrix: one row per output pixel,
 * one column per filter tap and input channel (Fig. 1, right). */
int64_t oracle_im2col_elems(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi,
                            int64_t Kh, int64_t Kw, int64_t s)
{
    int64_t Ho = oracle_out_extent(Hi, Kh, s);
    int64_t Wo = oracle_out_extent(Wi, Kw, s);
    if (N <= 0 || Ci <= 0 || Ho < 0 || Wo < 0)
        return -1;
    return N * Ho * Wo * Kh * Kw * Ci;
}

/*
 * Eq. (2) in NHWC element order:
 *   W[i][m][k*K_h + u][r] = I[i][m*s + u][k][r],
 * for i<N, m<H_o, k<W_i, u<K_h, r<C_i.  Each output row m gets one strip of
 * W_i*K_h*C_i elements: input column k of the K_h rows the output row needs,
 * stacked row after row, channels fastest.  Elements are copied as raw bytes
 * (`elt` bytes each), so the result is bit-exact for any element type.
 */
int oracle_im2win(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi,
                  int64_t Kh, int64_t s, int64_t elt,
                  const void *in, void *out)
{
    int64_t Ho = oracle_out_extent(Hi, Kh, s);
    if (N <= 0 || Ci <= 0 || Ho < 0 || elt <= 0)
        return -1;
    const unsigned char *src = (const unsigned char *)in;
    unsigned char *dst = (unsigned char *)out;

#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < N; ++i) {
        for (int64_t m = 0; m < Ho; ++m) {
            for (int64_t k = 0; k < Wi; ++k) {
                for (int64_t u = 0; u < Kh; ++u) {
                    for (int64_t r = 0; r < Ci; ++r) {
                        int64_t d = ((i * Ho + m) * (Wi * Kh) + (k * Kh + u)) * Ci + r;
                        int64_t x = ((i * Hi + (m * s + u)) * Wi + k) * Ci + r;
                        memcpy(dst + d * elt, src + x * elt, (size_t)elt);
                    }
                }
            }
        }
    }
    return 0;
}

/*
 * Eq. (3): the convolution read out of the window tensor.  The window of
 * output (i, m, n) lies in strip (i, m); tap (u, v) of input channel r sits at
 * strip element ((n*s + v)*K_h + u)*C_i + r.  The next output column moves
 * the window s*K_h*C_i elements along the strip; the next output row moves to
 * the next strip.
 */
int oracle_windowed_conv_f64(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi, int64_t Co,
                             int64_t Kh, int64_t Kw, int64_t s,
                             const double *win, const double *filt, double *out)
{
    int64_t Ho = oracle_out_extent(Hi, Kh, s);
    int64_t Wo = oracle_out_extent(Wi, Kw, s);
    if (N <= 0 || Ci <= 0 || Co <= 0 || Ho < 0 || Wo < 0)
        return -1;
    int64_t strip = Wi * Kh * Ci;

#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < N; ++i) {
        for (int64_t m = 0; m < Ho; ++m) {
            const double *w = win + (i * Ho + m) * strip;
            for (int64_t n = 0; n < Wo; ++n) {
                for (int64_t j = 0; j < Co; ++j) {
                    double acc = 0.0;
                    for (int64_t u = 0; u < Kh; ++u) {
                        for (int64_t v = 0; v < Kw; ++v) {
                            for (int64_t r = 0; r < Ci; ++r) {
                                double x = w[((n * s + v) * Kh + u) * Ci + r];
                                double f = filt[((u * Kw + v) * Ci + r) * Co + j];
                                acc += x * f;
                            }
                        }
                    }
                    out[((i * Ho + m) * Wo + n) * Co + j] = acc;
                }
            }
        }
    }
    return 0;
}

/*
 * Zero padding (not in the paper's layers: its Table I convolutions have
 * none).  The padded input is the input surrounded by ph zero rows above and
 * below and pw zero columns left and right:
 *   Ip[i][h][w][r] = I[i][h - ph][w - pw][r]  when 0 <= h - ph < H_i and
 *                                               0 <= w - pw < W_i,
 *                  = 0                          otherwise,
 * of extent (H_i + 2 ph) x (W_i + 2 pw).  Both functions below read Ip
 * through that rule; neither builds it.
 */
static int oracle_pad_tap(int64_t h, int64_t w, int64_t Hi, int64_t Wi)
{
    return h >= 0 && h < Hi && w >= 0 && w < Wi;
}

/*
 * Eq. (1) on the padded input: the sum over (u, v, r) of
 * Ip[i][m*s+u][n*s+v][r] * F[u][v][r][j], with H_o = floor((H_i + 2 ph -
 * K_h) / s) + 1 and W_o likewise; `absout` (may be NULL) gets the |x||w| sum.
 * Seven nested loops, fixed order (i, m, n, j, u, v, r), fp64.
 */
int oracle_conv_pad_f64(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi, int64_t Co,
                        int64_t Kh, int64_t Kw, int64_t s, int64_t ph, int64_t pw,
                        const double *in, const double *filt,
                        double *out, double *absout)
{
    if (ph < 0 || pw < 0 || Hi <= 0 || Wi <= 0)
        return -1;
    int64_t Ho = oracle_out_extent(Hi + 2 * ph, Kh, s);
    int64_t Wo = oracle_out_extent(Wi + 2 * pw, Kw, s);
    if (N <= 0 || Ci <= 0 || Co <= 0 || Ho < 0 || Wo < 0)
        return -1;

#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < N; ++i) {
        for (int64_t m = 0; m < Ho; ++m) {
            for (int64_t n = 0; n < Wo; ++n) {
                for (int64_t j = 0; j < Co; ++j) {
                    double acc = 0.0, aacc = 0.0;
                    for (int64_t u = 0; u < Kh; ++u) {
                        for (int64_t v = 0; v < Kw; ++v) {
                            int64_t h = m * s + u - ph, w = n * s + v - pw;
                            if (!oracle_pad_tap(h, w, Hi, Wi))
                                continue;  /* a zero of the padding adds 0 */
                            for (int64_t r = 0; r < Ci; ++r) {
                                double x = in[((i * Hi + h) * Wi + w) * Ci + r];
                                double f = filt[((u * Kw + v) * Ci + r) * Co + j];
                                acc += x * f;
                                aacc += fabs(x) * fabs(f);
                            }
                        }
                    }
                    int64_t o = ((i * Ho + m) * Wo + n) * Co + j;
                    out[o] = acc;
                    if (absout)
                        absout[o] = aacc;
                }
            }
        }
    }
    return 0;
}

/*
 * Eq. (2) on the padded input:
 *   W[i][m][k*K_h + u][r] = Ip[i][m*s + u][k][r]
 * for i<N, m<H_o, k<W_i+2pw, u<K_h, r<C_i; padded positions are all-zero
 * bytes (the zero of every element type used here).  Raw `elt`-byte copies.
 */
int oracle_im2win_pad(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi,
                      int64_t Kh, int64_t s, int64_t ph, int64_t pw, int64_t elt,
                      const void *in, void *out)
{
    if (ph < 0 || pw < 0 || Hi <= 0 || Wi <= 0)
        return -1;
    int64_t Hp = Hi + 2 * ph, Wp = Wi + 2 * pw;
    int64_t Ho = oracle_out_extent(Hp, Kh, s);
    if (N <= 0 || Ci <= 0 || Ho < 0 || elt <= 0)
        return -1;
    const unsigned char *src = (const unsigned char *)in;
    unsigned char *dst = (unsigned char *)out;

#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < N; ++i) {
        for (int64_t m = 0; m < Ho; ++m) {
            for (int64_t k = 0; k < Wp; ++k) {
                for (int64_t u = 0; u < Kh; ++u) {
                    int64_t h = m * s + u - ph, w = k - pw;
                    for (int64_t r = 0; r < Ci; ++r) {
                        int64_t d = ((i * Ho + m) * (Wp * Kh) + (k * Kh + u)) * Ci + r;
                        if (oracle_pad_tap(h, w, Hi, Wi))
                            memcpy(dst + d * elt, src + (((i * Hi + h) * Wi + w) * Ci + r) * elt,
                                   (size_t)elt);
                        else
                            memset(dst + d * elt, 0, (size_t)elt);
                    }
                }
            }
        }
    }
    return 0;
}

/*
 * Filter dilation d >= 1 (an extension; the paper's layers have none): tap
 * (u, v) of output (m, n) reads padded input row m*s + u*d and column
 * n*s + v*d.  The dilated filter spans E_h = (K_h - 1)*d + 1 rows and E_w
 * columns, so H_o = floor((H_i + 2 ph - E_h) / s) + 1 and W_o likewise.
 * d = 1 is the padded convolution above.
 */
static int64_t oracle_dil_extent(int64_t in, int64_t k, int64_t s, int64_t d)
{
    if (d <= 0 || k <= 0)
        return -1;
    return oracle_out_extent(in, (k - 1) * d + 1, s);
}

/* Eq. (1) with dilation d on the padded input; `absout` (may be NULL) gets
 * the |x||w| sum.  Loops (i, m, n, j, u, v, r), fp64. */
int oracle_conv_dil_f64(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi, int64_t Co,
                        int64_t Kh, int64_t Kw, int64_t s, int64_t ph, int64_t pw, int64_t d,
                        const double *in, const double *filt, double *out, double *absout)
{
    if (ph < 0 || pw < 0 || Hi <= 0 || Wi <= 0)
        return -1;
    int64_t Ho = oracle_dil_extent(Hi + 2 * ph, Kh, s, d);
    int64_t Wo = oracle_dil_extent(Wi + 2 * pw, Kw, s, d);
    if (N <= 0 || Ci <= 0 || Co <= 0 || Ho < 0 || Wo < 0)
        return -1;

#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < N; ++i) {
        for (int64_t m = 0; m < Ho; ++m) {
            for (int64_t n = 0; n < Wo; ++n) {
                for (int64_t j = 0; j < Co; ++j) {
                    double acc = 0.0, aacc = 0.0;
                    for (int64_t u = 0; u < Kh; ++u) {
                        for (int64_t v = 0; v < Kw; ++v) {
                            int64_t h = m * s + u * d - ph, w = n * s + v * d - pw;
                            if (!oracle_pad_tap(h, w, Hi, Wi))
                                continue;
                            for (int64_t r = 0; r < Ci; ++r) {
                                double x = in[((i * Hi + h) * Wi + w) * Ci + r];
                                double f = filt[((u * Kw + v) * Ci + r) * Co + j];
                                acc += x * f;
                                aacc += fabs(x) * fabs(f);
                            }
                        }
                    }
                    int64_t o = ((i * Ho + m) * Wo + n) * Co + j;
                    out[o] = acc;
                    if (absout)
                        absout[o] = aacc;
                }
            }
        }
    }
    return 0;
}

/*
 * Columns per residue group of a strip: Wq = ceil(Wp / d) for the padded
 * width Wp.  Strip position P (0 <= P < d*Wq) holds padded column
 *   k = (P mod Wq) * d + floor(P / Wq)        (group floor(P / Wq)),
 * or nothing (zero filler) when k >= Wp.  The window of output column n then
 * starts at position ((n*s) mod d) * Wq + floor(n*s / d) and its K_w columns
 * n*s + v*d are the K_w positions after it; d = 1 gives position n*s, Eq. 2's
 * order.
 */
int64_t oracle_dil_group_cols(int64_t Wp, int64_t d)
{
    if (Wp <= 0 || d <= 0)
        return -1;
    return (Wp + d - 1) / d;
}

int64_t oracle_dil_window_col(int64_t n, int64_t s, int64_t d, int64_t Wq)
{
    int64_t c = n * s;
    return (c % d) * Wq + c / d;
}

/*
 * Eq. (2) with dilation on the padded input:
 *   W[i][m][P*K_h + u][r] = Ip[i][m*s + u*d][k(P)][r]
 * for P < d*Wq, u < K_h, r < C_i; filler positions and padded taps are zero
 * bytes.  Raw `elt`-byte copies.
 */
int oracle_im2win_dil(int64_t N, int64_t Ci, int64_t Hi, int64_t Wi, int64_t Kh, int64_t s,
                      int64_t ph, int64_t pw, int64_t d, int64_t elt, const void *in, void *out)
{
    if (ph < 0 || pw < 0 || Hi <= 0 || Wi <= 0)
        return -1;
    int64_t Hp = Hi + 2 * ph, Wp = Wi + 2 * pw;
    int64_t Ho = oracle_dil_extent(Hp, Kh, s, d);
    int64_t Wq = oracle_dil_group_cols(Wp, d);
    if (N <= 0 || Ci <= 0 || Ho < 0 || Wq < 0 || elt <= 0)
        return -1;
    int64_t cols = d * Wq;
    const unsigned char *src = (const unsigned char *)in;
    unsigned char *dst = (unsigned char *)out;

#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < N; ++i) {
        for (int64_t m = 0; m < Ho; ++m) {
            for (int64_t P = 0; P < cols; ++P) {
                int64_t k = (P % Wq) * d + P / Wq;
                for (int64_t u = 0; u < Kh; ++u) {
                    int64_t h = m * s + u * d - ph, w = k - pw;
                    for (int64_t r = 0; r < Ci; ++r) {
                        int64_t o = ((i * Ho + m) * (cols * Kh) + (P * Kh + u)) * Ci + r;
                        if (k < Wp && oracle_pad_tap(h, w, Hi, Wi))
                            memcpy(dst + o * elt, src + (((i * Hi + h) * Wi + w) * Ci + r) * elt,
                                   (size_t)elt);
                        else
                            memset(dst + o * elt, 0, (size_t)elt);
                    }
                }
            }
        }
    }
    return 0;
}

/*
 * Eq. (3) with dilation: the sums of oracle_conv_dil_f64 read out of the
 * dilated window tensor `win` (as oracle_im2win_dil lays it out): the window
 * of (i, m, n) is the K = K_w*K_h*C_i elements of strip (i, m) from position
 * oracle_dil_window_col(n) on, in (v, u, r) order.  H_i, W_i are the padded
 * extents.
 */
int oracle_windowed_conv_dil_f64(int64_t N, int64_t Ci, int64_t Hp, int64_t Wp, int64_t Co,
                                 int64_t Kh, int64_t Kw, int64_t s, int64_t d,
                                 const double *win, const double *filt, double *out)
{
    int64_t Ho = oracle_dil_extent(Hp, Kh, s, d);
    int64_t Wo = oracle_dil_extent(Wp, Kw, s, d);
    int64_t Wq = oracle_dil_group_cols(Wp, d);
    if (N <= 0 || Ci <= 0 || Co <= 0 || Ho < 0 || Wo < 0 || Wq < 0)
        return -1;
    int64_t L = d * Wq * Kh * Ci;

#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < N; ++i) {
        for (int64_t m = 0; m < Ho; ++m) {
            const double *strip = win + (i * Ho + m) * L;
            for (int64_t n = 0; n < Wo; ++n) {
                const double *span = strip + oracle_dil_window_col(n, s, d, Wq) * Kh * Ci;
                for (int64_t j = 0; j < Co; ++j) {
                    double acc = 0.0;
                    for (int64_t v = 0; v < Kw; ++v)
                        for (int64_t u = 0; u < Kh; ++u)
                            for (int64_t r = 0; r < Ci; ++r)
                                acc += span[(v * Kh + u) * Ci + r] * filt[((u * Kw + v) * Ci + r) * Co + j];
                    out[((i * Ho + m) * Wo + n) * Co + j] = acc;
                }
            }
        }
    }
    return 0;
}
