/*
 * PIC synthesis decoder -- CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * statement of what the decoder's synthesis step computes.  Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg may load it; the
 * product library never links, loads or calls it, and it shares no source
 * with the HIP kernels.
 *
 * What is computed (PIC, Sec. 3.1 and App. A):
 *   - a pyramid of L single-channel latent grids; with level k = 0 the full
 *     resolution and level k scaled by 1/2^k (the paper's Eq. (2) indexes the
 *     same grids coarsest-first, i = L - k), H_k = ceil(H / 2^k) and
 *     W_k = ceil(W / 2^k) (Eq. (2) states H / 2^(L-i) for divisible sizes);
 *   - every level upsampled to H x W (Sec. 3.1: the pyramid is upsampled to
 *     the image resolution before synthesis; the kernel is not named there and
 *     is read as bilinear with half-pixel centres, edge replication and the
 *     nominal 2^k scale, i.e. the grid upsampled by exactly 2^k and cropped);
 *   - the upsampled C = L channel vector of each pixel, finest level first,
 *     fed to the synthesis MLP g_s: affine layers with ReLU between them and
 *     none after the last (Sec. 4.1 "Implementation Details", App. A: the last
 *     layer is MLP^i whose fused weights w', b' are all the decoder needs);
 *   - the three outputs are the RGB sample, clamped to [0, 1] and optionally
 *     quantised to 8 bits as floor(255 c + 1/2).
 *
 * Two entry points:
 *   pic_oracle_decode_f64  -- the definition, evaluated in double precision;
 *   pic_oracle_decode_f32  -- the same definition in binary32 with one stated
 *                             operation order (bias as the accumulator's start
 *                             value, one fused multiply-add per input in
 *                             increasing input index).  It exists because an
 *                             8-bit code is an integer decided by floating
 *                             point: a decision taken in binary32 is compared
 *                             with one taken in binary32.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared (see build.py).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_MAX_LEVELS 16
#define OR_MAX_LAYERS 16
#define OR_MAX_WIDTH 256

enum { OR_OUT_RAW = 0, OR_OUT_CLAMPED = 1, OR_OUT_U8 = 2 };
enum { OR_OK = 0, OR_E_INVALID = 1 };

/* Size of level k along an axis of n samples: ceil(n / 2^k). */
int pic_oracle_level_dim(int n, int k)
{
    long f = 1L << k;
    return (int)((n + f - 1) / f);
}

/* Value of a bf16 bit pattern: the top half of a binary32 pattern. */
static double bf16_value(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static int check_args(int H, int W, int L, int nl, const int *widths, int batch,
                      const float *const *latents, const void *weights,
                      const float *biases, const void *out, int out_kind)
{
    if (H < 1 || W < 1 || L < 1 || L > OR_MAX_LEVELS || nl < 1 || nl > OR_MAX_LAYERS)
        return OR_E_INVALID;
    if (batch < 0 || !widths || !latents || !weights || !biases || !out)
        return OR_E_INVALID;
    if (widths[0] != L || widths[nl] != 3)
        return OR_E_INVALID;
    for (int l = 0; l <= nl; ++l)
        if (widths[l] < 1 || widths[l] > OR_MAX_WIDTH)
            return OR_E_INVALID;
    for (int k = 0; k < L; ++k)
        if (!latents[k])
            return OR_E_INVALID;
    if (out_kind < OR_OUT_RAW || out_kind > OR_OUT_U8)
        return OR_E_INVALID;
    return OR_OK;
}

/* ------------------------------------------------------------------ fp64 */

/*
 * Upsampled value of level k at output pixel (y, x), in double precision.
 * Bilinear interpolation with half-pixel centres: the source coordinate of
 * output index y is (y + 1/2) / 2^k - 1/2, clamped below at 0; the two taps
 * are floor of it and the next sample, the latter clamped to the last row
 * (edge replication); the weights are the fractional part and its complement.
 */
static double upsample_f64(const float *grid, int hk, int wk, int k, int y, int x)
{
    if (k == 0)
        return (double)grid[(size_t)y * wk + x];
    double f = (double)(1L << k);
    double sy = ((double)y + 0.5) / f - 0.5;
    double sx = ((double)x + 0.5) / f - 0.5;
    if (sy < 0.0) sy = 0.0;
    if (sx < 0.0) sx = 0.0;
    int y0 = (int)floor(sy), x0 = (int)floor(sx);
    int y1 = y0 + 1 < hk ? y0 + 1 : hk - 1;
    int x1 = x0 + 1 < wk ? x0 + 1 : wk - 1;
    double ly = sy - y0, lx = sx - x0;
    double a = grid[(size_t)y0 * wk + x0], b = grid[(size_t)y0 * wk + x1];
    double c = grid[(size_t)y1 * wk + x0], d = grid[(size_t)y1 * wk + x1];
    double top = (1.0 - lx) * a + lx * b;
    double bot = (1.0 - lx) * c + lx * d;
    return (1.0 - ly) * top + ly * bot;
}

/*
 * Decode `batch` images in double precision.
 *   latents[k]  : level k, float32 [batch][H_k][W_k] row-major
 *   weights     : per image, layer l's matrix [widths[l+1]][widths[l]] row-major,
 *                 layers concatenated; float32 if weights_are_bf16 == 0, else
 *                 uint16 bf16 bit patterns; image b starts at b * w_stride
 *                 elements (0: all images share one set)
 *   biases      : float32, per image, layer l's widths[l+1] values concatenated;
 *                 image b starts at b * b_stride
 *   out         : [batch][3][y_end - y_begin][W] planar, double for raw /
 *                 clamped output, uint8 for 8-bit output
 *   nthreads    : OpenMP threads (<= 0: the runtime's default)
 *   y_begin, y_end : the output rows computed (0 and H for the whole image);
 *                 a row's values do not depend on which other rows are computed
 * Returns 0, or 1 on invalid arguments (nothing written).
 */
int pic_oracle_decode_f64(int H, int W, int L, int nl, const int *widths, int batch,
                          const float *const *latents,
                          const void *weights, int weights_are_bf16, long w_stride,
                          const float *biases, long b_stride,
                          int out_kind, void *out, int nthreads, int y_begin, int y_end)
{
    if (check_args(H, W, L, nl, widths, batch, latents, weights, biases, out, out_kind))
        return OR_E_INVALID;
    if (y_begin < 0 || y_end > H || y_begin >= y_end)
        return OR_E_INVALID;
    const int R = y_end - y_begin;
    int hk[OR_MAX_LEVELS], wk[OR_MAX_LEVELS];
    for (int k = 0; k < L; ++k) {
        hk[k] = pic_oracle_level_dim(H, k);
        wk[k] = pic_oracle_level_dim(W, k);
    }
    long rows = (long)batch * R;
#ifdef _OPENMP
    int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
#endif
    for (long r = 0; r < rows; ++r) {
        int b = (int)(r / R), y = y_begin + (int)(r % R);
        const float *fw = (const float *)weights + (weights_are_bf16 ? 0 : b * w_stride);
        const uint16_t *hw = (const uint16_t *)weights + (weights_are_bf16 ? b * w_stride : 0);
        const float *bias = biases + b * b_stride;
        double h[OR_MAX_WIDTH], g[OR_MAX_WIDTH];
        for (int x = 0; x < W; ++x) {
            for (int k = 0; k < L; ++k) {
                const float *grid = latents[k] + (size_t)b * hk[k] * wk[k];
                h[k] = upsample_f64(grid, hk[k], wk[k], k, y, x);
            }
            long wo = 0, bo = 0;
            for (int l = 0; l < nl; ++l) {
                int fin = widths[l], fout = widths[l + 1];
                for (int j = 0; j < fout; ++j) {
                    double acc = 0.0;
                    for (int i = 0; i < fin; ++i) {
                        long idx = wo + (long)j * fin + i;
                        double wv = weights_are_bf16 ? bf16_value(hw[idx]) : (double)fw[idx];
                        acc += wv * h[i];
                    }
                    acc += (double)bias[bo + j];
                    g[j] = (l < nl - 1 && acc < 0.0) ? 0.0 : acc;   /* ReLU except after the last layer */
                }
                memcpy(h, g, sizeof(double) * fout);
                wo += (long)fin * fout;
                bo += fout;
            }
            for (int c = 0; c < 3; ++c) {
                size_t o = (((size_t)b * 3 + c) * R + (y - y_begin)) * (size_t)W + x;
                double v = h[c];
                double cl = v < 0.0 ? 0.0 : (v > 1.0 ? 1.0 : v);
                if (out_kind == OR_OUT_RAW)
                    ((double *)out)[o] = v;
                else if (out_kind == OR_OUT_CLAMPED)
                    ((double *)out)[o] = cl;
                else
                    ((uint8_t *)out)[o] = (uint8_t)floor(255.0 * cl + 0.5);
            }
        }
    }
    return OR_OK;
}

/* ------------------------------------------------------------------ fp32 */

/* The upsample of upsample_f64, every operation rounded to binary32. */
static float upsample_f32(const float *grid, int hk, int wk, int k, int y, int x)
{
    if (k == 0)
        return grid[(size_t)y * wk + x];
    float inv = ldexpf(1.0f, -k);
    float sy = ((float)y + 0.5f) * inv - 0.5f;
    float sx = ((float)x + 0.5f) * inv - 0.5f;
    if (sy < 0.0f) sy = 0.0f;
    if (sx < 0.0f) sx = 0.0f;
    int y0 = (int)floorf(sy), x0 = (int)floorf(sx);
    int y1 = y0 + 1 < hk ? y0 + 1 : hk - 1;
    int x1 = x0 + 1 < wk ? x0 + 1 : wk - 1;
    float ly = sy - (float)y0, lx = sx - (float)x0;
    float a = grid[(size_t)y0 * wk + x0], b = grid[(size_t)y0 * wk + x1];
    float c = grid[(size_t)y1 * wk + x0], d = grid[(size_t)y1 * wk + x1];
    float top = (1.0f - lx) * a + lx * b;
    float bot = (1.0f - lx) * c + lx * d;
    return (1.0f - ly) * top + ly * bot;
}

/*
 * Same arguments and layouts as pic_oracle_decode_f64, but evaluated in
 * binary32: each layer output starts from its bias and adds one fused
 * multiply-add per input, inputs in increasing index; the 8-bit code is
 * floor(fma(c, 255, 1/2)) with c the clamped binary32 output.  Raw and
 * clamped outputs are written as float.
 */
int pic_oracle_decode_f32(int H, int W, int L, int nl, const int *widths, int batch,
                          const float *const *latents,
                          const void *weights, int weights_are_bf16, long w_stride,
                          const float *biases, long b_stride,
                          int out_kind, void *out, int nthreads, int y_begin, int y_end)
{
    if (check_args(H, W, L, nl, widths, batch, latents, weights, biases, out, out_kind))
        return OR_E_INVALID;
    if (y_begin < 0 || y_end > H || y_begin >= y_end)
        return OR_E_INVALID;
    const int R = y_end - y_begin;
    int hk[OR_MAX_LEVELS], wk[OR_MAX_LEVELS];
    for (int k = 0; k < L; ++k) {
        hk[k] = pic_oracle_level_dim(H, k);
        wk[k] = pic_oracle_level_dim(W, k);
    }
    long rows = (long)batch * R;
#ifdef _OPENMP
    int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
#endif
    for (long r = 0; r < rows; ++r) {
        int b = (int)(r / R), y = y_begin + (int)(r % R);
        const float *fw = (const float *)weights + (weights_are_bf16 ? 0 : b * w_stride);
        const uint16_t *hw = (const uint16_t *)weights + (weights_are_bf16 ? b * w_stride : 0);
        const float *bias = biases + b * b_stride;
        float h[OR_MAX_WIDTH], g[OR_MAX_WIDTH];
        for (int x = 0; x < W; ++x) {
            for (int k = 0; k < L; ++k) {
                const float *grid = latents[k] + (size_t)b * hk[k] * wk[k];
                h[k] = upsample_f32(grid, hk[k], wk[k], k, y, x);
            }
            long wo = 0, bo = 0;
            for (int l = 0; l < nl; ++l) {
                int fin = widths[l], fout = widths[l + 1];
                for (int j = 0; j < fout; ++j) {
                    float acc = bias[bo + j];
                    for (int i = 0; i < fin; ++i) {
                        long idx = wo + (long)j * fin + i;
                        float wv = weights_are_bf16 ? (float)bf16_value(hw[idx]) : fw[idx];
                        acc = fmaf(wv, h[i], acc);
                    }
                    g[j] = (l < nl - 1) ? fmaxf(acc, 0.0f) : acc;
                }
                memcpy(h, g, sizeof(float) * fout);
                wo += (long)fin * fout;
                bo += fout;
            }
            for (int c = 0; c < 3; ++c) {
                size_t o = (((size_t)b * 3 + c) * R + (y - y_begin)) * (size_t)W + x;
                float v = h[c];
                float cl = fminf(fmaxf(v, 0.0f), 1.0f);
                if (out_kind == OR_OUT_RAW)
                    ((float *)out)[o] = v;
                else if (out_kind == OR_OUT_CLAMPED)
                    ((float *)out)[o] = cl;
                else
                    ((uint8_t *)out)[o] = (uint8_t)floorf(fmaf(cl, 255.0f, 0.5f));
            }
        }
    }
    return OR_OK;
}

/*
 * The upsampled pyramid alone (the MLP's input, Sec. 3.1): out is double
 * [batch][L][H][W], channel k = level k.  Exposed so the upsample can be
 * checked on its own; decode uses the same routine.
 */
int pic_oracle_upsample_f64(int H, int W, int L, int batch,
                            const float *const *latents, double *out, int nthreads)
{
    if (H < 1 || W < 1 || L < 1 || L > OR_MAX_LEVELS || batch < 0 || !latents || !out)
        return OR_E_INVALID;
    for (int k = 0; k < L; ++k)
        if (!latents[k])
            return OR_E_INVALID;
    int hk[OR_MAX_LEVELS], wk[OR_MAX_LEVELS];
    for (int k = 0; k < L; ++k) {
        hk[k] = pic_oracle_level_dim(H, k);
        wk[k] = pic_oracle_level_dim(W, k);
    }
    long rows = (long)batch * H;
#ifdef _OPENMP
    int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(static) num_threads(nt)
#endif
    for (long r = 0; r < rows; ++r) {
        int b = (int)(r / H), y = (int)(r % H);
        for (int k = 0; k < L; ++k) {
            const float *grid = latents[k] + (size_t)b * hk[k] * wk[k];
            double *o = out + (((size_t)b * L + k) * H + y) * (size_t)W;
            for (int x = 0; x < W; ++x)
                o[x] = upsample_f64(grid, hk[k], wk[k], k, y, x);
        }
    }
    return OR_OK;
}

/*
 * Folding of instance normalisation and channel modulation into the next
 * linear layer (App. A), in double precision.  The layer's input is
 * f~[c] = gamma[c] * (f[c] - mu[c]) / sigma[c] + beta[c]; writing its
 * output W f~ + b as a layer on the raw features f gives
 *   W'[o][c] = W[o][c] * gamma[c] / sigma[c]
 *   b'[o]    = b[o] + sum_c W[o][c] * beta[c] - sum_c W[o][c] * gamma[c] * mu[c] / sigma[c]
 * (App. A's w is the transpose of W).  One image; W is [out][in].
 */
int pic_oracle_fuse_modulation_f64(int in, int out, const float *W, const float *b, const float *gamma,
                                   const float *beta, const float *mu, const float *sigma,
                                   double *w_fused, double *b_fused)
{
    if (in < 1 || out < 1 || !W || !b || !gamma || !beta || !mu || !sigma || !w_fused || !b_fused)
        return OR_E_INVALID;
    for (int o = 0; o < out; ++o) {
        double shift = 0.0, mod = 0.0;
        for (int c = 0; c < in; ++c) {
            double w = W[(size_t)o * in + c];
            w_fused[(size_t)o * in + c] = w * (double)gamma[c] / (double)sigma[c];
            mod += w * (double)beta[c];
            shift += w * (double)gamma[c] * (double)mu[c] / (double)sigma[c];
        }
        b_fused[o] = (double)b[o] + mod - shift;
    }
    return OR_OK;
}
