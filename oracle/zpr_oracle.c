/*
 * PIC latent decoding from the ZpR symbol stream -- CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  The plain, slow statement of the decoder step
 * that turns the entropy-decoded symbol stream back into the latent pyramid.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load it; the product library never links, loads or calls it, and it
 * shares no source with the HIP kernels.
 *
 * What is computed (PIC, Fig. 1, Sec. 3.2 Eq. (5)-(7), Sec. 3.3 and Fig. 2,
 * App. B Alg. 1):
 *   - the encoder cut every latent grid into 8x8 patches, concatenated them
 *     (Eq. (6)), took the 2-D DCT of each patch (Eq. (7)), quantised, and
 *     coded each block's 64 coefficients with ZpR (Fig. 2): zigzag order,
 *     trailing zeros dropped, zero runs replaced by run codes; every block's
 *     code ends with the end-of-block marker eob;
 *   - the decoder finds the eob positions (App. B: a copy_if over the stream),
 *     expands each block (Alg. 1): a symbol s >= eob - 16 is a run of
 *     s - eob + 17 zeros (1 .. 16), any smaller symbol is one coefficient;
 *     the p-th coefficient produced goes to natural position ZIGZAG[p]; what a
 *     block does not produce is zero (the trimmed tail);
 *   - each 64-coefficient block goes through the inverse 2-D DCT and lands in
 *     its latent grid at its patch position (un-patchify, the inverse of
 *     Eq. (6)); samples of padding patches outside the grid are dropped.
 *
 * Readings where the paper is silent:
 *   - quantisation has unit step: the symbols are the coefficients (Eq. (8)
 *     relaxes rounding with uniform noise on (-1/2, 1/2));
 *   - the DCT is the orthonormal DCT-II, so its inverse is the orthonormal
 *     DCT-III written out below;
 *   - block order: image by image; within an image the paper's level order
 *     y_1 .. y_L of Eq. (5), i.e. coarsest grid first (level k = L-1 down to
 *     k = 0 in the finest-first numbering used everywhere else); within a
 *     level the patches row by row, left to right; within a patch row-major;
 *     level k's grid is ceil(H / 2^k) x ceil(W / 2^k), padded at the bottom
 *     and right to whole patches;
 *   - the zigzag order is JPEG's;
 *   - one eob value serves the whole stream of a call.
 *
 * Error flags (bitwise or), returned by the expansion and the whole decode:
 *   1  the stream holds a different number of eob markers than blocks, or
 *      symbols follow the last marker;
 *   2  a block produces more than 64 coefficients (the excess is dropped) or
 *      holds more than 64 symbols;
 *   4  a symbol is greater than eob (it is skipped).
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared (see build.py).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ZO_MAX_LEVELS 16

enum { ZO_ERR_COUNT = 1, ZO_ERR_OVERFLOW = 2, ZO_ERR_SYMBOL = 4 };

static int zo_dim(int n, int k)
{
    long f = 1L << k;
    return (int)((n + f - 1) / f);
}

/* JPEG zigzag scan: zz[p] is the row-major index of the p-th coefficient.
 * The scan walks the anti-diagonals d = r + c = 0 .. 14; on odd d it goes
 * down-left (row increasing), on even d up-right (row decreasing). */
void pic_oracle_zigzag(int32_t zz[64])
{
    int p = 0;
    for (int d = 0; d <= 14; ++d) {
        int rlo = d - 7 > 0 ? d - 7 : 0;
        int rhi = d < 7 ? d : 7;
        if (d % 2 == 1) {
            for (int r = rlo; r <= rhi; ++r)
                zz[p++] = r * 8 + (d - r);
        } else {
            for (int r = rhi; r >= rlo; --r)
                zz[p++] = r * 8 + (d - r);
        }
    }
}

/* Number of 8x8 blocks of one image: sum over levels of the patch grid. */
long pic_oracle_zpr_blocks(int H, int W, int L)
{
    long n = 0;
    for (int k = 0; k < L; ++k)
        n += (long)((zo_dim(H, k) + 7) / 8) * ((zo_dim(W, k) + 7) / 8);
    return n;
}

/* The copy_if of App. B: positions i with symbols[i] == eob, increasing.
 * Writes at most max_out of them; returns how many there are. */
long pic_oracle_eob_offsets(const int32_t *symbols, long n, int32_t eob, long *offsets, long max_out)
{
    long m = 0;
    for (long i = 0; i < n; ++i) {
        if (symbols[i] == eob) {
            if (m < max_out)
                offsets[m] = i;
            ++m;
        }
    }
    return m;
}

/* Alg. 1 for blocks 0 .. n_blocks-1, given their eob offsets.  Block g reads
 * symbols offsets[g-1]+1 .. offsets[g]-1 (from 0 for g = 0) and writes its 64
 * coefficients, row-major, at coeffs + 64 g; the rest stays zero. */
int pic_oracle_expand_symbols(const int32_t *symbols, int32_t eob, const long *offsets, long n_blocks,
                              int32_t *coeffs)
{
    int32_t zz[64];
    pic_oracle_zigzag(zz);
    int err = 0;
    memset(coeffs, 0, (size_t)n_blocks * 64 * sizeof(int32_t));
    for (long g = 0; g < n_blocks; ++g) {
        long begin = g == 0 ? 0 : offsets[g - 1] + 1;
        long end = offsets[g];
        int32_t *blk = coeffs + (size_t)g * 64;
        int produced = 0;
        for (long i = begin; i < end; ++i) {
            int32_t s = symbols[i];
            if (s > eob) {
                err |= ZO_ERR_SYMBOL;
                continue;
            }
            if (s >= eob - 16) {
                int run = s - eob + 17;          /* zeros; the block is pre-zeroed */
                produced += run;
            } else {
                if (produced < 64)
                    blk[zz[produced]] = s;
                produced += 1;
            }
        }
        if (produced > 64 || end - begin > 64)
            err |= ZO_ERR_OVERFLOW;
    }
    return err;
}

/* Basis of the orthonormal 8-point DCT: C[x][u] = a(u) cos((2x+1) u pi / 16)
 * with a(0) = sqrt(1/8) and a(u) = sqrt(2/8) = 1/2 otherwise. */
static void idct_basis(double C[8][8])
{
    const double pi = 3.14159265358979323846;
    for (int x = 0; x < 8; ++x) {
        for (int u = 0; u < 8; ++u) {
            double a = u == 0 ? sqrt(1.0 / 8.0) : 0.5;
            C[x][u] = a * cos((2 * x + 1) * u * pi / 16.0);
        }
    }
}

/* Orthonormal 8x8 inverse DCT (DCT-III), the definition:
 *   f[x][y] = sum_u sum_v C[x][u] C[y][v] S[u][v]
 * u indexes rows (vertical frequency), v columns; S and f are row-major. */
static void idct8x8(const double C[8][8], const double *S, double *f)
{
    for (int x = 0; x < 8; ++x) {
        for (int y = 0; y < 8; ++y) {
            double acc = 0.0;
            for (int u = 0; u < 8; ++u)
                for (int v = 0; v < 8; ++v)
                    acc += C[x][u] * C[y][v] * S[u * 8 + v];
            f[x * 8 + y] = acc;
        }
    }
}

void pic_oracle_idct8x8_f64(const double *S, double *f)
{
    double C[8][8];
    idct_basis(C);
    idct8x8(C, S, f);
}

/* Offset of level k's grid in the concatenated output of `batch` images:
 * levels k = 0 .. L-1 one after another, each [batch][h_k][w_k]. */
static size_t level_base(int H, int W, int batch, int k)
{
    size_t o = 0;
    for (int j = 0; j < k; ++j)
        o += (size_t)batch * zo_dim(H, j) * zo_dim(W, j);
    return o;
}

/* Un-patchify: place block g's 64 samples (row-major 8x8 at blocks + 64 g)
 * into the concatenated pyramid `out` (see level_base), dropping samples
 * outside the grid.  Block order as in the file header. */
int pic_oracle_unpatchify_f64(int H, int W, int L, int batch, const double *blocks, double *out)
{
    if (H < 1 || W < 1 || L < 1 || L > ZO_MAX_LEVELS || batch < 0)
        return 1;
    long g = 0;
    for (int b = 0; b < batch; ++b) {
        for (int k = L - 1; k >= 0; --k) {
            int hk = zo_dim(H, k), wk = zo_dim(W, k);
            int ph = (hk + 7) / 8, pw = (wk + 7) / 8;
            double *grid = out + level_base(H, W, batch, k) + (size_t)b * hk * wk;
            for (int py = 0; py < ph; ++py) {
                for (int px = 0; px < pw; ++px, ++g) {
                    const double *blk = blocks + (size_t)g * 64;
                    for (int r = 0; r < 8; ++r) {
                        for (int c = 0; c < 8; ++c) {
                            int y = py * 8 + r, x = px * 8 + c;
                            if (y < hk && x < wk)
                                grid[(size_t)y * wk + x] = blk[r * 8 + c];
                        }
                    }
                }
            }
        }
    }
    return 0;
}

/* The whole step for `batch` images: eob offsets, Alg. 1, inverse DCT and
 * un-patchify into the concatenated fp64 pyramid `out` (see level_base;
 * grids not covered by a decoded block are left as they were).  Returns the
 * error flags, or -1 for invalid sizes or a failed allocation. */
int pic_oracle_zpr_decode_f64(int H, int W, int L, int batch, const int32_t *symbols, long n, int32_t eob,
                              double *out)
{
    if (H < 1 || W < 1 || L < 1 || L > ZO_MAX_LEVELS || batch < 0 || n < 0)
        return -1;
    long nb = pic_oracle_zpr_blocks(H, W, L) * batch;
    long *offsets = malloc(sizeof(long) * (size_t)(nb > 0 ? nb : 1));
    int32_t *coeffs = malloc(sizeof(int32_t) * 64 * (size_t)(nb > 0 ? nb : 1));
    double *blocks = malloc(sizeof(double) * 64 * (size_t)(nb > 0 ? nb : 1));
    if (!offsets || !coeffs || !blocks) {
        free(offsets);
        free(coeffs);
        free(blocks);
        return -1;
    }
    int err = 0;
    long m = pic_oracle_eob_offsets(symbols, n, eob, offsets, nb);
    if (m != nb || (n > 0 && symbols[n - 1] != eob))
        err |= ZO_ERR_COUNT;
    long dec = m < nb ? m : nb;                  /* blocks the stream delimits */
    err |= pic_oracle_expand_symbols(symbols, eob, offsets, dec, coeffs);
    double C[8][8];
    idct_basis(C);
#pragma omp parallel for schedule(static)
    for (long g = 0; g < dec; ++g) {
        double S[64];
        for (int i = 0; i < 64; ++i)
            S[i] = (double)coeffs[(size_t)g * 64 + i];
        idct8x8((const double(*)[8])C, S, blocks + (size_t)g * 64);
    }
    /* blocks past `dec` are absent: place only the decoded ones */
    if (dec == nb) {
        pic_oracle_unpatchify_f64(H, W, L, batch, blocks, out);
    } else {
        double *full = malloc(sizeof(double) * 64 * (size_t)(nb > 0 ? nb : 1));
        double *tmp = malloc(sizeof(double) * level_base(H, W, batch, L) + 1);
        if (!full || !tmp) {
            free(full);
            free(tmp);
            free(offsets);
            free(coeffs);
            free(blocks);
            return -1;
        }
        for (long i = 0; i < nb * 64; ++i)
            full[i] = NAN;
        memcpy(full, blocks, sizeof(double) * 64 * (size_t)dec);
        pic_oracle_unpatchify_f64(H, W, L, batch, full, tmp);
        size_t tot = level_base(H, W, batch, L);
        for (size_t i = 0; i < tot; ++i)
            if (!isnan(tmp[i]))
                out[i] = tmp[i];
        free(full);
        free(tmp);
    }
    free(offsets);
    free(coeffs);
    free(blocks);
    return err;
}
