/*
 * pic_zpr.h -- C ABI of the PIC latent decoding step on AMD Instinct MI355X
 * (gfx950): from the entropy-decoded symbol stream to the latent pyramid that
 * pic_decode_run synthesises.
 *
 * The operation (PIC, Fig. 1; Sec. 3.2 Eq. (5)-(7); Sec. 3.3 with Fig. 2;
 * App. B, Alg. 1 and the copy_if of eob offsets before it): the encoder cut
 * each latent grid into 8x8 patches (Eq. (6)), transformed them with the 2-D
 * DCT (Eq. (7)), and ZpR-coded every block (Fig. 2): zigzag order, trailing
 * zeros dropped, each zero run replaced by run codes, an end-of-block marker
 * (eob) last.  The decoder
 *   1. finds every block's marker (the offsets Alg. 1 needs),
 *   2. expands each block (Alg. 1): a symbol s with eob - 16 <= s < eob is a
 *      run of s - eob + 17 zeros (1 .. 16); any smaller symbol is one
 *      coefficient; the p-th coefficient produced lands at row-major position
 *      ZIGZAG[p] of the 8x8 block; positions not produced are zero,
 *   3. applies the orthonormal 2-D inverse DCT to each block, and
 *   4. writes the 64 samples to the block's patch of its latent grid
 *      (un-patchify), dropping samples of padding patches outside the grid.
 *
 * Conventions fixed by this ABI where the paper leaves them open:
 *   - coefficients are the symbols themselves (unit quantisation step);
 *   - the DCT is orthonormal: sample (x, y) of a block is
 *       sum_{u,v} a(u) a(v) S[u][v] cos((2x+1) u pi/16) cos((2y+1) v pi/16)
 *     with a(0) = sqrt(1/8), a(u > 0) = 1/2, u the row (vertical) frequency;
 *   - ZIGZAG is the JPEG scan order (ITU-T T.81, Fig. A.6);
 *   - block order: image by image; within an image the paper's level order of
 *     Eq. (5), coarsest grid first (level k = L-1 down to 0 in the numbering of
 *     pic_decode.h); within a level patches row by row, left to right; level
 *     k's grid is ceil(H / 2^k) x ceil(W / 2^k), padded at the bottom and right
 *     to whole patches;
 *   - one eob value serves the whole stream of a call (an encoder uses the
 *     largest symbol of its alphabet; streams coded with other markers are
 *     re-marked by shifting their run codes and markers).
 *
 * Link against libpic_decode.so (same library, same status codes).
 */
#ifndef PIC_ZPR_H
#define PIC_ZPR_H

#include <stdint.h>

#include "pic_decode.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Opaque handle: the pyramid shape, the device it was created on and a small
 * device scratch buffer (per-chunk marker counts, 4 bytes per 256 symbols of
 * the longest accepted stream), so runs neither allocate nor synchronise.
 * Runs on one handle must not overlap: enqueue them on one stream, or
 * synchronise between them. */
typedef struct pic_zpr pic_zpr;

/* Bits of the status word a run writes (0: the stream is well formed). */
enum {
    PIC_ZPR_ERR_COUNT = 1,      /* marker count differs from the number of blocks, or
                                   symbols follow the last marker                  */
    PIC_ZPR_ERR_OVERFLOW = 2,   /* a block holds more than 64 symbols or produces more
                                   than 64 coefficients; the excess is dropped      */
    PIC_ZPR_ERR_SYMBOL = 4      /* a symbol greater than eob (it is skipped)        */
};

/* Zero-initialise, then set struct_size = sizeof(pic_zpr_desc). */
typedef struct pic_zpr_desc {
    uint32_t struct_size;
    int32_t height, width;      /* H, W >= 1, H * W < 2^31                          */
    int32_t num_levels;         /* L in [1, PIC_MAX_LEVELS]                          */
    int32_t max_batch;          /* largest batch passed to a run, 1 .. PIC_MAX_BATCH;
                                   max_batch * blocks per image must be < 2^31       */
} pic_zpr_desc;

typedef struct pic_zpr_info {
    uint32_t struct_size;       /* set by the caller: sizeof(pic_zpr_info)           */
    int32_t device;             /* HIP device ordinal of the handle                 */
    int64_t blocks_per_image;   /* sum over levels of ceil(h_k/8) * ceil(w_k/8)     */
    int64_t max_symbols;        /* longest stream a run accepts at max_batch:
                                   min(65 * blocks_per_image * max_batch, 2^31 - 1)  */
    int64_t scratch_bytes;      /* device memory the handle holds                   */
    int32_t symbols_per_chunk;  /* symbols one workgroup scans on short streams (long
                                   streams, from 2^18 symbols, use 4 times as many)  */
} pic_zpr_info;

/*
 * pic_zpr_create -- validate `desc` and build a handle on the current HIP
 * device; allocates its device scratch (hipMalloc).
 * Returns PIC_OK; PIC_E_INVALID for a malformed descriptor or NULL `out`;
 * PIC_E_UNSUPPORTED when max_batch * blocks per image reaches 2^31;
 * PIC_E_NODEVICE when no gfx950 device is current; PIC_E_NOMEM when the handle
 * cannot be allocated; PIC_E_HIP when the device scratch cannot.
 */
PIC_API pic_status pic_zpr_create(const pic_zpr_desc *desc, pic_zpr **out);

/*
 * pic_zpr_decode -- enqueue steps 1-4 for `batch` images on `stream`.
 *   batch     : 0 .. max_batch (0 enqueues nothing and leaves *status alone;
 *               `latents` may then be NULL).
 *   symbols   : device, int32 [n_symbols], the images' streams concatenated
 *               in block order (see above); may be NULL when n_symbols == 0.
 *   n_symbols : 0 .. min(65 * blocks_per_image * batch, 2^31 - 1) (a well-formed
 *               block has at most 64 symbols and its marker).
 *   eob       : the end-of-block marker, in [INT32_MIN + 17, INT32_MAX - 1].
 *   latents   : host array of num_levels device pointers; latents[k] receives
 *               fp32 [batch][ceil(H/2^k)][ceil(W/2^k)] (the layout pic_decode_run
 *               reads).  Every sample of a well-formed stream is written;
 *               blocks a malformed stream does not delimit are left as they were.
 *   status    : device int32, receives the PIC_ZPR_ERR_* bits of this run (no
 *               need to clear it first; readable after the stream reaches it).
 *   stream    : hipStream_t (NULL: the null stream).
 * Pointers must be 4-byte aligned and must not overlap.  Asynchronous: no
 * allocation, no synchronisation.  Returns PIC_E_INVALID for a bad argument
 * (nothing enqueued), PIC_E_HIP for a failed launch.
 */
PIC_API pic_status pic_zpr_decode(pic_zpr *h, int32_t batch, const int32_t *symbols, int64_t n_symbols,
                                  int32_t eob, float *const *latents, int32_t *status, void *stream);

/*
 * pic_zpr_expand -- steps 1-2 only (Alg. 1's output): every block's 64
 * coefficients, row-major, as int32 [batch * blocks_per_image][64] at `coeffs`
 * (device, 16-byte aligned).  Blocks a malformed stream does not delimit are
 * left as they were.  Other arguments, errors and ownership as pic_zpr_decode.
 */
PIC_API pic_status pic_zpr_expand(pic_zpr *h, int32_t batch, const int32_t *symbols, int64_t n_symbols,
                                  int32_t eob, int32_t *coeffs, int32_t *status, void *stream);

/* pic_zpr_query -- describe the handle.  PIC_E_INVALID for NULL arguments or
 * an unknown info->struct_size. */
PIC_API pic_status pic_zpr_query(const pic_zpr *h, pic_zpr_info *info);

/* pic_zpr_destroy -- free the handle and its device scratch (NULL is
 * accepted).  Synchronises the handle's device first, so work enqueued with
 * the handle completes before the scratch is released. */
PIC_API void pic_zpr_destroy(pic_zpr *h);

#ifdef __cplusplus
}
#endif

#endif /* PIC_ZPR_H */
