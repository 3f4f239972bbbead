/*
 * pic_decode.h -- C ABI of the PIC synthesis decoder on AMD Instinct MI355X
 * (gfx950).
 *
 * The operation (PIC: "Revisiting INR for Image Coding with Fast Encoding and
 * Sub-Millisecond Decoding", Sec. 3.1 with Eq. (2), Sec. 4.1 "Implementation
 * Details", App. A): the decoder holds a pyramid of L single-channel latent
 * grids and the weights of the per-image synthesis MLP g_s.  Every level is
 * upsampled to the H x W image, the L upsampled values of a pixel form the
 * MLP's input vector, and the MLP (affine layers, ReLU between them, none
 * after the last) maps it to the pixel's RGB value.
 *
 * Conventions fixed by this ABI where the paper leaves them open:
 *   - level k (k = 0 .. L-1) is the grid at scale 1/2^k, finest first; its
 *     size is ceil(H / 2^k) x ceil(W / 2^k) (Eq. (2) gives H / 2^k when 2^k
 *     divides H; the paper numbers the same grids coarsest first, i = L - k);
 *     input channel c of the MLP is level k = c;
 *   - upsampling is bilinear with half-pixel sample centres and edge
 *     replication at the nominal scale 2^k: output row y samples source row
 *     max((y + 1/2) / 2^k - 1/2, 0), the lower tap clamped to the last row;
 *   - layer l's weights are a [widths[l+1]][widths[l]] row-major matrix
 *     (output-major, the transpose of the paper's w in App. A), its bias a
 *     vector of widths[l+1] values;
 *   - the output is planar RGB, [batch][3][H][W], clamped to [0, 1]; the 8-bit
 *     form stores floor(255 c + 1/2).
 *
 * All entry points are plain C: no exceptions cross this boundary, no torch
 * or HIP runtime types appear in a signature (streams are passed as void*).
 * Link against libpic_decode.so.
 */
#ifndef PIC_DECODE_H
#define PIC_DECODE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PIC_DECODE_ABI_VERSION 1

/* Symbols of this header are the library's only exports. */
#if defined(__GNUC__) || defined(__clang__)
#define PIC_API __attribute__((visibility("default")))
#else
#define PIC_API
#endif

/* Opaque decoder handle: the validated descriptor, the chosen kernel variant,
 * the device it was created on, and 8 bytes of device memory per image of
 * max_batch, at least 64 bytes (the matrix-core kernels' tile counters:
 * workgroups take tiles from a per-image counter, or from one per XCD for a
 * single image, and each run clears the next run's).  Runs on one handle must
 * not overlap: enqueue them on one stream, or synchronise between them. */
typedef struct pic_decoder pic_decoder;

typedef enum pic_status {
    PIC_OK = 0,
    PIC_E_INVALID = 1,      /* an argument is out of range or a pointer is NULL   */
    PIC_E_UNSUPPORTED = 2,  /* valid request the library does not handle          */
    PIC_E_NODEVICE = 3,     /* no HIP device, or the current device is not gfx950 */
    PIC_E_HIP = 4,          /* the HIP runtime reported an error (launch failure) */
    PIC_E_NOMEM = 5         /* host allocation of the handle failed               */
} pic_status;

typedef enum pic_dtype {
    PIC_F32 = 0,            /* IEEE binary32                                      */
    PIC_BF16 = 1,           /* bfloat16 (weights only)                            */
    PIC_U8 = 2              /* unsigned 8-bit code (output only)                  */
} pic_dtype;

/* Kernel family.  AUTO picks MFMA_F32 for fp32 weights and MFMA_BF16 for
 * bf16 weights where that family covers the shape, VALU otherwise, and VALU
 * also for fp32 nets whose hidden layers are all at most 8 wide (the matrix
 * family would pad them to 16-neuron blocks).  VALU is
 * the reference family: plain binary32 arithmetic in a
 * fixed order (bias first, then one fused multiply-add per input in
 * increasing index), so its results are reproducible bit for bit. */
typedef enum pic_variant {
    PIC_VARIANT_AUTO = 0,
    PIC_VARIANT_VALU = 1,       /* fp32 vector ALU, canonical order                 */
    PIC_VARIANT_MFMA_F32 = 2,   /* fp32 matrix cores (v_mfma_f32_16x16x4_f32)       */
    PIC_VARIANT_MFMA_BF16 = 3,  /* bf16 matrix cores; requires PIC_BF16 weights;
                                   activations split into bf16 high + low parts    */
    PIC_VARIANT_MFMA_F16X3 = 4  /* fp16 matrix cores (v_mfma_f32_16x16x32_f16) at
                                   binary32 accuracy: each fp32 weight and
                                   activation is scaled by a power of two, split
                                   into two fp16 parts, and every product is
                                   formed from three partial products; requires
                                   PIC_F32 weights                                 */
} pic_variant;

enum {
    PIC_MAX_LEVELS = 12,    /* L                                                  */
    PIC_MAX_LAYERS = 8,     /* linear layers                                      */
    PIC_MAX_WIDTH = 128,    /* hidden width                                       */
    PIC_MAX_BATCH = 65535,  /* images per call                                    */
    PIC_NOALLOC_MAX_BATCH = 4096  /* images per pic_decode_run_noalloc call       */
};

/* desc.flags */
enum {
    PIC_FLAG_NO_CLAMP = 1u  /* fp32 output holds the raw last-layer value (no
                               clamp); meant for testing.  Invalid with PIC_U8. */
};

/* Decoder description.  Zero-initialise, then set struct_size to
 * sizeof(pic_decode_desc) (the library rejects sizes it does not know). */
typedef struct pic_decode_desc {
    uint32_t struct_size;
    int32_t height, width;                  /* H, W in [1, 2^23), H * W < 2^31  */
    int32_t num_levels;                     /* L in [1, PIC_MAX_LEVELS]          */
    int32_t num_layers;                     /* linear layers in [1, PIC_MAX_LAYERS] */
    int32_t widths[PIC_MAX_LAYERS + 1];     /* widths[0] == L, widths[num_layers] == 3,
                                               widths in between in [1, PIC_MAX_WIDTH] */
    int32_t weight_dtype;                   /* PIC_F32 or PIC_BF16 (biases are fp32) */
    int32_t out_dtype;                      /* PIC_F32 or PIC_U8                  */
    uint32_t flags;                         /* PIC_FLAG_*                          */
    int32_t max_batch;                      /* largest batch passed to run, >= 1  */
    int32_t variant;                        /* pic_variant                         */
} pic_decode_desc;

/* Introspection record filled by pic_decode_query. */
typedef struct pic_decode_info {
    uint32_t struct_size;                   /* set by the caller: sizeof(pic_decode_info) */
    int32_t variant;                        /* the variant actually used          */
    int64_t weights_per_image;              /* sum of widths[l] * widths[l+1]     */
    int64_t biases_per_image;               /* sum of widths[l+1]                 */
    int32_t device;                         /* HIP device ordinal of the handle   */
    int32_t pixels_per_wave_step;           /* pixels one wavefront handles per step */
    char kernel_name[64];                   /* NUL-terminated                      */
} pic_decode_info;

/*
 * pic_decode_create -- validate `desc` and build a handle for the current HIP
 * device.
 *   desc : read only, not retained.
 *   out  : receives the handle (set to NULL on failure).
 * Returns PIC_OK; PIC_E_INVALID for a malformed descriptor (sizes, widths,
 * dtypes, flags out of range); PIC_E_UNSUPPORTED for a valid combination no
 * kernel implements (e.g. MFMA_BF16 with fp32 weights); PIC_E_NODEVICE when no
 * gfx950 device is current; PIC_E_NOMEM when the handle cannot be allocated;
 * PIC_E_HIP when its device memory cannot (allocated and cleared here, once;
 * the clear runs on a private stream and waits for itself alone, not for work
 * queued on other streams).
 * Defines: Sec. 3.1 (pyramid and upsample), Sec. 4.1 / App. A (MLP).
 */
PIC_API pic_status pic_decode_create(const pic_decode_desc *desc, pic_decoder **out);

/*
 * pic_decode_run -- enqueue the synthesis of `batch` images on `stream`.
 *   batch      : 0 .. max_batch images (0 enqueues nothing).
 *   latents    : host array of num_levels device pointers; latents[k] points to
 *                fp32 [batch][ceil(H/2^k)][ceil(W/2^k)], row-major, image-major.
 *   weights    : device pointer; one image's parameters are every layer's
 *                [out][in] row-major matrix, layers concatenated
 *                (weights_per_image elements of weight_dtype); image b's start
 *                at weights + b * weights_img_stride elements.  A stride of 0
 *                shares one set across the batch (the paper's shared MLP^s).
 *   biases     : device pointer, fp32; per image every layer's bias vector
 *                concatenated (biases_per_image values), image b at
 *                biases + b * biases_img_stride (0: shared).
 *   out        : device pointer, [batch][3][H][W] of out_dtype (planar RGB).
 *   stream     : a hipStream_t (NULL: the null stream).
 * Buffers stay owned by the caller and must stay valid until the enqueued
 * work completes; inputs and output must not overlap.  Pointers must be
 * 4-byte aligned (2-byte for bf16 weights, 1-byte for u8 output).  The call
 * is asynchronous: it neither synchronises nor allocates.  On a validation
 * error nothing is enqueued; a failed launch returns PIC_E_HIP.  Faults of
 * the enqueued kernels surface at the caller's next synchronisation.
 * A handle must not be used by two threads at once.
 */
PIC_API pic_status pic_decode_run(pic_decoder *dec, int32_t batch,
                                  const float *const *latents,
                                  const void *weights, int64_t weights_img_stride,
                                  const float *biases, int64_t biases_img_stride,
                                  void *out, void *stream);

/*
 * pic_decode_run_noalloc -- pic_decode_run without a handle, for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation.  It validates `desc` (as
 * pic_decode_create does) and enqueues the same kernels pic_decode_run would,
 * and it calls no hipMalloc, hipFree or other allocating routine.
 *   desc       : read only, not retained; desc->max_batch bounds `batch`.
 *   other arguments, layouts and ownership: as pic_decode_run.
 * The matrix-core kernels' tile counters live in the library's own device
 * array (16 KiB: PIC_NOALLOC_MAX_BATCH 4-byte counters, held by each GPU the
 * library runs on until the process ends).  Each call first enqueues a small
 * kernel that clears the counters it uses, then the decode, on `stream`.
 * Every call on one GPU shares that array: calls that overlap on one GPU
 * (other streams without synchronisation, or other threads) race on it and
 * must not be made.  The first call on a device, with that device current,
 * looks up the array's device address and the device's properties.
 * Returns as pic_decode_run, plus PIC_E_UNSUPPORTED for batch above
 * PIC_NOALLOC_MAX_BATCH (nothing is enqueued) and the statuses of
 * pic_decode_create for the descriptor (PIC_E_INVALID, PIC_E_UNSUPPORTED,
 * PIC_E_NODEVICE); PIC_E_HIP if the array's address cannot be found.
 */
PIC_API pic_status pic_decode_run_noalloc(const pic_decode_desc *desc, int32_t batch,
                                          const float *const *latents,
                                          const void *weights, int64_t weights_img_stride,
                                          const float *biases, int64_t biases_img_stride,
                                          void *out, void *stream);

/*
 * pic_decode_run_layers -- pic_decode_run with one parameter pointer and one
 * per-image stride per layer, so some layers can be shared by every image
 * and others given per image (the paper's split of g_s into a shared MLP^s
 * and a per-image MLP^i, Sec. 3.1 and App. A).
 *   layer_weights[l]        : device pointer to image 0's layer-l matrix,
 *                             [widths[l+1]][widths[l]] row-major, weight_dtype
 *   layer_weight_strides[l] : elements from image b's matrix to image b+1's
 *                             (0: one matrix shared by the batch)
 *   layer_biases[l]         : device pointer to image 0's layer-l bias (fp32)
 *   layer_bias_strides[l]   : the same for biases
 * The four arrays are host arrays of num_layers entries.  Other arguments,
 * ownership and errors as pic_decode_run.
 */
PIC_API pic_status pic_decode_run_layers(pic_decoder *dec, int32_t batch, const float *const *latents,
                                         const void *const *layer_weights, const int64_t *layer_weight_strides,
                                         const float *const *layer_biases, const int64_t *layer_bias_strides,
                                         void *out, void *stream);

/*
 * pic_fuse_modulation -- fold instance normalisation and channel modulation
 * into the following linear layer (App. A).  For a layer out = W f~ + b whose
 * input is f~ = gamma * (f - mu) / sigma + beta (per input channel c), the
 * fused layer out = W' f + b' has
 *     W'[o][c] = W[o][c] * gamma[c] / sigma[c]
 *     b'[o]    = b[o] + sum_c W[o][c] * (beta[c] - gamma[c] * mu[c] / sigma[c])
 * (App. A writes the same with w = W^T).  Computed per image, in double
 * precision, rounded once to fp32.
 *   in, out      : layer input / output widths, 1 .. PIC_MAX_WIDTH
 *   batch        : images (0 enqueues nothing)
 *   w, b         : device, image b's W at w + b*w_stride ([out][in] row-major),
 *                  its bias at b + b*b_stride (strides 0: shared)
 *   gamma, beta, mu, sigma : device, image b's vectors of `in` values at
 *                  + b*stat_stride; sigma must be nonzero
 *   w_fused      : device, [batch][out][in] fp32 (written)
 *   b_fused      : device, [batch][out] fp32 (written)
 *   stream       : hipStream_t (NULL: null stream); asynchronous
 * Returns PIC_E_INVALID for bad sizes or NULL/misaligned pointers,
 * PIC_E_NODEVICE without a HIP device, PIC_E_HIP for a failed launch.
 * Outputs must not overlap the inputs.
 */
PIC_API pic_status pic_fuse_modulation(int32_t in, int32_t out, int32_t batch,
                                       const float *w, int64_t w_stride, const float *b, int64_t b_stride,
                                       const float *gamma, const float *beta, const float *mu,
                                       const float *sigma, int64_t stat_stride,
                                       float *w_fused, float *b_fused, void *stream);

/* pic_decode_query -- describe the handle (variant, kernel, parameter counts).
 * Returns PIC_E_INVALID for NULL arguments or an unknown info->struct_size. */
PIC_API pic_status pic_decode_query(const pic_decoder *dec, pic_decode_info *info);

/* pic_decode_destroy -- free the handle and its device memory (NULL is
 * accepted).  Synchronises the handle's device first. */
PIC_API void pic_decode_destroy(pic_decoder *dec);

/* pic_status_string -- static description of a status code (never NULL).
 * `status` is a pic_status value; any other int32_t gives "unknown status"
 * (the parameter is an int32_t so that a value outside the enumeration is
 * well defined to pass). */
PIC_API const char *pic_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* PIC_DECODE_H */
