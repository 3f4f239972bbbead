// C ABI of the PIC synthesis decoder: argument validation, variant choice and
// launch on the caller's stream.  The kernels live in k_*.hip.
#include <hip/hip_runtime.h>

#include <mutex>
#include <new>
#include <stdio.h>
#include <string.h>

#include "pic_decode.h"
#include "pic_internal.h"

struct pic_decoder {
    pic_decode_desc desc;
    int32_t variant;            // resolved pic_variant (never AUTO)
    int32_t device;
    int32_t num_cus;
    int64_t weights_per_image;
    int64_t biases_per_image;
    int32_t px_per_step;
    char kernel_name[64];
    int32_t *d_ctr;             // [2][tile_counters(max_batch)] tile counters, used by alternate runs
    uint32_t runs;              // matrix-core runs launched so far
};

// Tile counters of pic_decode_run_noalloc: one slot of tile_counters(batch)
// per device (each GPU the library runs on holds its own copy of the array
// until the process ends).  Host code never passes this name to a kernel or a
// copy: it is a host-side stand-in; the device address comes from
// hipGetSymbolAddress, once per device (noalloc_state below).
static __device__ __align__(256) int32_t scratch[PIC_NOALLOC_MAX_BATCH];

namespace {

int32_t level_dim(int32_t n, int k) { return (int32_t)(((int64_t)n + (1LL << k) - 1) >> k); }

pic_status validate_desc(const pic_decode_desc *d)
{
    if (!d || d->struct_size != sizeof(pic_decode_desc))
        return PIC_E_INVALID;
    if (d->height < 1 || d->width < 1 || d->height >= (1 << 23) || d->width >= (1 << 23) ||
        (int64_t)d->height * d->width >= (1LL << 31))
        return PIC_E_INVALID;
    if (d->num_levels < 1 || d->num_levels > PIC_MAX_LEVELS)
        return PIC_E_INVALID;
    if (d->num_layers < 1 || d->num_layers > PIC_MAX_LAYERS)
        return PIC_E_INVALID;
    if (d->widths[0] != d->num_levels || d->widths[d->num_layers] != 3)
        return PIC_E_INVALID;
    for (int l = 1; l < d->num_layers; ++l)
        if (d->widths[l] < 1 || d->widths[l] > PIC_MAX_WIDTH)
            return PIC_E_INVALID;
    if (d->weight_dtype != PIC_F32 && d->weight_dtype != PIC_BF16)
        return PIC_E_INVALID;
    if (d->out_dtype != PIC_F32 && d->out_dtype != PIC_U8)
        return PIC_E_INVALID;
    if (d->flags & ~(uint32_t)PIC_FLAG_NO_CLAMP)
        return PIC_E_INVALID;
    if ((d->flags & PIC_FLAG_NO_CLAMP) && d->out_dtype != PIC_F32)
        return PIC_E_INVALID;
    if (d->max_batch < 1 || d->max_batch > PIC_MAX_BATCH)
        return PIC_E_INVALID;
    if (d->variant < PIC_VARIANT_AUTO || d->variant > PIC_VARIANT_MFMA_F16X3)
        return PIC_E_INVALID;
    return PIC_OK;
}

// The kernel family for a valid descriptor (AUTO resolved), or
// PIC_E_UNSUPPORTED.
pic_status resolve_variant(const pic_decode_desc *desc, int32_t *out)
{
    const int L = desc->num_levels, nl = desc->num_layers;
    int32_t variant = desc->variant;
    if (variant == PIC_VARIANT_AUTO) {
        // Matrix cores where the family covers the shape, else the reference
        // family.  An fp32 net whose hidden layers are all at most 8 wide
        // runs on the reference family too: the matrix family pads each layer
        // to a 16-neuron block, four times the multiply-adds of the hidden
        // layers, where the vector family evaluates one pixel per lane
        // unpadded (768x512, 8 -> 8 -> 8 -> 8 -> 3: 10.0 against 13.4 us).
        int widest = 0;
        for (int l = 1; l < nl; ++l)
            widest = desc->widths[l] > widest ? desc->widths[l] : widest;
        if (desc->weight_dtype == PIC_BF16 && pic::mfma_bf16_supports(L, nl, desc->widths))
            variant = PIC_VARIANT_MFMA_BF16;
        else if (desc->weight_dtype == PIC_F32 && widest > 8 && pic::mfma_f32_supports(L, nl, desc->widths))
            variant = PIC_VARIANT_MFMA_F32;
        else
            variant = PIC_VARIANT_VALU;
    }
    bool ok = false;
    switch (variant) {
    case PIC_VARIANT_VALU: ok = pic::valu_supports(L, nl, desc->widths); break;
    case PIC_VARIANT_MFMA_F32: ok = pic::mfma_f32_supports(L, nl, desc->widths); break;
    case PIC_VARIANT_MFMA_BF16:
        ok = desc->weight_dtype == PIC_BF16 && pic::mfma_bf16_supports(L, nl, desc->widths);
        break;
    case PIC_VARIANT_MFMA_F16X3:
        ok = desc->weight_dtype == PIC_F32 && pic::mfma_f16x3_supports(L, nl, desc->widths);
        break;
    }
    if (!ok)
        return PIC_E_UNSUPPORTED;
    *out = variant;
    return PIC_OK;
}

// Compute units of device dev if it is a gfx950 (else PIC_E_NODEVICE).
pic_status gfx950_cus(int dev, int *num_cus)
{
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
        (void)hipGetLastError();
        return PIC_E_NODEVICE;
    }
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return PIC_E_NODEVICE;
    *num_cus = prop.multiProcessorCount;
    return PIC_OK;
}

// The current device, if there is one.
pic_status current_device(int *dev)
{
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1 || hipGetDevice(dev) != hipSuccess) {
        (void)hipGetLastError();
        return PIC_E_NODEVICE;
    }
    return PIC_OK;
}

// A handle's host fields for a validated descriptor.
void init_handle(pic_decoder *d, const pic_decode_desc *desc, int32_t variant, int dev, int num_cus)
{
    memset(d, 0, sizeof *d);
    d->desc = *desc;
    d->variant = variant;
    d->device = dev;
    d->num_cus = num_cus;
    for (int l = 0; l < desc->num_layers; ++l) {
        d->weights_per_image += (int64_t)desc->widths[l] * desc->widths[l + 1];
        d->biases_per_image += desc->widths[l + 1];
    }
}

}  // namespace

extern "C" {

const char *pic_status_string(int32_t status)
{
    switch (status) {
    case PIC_OK: return "ok";
    case PIC_E_INVALID: return "invalid argument";
    case PIC_E_UNSUPPORTED: return "unsupported configuration";
    case PIC_E_NODEVICE: return "no gfx950 HIP device";
    case PIC_E_HIP: return "HIP runtime error";
    case PIC_E_NOMEM: return "out of host memory";
    }
    return "unknown status";
}

pic_status pic_decode_create(const pic_decode_desc *desc, pic_decoder **out)
{
    if (!out)
        return PIC_E_INVALID;
    *out = nullptr;
    pic_status st = validate_desc(desc);
    if (st != PIC_OK)
        return st;
    int32_t variant = 0;
    st = resolve_variant(desc, &variant);
    if (st != PIC_OK)
        return st;
    int dev = 0, num_cus = 0;
    st = current_device(&dev);
    if (st == PIC_OK)
        st = gfx950_cus(dev, &num_cus);
    if (st != PIC_OK)
        return st;

    pic_decoder *d = new (std::nothrow) pic_decoder;
    if (!d)
        return PIC_E_NOMEM;
    init_handle(d, desc, variant, dev, num_cus);
    const size_t ctr_bytes = sizeof(int32_t) * 2 * (size_t)pic::tile_counters(desc->max_batch);
    void *mem = nullptr;
    if (hipMalloc(&mem, ctr_bytes) != hipSuccess || pic::zero_device_memory(mem, ctr_bytes) != hipSuccess) {
        (void)hipGetLastError();
        if (mem)
            (void)hipFree(mem);
        delete d;
        return PIC_E_HIP;
    }
    d->d_ctr = static_cast<int32_t *>(mem);
    *out = d;
    return PIC_OK;
}

}  // extern "C"

namespace {

// Checks shared by both run entry points and the parts of the kernel
// argument they have in common (latents, sizes, output).
pic_status prepare(const pic_decoder *dec, int32_t batch, const float *const *latents, void *out,
                   pic::DecodeParams &p)
{
    const pic_decode_desc &d = dec->desc;
    if (!latents || !out)
        return PIC_E_INVALID;
    if (d.out_dtype == PIC_F32 && ((uintptr_t)out % 4))
        return PIC_E_INVALID;
    memset(&p, 0, sizeof p);
    for (int k = 0; k < d.num_levels; ++k) {
        if (!latents[k] || ((uintptr_t)latents[k] % 4))
            return PIC_E_INVALID;
        p.lat[k] = latents[k];
        p.hk[k] = level_dim(d.height, k);
        p.wk[k] = level_dim(d.width, k);
    }
    for (int k = d.num_levels; k < PIC_MAX_LEVELS; ++k) {   // unused slots repeat level 0
        p.lat[k] = p.lat[0];
        p.hk[k] = p.hk[0];
        p.wk[k] = p.wk[0];
    }
    p.H = d.height;
    p.W = d.width;
    p.L = d.num_levels;
    p.nl = d.num_layers;
    for (int l = 0; l <= d.num_layers; ++l)
        p.widths[l] = d.widths[l];
    p.out = out;
    p.out_kind = d.out_dtype == PIC_U8 ? pic::OUT_U8
               : (d.flags & PIC_FLAG_NO_CLAMP) ? pic::OUT_RAW_F32 : pic::OUT_CLAMPED_F32;
    p.weights_bf16 = d.weight_dtype == PIC_BF16;
    p.batch = batch;
    p.groups_per_image = (int32_t)(((int64_t)d.height * d.width + 15) / 16);
    return PIC_OK;
}

// The checks of pic_decode_run and the rest of its kernel argument.  PIC_OK
// with nothing to enqueue when batch is 0.
pic_status run_params(const pic_decoder *dec, int32_t batch, const float *const *latents, const void *weights,
                      int64_t weights_img_stride, const float *biases, int64_t biases_img_stride, void *out,
                      pic::DecodeParams &p)
{
    const pic_decode_desc &d = dec->desc;
    if (batch < 0 || batch > d.max_batch)
        return PIC_E_INVALID;
    if (weights_img_stride < 0 || biases_img_stride < 0)
        return PIC_E_INVALID;
    if (batch == 0)
        return PIC_OK;
    if (!weights || !biases)
        return PIC_E_INVALID;
    const size_t esize = d.weight_dtype == PIC_BF16 ? 2 : 4;
    if (((uintptr_t)weights % esize) || ((uintptr_t)biases % 4))
        return PIC_E_INVALID;
    // Per-image parameter blocks must not overlap unless shared.
    if (weights_img_stride != 0 && weights_img_stride < dec->weights_per_image)
        return PIC_E_INVALID;
    if (biases_img_stride != 0 && biases_img_stride < dec->biases_per_image)
        return PIC_E_INVALID;
    pic_status st = prepare(dec, batch, latents, out, p);
    if (st != PIC_OK)
        return st;
    int64_t wo = 0, bo = 0;
    for (int l = 0; l < d.num_layers; ++l) {
        p.wl[l] = static_cast<const char *>(weights) + wo * esize;
        p.wls[l] = weights_img_stride;
        p.bl[l] = biases + bo;
        p.bls[l] = biases_img_stride;
        wo += (int64_t)d.widths[l] * d.widths[l + 1];
        bo += d.widths[l + 1];
    }
    return PIC_OK;
}

__global__ void k_clear_counters(int32_t *c, int n)
{
    for (int i = threadIdx.x; i < n; i += blockDim.x)
        c[i] = 0;
}

// Enqueue the decode.  A handle's run uses one of its two counter slots
// (cleared by the previous run, or at create) and has the kernel clear the
// other.  With clear_here (pic_decode_run_noalloc: dec->d_ctr is one slot of
// the library's per-device array, whose contents the previous call left), a
// fill kernel clears the counters on the stream first and the decode kernel
// clears nothing.
pic_status launch(pic_decoder *dec, const pic::DecodeParams &params, void *stream, bool clear_here)
{
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess || cur != dec->device) {
        (void)hipGetLastError();
        return PIC_E_INVALID;   // the handle belongs to another device
    }
    pic::DecodeParams p = params;
    hipStream_t s = (hipStream_t)stream;
    if (clear_here) {
        p.tile_ctr = dec->d_ctr;
        p.tile_ctr_next = dec->d_ctr;
        p.tile_ctr_len = 0;
        if (dec->variant != PIC_VARIANT_VALU) {   // (the reference family takes no tiles)
            hipLaunchKernelGGL(k_clear_counters, dim3(1), dim3(256), 0, s, dec->d_ctr,
                               pic::tile_counters(params.batch));
            if (hipGetLastError() != hipSuccess)
                return PIC_E_HIP;
        }
    } else {
        const int32_t mb = pic::tile_counters(dec->desc.max_batch);
        p.tile_ctr = dec->d_ctr + (dec->runs & 1u) * mb;
        p.tile_ctr_next = dec->d_ctr + ((dec->runs + 1u) & 1u) * mb;
        p.tile_ctr_len = mb;
    }
    const char *name = nullptr;
    int pxs = 0;
    hipError_t e = hipErrorInvalidValue;
    switch (dec->variant) {
    case PIC_VARIANT_VALU: e = pic::launch_valu(p, s, &name, &pxs); break;
    case PIC_VARIANT_MFMA_F32: e = pic::launch_mfma_f32(p, s, &name, &pxs, dec->num_cus); break;
    case PIC_VARIANT_MFMA_BF16: e = pic::launch_mfma_bf16(p, s, &name, &pxs, dec->num_cus); break;
    case PIC_VARIANT_MFMA_F16X3: e = pic::launch_mfma_f16x3(p, s, &name, &pxs, dec->num_cus); break;
    }
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return PIC_E_HIP;
    }
    if (dec->variant != PIC_VARIANT_VALU && !clear_here)
        ++dec->runs;
    if (name) {
        strncpy(dec->kernel_name, name, sizeof dec->kernel_name - 1);
        dec->px_per_step = pxs;
    }
    return PIC_OK;
}

// Per-device state of pic_decode_run_noalloc, set up on its first call on a
// device (with that device current): the device address of `scratch` and the
// compute-unit count.
constexpr int kMaxDevices = 64;
struct NoAllocDevice {
    bool ready;
    pic_status status;     // of the set-up (PIC_OK, PIC_E_NODEVICE or PIC_E_HIP)
    int32_t *scratch;      // device address of this device's copy of `scratch`
    int num_cus;
};
std::mutex g_noalloc_mu;
NoAllocDevice g_noalloc[kMaxDevices];

pic_status noalloc_state(int dev, NoAllocDevice *out)
{
    if (dev < 0 || dev >= kMaxDevices)
        return PIC_E_NODEVICE;
    std::lock_guard<std::mutex> lock(g_noalloc_mu);
    NoAllocDevice &st = g_noalloc[dev];
    if (!st.ready) {
        st.status = gfx950_cus(dev, &st.num_cus);
        if (st.status == PIC_OK) {
            void *ptr = nullptr;
            if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
                (void)hipGetLastError();
                st.status = PIC_E_HIP;
            } else {
                st.scratch = static_cast<int32_t *>(ptr);
            }
        }
        st.ready = true;
    }
    *out = st;
    return st.status;
}

}  // namespace

extern "C" {

pic_status pic_decode_run(pic_decoder *dec, int32_t batch, const float *const *latents,
                          const void *weights, int64_t weights_img_stride,
                          const float *biases, int64_t biases_img_stride,
                          void *out, void *stream)
{
    if (!dec)
        return PIC_E_INVALID;
    pic::DecodeParams p;
    const pic_status st = run_params(dec, batch, latents, weights, weights_img_stride, biases,
                                     biases_img_stride, out, p);
    if (st != PIC_OK || batch == 0)
        return st;
    return launch(dec, p, stream, false);
}

pic_status pic_decode_run_noalloc(const pic_decode_desc *desc, int32_t batch, const float *const *latents,
                                  const void *weights, int64_t weights_img_stride,
                                  const float *biases, int64_t biases_img_stride,
                                  void *out, void *stream)
{
    pic_status st = validate_desc(desc);
    if (st != PIC_OK)
        return st;
    if (batch > PIC_NOALLOC_MAX_BATCH && batch <= desc->max_batch)
        return PIC_E_UNSUPPORTED;    // beyond the library's counter array
    int32_t variant = 0;
    st = resolve_variant(desc, &variant);
    if (st != PIC_OK)
        return st;
    // a handle on the stack: host fields only, its counters the array's
    pic_decoder dec;
    init_handle(&dec, desc, variant, 0, 0);
    pic::DecodeParams p;
    st = run_params(&dec, batch, latents, weights, weights_img_stride, biases, biases_img_stride, out, p);
    if (st != PIC_OK || batch == 0)
        return st;
    int dev = 0;
    st = current_device(&dev);
    if (st != PIC_OK)
        return st;
    NoAllocDevice nd;
    st = noalloc_state(dev, &nd);
    if (st != PIC_OK)
        return st;
    dec.device = dev;
    dec.num_cus = nd.num_cus;
    dec.d_ctr = nd.scratch;
    return launch(&dec, p, stream, true);
}

pic_status pic_decode_run_layers(pic_decoder *dec, int32_t batch, const float *const *latents,
                                 const void *const *layer_weights, const int64_t *layer_weight_strides,
                                 const float *const *layer_biases, const int64_t *layer_bias_strides,
                                 void *out, void *stream)
{
    if (!dec)
        return PIC_E_INVALID;
    const pic_decode_desc &d = dec->desc;
    if (batch < 0 || batch > d.max_batch)
        return PIC_E_INVALID;
    if (!layer_weights || !layer_weight_strides || !layer_biases || !layer_bias_strides)
        return PIC_E_INVALID;
    const size_t esize = d.weight_dtype == PIC_BF16 ? 2 : 4;
    for (int l = 0; l < d.num_layers; ++l) {
        const int64_t nw = (int64_t)d.widths[l] * d.widths[l + 1], nb = d.widths[l + 1];
        if (!layer_weights[l] || !layer_biases[l] || ((uintptr_t)layer_weights[l] % esize) ||
            ((uintptr_t)layer_biases[l] % 4))
            return PIC_E_INVALID;
        if (layer_weight_strides[l] < 0 || layer_bias_strides[l] < 0 ||
            (layer_weight_strides[l] != 0 && layer_weight_strides[l] < nw) ||
            (layer_bias_strides[l] != 0 && layer_bias_strides[l] < nb))
            return PIC_E_INVALID;
    }
    if (batch == 0)
        return PIC_OK;
    pic::DecodeParams p;
    pic_status st = prepare(dec, batch, latents, out, p);
    if (st != PIC_OK)
        return st;
    for (int l = 0; l < d.num_layers; ++l) {
        p.wl[l] = layer_weights[l];
        p.wls[l] = layer_weight_strides[l];
        p.bl[l] = layer_biases[l];
        p.bls[l] = layer_bias_strides[l];
    }
    return launch(dec, p, stream, false);
}

pic_status pic_decode_query(const pic_decoder *dec, pic_decode_info *info)
{
    if (!dec || !info || info->struct_size != sizeof(pic_decode_info))
        return PIC_E_INVALID;
    info->variant = dec->variant;
    info->weights_per_image = dec->weights_per_image;
    info->biases_per_image = dec->biases_per_image;
    info->device = dec->device;
    info->pixels_per_wave_step = dec->px_per_step;
    memset(info->kernel_name, 0, sizeof info->kernel_name);
    strncpy(info->kernel_name, dec->kernel_name, sizeof info->kernel_name - 1);
    return PIC_OK;
}

void pic_decode_destroy(pic_decoder *dec)
{
    if (!dec)
        return;
    int cur = -1;
    const bool switch_dev = hipGetDevice(&cur) == hipSuccess && cur != dec->device;
    if (switch_dev)
        (void)hipSetDevice(dec->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(dec->d_ctr);
    if (switch_dev)
        (void)hipSetDevice(cur);
    (void)hipGetLastError();
    delete dec;
}

}  // extern "C"
