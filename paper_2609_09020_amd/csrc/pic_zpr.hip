// C ABI of the latent-decoding step (include/pic_zpr.h): validation, the
// stream-order level table, device scratch and launch on the caller's stream.
// The kernels live in k_zpr.hip.
#include <hip/hip_runtime.h>

#include <new>
#include <string.h>

#include "pic_internal.h"
#include "pic_zpr.h"

struct pic_zpr {
    pic_zpr_desc desc;
    int32_t device;
    int64_t blocks_per_image;
    int64_t max_symbols;
    int32_t max_chunks;
    int64_t scratch_bytes;
    int32_t *d_counts;          // [max_chunks]
    // levels in stream order (coarsest first)
    int32_t first[PIC_MAX_LEVELS + 1];
    int32_t hk[PIC_MAX_LEVELS], wk[PIC_MAX_LEVELS], pw[PIC_MAX_LEVELS];
};

namespace {

constexpr int64_t kMaxSymbolsPerBlock = 65;   // 64 coefficients and the marker
constexpr int64_t kInt31 = (1LL << 31) - 1;
// Up to this many chunks the decoding kernel sums the earlier chunks' marker
// counts itself; beyond it a one-workgroup scan kernel runs first.
constexpr int32_t kPrefixInKernelMax = 16384;

int32_t level_dim(int32_t n, int k) { return (int32_t)(((int64_t)n + (1LL << k) - 1) >> k); }

pic_status check_device(int32_t *dev_out)
{
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
        (void)hipGetLastError();
        return PIC_E_NODEVICE;
    }
    int dev = 0;
    hipDeviceProp_t prop;
    if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess) {
        (void)hipGetLastError();
        return PIC_E_NODEVICE;
    }
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return PIC_E_NODEVICE;
    *dev_out = dev;
    return PIC_OK;
}

// Shared checks of both run entry points; fills everything but the output.
pic_status prepare(const pic_zpr *h, int32_t batch, const int32_t *symbols, int64_t n_symbols, int32_t eob,
                   int32_t *status, pic::ZprParams &p)
{
    if (!h || batch < 0 || batch > h->desc.max_batch || n_symbols < 0 || !status)
        return PIC_E_INVALID;
    if ((uintptr_t)status % 4 || (n_symbols > 0 && (!symbols || (uintptr_t)symbols % 4)))
        return PIC_E_INVALID;
    if (eob < INT32_MIN + 17 || eob == INT32_MAX)
        return PIC_E_INVALID;
    const int64_t blocks = h->blocks_per_image * batch;
    int64_t cap = kMaxSymbolsPerBlock * blocks;
    if (cap > kInt31)
        cap = kInt31;
    if (batch > 0 && n_symbols > cap)
        return PIC_E_INVALID;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess || cur != h->device) {
        (void)hipGetLastError();
        return PIC_E_INVALID;   // the handle belongs to another device
    }
    memset(&p, 0, sizeof p);
    p.sym = symbols;
    p.n = n_symbols;
    p.eob = eob;
    p.chunk = n_symbols >= pic::kZprLargeFrom ? pic::kZprChunkLarge : pic::kZprChunkSmall;
    p.nchunks = (int32_t)((n_symbols + p.chunk - 1) / p.chunk);
    if (p.nchunks < 1)
        p.nchunks = 1;
    p.expected = (int32_t)blocks;
    p.blocks_per_image = (int32_t)h->blocks_per_image;
    p.L = h->desc.num_levels;
    p.counts = h->d_counts;
    p.counts_are_prefix = p.nchunks > kPrefixInKernelMax;
    p.status = status;
    for (int i = 0; i <= PIC_MAX_LEVELS; ++i)   // past the end: no block reaches these
        p.first[i] = i <= p.L ? h->first[i] : INT32_MAX;
    for (int i = 0; i < p.L; ++i) {
        p.hk[i] = h->hk[i];
        p.wk[i] = h->wk[i];
        p.pw[i] = h->pw[i];
        int k = 24;
        while ((1 << (k - 24)) < h->pw[i])
            ++k;
        p.pw_shift[i] = k;
        p.pw_recip[i] = (int32_t)(((1ULL << k) + (uint64_t)h->pw[i] - 1) / (uint64_t)h->pw[i]);
    }
    return PIC_OK;
}

}  // namespace

extern "C" {

pic_status pic_zpr_create(const pic_zpr_desc *d, pic_zpr **out)
{
    if (!out)
        return PIC_E_INVALID;
    *out = nullptr;
    if (!d || d->struct_size != sizeof(pic_zpr_desc))
        return PIC_E_INVALID;
    if (d->height < 1 || d->width < 1 || (int64_t)d->height * d->width >= (1LL << 31))
        return PIC_E_INVALID;
    if (d->num_levels < 1 || d->num_levels > PIC_MAX_LEVELS)
        return PIC_E_INVALID;
    if (d->max_batch < 1 || d->max_batch > PIC_MAX_BATCH)
        return PIC_E_INVALID;

    pic_zpr tmp;
    memset(&tmp, 0, sizeof tmp);
    tmp.desc = *d;
    const int L = d->num_levels;
    int64_t nb = 0;
    for (int i = 0; i < L; ++i) {               // stream order: level k = L - 1 - i
        const int k = L - 1 - i;
        tmp.hk[i] = level_dim(d->height, k);
        tmp.wk[i] = level_dim(d->width, k);
        tmp.pw[i] = (tmp.wk[i] + 7) / 8;
        tmp.first[i] = (int32_t)nb;
        nb += (int64_t)((tmp.hk[i] + 7) / 8) * tmp.pw[i];
    }
    tmp.first[L] = (int32_t)nb;
    // the kernels divide patch indices (< 2^24 per level) by patches per row
    // (< 2^16) with a fixed-point reciprocal, exact in that range
    for (int i = 0; i < L; ++i)
        if (tmp.pw[i] >= (1 << 16) || tmp.first[i + 1] - tmp.first[i] >= (1 << 24))
            return PIC_E_UNSUPPORTED;
    tmp.blocks_per_image = nb;
    if (nb * d->max_batch > kInt31)
        return PIC_E_UNSUPPORTED;
    tmp.max_symbols = kMaxSymbolsPerBlock * nb * d->max_batch;
    if (tmp.max_symbols > kInt31)
        tmp.max_symbols = kInt31;
    tmp.max_chunks = (int32_t)((tmp.max_symbols + pic::kZprChunkSmall - 1) / pic::kZprChunkSmall);

    pic_status st = check_device(&tmp.device);
    if (st != PIC_OK)
        return st;

    pic_zpr *h = new (std::nothrow) pic_zpr;
    if (!h)
        return PIC_E_NOMEM;
    *h = tmp;
    // per-chunk marker counts (every run writes them before reading them)
    h->scratch_bytes = (int64_t)(((size_t)h->max_chunks * sizeof(int32_t) + 255) & ~(size_t)255);
    void *mem = nullptr;
    if (hipMalloc(&mem, (size_t)h->scratch_bytes) != hipSuccess) {
        (void)hipGetLastError();
        delete h;
        return PIC_E_HIP;
    }
    h->d_counts = static_cast<int32_t *>(mem);
    *out = h;
    return PIC_OK;
}

pic_status pic_zpr_decode(pic_zpr *h, int32_t batch, const int32_t *symbols, int64_t n_symbols, int32_t eob,
                          float *const *latents, int32_t *status, void *stream)
{
    pic::ZprParams p;
    pic_status st = prepare(h, batch, symbols, n_symbols, eob, status, p);
    if (st != PIC_OK)
        return st;
    if (batch == 0)
        return PIC_OK;
    if (!latents)
        return PIC_E_INVALID;
    for (int i = 0; i < p.L; ++i) {
        float *lk = latents[p.L - 1 - i];          // stream level i is level k = L - 1 - i
        if (!lk || (uintptr_t)lk % 4)
            return PIC_E_INVALID;
        p.lat[i] = lk;
    }
    if (pic::launch_zpr(p, false, (hipStream_t)stream) != hipSuccess) {
        (void)hipGetLastError();
        return PIC_E_HIP;
    }
    return PIC_OK;
}

pic_status pic_zpr_expand(pic_zpr *h, int32_t batch, const int32_t *symbols, int64_t n_symbols, int32_t eob,
                          int32_t *coeffs, int32_t *status, void *stream)
{
    pic::ZprParams p;
    pic_status st = prepare(h, batch, symbols, n_symbols, eob, status, p);
    if (st != PIC_OK)
        return st;
    if (batch == 0)
        return PIC_OK;
    if (!coeffs || (uintptr_t)coeffs % 16)
        return PIC_E_INVALID;
    p.coeffs = coeffs;
    if (pic::launch_zpr(p, true, (hipStream_t)stream) != hipSuccess) {
        (void)hipGetLastError();
        return PIC_E_HIP;
    }
    return PIC_OK;
}

pic_status pic_zpr_query(const pic_zpr *h, pic_zpr_info *info)
{
    if (!h || !info || info->struct_size != sizeof(pic_zpr_info))
        return PIC_E_INVALID;
    info->device = h->device;
    info->blocks_per_image = h->blocks_per_image;
    info->max_symbols = h->max_symbols;
    info->scratch_bytes = h->scratch_bytes;
    info->symbols_per_chunk = pic::kZprChunkSmall;
    return PIC_OK;
}

void pic_zpr_destroy(pic_zpr *h)
{
    if (!h)
        return;
    int cur = -1;
    const bool switch_dev = hipGetDevice(&cur) == hipSuccess && cur != h->device;
    if (switch_dev)
        (void)hipSetDevice(h->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(h->d_counts);
    if (switch_dev)
        (void)hipSetDevice(cur);
    (void)hipGetLastError();
    delete h;
}

}  // extern "C"
