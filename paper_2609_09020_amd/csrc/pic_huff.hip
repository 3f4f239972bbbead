// C ABI of the entropy-decoding step (include/pic_huff.h): validation, device
// scratch and launch on the caller's stream.  The kernels live in k_huff.hip.
#include <hip/hip_runtime.h>

#include <new>
#include <string.h>

#include "pic_huff.h"
#include "pic_internal.h"

struct pic_huff {
    pic_huff_desc desc;
    int32_t device;
    int32_t max_nsub;
    int64_t scratch_bytes;
    char *d_scratch;
    // offsets of the scratch arrays
    size_t o_mask, o_end, o_cnt, o_fail, o_flags, o_blk, o_bnd, o_sync;
};

namespace {

constexpr int64_t kInt31 = (1LL << 31) - 1;

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

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

}  // namespace

extern "C" {

pic_status pic_huff_create(const pic_huff_desc *d, pic_huff **out)
{
    if (!out)
        return PIC_E_INVALID;
    *out = nullptr;
    if (!d || d->struct_size != sizeof(pic_huff_desc) || d->reserved != 0)
        return PIC_E_INVALID;
    if (d->max_bits < 1 || d->max_bits > kInt31)
        return PIC_E_INVALID;
    int32_t dev = 0;
    pic_status st = check_device(&dev);
    if (st != PIC_OK)
        return st;
    pic_huff *h = new (std::nothrow) pic_huff;
    if (!h)
        return PIC_E_NOMEM;
    memset(h, 0, sizeof *h);
    h->desc = *d;
    h->device = dev;
    h->max_nsub = (int32_t)((d->max_bits + pic::kHuffSub - 1) / pic::kHuffSub);
    const size_t nblk = (size_t)(h->max_nsub + pic::kHuffOwn - 1) / pic::kHuffOwn;
    size_t o = 0;
    h->o_mask = o;   o += align256(sizeof(uint64_t) * (size_t)h->max_nsub);
    h->o_end = o;    o += align256(sizeof(int32_t) * (size_t)h->max_nsub);
    h->o_cnt = o;    o += align256(sizeof(int32_t) * (size_t)h->max_nsub);
    h->o_fail = o;   o += align256(sizeof(uint32_t) * 8 * nblk);       // two words per wave
    h->o_flags = o;  o += align256(sizeof(int32_t) * 4);
    h->o_blk = o;    o += align256(sizeof(int32_t) * nblk);
    h->o_bnd = o;    o += align256(sizeof(int32_t) * nblk);
    h->o_sync = o;   o += align256(2 * sizeof(uint64_t));   // hand-off and leave words
    h->scratch_bytes = (int64_t)o;
    void *mem = nullptr;
    if (hipMalloc(&mem, o) != hipSuccess) {
        (void)hipGetLastError();
        delete h;
        return PIC_E_HIP;
    }
    h->d_scratch = static_cast<char *>(mem);
    // the one-launch path's hand-off word starts at zero; each launch leaves
    // it ready for the next
    if (pic::zero_device_memory(h->d_scratch + h->o_sync, 2 * sizeof(uint64_t)) != hipSuccess) {
        (void)hipGetLastError();
        (void)hipFree(mem);
        delete h;
        return PIC_E_HIP;
    }
    *out = h;
    return PIC_OK;
}

pic_status pic_huff_decode(pic_huff *h, const uint8_t *data, int64_t n_bits, const int32_t *values,
                           const uint8_t *lengths, int32_t n_table, int64_t n_symbols, int32_t *out,
                           int32_t *status, void *stream)
{
    if (!h || n_bits < 0 || n_bits > h->desc.max_bits || n_symbols < 0 || n_symbols > kInt31)
        return PIC_E_INVALID;
    if (n_table < 1 || n_table > PIC_HUFF_MAX_TABLE)
        return PIC_E_INVALID;
    if (n_symbols == 0)
        return PIC_OK;
    if ((n_bits > 0 && !data) || !values || !lengths || !out || !status)
        return PIC_E_INVALID;
    if ((uintptr_t)values % 4 || (uintptr_t)out % 4 || (uintptr_t)status % 4)
        return PIC_E_INVALID;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess || cur != h->device) {
        (void)hipGetLastError();
        return PIC_E_INVALID;   // the handle belongs to another device
    }
    pic::HuffParams p;
    memset(&p, 0, sizeof p);
    p.data = data;
    p.n_bits = (int32_t)n_bits;
    p.nsub = (int32_t)((n_bits + pic::kHuffSub - 1) / pic::kHuffSub);
    if (p.nsub < 1)
        p.nsub = 1;
    p.n_symbols = (int32_t)n_symbols;
    p.n_table = n_table;
    p.values = values;
    p.lengths = lengths;
    p.out = out;
    p.status = status;
    p.mask = reinterpret_cast<uint64_t *>(h->d_scratch + h->o_mask);
    p.end = reinterpret_cast<int32_t *>(h->d_scratch + h->o_end);
    p.cnt = reinterpret_cast<int32_t *>(h->d_scratch + h->o_cnt);
    p.fail = reinterpret_cast<uint32_t *>(h->d_scratch + h->o_fail);
    p.flags = reinterpret_cast<int32_t *>(h->d_scratch + h->o_flags);
    p.blk = reinterpret_cast<int32_t *>(h->d_scratch + h->o_blk);
    p.bnd = reinterpret_cast<int32_t *>(h->d_scratch + h->o_bnd);
    p.nblk = (p.nsub + pic::kHuffOwn - 1) / pic::kHuffOwn;
    p.blk_is_prefix = p.nblk > pic::kHuffPrefixInKernelMax;
    p.sync = reinterpret_cast<uint64_t *>(h->d_scratch + h->o_sync);
    p.wait_ticks = pic::kHuffWaitTicks;
    if (pic::launch_huff(p, (hipStream_t)stream) != hipSuccess) {
        (void)hipGetLastError();
        return PIC_E_HIP;
    }
    return PIC_OK;
}

pic_status pic_huff_query(const pic_huff *h, pic_huff_info *info)
{
    if (!h || !info || info->struct_size != sizeof(pic_huff_info))
        return PIC_E_INVALID;
    info->device = h->device;
    info->max_bits = h->desc.max_bits;
    info->scratch_bytes = h->scratch_bytes;
    info->bits_per_thread = pic::kHuffSub;
    info->lut_bits = pic::kHuffLutBits;
    return PIC_OK;
}

void pic_huff_destroy(pic_huff *h)
{
    if (!h)
        return;
    int cur = -1;
    const bool switch_dev = hipGetDevice(&cur) == hipSuccess && cur != h->device;
    if (switch_dev)
        (void)hipSetDevice(h->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(h->d_scratch);
    if (switch_dev)
        (void)hipSetDevice(cur);
    (void)hipGetLastError();
    delete h;
}

}  // extern "C"
