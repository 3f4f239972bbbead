// Internal interface between the C ABI (pic_decode.hip) and the kernel
// translation units.  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pic_decode.h"

namespace pic {

// Read one dword of every 64-byte line of the kernel arguments, all at once
// and waited for together, at kernel entry.  The arguments of a launch are
// written for that launch, so their lines start cold; read where first
// needed, they would cost a memory round trip per line, one after another
// (the address of the next load often depends on the previous one).
template <int BYTES>
__device__ __forceinline__ void warm_kernel_args()
{
    static_assert(BYTES <= 12 * 64, "one operand per line below");
    const unsigned *ka = (const unsigned *)__builtin_amdgcn_kernarg_segment_ptr();
    unsigned v[12];
#pragma unroll
    for (int i = 0; i < 12; ++i)
        v[i] = ka[(i * 64 < BYTES ? i * 64 : 0) / 4];
    // every value used at once: the loads go out together, one wait
    asm volatile("" ::"s"(v[0]), "s"(v[1]), "s"(v[2]), "s"(v[3]), "s"(v[4]), "s"(v[5]), "s"(v[6]), "s"(v[7]),
                 "s"(v[8]), "s"(v[9]), "s"(v[10]), "s"(v[11]));
}

// Inclusive sum of x over the 64 lanes of the wavefront (every lane active),
// by data-parallel moves between lanes instead of exchanges through LDS:
// shifts by 1, 2, 4 and 8 within each row of 16 lanes give each row's
// running sums (a lane with no source adds 0); then lane 15 into row 1 and
// lane 47 into row 3, and lane 31 into rows 2 and 3, carry the earlier rows'
// totals.  Sums wrap like integer additions (packed counters stay packed
// while no field overflows).
__device__ __forceinline__ int32_t wave_inclusive_sum(int32_t x)
{
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);   // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);   // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);   // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, false);   // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);   // row_bcast:15, rows 1 and 3
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);   // row_bcast:31, rows 2 and 3
    return x;
}

// Zero `bytes` of device memory and wait for that alone: on a private
// non-blocking stream (default priority), so that work already queued on the
// caller's streams is not waited for.  For handle set-up, never inside a
// captured stream.
inline hipError_t zero_device_memory(void *mem, size_t bytes)
{
    hipStream_t s = nullptr;
    hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
    if (e != hipSuccess)
        return e;
    e = hipMemsetAsync(mem, 0, bytes, s);
    const hipError_t w = hipStreamSynchronize(s);
    const hipError_t d = hipStreamDestroy(s);
    return e != hipSuccess ? e : (w != hipSuccess ? w : d);
}

// Tile counters a decode handle keeps per run: one per image, and at least
// one per XCD (a one-image grid schedules each XCD's tiles separately).
constexpr int kXcds = 8;
inline int tile_counters(int max_batch) { return max_batch > kXcds ? max_batch : kXcds; }

// Output encodings of the epilogue.
enum OutKind : int32_t { OUT_RAW_F32 = 0, OUT_CLAMPED_F32 = 1, OUT_U8 = 2 };

// Everything a decode kernel needs, passed by value as the kernel argument.
// Level slots L .. PIC_MAX_LEVELS - 1 repeat level 0, so that an unrolled
// level loop reads every slot at a constant index (a run-time index into the
// kernel arguments becomes one waited-for scalar load per level).
struct DecodeParams {
    const float *lat[PIC_MAX_LEVELS];   // level k base pointer, [batch][hk][wk]
    int32_t hk[PIC_MAX_LEVELS];         // ceil(H / 2^k)
    int32_t wk[PIC_MAX_LEVELS];         // ceil(W / 2^k)
    int32_t H, W, L, nl;                // image size, levels, linear layers
    int32_t widths[PIC_MAX_LAYERS + 1];
    const void *wl[PIC_MAX_LAYERS];     // layer l's [out][in] matrix of image 0 (fp32 or bf16)
    int64_t wls[PIC_MAX_LAYERS];        // elements between images' copies of layer l (0: shared)
    const float *bl[PIC_MAX_LAYERS];    // layer l's bias of image 0
    int64_t bls[PIC_MAX_LAYERS];        // elements between images' biases of layer l (0: shared)
    void *out;                          // [batch][3][H][W]
    int32_t out_kind;                   // OutKind
    int32_t weights_bf16;               // 1: weights are bf16 bit patterns
    int32_t batch;
    int32_t groups_per_image;           // 16-pixel groups per image (MFMA kernels)
    int32_t *tile_ctr;                  // [batch] tile counters of this run (zero at its start)
    int32_t *tile_ctr_next;             // [tile_ctr_len] the next run's counters, cleared by this run
    int32_t tile_ctr_len;               // counters per run (the handle's max_batch)
};

// Kernel launchers: return hipSuccess or the launch error.  Each checks that
// the shape it is asked for is one it was instantiated for (returns
// hipErrorInvalidValue otherwise, nothing launched).
hipError_t launch_valu(const DecodeParams &p, hipStream_t s, const char **name, int *px_per_step);
hipError_t launch_mfma_f32(const DecodeParams &p, hipStream_t s, const char **name, int *px_per_step,
                           int num_cus);
hipError_t launch_mfma_bf16(const DecodeParams &p, hipStream_t s, const char **name, int *px_per_step,
                            int num_cus);
hipError_t launch_mfma_f16x3(const DecodeParams &p, hipStream_t s, const char **name, int *px_per_step,
                             int num_cus);

// Shape support queries used at create time (no device needed).
bool valu_supports(int L, int nl, const int32_t *widths);
bool mfma_f32_supports(int L, int nl, const int32_t *widths);
bool mfma_bf16_supports(int L, int nl, const int32_t *widths);
bool mfma_f16x3_supports(int L, int nl, const int32_t *widths);

}  // namespace pic

// ------------------------------------------------------------------------
// Latent decoding from the ZpR symbol stream (k_zpr.hip, pic_zpr.hip).
namespace pic {

constexpr int kZprThreads = 256;
constexpr int kZprChunkSmall = 256;            // symbols per workgroup on short streams
constexpr int kZprChunkLarge = 1024;           // ... on long ones
constexpr int64_t kZprLargeFrom = 256 * 1024;  // stream length from which the large chunk is used

// Kernel argument of both latent-decoding kernels.
struct ZprParams {
    const int32_t *sym;             // the stream
    int64_t n;                      // symbols in it
    int32_t eob;                    // end-of-block marker
    int32_t chunk;                  // symbols per workgroup: kZprChunkSmall or kZprChunkLarge
    int32_t nchunks;                // ceil(n / chunk), at least 1
    int32_t expected;               // blocks the stream must hold
    int32_t blocks_per_image;
    int32_t L;
    int32_t *counts;                // [nchunks] scratch: marker counts (their exclusive prefix
                                    // when counts_are_prefix)
    int32_t counts_are_prefix;      // 1: the scan kernel ran (long streams)
    int32_t *status;                // PIC_ZPR_ERR_* bits of the run
    // levels in stream order, i = 0 the coarsest (level k = L - 1 - i)
    int32_t first[PIC_MAX_LEVELS + 1];   // first block of stream level i inside an image;
                                         // [L]: blocks per image; INT32_MAX past it
    int32_t hk[PIC_MAX_LEVELS];
    int32_t wk[PIC_MAX_LEVELS];
    int32_t pw[PIC_MAX_LEVELS];          // patches per row
    int32_t pw_shift[PIC_MAX_LEVELS];    // k = 24 + ceil(log2 pw)
    int32_t pw_recip[PIC_MAX_LEVELS];    // ceil(2^k / pw) (< 2^25): q / pw = (q * it) >> k for q < 2^24
    float *lat[PIC_MAX_LEVELS];          // [batch][hk][wk] of stream level i
    int32_t *coeffs;                     // [expected][64] row-major (expand only)
};

// Enqueue the two kernels; `coeff_only` writes the expanded blocks to
// p.coeffs instead of transforming and placing them.
hipError_t launch_zpr(const ZprParams &p, bool coeff_only, hipStream_t s);

}  // namespace pic

// ------------------------------------------------------------------------
// Huffman entropy decoding (k_huff.hip, pic_huff.hip).
namespace pic {

constexpr int kHuffThreads = 256;
constexpr int kHuffSub = 64;                   // bitstream bits per parsing thread
constexpr int kHuffOwn = kHuffThreads - 1;     // subsequences a workgroup owns (its first thread
                                               // re-parses the previous workgroup's last one)
constexpr int kHuffPrefixInKernelMax = 4096;   // more workgroups: the fix kernel turns the
                                               // per-workgroup counts into prefixes
constexpr int kHuffLutBits = 11;               // first-level decode table: 2^11 entries
constexpr int kHuffMaxLen = 24;
constexpr int kHuffMaxTable = 4096;
constexpr int kHuffOneLaunchMax = 64;          // workgroups: one launch (parse, repair, write)
constexpr uint64_t kHuffWaitTicks = 20000000;  // a waiter's limit: 0.2 s of the 100 MHz real-time counter

// Kernel argument of the entropy-decoding kernels.
struct HuffParams {
    const uint8_t *data;            // bitstream, MSB first
    int32_t n_bits;
    int32_t nsub;                   // subsequences: ceil(n_bits / kHuffSub), at least 1
    int32_t n_symbols;              // symbols to decode
    int32_t n_table;
    const int32_t *values;          // [n_table]
    const uint8_t *lengths;         // [n_table]
    int32_t *out;                   // [n_symbols]
    int32_t *status;
    // scratch
    uint64_t *mask;                 // [nsub]: codeword starts of the subsequence's parse (bit k: offset k)
    int32_t *end;                   // [nsub]: where that parse crosses into the next subsequence, -1 if it
                                    // met a pattern that is no codeword, n_bits if the stream ran out
    int32_t *cnt;                   // [nsub]: codewords of the true parse that start in the subsequence
    uint32_t *fail;                 // [8 per workgroup]: owned subsequences left out of step (bit l: the
                                    // workgroup's thread l)
    int32_t *flags;                 // [1]: first subsequence whose true parse meets a pattern that is no
                                    // codeword
    int32_t *blk;                   // [ceil(nsub / kHuffOwn)]: symbols per workgroup (exclusive prefixes
                                    // when blk_is_prefix)
    int32_t *bnd;                   // [ceil(nsub / kHuffOwn)]: bit 0: the workgroup's last crossing point
                                    // moved; bit 1: the workgroup left subsequences to the fix kernel
    int32_t nblk;                   // workgroups of the parse and write kernels
    int32_t blk_is_prefix;
    uint64_t *sync;                 // [2]: the one-launch path's hand-off word (generation << 32 |
                                    // arrivals) and leave word (error bits << 32 | departures), zero
                                    // at create
    uint64_t wait_ticks;            // how long a workgroup waits for the repair step at most (100 MHz ticks)
};

hipError_t launch_huff(const HuffParams &p, hipStream_t s);

}  // namespace pic
