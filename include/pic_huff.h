/*
 * pic_huff.h -- C ABI of the PIC entropy-decoding step on AMD Instinct MI355X
 * (gfx950): from the Huffman-coded bitstream to the ZpR symbol stream that
 * pic_zpr_decode (pic_zpr.h) expands.
 *
 * The operation (PIC, Fig. 1 "HD"; Sec. 3.3; Sec. 4.1): the encoder codes
 * an image's ZpR symbols with an image-specific Huffman code whose stored
 * table lists only the symbols used; the decoder maps every codeword back to
 * its symbol (Sec. 3.3 builds the decode table with 2^p entries, p the
 * longest code, so that one symbol costs one lookup; Sec. 4.1 decodes in
 * parallel on the GPU, after GPUHD).
 *
 * Conventions fixed by this ABI where the paper leaves them open:
 *   - the table is a list of (symbol value, code length) pairs, one per used
 *     symbol; the code is the canonical Huffman code of those lengths as
 *     DEFLATE defines it (RFC 1951, Sec. 3.2.2): codes of one length are
 *     consecutive integers in table order, shorter lengths first;
 *   - code lengths are 1 .. PIC_HUFF_MAX_LEN bits;
 *   - the bitstream is read most significant bit first: bit 7 of byte 0 is
 *     the first bit;
 *   - the number of symbols to decode is given (the container holds it).
 *
 * Link against libpic_decode.so (same library, same status codes).
 */
#ifndef PIC_HUFF_H
#define PIC_HUFF_H

#include <stdint.h>

#include "pic_decode.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Opaque handle: the device it was created on and its device scratch (the
 * per-subsequence parse records: about 16 bytes per 64 bits of the longest
 * accepted stream).  Runs on one handle must not overlap: enqueue them on one
 * stream, or synchronise between them. */
typedef struct pic_huff pic_huff;

enum {
    PIC_HUFF_MAX_LEN = 24,          /* longest codeword, bits                        */
    PIC_HUFF_MAX_TABLE = 4096       /* table entries (used symbols)                  */
};

/* Bits of the status word a run writes (0: decoded without error). */
enum {
    PIC_HUFF_ERR_BITS = 1,          /* the bits end before n_symbols codewords      */
    PIC_HUFF_ERR_CODE = 2,          /* a bit pattern that starts no codeword; the
                                       decoding stops there (BITS is then not set)  */
    PIC_HUFF_ERR_TABLE = 4,         /* a length outside 1 .. PIC_HUFF_MAX_LEN, or an
                                       over-subscribed code (Kraft sum above 1);
                                       nothing is decoded                           */
    PIC_HUFF_ERR_SYNC = 8           /* a short stream's one-launch decode: a
                                       workgroup gave up waiting (a bounded wait,
                                       about 0.2 s) for the repair step of the
                                       others; its symbols are not written. Calls
                                       on one handle must not overlap           */
};

/* Zero-initialise, then set struct_size = sizeof(pic_huff_desc). */
typedef struct pic_huff_desc {
    uint32_t struct_size;
    int32_t reserved;               /* 0                                             */
    int64_t max_bits;               /* longest bitstream a run accepts, 1 .. 2^31 - 1 */
} pic_huff_desc;

typedef struct pic_huff_info {
    uint32_t struct_size;           /* set by the caller: sizeof(pic_huff_info)      */
    int32_t device;                 /* HIP device ordinal of the handle              */
    int64_t max_bits;
    int64_t scratch_bytes;          /* device memory the handle holds                */
    int32_t bits_per_thread;        /* bitstream bits one thread parses              */
    int32_t lut_bits;               /* width of the first-level decode table         */
} pic_huff_info;

/*
 * pic_huff_create -- validate `desc` and build a handle on the current HIP
 * device; allocates its device scratch (hipMalloc).
 * Returns PIC_OK; PIC_E_INVALID for a malformed descriptor or NULL `out`;
 * PIC_E_NODEVICE when no gfx950 device is current; PIC_E_NOMEM when the handle
 * cannot be allocated; PIC_E_HIP when the device scratch cannot.
 */
PIC_API pic_status pic_huff_create(const pic_huff_desc *desc, pic_huff **out);

/*
 * pic_huff_decode -- enqueue the decoding of n_symbols symbols on `stream`.
 *   data      : device, the bitstream: ceil(n_bits / 8) bytes, MSB first
 *               (may be NULL when n_bits == 0).
 *   n_bits    : 0 .. max_bits; bits past it are not read.
 *   values    : device, int32 [n_table], the symbol of each table entry.
 *   lengths   : device, uint8 [n_table], the code length of each entry.
 *   n_table   : 1 .. PIC_HUFF_MAX_TABLE.
 *   n_symbols : symbols to decode, 0 .. 2^31 - 1 (0 enqueues nothing and
 *               leaves *status alone).
 *   out       : device, int32 [n_symbols]; entries past the decodable
 *               symbols of a malformed stream are left as they were.
 *   status    : device int32, receives the PIC_HUFF_ERR_* bits of this run (no
 *               need to clear it first; readable after the stream reaches it).
 *   stream    : hipStream_t (NULL: the null stream).
 * `values`, `out` and `status` must be 4-byte aligned; buffers must not
 * overlap.  Asynchronous: no allocation, no synchronisation.  A stream of up
 * to 64 * 255 * 64 bits (about 1 Mbit: one Kodak-size image) is decoded in
 * one launch of at most 64 workgroups that hand the repair step to the last
 * of them; the others wait for it at most about 0.2 s (PIC_HUFF_ERR_SYNC:
 * only when other work keeps some of the 64 from starting that long).  A
 * longer stream takes three launches.  Calls on one handle share its
 * scratch and must not overlap.  Returns PIC_E_INVALID for a bad argument
 * (nothing enqueued), PIC_E_HIP for a failed launch.
 */
PIC_API pic_status pic_huff_decode(pic_huff *h, const uint8_t *data, int64_t n_bits, const int32_t *values,
                                   const uint8_t *lengths, int32_t n_table, int64_t n_symbols, int32_t *out,
                                   int32_t *status, void *stream);

/* pic_huff_query -- describe the handle.  PIC_E_INVALID for NULL arguments
 * or an unknown info->struct_size. */
PIC_API pic_status pic_huff_query(const pic_huff *h, pic_huff_info *info);

/* pic_huff_destroy -- free the handle and its device scratch (NULL is
 * accepted).  Synchronises the handle's device first. */
PIC_API void pic_huff_destroy(pic_huff *h);

#ifdef __cplusplus
}
#endif

#endif /* PIC_HUFF_H */
