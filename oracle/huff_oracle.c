/*
 * PIC entropy decoding (Huffman) -- CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  The plain, slow statement of the decoder step
 * that turns the Huffman-coded bitstream back into the ZpR symbol stream.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load it; the product library never links, loads or calls it, and it
 * shares no source with the HIP kernels.
 *
 * What is computed (PIC, Fig. 1 "HD"; Sec. 3.3; Sec. 4.1): the encoder codes
 * the ZpR symbols of an image with an image-specific Huffman code, whose
 * stored table lists only the symbols used; the decoder maps every codeword
 * of the bitstream back to its symbol.
 *
 * Readings where the paper is silent:
 *   - the table is a list of (symbol value, code length) pairs, one per used
 *     symbol; the code is the canonical Huffman code of those lengths as
 *     DEFLATE defines it (RFC 1951, Sec. 3.2.2): codes of one length are
 *     consecutive integers in table order, and the first code of length l is
 *     (first code of length l - 1 + number of codes of length l - 1) << 1,
 *     starting from 0;
 *   - code lengths are 1 .. 24 bits;
 *   - the bitstream is read most significant bit first: bit 7 of byte 0 is
 *     the first bit;
 *   - the number of symbols is given (the container holds it); decoding
 *     stops after that many.
 *
 * Error flags (bitwise or):
 *   1  the bits end before all symbols are decoded (or inside a codeword);
 *   2  a bit pattern that starts no codeword (the code is incomplete);
 *   4  an invalid table: a length outside 1 .. 24, or more codes of some
 *      lengths than the code space holds (Kraft sum above 1).
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared (see build.py).
 */
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define HO_MAX_LEN 24

enum { HO_ERR_BITS = 1, HO_ERR_CODE = 2, HO_ERR_TABLE = 4 };

/* Canonical codes of `n` symbols with the given lengths (RFC 1951, Sec.
 * 3.2.2, steps 1-3).  codes[i] holds symbol i's code in its low lengths[i]
 * bits.  Returns 0, or HO_ERR_TABLE for a length outside 1 .. 24 or an
 * over-subscribed code. */
int pic_oracle_huffman_codes(const uint8_t *lengths, int n, uint32_t *codes)
{
    long count[HO_MAX_LEN + 1];
    memset(count, 0, sizeof count);
    for (int i = 0; i < n; ++i) {
        if (lengths[i] < 1 || lengths[i] > HO_MAX_LEN)
            return HO_ERR_TABLE;
        count[lengths[i]]++;
    }
    /* Kraft: sum 2^-l <= 1, i.e. sum count[l] * 2^(24 - l) <= 2^24 */
    long long kraft = 0;
    for (int l = 1; l <= HO_MAX_LEN; ++l)
        kraft += (long long)count[l] << (HO_MAX_LEN - l);
    if (kraft > (1LL << HO_MAX_LEN))
        return HO_ERR_TABLE;
    uint32_t next[HO_MAX_LEN + 1];
    uint32_t code = 0;
    next[0] = 0;
    for (int l = 1; l <= HO_MAX_LEN; ++l) {
        code = (code + (uint32_t)count[l - 1]) << 1;
        next[l] = code;
    }
    /* count[0] is 0, so the first code of the shortest length is 0 */
    for (int i = 0; i < n; ++i)
        codes[i] = next[lengths[i]]++;
    return 0;
}

/* Decode n_out symbols.  Bit k of the stream is bit 7 - (k % 8) of byte
 * k / 8; only the first n_bits bits exist.  A codeword is recognised by
 * reading bits one at a time and comparing the bits read so far with every
 * table entry of that length; bits that begin no codeword stop the decoding
 * with HO_ERR_CODE.  *n_decoded receives the number of symbols
 * written (n_out unless an error stopped the decoding; out[] beyond it is
 * untouched) and *bits_used the bits they took.  Returns the error flags. */
int pic_oracle_huffman_decode(const uint8_t *bits, long n_bits, const int32_t *values, const uint8_t *lengths,
                              int n_sym, long n_out, int32_t *out, long *n_decoded, long *bits_used)
{
    *n_decoded = 0;
    *bits_used = 0;
    if (n_sym < 1 || n_sym > 65536)
        return HO_ERR_TABLE;
    uint32_t *codes = malloc(sizeof(uint32_t) * (size_t)n_sym);
    if (!codes)
        return HO_ERR_TABLE;
    int err = pic_oracle_huffman_codes(lengths, n_sym, codes);
    if (err) {
        free(codes);
        return err;
    }
    long pos = 0;
    for (long s = 0; s < n_out; ++s) {
        uint32_t acc = 0;
        int len = 0, found = -1;
        while (found < 0) {
            if (pos >= n_bits) {
                free(codes);
                return HO_ERR_BITS;
            }
            acc = (acc << 1) | (uint32_t)((bits[pos >> 3] >> (7 - (pos & 7))) & 1u);
            ++pos;
            ++len;
            int longer = 0;     /* codewords that begin with the bits read so far */
            for (int i = 0; i < n_sym; ++i) {
                if (lengths[i] == len && codes[i] == acc) {
                    found = i;
                    break;
                }
                if (lengths[i] > len && (codes[i] >> (lengths[i] - len)) == acc)
                    longer = 1;
            }
            if (found < 0 && !longer) {
                free(codes);
                return HO_ERR_CODE;
            }
        }
        out[s] = values[found];
        *n_decoded = s + 1;
        *bits_used = pos;
    }
    free(codes);
    return 0;
}
