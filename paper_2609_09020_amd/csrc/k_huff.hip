// Huffman entropy decoding (PIC, Fig. 1 "HD"; Sec. 3.3: an image-specific
// canonical code, decoded with a table indexed by the next bits; Sec. 4.1:
// parallel decoding after GPUHD, which relies on Huffman codes
// resynchronising by themselves).
//
// The bitstream is cut into subsequences of 64 bits, one thread each.  A
// thread cannot know where the first codeword of its subsequence starts, so
// it parses from the subsequence's first bit anyway; a parse that starts
// inside a codeword soon falls onto a true codeword boundary, and from there
// on it equals the true parse.  Three steps, as three kernels for a long
// stream, and for a short one (one image) as one kernel, k_huff_one, whose
// workgroups hand the repair step to the last of them:
//
//   k_huff_parse  parses every subsequence from its first bit, then walks from
//                 where the previous subsequence's parse crossed into it until
//                 the walk meets its own parse: from there on the two agree,
//                 so the walk's codeword starts replace the parse's before
//                 that point.  A walk that meets nothing gives a new crossing
//                 point, and the next subsequence walks again, until none
//                 moves.  A workgroup owns 255 subsequences; its first thread
//                 re-parses the previous workgroup's last one, so all of this
//                 stays inside the workgroup.
//   k_huff_fix    (one workgroup, usually nothing to repair) writes the status
//                 and repeats the walk, in stream order and from the true
//                 crossing point, for what a workgroup could not settle: a
//                 first subsequence whose predecessor's crossing point moved,
//                 a pattern that is no codeword, a codeword past the stream's
//                 end.  It carries a changed crossing point on to the next
//                 subsequence, finds the first pattern that is no codeword and
//                 adjusts the counts.
//   k_huff_write  places each subsequence's symbols by a prefix of the counts
//                 and decodes the codewords its record marks, writing the
//                 values through LDS.
//
// Each workgroup builds the canonical decode tables in LDS from the (value,
// length) list: a 2^11-entry first-level table for codes of up to 11 bits
// (with the length of a second codeword when two fit, so that a parse often
// takes two codewords a step), and for longer codes the left-aligned limits
// of each length (the codes of one length fill one interval of the code
// space, shorter lengths first).
#include "huff_barrier.h"
#include "pic_huff.h"
#include "pic_internal.h"

namespace pic {
namespace {

constexpr int kWaves = kHuffThreads / 64;
constexpr int kLut = 1 << kHuffLutBits;
constexpr int kSubWords = kHuffSub / 32;
constexpr int kStageWords = kHuffThreads * kSubWords + 2;    // the workgroup's words and the codeword
                                                             // crossing the end
constexpr int kLong = kHuffMaxLen - kHuffLutBits;            // lengths beyond the first-level table
constexpr int kHuffFixList = 2048;                           // workgroups to repair listed in LDS
constexpr int kWriteLds = 6144;                              // ints: the table's values in code order,
                                                             // then the workgroup's symbols if they fit

// Big-endian 32-bit word w of the bitstream (bytes outside it read as 0).
__device__ __forceinline__ uint32_t stream_word(const uint8_t *data, int32_t n_bytes, int64_t w)
{
    // branch-free (a byte outside the stream reads byte 0 and is dropped), so
    // that the loads of all the words a thread stages are in flight together
    uint32_t v = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int64_t i = w * 4 + k;
        const bool in = i >= 0 && i < n_bytes;
        const uint32_t byte = data[in ? i : 0];
        v = (v << 8) | (in ? byte : 0u);
    }
    return v;
}

// Decode tables of one workgroup (LDS).
struct SharedTables {
    uint32_t lut[kLut];                  // index | length << 16 | length of a second codeword within
                                         // the slot's bits << 24; 0: a longer code, or none
    uint32_t lim[kHuffMaxLen + 1];       // end of the codes of length <= l, as 24-bit left-aligned values
    int32_t fc[kHuffMaxLen + 1];         // first code of length l
    int32_t fi[kHuffMaxLen + 1];         // code-order index of the first code of length l
    int32_t d[kHuffMaxLen + 1];          // fi - fc
    int32_t cnt[kHuffMaxLen + 1];
    int32_t run[kHuffMaxLen + 1];        // entries of each length ranked so far
    int32_t wcnt[kWaves][kHuffMaxLen + 1];
    int32_t valid;
};

// The length of table entry threadIdx.x (-1 past the table); read before
// other loads are waited for.
__device__ __forceinline__ int first_length(const HuffParams &p)
{
    // branch-free (the table has at least one entry), so that nothing waits
    // for the load before its use
    const bool in = (int)threadIdx.x < p.n_table;
    const int l = p.lengths[in ? threadIdx.x : 0];
    return in ? l : -1;
}

// The length counts, first codes, first indexes and limits of the canonical
// code (RFC 1951, Sec. 3.2.2), and whether the table is valid: every length
// in 1 .. kHuffMaxLen and the Kraft sum at most 1.  `len0` is
// first_length(p).  All threads.
__device__ void build_code(const HuffParams &p, SharedTables &s, int len0)
{
    const int t = threadIdx.x;
    if (t <= kHuffMaxLen) {
        s.cnt[t] = 0;
        s.run[t] = 0;
    }
    if (t == 0)
        s.valid = 1;
    __syncthreads();
    // entry t from len0 outside the loop, so that only that load is waited
    // for here, not the ones issued after it
    if (t < p.n_table) {
        if (len0 < 1 || len0 > kHuffMaxLen)
            s.valid = 0;
        else
            atomicAdd(&s.cnt[len0], 1);
    }
    for (int i = t + kHuffThreads; i < p.n_table; i += kHuffThreads) {
        const int l = p.lengths[i];
        if (l < 1 || l > kHuffMaxLen)
            s.valid = 0;
        else
            atomicAdd(&s.cnt[l], 1);
    }
    __syncthreads();
    if (t < 32) {
        // lane l holds length l; prefix sums across the lanes give the first
        // index of each length and the limits (the Kraft sums: the codes of
        // length l fill [lim[l - 1], lim[l]) of the 24-bit code space, so the
        // first code of length l is lim[l - 1] >> (24 - l))
        const int c = t >= 1 && t <= kHuffMaxLen ? s.cnt[t] : 0;
        // more than 2^l codes of length l over-subscribe the code by
        // themselves; clamped so the sums stay in 32 bits
        const uint32_t w = t >= 1 && t <= kHuffMaxLen
                               ? (uint32_t)min(c, (1 << t) + 1) << (kHuffMaxLen - t) : 0u;
        // inclusive sums over lanes 0..31 by data-parallel moves: shifts by
        // 1, 2, 4, 8 within each row of 16 lanes (a lane with no source adds
        // 0), then row 0's total into row 1
        auto prefix = [](uint32_t x) {
            x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);   // row_shr:1
            x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);   // row_shr:2
            x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);   // row_shr:4
            x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);   // row_shr:8
            x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);   // row_bcast:15
            return x;
        };
        int32_t fi = (int32_t)prefix((uint32_t)c);
        const uint32_t lim = prefix(w);
        fi -= c;                           // exclusive
        // lim of the lane before (wave_shr:1; lane 0 reads 0 and is not used)
        const uint32_t below = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)lim, 0x138, 0xF, 0xF, false);
        const int32_t fc = t >= 1 ? (int32_t)(below >> (kHuffMaxLen - t)) : 0;
        if (t <= kHuffMaxLen) {
            s.fi[t] = fi;
            s.fc[t] = fc;
            s.d[t] = fi - fc;
            s.lim[t] = lim;
        }
        if (t == kHuffMaxLen && lim > (1u << kHuffMaxLen))
            s.valid = 0;
    }
    __syncthreads();
}

// The first-level table: slot k holds the code of up to kHuffLutBits bits
// that the bits k begin with, and the length of the codeword after it when
// that one ends within the kHuffLutBits bits too.  Needs build_code; all
// threads.
__device__ void build_lut(SharedTables &s)
{
    constexpr int kPer = kLut / kHuffThreads;
    uint32_t lim[kHuffLutBits + 1];
#pragma unroll
    for (int l = 1; l <= kHuffLutBits; ++l)
        lim[l] = s.lim[l];
    uint32_t ent[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int k = threadIdx.x + j * kHuffThreads;
        const uint32_t v = (uint32_t)k << (kHuffMaxLen - kHuffLutBits);
        // The limits grow with the length, so the first codeword's length is
        // one more than the number of limits at or below v (12: longer than
        // the table's bits); its index is its code plus d[length].
        int c = 0;
#pragma unroll
        for (int l = 1; l <= kHuffLutBits; ++l)
            c += v >= lim[l] ? 1 : 0;
        const int len = c < kHuffLutBits ? c + 1 : kHuffLutBits;
        const uint32_t idx = (uint32_t)(s.d[len] + (k >> (kHuffLutBits - len)));
        const uint32_t e = c < kHuffLutBits ? idx | (uint32_t)len << 16 : 0u;
        ent[j] = e;
        s.lut[k] = e;
    }
    __syncthreads();
    // the bits after the first codeword, padded with zeros, begin the second
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int k = threadIdx.x + j * kHuffThreads;
        const int len1 = (int)(ent[j] >> 16);
        if (len1 > 0 && len1 < kHuffLutBits) {
            const int len2 = (int)(s.lut[(k << len1) & (kLut - 1)] >> 16);
            if (len2 > 0 && len1 + len2 <= kHuffLutBits)
                ent[j] |= (uint32_t)len2 << 24;
        }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kPer; ++j)
        s.lut[threadIdx.x + j * kHuffThreads] = ent[j];
    __syncthreads();
}

// The table's values in code order (by length, then table order).  Needs
// build_code; all threads.  `len0` and `val0` are entry threadIdx.x's length
// (first_length) and value, loaded before anything was waited for.
__device__ void build_sorted(const HuffParams &p, SharedTables &s, int32_t *sorted, int len0, int32_t val0)
{
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    // one pass per kHuffThreads entries: entry i has length l (0: none) and
    // value v; its rank among the entries of its length continues s.run
    auto pass = [&](int l, int32_t v) {
        int in_wave = 0;
        for (int k = 1; k <= kHuffMaxLen; ++k) {
            const uint64_t m = __ballot(l == k);
            if (l == k)
                in_wave = __popcll(m & ((1ull << lane) - 1));
            if (lane == 0)
                s.wcnt[wave][k] = __popcll(m);
        }
        __syncthreads();
        if (l > 0) {
            int rank = s.run[l] + in_wave;
            for (int w = 0; w < wave; ++w)
                rank += s.wcnt[w][l];
            sorted[s.fi[l] + rank] = v;
        }
        __syncthreads();
        if (t >= 1 && t <= kHuffMaxLen)
            for (int w = 0; w < kWaves; ++w)
                s.run[t] += s.wcnt[w][t];
        __syncthreads();
    };
    // the first entries from len0 / val0, outside the loop, so that only
    // those loads are waited for here
    pass(t < p.n_table ? len0 : 0, val0);
    for (int base = kHuffThreads; base < p.n_table; base += kHuffThreads) {
        const int i = base + t;
        const bool in = i < p.n_table;
        pass(in ? (int)p.lengths[i] : 0, in ? p.values[i] : 0);
    }
}

// Per-thread view of the tables: the limits of the long lengths in registers.
struct Decoder {
    const uint32_t *lut;
    const int32_t *d;
    uint32_t lim[kLong];                 // lim[j]: limit of length kHuffLutBits + 1 + j; lim[kLong - 1]
                                         // (length kHuffMaxLen) is the end of the whole code
};

__device__ __forceinline__ Decoder decoder_of(const SharedTables &s)
{
    Decoder dc;
    dc.lut = s.lut;
    dc.d = s.d;
#pragma unroll
    for (int j = 0; j < kLong; ++j)
        dc.lim[j] = s.lim[kHuffLutBits + 1 + j];
    return dc;
}

// Length of a codeword longer than the first-level table at the top of
// `win` (0: no codeword starts there).
__device__ __forceinline__ int decode_long(uint32_t win, const Decoder &dc)
{
    const uint32_t v = win >> (32 - kHuffMaxLen);
    if (v >= dc.lim[kLong - 1])
        return 0;                        // past the last code: no codeword has these bits
    // the length whose interval holds v: one past the lengths whose limit is <= v
    int len = kHuffLutBits + 1;
#pragma unroll
    for (int j = 0; j < kLong - 1; ++j)
        len += v >= dc.lim[j] ? 1 : 0;
    return len;
}

// Length of the codeword at the top of `win` (0: no codeword starts there)
// and its index in code order.
__device__ __forceinline__ int decode_one(uint32_t win, const Decoder &dc, int *idx)
{
    const uint32_t e = dc.lut[win >> (32 - kHuffLutBits)];
    if (e) {
        *idx = (int)(e & 0xfffu);
        return (int)((e >> 16) & 0xffu);
    }
    const int len = decode_long(win, dc);
    *idx = len ? (int)(win >> (32 - len)) + dc.d[len] : 0;
    return len;
}

// The bitstream words [w0, w0 + kStageWords) a workgroup stages in LDS, in
// two steps: load_words issues the loads into registers (nothing waits for
// them, so the tables can be built meanwhile), store_words writes them.
constexpr int kStagePer = (kStageWords + kHuffThreads - 1) / kHuffThreads;
struct StagedWords {
    uint32_t v[kStagePer];
};

__device__ __forceinline__ StagedWords load_words(const HuffParams &p, int64_t w0)
{
    const int32_t n_bytes = (int32_t)(((int64_t)p.n_bits + 7) >> 3);
    StagedWords sw;
#pragma unroll
    for (int j = 0; j < kStagePer; ++j) {
        const int i = threadIdx.x + j * kHuffThreads;
        sw.v[j] = stream_word(p.data, n_bytes, w0 + i);   // (i >= kStageWords: not stored)
    }
    return sw;
}

__device__ __forceinline__ void store_words(uint32_t *words, const StagedWords &sw)
{
#pragma unroll
    for (int j = 0; j < kStagePer; ++j) {
        const int i = threadIdx.x + j * kHuffThreads;
        if (i < kStageWords)
            words[i] = sw.v[j];
    }
}

// The bits of one subsequence (two words) and the word after it.
struct SubBits {
    uint32_t w0, w1, w2;
    // the 32 bits from bit offset `off` of the subsequence (0 <= off < 64)
    __device__ __forceinline__ uint32_t window(int off) const
    {
        const uint64_t two = off < 32 ? (uint64_t)w0 << 32 | w1 : (uint64_t)w1 << 32 | w2;
        return (uint32_t)(two << (off & 31) >> 32);
    }
};

static_assert(kSubWords == 2, "a subsequence is two words");

// From the workgroup's staged words, starting at word `first`.
__device__ __forceinline__ SubBits lds_sub(const uint32_t *words, int first)
{
    return SubBits{words[first], words[first + 1], words[first + 2]};
}

// Subsequence `t` straight from the bitstream.
__device__ __forceinline__ SubBits global_sub(const HuffParams &p, int t)
{
    const int32_t n_bytes = (int32_t)(((int64_t)p.n_bits + 7) >> 3);
    const int64_t w = (int64_t)t * kSubWords;
    return SubBits{stream_word(p.data, n_bytes, w), stream_word(p.data, n_bytes, w + 1),
                   stream_word(p.data, n_bytes, w + 2)};
}

// A record of codeword starts: bit k for bit offset k of a subsequence.
__device__ __forceinline__ bool mask_has(uint64_t m, int off) { return (m >> (off & 63)) & 1u; }

// The bits of `m` at offsets >= off (0 <= off <= 64).
__device__ __forceinline__ uint64_t mask_from(uint64_t m, int off)
{
    return off >= 64 ? 0ull : m & (~0ull << off);
}

// How a walk ends.
enum { kReached = 0, kMet = 1, kInvalid = 2, kPastEnd = 3 };

// Parse from bit *pos of the subsequence that starts at bit `start` and ends
// before `lim`, setting each codeword start in `m`; with MEET, stop at the
// first position that `old` holds already.  *pos receives where the walk
// stopped.
template <bool MEET>
__device__ __forceinline__ int walk(const SubBits &bits, const Decoder &dc, int32_t start, int32_t lim,
                                    int32_t n_bits, uint64_t old, uint64_t &m, int32_t *pos_io)
{
    int32_t pos = *pos_io;
    int state = kReached;
    while (pos < lim) {
        const int off = pos - start;
        if (MEET && mask_has(old, off)) {
            state = kMet;
            break;
        }
        const uint32_t win = bits.window(off);
        const uint32_t e = dc.lut[win >> (32 - kHuffLutBits)];
        int len = (int)((e >> 16) & 0xffu);
        if (len == 0)
            len = decode_long(win, dc);
        if (len == 0) {
            state = kInvalid;
            break;
        }
        if (len > n_bits - pos) {
            state = kPastEnd;
            break;
        }
        // the table's second codeword too, when it starts inside the
        // subsequence, ends inside the stream and (walking to meet `old`)
        // starts before the meeting point
        const int len2 = (int)(e >> 24);
        const int off2 = off + len;
        const bool two = len2 > 0 && pos + len < lim && len2 <= n_bits - pos - len &&
                         !(MEET && mask_has(old, off2));
        m |= 1ull << off | (two ? 1ull << (off2 & 63) : 0ull);
        pos += two ? len + len2 : len;
    }
    *pos_io = pos;
    return state;
}

// Where a parse that stopped in `state` at `pos` crosses into the next
// subsequence: pos itself; -1 after a pattern that is no codeword; n_bits when
// a codeword would run past the stream.
__device__ __forceinline__ int32_t crossing(int state, int32_t pos, int32_t n_bits)
{
    return state == kInvalid ? -1 : state == kPastEnd ? n_bits : pos;
}

__device__ __forceinline__ int32_t block_sum_incl(int32_t v, int32_t *s_wsum, int32_t *total)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int32_t incl = wave_inclusive_sum(v);
    if (lane == 63)
        s_wsum[wave] = incl;
    __syncthreads();
    int32_t off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        off += w < wave ? s_wsum[w] : 0;
        tot += s_wsum[w];
    }
    __syncthreads();
    *total = tot;
    return off + incl;
}

// The parse of a workgroup's subsequences, the in-step check and repair, and
// its records.  All threads; the tables and the staged words are ready in LDS.
// The workgroup's summary word (what the repair step has to look at: 0 when
// nothing) also goes to *s_summary, visible to the workgroup after its next
// barrier.
__device__ __forceinline__ void parse_phase(const HuffParams &p, const SharedTables &s_tab,
                                            const uint32_t *s_words, int32_t *s_end, int32_t *s_moved,
                                            int32_t *s_wsum, int blk, int32_t *s_summary)
{
    const int l = threadIdx.x;
    const int32_t t0 = blk * kHuffOwn;           // first owned subsequence
    const Decoder dc = decoder_of(s_tab);
    const int32_t t = t0 + l - 1;
    const bool live = t >= 0 && t < p.nsub;
    const int32_t start = t * kHuffSub;
    const int32_t lim = start + kHuffSub < p.n_bits ? start + kHuffSub : p.n_bits;
    const SubBits bits = lds_sub(s_words, l * kSubWords);
    uint64_t m = 0;
    int32_t end = 0;
    if (live) {
        int32_t pos = start;
        const int st = walk<false>(bits, dc, start, lim, p.n_bits, 0ull, m, &pos);
        end = crossing(st, pos, p.n_bits);
    }
    const int32_t nominal_end = end;
    s_end[l] = end;
    __syncthreads();
    // Walk from the previous subsequence's crossing point to the first
    // codeword start the walk shares with this subsequence's parse; from there
    // on the two agree, so the walk's starts replace the parse's before it.
    // A walk that meets nothing ends at a new crossing point, and the next
    // subsequence walks again, until no crossing point moves.  Subsequences
    // whose walk meets a pattern that is no codeword, runs past the stream or
    // follows such a one are left to the fix kernel, which decides in stream
    // order.
    bool bad = false, redo = live && l > 0;
    int32_t n = 0;
    while (true) {
        bool moved = false;
        if (redo) {
            const int32_t b = t == 0 ? 0 : s_end[l - 1];
            if (b < 0) {
                bad = true;
            } else if (b >= p.n_bits) {
                n = 0;                     // the stream ended before this subsequence
            } else {
                uint64_t w = 0;
                int32_t pos = b;
                const int st = walk<true>(bits, dc, start, lim, p.n_bits, m, w, &pos);
                if (st == kMet) {
                    m = w | mask_from(m, pos - start);
                    bad = end < 0;
                } else if (st == kReached) {
                    m = w;
                    moved = pos != end;
                    end = pos;
                } else {
                    bad = true;
                }
                n = __popcll(m);
            }
        }
        __syncthreads();                   // every read of s_end is done
        s_end[l] = end;
        s_moved[l] = moved;
        if (!__syncthreads_or(moved))
            break;   // uniform
        redo = live && l > 0 && !bad && s_moved[l - 1];
    }
    // the workgroup's sums first: their barriers then wait for no stores
    int32_t total;
    (void)block_sum_incl(n, s_wsum, &total);
    const bool any_bad = __syncthreads_or(bad);
    if (live && l > 0) {
        p.mask[t] = m;
        p.end[t] = end;
        p.cnt[t] = n;
    }
    const uint64_t fail = __ballot(bad);
    const int lane = l & 63, wave = l >> 6;
    if (lane == 0) {
        p.fail[blk * 8 + wave * 2] = (uint32_t)fail;
        p.fail[blk * 8 + wave * 2 + 1] = (uint32_t)(fail >> 32);
    }
    if (l == 0)
        p.blk[blk] = total;
    // bit 0: the next workgroup took this one's last nominal crossing point,
    // and it moved; bit 1: a subsequence here was left to the fix kernel
    if (l == kHuffThreads - 1) {
        const int32_t summary = (live && end != nominal_end ? 1 : 0) | (any_bad ? 2 : 0);
        p.bnd[blk] = summary;
        *s_summary = summary;
    }
}

__global__ __launch_bounds__(kHuffThreads) void k_huff_parse(HuffParams p)
{
    warm_kernel_args<sizeof(HuffParams)>();
    __shared__ SharedTables s_tab;
    __shared__ uint32_t s_words[kStageWords];
    __shared__ int32_t s_end[kHuffThreads];
    __shared__ int32_t s_moved[kHuffThreads];
    __shared__ int32_t s_wsum[kWaves];
    const int l = threadIdx.x;
    const int32_t t0 = (int32_t)blockIdx.x * kHuffOwn;           // first owned subsequence
    const int64_t w0 = ((int64_t)t0 - 1) * kSubWords;            // staged from the one before
    // every global load goes out first; the tables are built while the
    // bitstream words are on their way
    const int len0 = first_length(p);
    const StagedWords sw = load_words(p, w0);
    build_code(p, s_tab, len0);
    if (blockIdx.x == 0 && l == 0) {       // the call's status starts here
        *p.status = s_tab.valid ? 0 : PIC_HUFF_ERR_TABLE;
        p.flags[1] = 0x7fffffff;           // first subsequence whose true parse meets no codeword
    }
    if (!s_tab.valid)
        return;   // uniform
    build_lut(s_tab);
    store_words(s_words, sw);
    __syncthreads();
    __shared__ int32_t s_summary;
    parse_phase(p, s_tab, s_words, s_end, s_moved, s_wsum, (int)blockIdx.x, &s_summary);
}

// Walk subsequence u again from the true crossing point of its predecessor
// until it meets its recorded parse, and update its record and count.
// Returns true when u's crossing point changed (u + 1 must be walked again);
// *corrupt is set when the true parse meets a pattern that is no codeword.
__device__ bool refix(const HuffParams &p, const Decoder &dc, int u, bool *corrupt)
{
    *corrupt = false;
    // every load first, in one round trip
    const int32_t b = u == 0 ? 0 : p.end[u - 1];
    const SubBits bits = global_sub(p, u);
    uint64_t m = p.mask[u];
    const int32_t end = p.end[u];
    const int32_t old = p.cnt[u];
    if (b < 0)
        return false;                      // cannot happen: the fix stops at the first such pattern
    const int32_t start = u * kHuffSub;
    const int32_t lim = start + kHuffSub < p.n_bits ? start + kHuffSub : p.n_bits;
    bool carry = false;
    int32_t n = 0;
    if (b < p.n_bits) {
        uint64_t w = 0;
        int32_t pos = b;
        const int st = walk<true>(bits, dc, start, lim, p.n_bits, m, w, &pos);
        if (st == kMet) {
            m = w | mask_from(m, pos - start);
            *corrupt = end < 0;
        } else {
            m = w;
            const int32_t e = crossing(st, pos, p.n_bits);
            carry = e != end;
            *corrupt = st == kInvalid;
            p.end[u] = e;
        }
        p.mask[u] = m;
        n = __popcll(m);
    }
    if (n != old) {
        p.cnt[u] = n;
        p.blk[u / kHuffOwn] += n - old;
    }
    return carry;
}

// Workgroups to repair, in stream order, repaired by one thread (see
// k_huff_fix), and the per-workgroup counts turned into prefixes when
// blk_is_prefix.  All threads of one workgroup; `s_list` holds kHuffFixList
// ints.  With `tables_ready` the tables are already in `s_tab` (valid).
__device__ __forceinline__ void fix_phase(const HuffParams &p, SharedTables &s_tab, bool tables_ready,
                                          int32_t *s_list, int32_t *s_wsum)
{
    // Workgroups to repair: those that left subsequences to this kernel, and
    // those whose first subsequence (thread 1) started from a crossing point
    // that moved in the previous workgroup.  Each thread takes a segment of
    // workgroups (eight loads in flight at a time) and the workgroup lists
    // them in stream order; one thread then repairs them.
    const int nblk = p.nblk;
    auto needs_fix = [&](int g) { return (p.bnd[g] & 2) || (g > 0 && (p.bnd[g - 1] & 1)); };
    const int seg = (nblk + kHuffThreads - 1) / kHuffThreads;
    const int seg_lo = threadIdx.x * seg, seg_hi = seg_lo + seg < nblk ? seg_lo + seg : nblk;
    const int len0 = first_length(p);
    const int32_t status0 = *p.status;     // the parse kernel's: whether the table is valid
    int32_t count = 0;
    uint32_t mine = 0;                     // the segment's workgroups to repair, while seg <= 32
    for (int g = seg_lo; g < seg_hi; g += 8) {
        int32_t f[8], b[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            f[j] = g + j < seg_hi ? p.bnd[g + j] & 2 : 0;
            b[j] = g + j < seg_hi && g + j > 0 ? p.bnd[g + j - 1] & 1 : 0;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (f[j] | b[j]) {
                ++count;
                if (g + j - seg_lo < 32)
                    mine |= 1u << (g + j - seg_lo);
            }
    }
    if (status0 & PIC_HUFF_ERR_TABLE)
        return;   // uniform: nothing was parsed
    int32_t total;
    const int32_t at = block_sum_incl(count, s_wsum, &total) - count;
    if (total > 0) {   // uniform; the tables are needed only to repair
        if (!tables_ready)
            build_code(p, s_tab, len0);
        const bool listed = total <= kHuffFixList && seg <= 32;
        if (listed)
            for (uint32_t b = mine; b; b &= b - 1u)
                s_list[at + __popc(mine & ((1u << __builtin_ctz(b)) - 1u))] = seg_lo + __builtin_ctz(b);
        if (!tables_ready)
            build_lut(s_tab);              // its barriers also publish the list
        else
            __syncthreads();               // publishes the list
        const Decoder dc = decoder_of(s_tab);
        if (threadIdx.x == 0) {
            // one workgroup's records, then the chain from each
            auto repair = [&](int g) -> bool {
                const uint4 lo = reinterpret_cast<const uint4 *>(p.fail)[g * 2];
                const uint4 hi = reinterpret_cast<const uint4 *>(p.fail)[g * 2 + 1];
                const uint32_t words[8] = {lo.x | (g > 0 && (p.bnd[g - 1] & 1) ? 2u : 0u), lo.y, lo.z, lo.w,
                                           hi.x, hi.y, hi.z, hi.w};
#pragma unroll 1
                for (int w = 0; w < 8; ++w)
                    for (uint32_t bm = words[w]; bm; bm &= bm - 1u) {
                        const int l = w * 32 + __builtin_ctz(bm);
                        // repair, then carry a changed crossing point onwards
                        for (int u = g * kHuffOwn + l - 1; u < p.nsub; ++u) {
                            bool corrupt;
                            const bool carry = refix(p, dc, u, &corrupt);
                            if (corrupt) {
                                atomicOr(p.status, PIC_HUFF_ERR_CODE);
                                p.flags[1] = u;
                                return true;
                            }
                            if (!carry)
                                break;
                        }
                    }
                return false;
            };
            if (listed) {
                for (int k = 0; k < total; ++k)
                    if (repair(s_list[k]))
                        break;
            } else {
                for (int g = 0; g < nblk; ++g)
                    if (needs_fix(g) && repair(g))
                        break;
            }
        }
    }
    if (p.blk_is_prefix) {
        // exclusive prefixes of the per-workgroup counts, a segment per thread
        __syncthreads();
        const int seg = (p.nblk + kHuffThreads - 1) / kHuffThreads;
        const int lo = threadIdx.x * seg, hi = lo + seg < p.nblk ? lo + seg : p.nblk;
        int32_t sum = 0;
        for (int g = lo; g < hi; ++g)
            sum += p.blk[g];
        int32_t total;
        int32_t run = block_sum_incl(sum, s_wsum, &total) - sum;
        for (int g = lo; g < hi; ++g) {
            const int32_t v = p.blk[g];
            p.blk[g] = run;
            run += v;
        }
    }
}

__global__ __launch_bounds__(kHuffThreads) void k_huff_fix(HuffParams p)
{
    warm_kernel_args<sizeof(HuffParams)>();
    __shared__ SharedTables s_tab;
    __shared__ int32_t s_list[kHuffFixList];
    __shared__ int32_t s_wsum[kWaves];
    fix_phase(p, s_tab, false, s_list, s_wsum);
}

// The records a workgroup's write needs (issued together, nothing waits).
struct WriteRecs {
    int32_t last_good, cnt_t, blk_before;
    uint64_t mask_t;
    int32_t pre[8];
};

__device__ __forceinline__ WriteRecs load_write_recs(const HuffParams &p, int blk)
{
    const int l = threadIdx.x;
    const int32_t t0 = blk * kHuffOwn;
    const int32_t t = t0 + l - 1;
    const bool rec = l > 0 && t < p.nsub;        // a subsequence this thread owns
    WriteRecs r;
    r.last_good = p.flags[1];
    r.cnt_t = p.cnt[rec ? t : 0];                // (unused unless rec)
    r.mask_t = p.mask[rec ? t : 0];
    r.blk_before = p.blk_is_prefix ? p.blk[blk] : 0;
    // the counts of up to 8 x kHuffThreads workgroups before this one, for
    // the symbols before it (branch-free: an index past them reads entry 0
    // and is dropped)
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int j = l + u * kHuffThreads;
        const bool in = !p.blk_is_prefix && j < blk;
        const int32_t v = p.blk[in ? j : 0];
        r.pre[u] = in ? v : 0;
    }
    return r;
}

// Decode and write a workgroup's symbols.  All threads; the tables, the
// values in code order (s_vals) and the staged words are ready in LDS.
__device__ __forceinline__ void write_phase(const HuffParams &p, const SharedTables &s_tab,
                                            const uint32_t *s_words, int32_t *s_vals, int32_t *s_wsum,
                                            int blk, const WriteRecs &r)
{
    const int l = threadIdx.x;
    const int32_t t0 = blk * kHuffOwn;
    const int32_t t = t0 + l - 1;
    const bool rec = l > 0 && t < p.nsub;
    const int32_t last_good = r.last_good, cnt_t = r.cnt_t, blk_before = r.blk_before;
    const uint64_t mask_t = r.mask_t;
    const int32_t *pre = r.pre;
    const Decoder dc = decoder_of(s_tab);
    // symbols before this workgroup's subsequences
    int32_t before;
    if (p.blk_is_prefix) {
        before = blk_before;
    } else {
        int32_t a[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            a[u] = pre[u];
        for (int j = l + 8 * kHuffThreads; j < blk; j += 8 * kHuffThreads) {
#pragma unroll
            for (int u = 0; u < 8; ++u)
                a[u] += j + u * kHuffThreads < blk ? p.blk[j + u * kHuffThreads] : 0;
        }
        (void)block_sum_incl(((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7])), s_wsum,
                             &before);
    }
    // subsequences after the first one whose true parse meets a pattern
    // that is no codeword hold nothing decodable
    const int32_t n = rec && t <= last_good ? cnt_t : 0;
    int32_t blk_total;
    const int32_t o = before + block_sum_incl(n, s_wsum, &blk_total) - n;
    // too few codewords: the bits ran out (unless a pattern that is no
    // codeword ended the decoding first, already reported)
    if (blk == p.nblk - 1 && l == 0 && (int64_t)before + blk_total < p.n_symbols &&
        !(*p.status & PIC_HUFF_ERR_CODE))
        atomicOr(p.status, PIC_HUFF_ERR_BITS);
    // the workgroup's symbols go through LDS when they fit, so that the
    // stores are contiguous (uniform)
    const bool staged = blk_total <= kWriteLds - p.n_table;
    if (n == 0 || o >= p.n_symbols) {
        if (!staged)
            return;
    } else {
    // the record marks every codeword start of the true parse: the codewords
    // are decoded independently, four at a time
    const SubBits bits = lds_sub(s_words, l * kSubWords);
    uint64_t m = mask_t;
    const int32_t k_end = o + n < p.n_symbols ? n : p.n_symbols - o;
    int32_t *out = staged ? s_vals + p.n_table + (o - before) : p.out + o;
    for (int32_t k = 0; k < k_end; k += 4) {
        uint32_t win[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int off = __builtin_ctzll(m | 1ull << 63);   // past the last start: unused
            m &= m - 1;
            win[j] = bits.window(off);
        }
        // the four table reads first, then the rare long codes, then the
        // four value reads
        uint32_t e[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            e[j] = dc.lut[win[j] >> (32 - kHuffLutBits)];
        int idx[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            idx[j] = (int)(e[j] & 0xfffu);
            if (e[j] == 0u) {
                const int len = decode_long(win[j], dc);
                idx[j] = len ? (int)(win[j] >> (32 - len)) + dc.d[len] : 0;
            }
        }
        int32_t v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            v[j] = s_vals[idx[j]];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (k + j < k_end)
                out[k + j] = v[j];
    }
    }
    if (staged) {
        __syncthreads();
        const int32_t count = before >= p.n_symbols ? 0 : min(blk_total, p.n_symbols - before);
        for (int32_t i = l; i < count; i += kHuffThreads)
            p.out[before + i] = s_vals[p.n_table + i];
    }
}

__global__ __launch_bounds__(kHuffThreads) void k_huff_write(HuffParams p)
{
    warm_kernel_args<sizeof(HuffParams)>();
    __shared__ SharedTables s_tab;
    __shared__ uint32_t s_words[kStageWords];
    __shared__ int32_t s_vals[kWriteLds];
    __shared__ int32_t s_wsum[kWaves];
    static_assert(kWriteLds > kHuffMaxTable, "room for the values");
    const int l = threadIdx.x;
    const int32_t t0 = (int32_t)blockIdx.x * kHuffOwn;
    const int64_t w0 = ((int64_t)t0 - 1) * kSubWords;
    // every global load whose address is known goes out first; the tables
    // are built while they are on their way
    const int len0 = first_length(p);
    const int32_t val0 = p.values[l < p.n_table ? l : 0];   // (unused past the table)
    const StagedWords sw = load_words(p, w0);
    const WriteRecs r = load_write_recs(p, (int)blockIdx.x);
    build_code(p, s_tab, len0);
    if (!s_tab.valid)
        return;   // uniform
    build_lut(s_tab);
    build_sorted(p, s_tab, s_vals, len0, val0);
    store_words(s_words, sw);
    __syncthreads();
    write_phase(p, s_tab, s_words, s_vals, s_wsum, (int)blockIdx.x, r);
}

// The three steps in one launch, for streams of at most kHuffOneLaunchMax
// workgroups.  Each workgroup builds the tables and stages its words once,
// parses, and arrives at the hand-off (huff_barrier.h); the last to arrive
// runs the repair step, then releases the others, which wait at most
// p.wait_ticks of the real-time counter (a workgroup that gives up sets PIC_HUFF_ERR_SYNC and
// writes nothing).  At most 64 workgroups of 36 KB of LDS (four fit on one
// CU) are resident together on an otherwise idle device; only another
// kernel that holds the CUs past the wait bound makes a waiter give up, and
// every wait ends either way.  Records cross workgroups, and XCDs, through
// device-scope release and acquire fences around the hand-off.
__global__ __launch_bounds__(kHuffThreads) void k_huff_one(HuffParams p)
{
    warm_kernel_args<sizeof(HuffParams)>();
    __shared__ SharedTables s_tab;
    __shared__ uint32_t s_words[kStageWords];
    // one phase's scratch at a time: the parse's crossing points, the
    // repair's list, the values in code order and the symbols
    __shared__ union {
        struct {
            int32_t end[kHuffThreads];
            int32_t moved[kHuffThreads];
        } parse;
        int32_t list[kHuffFixList];
        int32_t vals[kWriteLds];
    } s_u;
    __shared__ int32_t s_wsum[kWaves];
    __shared__ int32_t s_last, s_ok, s_flagged, s_summary;
    __shared__ uint32_t s_gen;
    const int l = threadIdx.x;
    const int blk = (int)blockIdx.x;
    const int32_t t0 = blk * kHuffOwn;
    const int64_t w0 = ((int64_t)t0 - 1) * kSubWords;
    const int len0 = first_length(p);
    const int32_t val0 = p.values[l < p.n_table ? l : 0];   // (unused past the table)
    const StagedWords sw = load_words(p, w0);
    build_code(p, s_tab, len0);
    if (blk == 0 && l == 0) {              // the call's status starts here
        *p.status = s_tab.valid ? 0 : PIC_HUFF_ERR_TABLE;
        p.flags[1] = 0x7fffffff;           // first subsequence whose true parse meets no codeword
    }
    const bool valid = s_tab.valid;        // uniform
    if (valid) {
        build_lut(s_tab);
        store_words(s_words, sw);
        __syncthreads();
        parse_phase(p, s_tab, s_words, s_u.parse.end, s_u.parse.moved, s_wsum, blk, &s_summary);
    }
    // hand-off: every workgroup arrives, also with an invalid table, so that
    // the word's count comes back to zero.  Each wavefront waits for its
    // record stores to reach the L2, then one write-back of the L2 publishes
    // them all (one per workgroup, not one per wavefront).
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (l < 64)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (l == 0) {
        // flagged: this workgroup left something to the repair step (with an
        // invalid table nothing was parsed and there is nothing to repair)
        const huff_barrier::Arrival a =
            huff_barrier::arrive<huff_barrier::DeviceOps>(p.sync, (uint32_t)p.nblk, valid && s_summary != 0);
        s_last = a.last;
        s_flagged = a.flagged;
        s_gen = a.generation;
    }
    __syncthreads();
    huff_barrier::Arrival a;
    a.generation = s_gen;
    a.last = s_last != 0;
    a.flagged = s_flagged != 0;
    if (a.last) {                          // uniform
        // The repair step only when a workgroup flagged it (a moved crossing
        // point or a subsequence it could not settle); otherwise the last
        // arrival reads and writes nothing the others need, so it releases
        // at once, without the fences.
        if (a.flagged) {                   // uniform
            // one invalidate per workgroup: its wavefronts share one CU
            if (l < 64)
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            __syncthreads();
            fix_phase(p, s_tab, valid, s_u.list, s_wsum);
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
            if (l < 64)
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            __syncthreads();
        }
        if (l == 0)
            huff_barrier::release<huff_barrier::DeviceOps>(p.sync, a);
    } else {
        if (l == 0)
            s_ok = huff_barrier::wait<huff_barrier::DeviceOps>(p.sync, a, p.wait_ticks);
        __syncthreads();
        if (s_ok && l < 64)
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        __syncthreads();
    }
    const bool go = a.last || s_ok;        // uniform: false for a waiter that gave up
    if (go && valid) {
        const WriteRecs r = load_write_recs(p, blk);
        build_sorted(p, s_tab, s_u.vals, len0, val0);
        write_phase(p, s_tab, s_words, s_u.vals, s_wsum, blk, r);
    }
    // leave (huff_barrier.h): the last to leave reports a give-up; the first
    // workgroup's clear of the status came before its arrival, so before this
    __syncthreads();
    if (l == 0) {
        uint32_t all = 0;
        if (huff_barrier::leave<huff_barrier::DeviceOps>(p.sync + 1, (uint32_t)p.nblk,
                                                         go ? 0u : (uint32_t)PIC_HUFF_ERR_SYNC, &all) && all)
            atomicOr(p.status, (int32_t)all);
    }
}

}  // namespace

hipError_t launch_huff(const HuffParams &p, hipStream_t s)
{
    if (p.nsub < 1 || p.nblk != (p.nsub + kHuffOwn - 1) / kHuffOwn)
        return hipErrorInvalidValue;
    const dim3 block(kHuffThreads);
    const dim3 grid((unsigned)p.nblk);
    if (p.nblk <= kHuffOneLaunchMax && p.sync) {
        // an ordinary launch: a cooperative one measured 18 us more per call
        hipLaunchKernelGGL(k_huff_one, grid, block, 0, s, p);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(k_huff_parse, grid, block, 0, s, p);
    hipLaunchKernelGGL(k_huff_fix, dim3(1), block, 0, s, p);
    hipLaunchKernelGGL(k_huff_write, grid, block, 0, s, p);
    return hipGetLastError();
}

}  // namespace pic
