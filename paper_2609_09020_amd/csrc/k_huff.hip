// Huffman entropy decoding (PIC, Fig. 1 "HD"; Sec. 3.3: an image-specific
// canonical code, decoded with a table indexed by the next bits; Sec. 4.1:
// parallel decoding after GPUHD, which relies on Huffman codes
// resynchronising by themselves).
//
// The bitstream is cut into subsequences of 128 bits, one thread each.  A
// thread cannot know where the first codeword of its subsequence starts, so
// it parses from the subsequence's first bit anyway; a parse that starts
// inside a codeword soon falls onto a true codeword boundary, and from there
// on it equals the true parse.  Four kernels:
//
//   k_huff_table  (one workgroup) checks the table and builds the canonical
//                 decode tables: a 2^11-entry first-level table (codes of up
//                 to 11 bits), per length the first code, the count and the
//                 first index (longer codes), and the values in code order.
//   k_huff_parse  parses every subsequence from its first bit (tables and the
//                 workgroup's slice of the bitstream in LDS), then walks from
//                 where the previous subsequence's parse crossed into it until
//                 the walk meets its own parse: from there on the two agree,
//                 so the walk's codeword starts replace the parse's before
//                 that point.  A workgroup owns 255 subsequences; its first
//                 thread re-parses the previous workgroup's last one, so the
//                 whole check stays inside the workgroup.  A walk that does
//                 not meet the parse before the subsequence ends is recorded.
//   k_huff_fix    (one workgroup, usually nothing to do) repeats the walk for
//                 the recorded subsequences in stream order, from the true
//                 crossing point, carrying a changed crossing point on to the
//                 next subsequence; finds the first pattern that is no
//                 codeword; adjusts the counts.
//   k_huff_write  places each subsequence's symbols by a prefix of the counts
//                 and decodes them again, writing the values.
#include "pic_huff.h"
#include "pic_internal.h"

namespace pic {
namespace {

constexpr int kWaves = kHuffThreads / 64;
constexpr int kLut = 1 << kHuffLutBits;
constexpr int kBlockWords = kHuffThreads * kHuffSub / 32;     // bitstream words of one workgroup
constexpr int kStageWords = kBlockWords + 2;                  // plus the codeword crossing the end
constexpr int kTabFirst = 8, kTabCount = 40, kTabIndex = 72;

// Big-endian 32-bit word w of the bitstream (bytes outside it read as 0).
__device__ __forceinline__ uint32_t stream_word(const uint8_t *data, int32_t n_bytes, int64_t w)
{
    uint32_t v = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int64_t i = w * 4 + k;
        v = (v << 8) | (i >= 0 && i < n_bytes ? (uint32_t)data[i] : 0u);
    }
    return v;
}

// The 32 bits from bit position `pos` of a word array (MSB first).
__device__ __forceinline__ uint32_t window32(const uint32_t *words, int32_t pos)
{
    const int i = pos >> 5, o = pos & 31;
    const uint64_t two = ((uint64_t)words[i] << 32) | words[i + 1];
    return (uint32_t)((two << o) >> 32);
}

// The same straight from the bitstream in global memory.
__device__ __forceinline__ uint32_t window32_global(const uint8_t *data, int32_t n_bytes, int32_t pos)
{
    const int64_t i = pos >> 5;
    const uint64_t two = ((uint64_t)stream_word(data, n_bytes, i) << 32) | stream_word(data, n_bytes, i + 1);
    return (uint32_t)((two << (pos & 31)) >> 32);
}

// Decode tables of one workgroup.
struct Tables {
    const uint32_t *lut;
    const int32_t *fc, *cnt, *fi;     // per length: first code, count, first index
    int max_len;
};

// Length of the codeword at the top of `win` (0: no codeword) and its index
// in code order.
__device__ __forceinline__ int decode_one(uint32_t win, const Tables &t, int *idx)
{
    const uint32_t e = t.lut[win >> (32 - kHuffLutBits)];
    if (e) {
        *idx = (int)(e & 0xffffu);
        return (int)(e >> 16);
    }
    for (int l = kHuffLutBits + 1; l <= t.max_len; ++l) {
        const uint32_t d = (win >> (32 - l)) - (uint32_t)t.fc[l];
        if (d < (uint32_t)t.cnt[l]) {
            *idx = t.fi[l] + (int)d;
            return l;
        }
    }
    return 0;
}

// LDS copies of the decode tables, filled by load_tables.
struct SharedTables {
    uint32_t lut[kLut];
    int32_t fc[kHuffMaxLen + 1], cnt[kHuffMaxLen + 1], fi[kHuffMaxLen + 1];
    int32_t valid, max_len;
};

__device__ __forceinline__ void load_tables(const HuffParams &p, SharedTables &s)
{
    for (int i = threadIdx.x; i < kLut; i += kHuffThreads)
        s.lut[i] = p.lut[i];
    if (threadIdx.x <= kHuffMaxLen) {
        s.fc[threadIdx.x] = p.tab[kTabFirst + threadIdx.x];
        s.cnt[threadIdx.x] = p.tab[kTabCount + threadIdx.x];
        s.fi[threadIdx.x] = p.tab[kTabIndex + threadIdx.x];
    }
    if (threadIdx.x == 0) {
        s.valid = p.tab[0];
        s.max_len = p.tab[1];
    }
}

__device__ __forceinline__ Tables tables_of(const SharedTables &s)
{
    return Tables{s.lut, s.fc, s.cnt, s.fi, s.max_len};
}

// Stage the bitstream words [w0, w0 + kStageWords) in LDS.
__device__ __forceinline__ void stage_words(const HuffParams &p, uint32_t *words, int64_t w0)
{
    const int32_t n_bytes = (int32_t)(((int64_t)p.n_bits + 7) >> 3);
    for (int i = threadIdx.x; i < kStageWords; i += kHuffThreads)
        words[i] = stream_word(p.data, n_bytes, w0 + i);
}

__global__ __launch_bounds__(kHuffThreads) void k_huff_table(HuffParams p)
{
    __shared__ int32_t s_count[kHuffMaxLen + 1], s_fc[kHuffMaxLen + 1], s_fi[kHuffMaxLen + 1];
    __shared__ int32_t s_run[kHuffMaxLen + 1];              // entries of each length in earlier tiles
    __shared__ int32_t s_wcnt[kWaves][kHuffMaxLen + 1];
    __shared__ uint32_t s_lut[kLut];
    __shared__ int32_t s_bad;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    if (t <= kHuffMaxLen) {
        s_count[t] = 0;
        s_run[t] = 0;
    }
    if (t == 0)
        s_bad = 0;
    for (int i = t; i < kLut; i += kHuffThreads)
        s_lut[i] = 0;
    __syncthreads();
    for (int i = t; i < p.n_table; i += kHuffThreads) {
        const int l = p.lengths[i];
        if (l < 1 || l > kHuffMaxLen)
            s_bad = 1;
        else
            atomicAdd(&s_count[l], 1);
    }
    __syncthreads();
    if (t == 0) {
        // canonical code (RFC 1951, Sec. 3.2.2) and the Kraft sum
        int64_t kraft = 0;
        uint32_t code = 0;
        int32_t idx = 0, max_len = 0;
        s_count[0] = 0;
        s_fc[0] = 0;
        s_fi[0] = 0;
        for (int l = 1; l <= kHuffMaxLen; ++l) {
            kraft += (int64_t)s_count[l] << (kHuffMaxLen - l);
            code = (code + (uint32_t)s_count[l - 1]) << 1;
            s_fc[l] = (int32_t)code;
            s_fi[l] = idx;
            idx += s_count[l];
            if (s_count[l])
                max_len = l;
        }
        if (kraft > (1LL << kHuffMaxLen))
            s_bad = 1;
        p.tab[0] = !s_bad;
        p.tab[1] = max_len;
        *p.status = s_bad ? PIC_HUFF_ERR_TABLE : 0;
        p.flags[0] = 0;
        p.flags[1] = 0x7fffffff;      // first subsequence whose true parse meets no codeword
    }
    __syncthreads();
    if (t <= kHuffMaxLen) {
        p.tab[kTabFirst + t] = s_fc[t];
        p.tab[kTabCount + t] = s_count[t];
        p.tab[kTabIndex + t] = s_fi[t];
    }
    if (s_bad)
        return;   // uniform

    // Rank of each entry among the entries of its length before it (table
    // order), 256 entries at a time: per wave a ballot per length.
    for (int base = 0; base < p.n_table; base += kHuffThreads) {
        const int i = base + t;
        const int l = i < p.n_table ? p.lengths[i] : 0;
        int in_wave = 0;
        for (int k = 1; k <= kHuffMaxLen; ++k) {
            const uint64_t m = __ballot(l == k);
            if (l == k)
                in_wave = __popcll(m & ((1ull << lane) - 1));
            if (lane == 0)
                s_wcnt[wave][k] = __popcll(m);
        }
        __syncthreads();
        if (l > 0) {
            int rank = s_run[l] + in_wave;
            for (int w = 0; w < wave; ++w)
                rank += s_wcnt[w][l];
            const int si = s_fi[l] + rank;
            const uint32_t code = (uint32_t)s_fc[l] + (uint32_t)rank;
            p.sorted[si] = p.values[i];
            if (l <= kHuffLutBits) {
                const uint32_t first = code << (kHuffLutBits - l), n = 1u << (kHuffLutBits - l);
                for (uint32_t k = 0; k < n; ++k)
                    s_lut[first + k] = (uint32_t)si | (uint32_t)l << 16;
            }
        }
        __syncthreads();
        if (t >= 1 && t <= kHuffMaxLen)
            for (int w = 0; w < kWaves; ++w)
                s_run[t] += s_wcnt[w][t];
        __syncthreads();
    }
    for (int i = t; i < kLut; i += kHuffThreads)
        p.lut[i] = s_lut[i];
}

// The 32 bits from absolute bit position `pos`: from the workgroup's staged
// words (LdsBits) or straight from the bitstream (GlobalBits).
struct LdsBits {
    const uint32_t *words;
    int32_t base;                     // bit position of words[0]
    __device__ __forceinline__ uint32_t operator()(int32_t pos) const { return window32(words, pos - base); }
};

struct GlobalBits {
    const uint8_t *data;
    int32_t n_bytes;
    __device__ __forceinline__ uint32_t operator()(int32_t pos) const
    {
        return window32_global(data, n_bytes, pos);
    }
};

// 128 bits, one per bit offset of a subsequence.
struct Mask {
    uint64_t lo, hi;
};

__device__ __forceinline__ bool mask_has(const Mask &m, int off)
{
    return ((off < 64 ? m.lo : m.hi) >> (off & 63)) & 1u;
}

__device__ __forceinline__ void mask_set(Mask &m, int off)
{
    const uint64_t bit = 1ull << (off & 63);
    if (off < 64)
        m.lo |= bit;
    else
        m.hi |= bit;
}

// The bits of `m` at offsets >= off (0 <= off <= 128).
__device__ __forceinline__ Mask mask_from(const Mask &m, int off)
{
    const uint64_t keep = ~0ull << (off & 63);
    Mask r;
    r.lo = off >= 64 ? 0ull : m.lo & keep;
    r.hi = off >= 128 ? 0ull : off < 64 ? m.hi : m.hi & keep;
    return r;
}

__device__ __forceinline__ int mask_count(const Mask &m) { return __popcll(m.lo) + __popcll(m.hi); }

__device__ __forceinline__ Mask load_mask(const HuffParams &p, int t)
{
    const uint4 v = reinterpret_cast<const uint4 *>(p.mask)[t];
    return Mask{(uint64_t)v.y << 32 | v.x, (uint64_t)v.w << 32 | v.z};
}

__device__ __forceinline__ void store_mask(const HuffParams &p, int t, const Mask &m)
{
    reinterpret_cast<uint4 *>(p.mask)[t] =
        make_uint4((uint32_t)m.lo, (uint32_t)(m.lo >> 32), (uint32_t)m.hi, (uint32_t)(m.hi >> 32));
}

// How a walk ends.
enum { kReached = 0, kMet = 1, kInvalid = 2, kPastEnd = 3 };

// Parse from bit *pos of the subsequence that starts at bit `start` and ends
// before `lim`, setting each codeword start in `m`; with MEET, stop at the
// first position that `old` holds already.  *pos receives where the walk
// stopped.
template <bool MEET, class Bits>
__device__ __forceinline__ int walk(const Bits &bits, const Tables &tab, int32_t start, int32_t lim,
                                    int32_t n_bits, const Mask &old, Mask &m, int32_t *pos_io)
{
    int32_t pos = *pos_io;
    int state = kReached;
    while (pos < lim) {
        const int off = pos - start;
        if (MEET && mask_has(old, off)) {
            state = kMet;
            break;
        }
        int idx;
        const int len = decode_one(bits(pos), tab, &idx);
        if (len == 0) {
            state = kInvalid;
            break;
        }
        if (len > n_bits - pos) {
            state = kPastEnd;
            break;
        }
        mask_set(m, off);
        pos += len;
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
    int32_t incl = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int32_t o = __shfl_up(incl, d, 64);
        if (lane >= d)
            incl += o;
    }
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

__global__ __launch_bounds__(kHuffThreads) void k_huff_parse(HuffParams p)
{
    __shared__ SharedTables s_tab;
    __shared__ uint32_t s_words[kStageWords];
    __shared__ int32_t s_end[kHuffThreads];
    __shared__ int32_t s_wsum[kWaves];
    const int l = threadIdx.x;
    const int32_t t0 = (int32_t)blockIdx.x * kHuffOwn;           // first owned subsequence
    const int64_t w0 = ((int64_t)t0 - 1) * (kHuffSub / 32);      // staged from the one before
    load_tables(p, s_tab);
    stage_words(p, s_words, w0);
    __syncthreads();
    if (!s_tab.valid)
        return;   // uniform
    const Tables tab = tables_of(s_tab);
    const LdsBits bits{s_words, (int32_t)(w0 * 32)};
    const int32_t t = t0 + l - 1;
    const bool live = t >= 0 && t < p.nsub;
    const int32_t start = t * kHuffSub;
    const int32_t lim = start + kHuffSub < p.n_bits ? start + kHuffSub : p.n_bits;
    Mask m{0ull, 0ull};
    int32_t end = 0;
    if (live) {
        int32_t pos = start;
        const int st = walk<false>(bits, tab, start, lim, p.n_bits, m, m, &pos);
        end = crossing(st, pos, p.n_bits);
    }
    s_end[l] = end;
    __syncthreads();
    // Walk from the previous parse's crossing point to the first codeword
    // start the two parses share; if the previous parse was true, so is this
    // one from there on, and the walk's starts replace the parse's before it.
    bool out_of_step = false;
    int32_t n = 0;
    if (live && l > 0) {
        const int32_t b = t == 0 ? 0 : s_end[l - 1];
        if (b < 0) {
            out_of_step = true;            // the previous parse met a pattern that is no codeword
        } else if (b < p.n_bits) {
            Mask w{0ull, 0ull};
            int32_t pos = b;
            const int st = walk<true>(bits, tab, start, lim, p.n_bits, m, w, &pos);
            if (st == kMet) {
                const Mask rest = mask_from(m, pos - start);
                m = Mask{w.lo | rest.lo, w.hi | rest.hi};
                // a parse that ends in a pattern that is no codeword: the
                // fix kernel decides, in stream order, where decoding stops
                out_of_step = end < 0;
            } else if (st == kReached && pos == end) {
                m = w;                     // no shared start, but the same crossing point
            } else {
                out_of_step = true;
            }
            n = mask_count(m);
        }
        // b >= n_bits: the stream ended before this subsequence; no codewords
        store_mask(p, t, m);
        p.end[t] = end;
        p.cnt[t] = n;
    }
    const uint64_t bad = __ballot(out_of_step);
    const int lane = l & 63, wave = l >> 6;
    if (lane == 0) {
        p.fail[blockIdx.x * 8 + wave * 2] = (uint32_t)bad;
        p.fail[blockIdx.x * 8 + wave * 2 + 1] = (uint32_t)(bad >> 32);
        if (bad)
            atomicOr(&p.flags[0], 1);
    }
    int32_t total;
    (void)block_sum_incl(n, s_wsum, &total);
    if (l == 0)
        p.blk[blockIdx.x] = total;
}

// Walk subsequence u again from the true crossing point of its predecessor
// until it meets its recorded parse, and update its record and count.
// Returns true when u's crossing point changed (u + 1 must be walked again);
// *corrupt is set when the true parse meets a pattern that is no codeword.
__device__ bool refix(const HuffParams &p, const Tables &tab, const GlobalBits &bits, int u, bool *corrupt)
{
    *corrupt = false;
    const int32_t b = u == 0 ? 0 : p.end[u - 1];
    if (b < 0)
        return false;                      // cannot happen: the fix stops at the first such pattern
    const int32_t start = u * kHuffSub;
    const int32_t lim = start + kHuffSub < p.n_bits ? start + kHuffSub : p.n_bits;
    bool carry = false;
    int32_t n = 0;
    if (b < p.n_bits) {
        Mask m = load_mask(p, u);
        const int32_t end = p.end[u];
        Mask w{0ull, 0ull};
        int32_t pos = b;
        const int st = walk<true>(bits, tab, start, lim, p.n_bits, m, w, &pos);
        if (st == kMet) {
            const Mask rest = mask_from(m, pos - start);
            m = Mask{w.lo | rest.lo, w.hi | rest.hi};
            *corrupt = end < 0;
        } else {
            m = w;
            const int32_t e = crossing(st, pos, p.n_bits);
            carry = e != end;
            *corrupt = st == kInvalid;
            p.end[u] = e;
        }
        store_mask(p, u, m);
        n = mask_count(m);
    }
    const int32_t old = p.cnt[u];
    if (n != old) {
        p.cnt[u] = n;
        p.blk[u / kHuffOwn] += n - old;
    }
    return carry;
}

__global__ __launch_bounds__(kHuffThreads) void k_huff_fix(HuffParams p)
{
    __shared__ SharedTables s_tab;
    __shared__ int32_t s_any, s_stop;
    __shared__ int32_t s_list[kHuffThreads];
    __shared__ int32_t s_wn[kWaves];
    __shared__ int32_t s_wsum[kWaves];
    if (threadIdx.x == 0) {
        s_any = p.flags[0];
        s_stop = 0;
    }
    load_tables(p, s_tab);
    __syncthreads();
    if (!s_tab.valid)
        return;   // uniform
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (s_any) {
        const Tables tab = tables_of(s_tab);
        const GlobalBits bits{p.data, (int32_t)(((int64_t)p.n_bits + 7) >> 3)};
        const int nwords = p.nblk * 8;
        // Walk the bitmap in stream order, 256 words at a time: the slice's
        // nonzero words are listed in order, then one thread repairs.
        for (int base = 0; base < nwords; base += kHuffThreads) {
            const int wd = base + threadIdx.x;
            const uint32_t word = wd < nwords ? p.fail[wd] : 0u;
            const uint64_t nz = __ballot(word != 0u);
            if (lane == 0)
                s_wn[wave] = __popcll(nz);
            __syncthreads();
            int at = __popcll(nz & ((1ull << lane) - 1));
            for (int k = 0; k < wave; ++k)
                at += s_wn[k];
            if (word)
                s_list[at] = wd;
            __syncthreads();
            if (threadIdx.x == 0) {
                const int nlist = s_wn[0] + s_wn[1] + s_wn[2] + s_wn[3];
                for (int k = 0; k < nlist && !s_stop; ++k) {
                    const int w = s_list[k];
                    uint32_t bm = p.fail[w];
                    while (bm && !s_stop) {
                        const int l = (w & 7) * 32 + __builtin_ctz(bm);
                        bm &= bm - 1u;
                        // repair, then carry a changed crossing point onwards
                        for (int u = (w >> 3) * kHuffOwn + l - 1; u < p.nsub; ++u) {
                            bool corrupt;
                            const bool carry = refix(p, tab, bits, u, &corrupt);
                            if (corrupt) {
                                atomicOr(p.status, PIC_HUFF_ERR_CODE);
                                p.flags[1] = u;
                                s_stop = 1;
                                break;
                            }
                            if (!carry)
                                break;
                        }
                    }
                }
            }
            __syncthreads();
            if (s_stop)
                break;   // uniform
        }
    }
    if (p.blk_is_prefix) {
        // exclusive prefixes of the per-workgroup counts, a segment per thread
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

__global__ __launch_bounds__(kHuffThreads) void k_huff_write(HuffParams p)
{
    __shared__ SharedTables s_tab;
    __shared__ uint32_t s_words[kStageWords];
    __shared__ int32_t s_sorted[kHuffMaxTable];
    __shared__ int32_t s_wsum[kWaves];
    const int l = threadIdx.x;
    const int32_t t0 = (int32_t)blockIdx.x * kHuffOwn;
    const int64_t w0 = ((int64_t)t0 - 1) * (kHuffSub / 32);
    load_tables(p, s_tab);
    stage_words(p, s_words, w0);
    for (int i = l; i < p.n_table; i += kHuffThreads)
        s_sorted[i] = p.sorted[i];
    __syncthreads();
    if (!s_tab.valid)
        return;   // uniform
    const Tables tab = tables_of(s_tab);
    // symbols before this workgroup's subsequences
    int32_t before;
    if (p.blk_is_prefix) {
        before = p.blk[blockIdx.x];
    } else {
        int32_t a[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int j = l; j < (int)blockIdx.x; j += 8 * kHuffThreads) {
#pragma unroll
            for (int u = 0; u < 8; ++u)
                a[u] += j + u * kHuffThreads < (int)blockIdx.x ? p.blk[j + u * kHuffThreads] : 0;
        }
        (void)block_sum_incl(((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7])), s_wsum,
                             &before);
    }
    const int32_t t = t0 + l - 1;
    // subsequences after the first one whose true parse meets a pattern
    // that is no codeword hold nothing decodable
    const int32_t n = l > 0 && t < p.nsub && t <= p.flags[1] ? p.cnt[t] : 0;
    int32_t blk_total;
    const int32_t o = before + block_sum_incl(n, s_wsum, &blk_total) - n;
    // too few codewords: the bits ran out (unless a pattern that is no
    // codeword ended the decoding first, already reported)
    if (blockIdx.x == gridDim.x - 1 && l == 0 && (int64_t)before + blk_total < p.n_symbols &&
        !(*p.status & PIC_HUFF_ERR_CODE))
        atomicOr(p.status, PIC_HUFF_ERR_BITS);
    if (n == 0 || o >= p.n_symbols)
        return;
    const LdsBits bits{s_words, (int32_t)(w0 * 32)};
    int32_t pos = t == 0 ? 0 : p.end[t - 1];
    const int32_t k_end = o + n < p.n_symbols ? n : p.n_symbols - o;
    for (int32_t k = 0; k < k_end; ++k) {
        int idx;
        const int len = decode_one(bits(pos), tab, &idx);
        if (len == 0)
            break;                         // cannot happen: the count came from this parse
        p.out[o + k] = s_sorted[idx];
        pos += len;
    }
}

}  // namespace

hipError_t launch_huff(const HuffParams &p, hipStream_t s)
{
    if (p.nsub < 1 || p.nblk != (p.nsub + kHuffOwn - 1) / kHuffOwn)
        return hipErrorInvalidValue;
    const dim3 block(kHuffThreads);
    const dim3 grid((unsigned)p.nblk);
    hipLaunchKernelGGL(k_huff_table, dim3(1), block, 0, s, p);
    hipLaunchKernelGGL(k_huff_parse, grid, block, 0, s, p);
    hipLaunchKernelGGL(k_huff_fix, dim3(1), block, 0, s, p);
    hipLaunchKernelGGL(k_huff_write, grid, block, 0, s, p);
    return hipGetLastError();
}

}  // namespace pic
