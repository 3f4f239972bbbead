// Huffman entropy decoding (PIC, Fig. 1 "HD"; Sec. 3.3: an image-specific
// canonical code, decoded with a table indexed by the next bits; Sec. 4.1:
// parallel decoding after GPUHD, which relies on Huffman codes
// resynchronising by themselves).
//
// The bitstream is cut into subsequences of 128 bits, one thread each.  A
// thread cannot know where the first codeword of its subsequence starts, so
// it parses from the subsequence's first bit anyway; a parse that starts
// inside a codeword soon falls onto a true codeword boundary, and from there
// on it equals the true parse.  Six kernels:
//
//   k_huff_table  (one workgroup) checks the table and builds the canonical
//                 decode tables: a 2^11-entry first-level table (codes of up
//                 to 11 bits), per length the first code, the count and the
//                 first index (longer codes), and the values in code order.
//   k_huff_parse  parses every subsequence from its first bit (LUT and the
//                 workgroup's slice of the bitstream in LDS) and records a
//                 128-bit mask of the codeword starts it visited and where the
//                 parse crossed into the next subsequence.
//   k_huff_check  subsequence t is in step if the parse of t - 1 crossed into
//                 it at a position t's own parse visited; the others are
//                 recorded in a bitmap.
//   k_huff_fix    (one workgroup, usually nothing to do) re-parses each
//                 subsequence that was not in step from the true start, in
//                 stream order, until its successor is in step again.
//   k_huff_count  counts each subsequence's codewords from its true start.
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

// Big-endian 32-bit word w of the bitstream (bytes past the end read as 0).
__device__ __forceinline__ uint32_t stream_word(const uint8_t *data, int32_t n_bytes, int64_t w)
{
    uint32_t v = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int64_t i = w * 4 + k;
        v = (v << 8) | (i < n_bytes ? (uint32_t)data[i] : 0u);
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

__global__ __launch_bounds__(kHuffThreads) void k_huff_parse(HuffParams p)
{
    __shared__ SharedTables s_tab;
    __shared__ uint32_t s_words[kStageWords];
    const int64_t w0 = (int64_t)blockIdx.x * kBlockWords;
    load_tables(p, s_tab);
    stage_words(p, s_words, w0);
    __syncthreads();
    if (!s_tab.valid)
        return;
    const Tables tab = tables_of(s_tab);
    const int t = blockIdx.x * kHuffThreads + threadIdx.x;
    if (t >= p.nsub)
        return;
    const int32_t start = t * kHuffSub;
    const int32_t lim = start + kHuffSub < p.n_bits ? start + kHuffSub : p.n_bits;
    const int32_t local0 = (int32_t)(start - w0 * 32);
    uint32_t m[4] = {0u, 0u, 0u, 0u};
    int32_t pos = start, end;
    while (true) {
        if (pos >= lim) {
            end = pos;
            break;
        }
        int idx;
        const int len = decode_one(window32(s_words, local0 + (pos - start)), tab, &idx);
        if (len == 0) {
            end = -1;                 // no codeword starts here
            break;
        }
        if (pos + len > p.n_bits) {   // the codeword would run past the stream
            end = p.n_bits;
            break;
        }
        const int off = pos - start;
        m[off >> 5] |= 1u << (off & 31);
        pos += len;
    }
    reinterpret_cast<uint4 *>(p.mask)[t] = make_uint4(m[0], m[1], m[2], m[3]);
    p.end[t] = end;
}

// Is subsequence t in step: did the previous parse cross into it at a
// codeword start of its own parse?
__device__ __forceinline__ bool in_step(const HuffParams &p, int t, int32_t b)
{
    if (t == 0)
        return true;
    if (b < 0)
        return false;                 // the previous parse met a pattern that is no codeword
    if (b >= p.n_bits)
        return true;                  // nothing left of the stream here
    const uint4 mk = reinterpret_cast<const uint4 *>(p.mask)[t];
    const int off = b - t * kHuffSub;
    const uint32_t word = off < 32 ? mk.x : off < 64 ? mk.y : off < 96 ? mk.z : mk.w;
    return (word >> (off & 31)) & 1u;
}

__global__ __launch_bounds__(kHuffThreads) void k_huff_check(HuffParams p)
{
    __shared__ int32_t s_valid;
    if (threadIdx.x == 0)
        s_valid = p.tab[0];
    __syncthreads();
    if (!s_valid)
        return;
    const int t = blockIdx.x * kHuffThreads + threadIdx.x;
    bool ok = true;
    if (t < p.nsub && t > 0)
        ok = in_step(p, t, p.end[t - 1]);
    const uint64_t bad = __ballot(!ok);
    const int lane = threadIdx.x & 63;
    const int word0 = (blockIdx.x * kHuffThreads + (threadIdx.x & ~63)) >> 5;   // two words per wave
    if (lane == 0) {
        p.fail[word0] = (uint32_t)bad;
        p.fail[word0 + 1] = (uint32_t)(bad >> 32);
        if (bad)
            atomicOr(&p.flags[0], 1);
    }
}

// Re-parse subsequence t from the true start b (one thread), updating its
// mask and crossing point.
__device__ void reparse(const HuffParams &p, const Tables &tab, int t, int32_t b)
{
    const int32_t n_bytes = (int32_t)(((int64_t)p.n_bits + 7) >> 3);
    const int32_t start = t * kHuffSub;
    const int32_t lim = start + kHuffSub < p.n_bits ? start + kHuffSub : p.n_bits;
    uint32_t m[4] = {0u, 0u, 0u, 0u};
    int32_t pos = b, end;
    while (true) {
        if (pos >= lim) {
            end = pos;
            break;
        }
        int idx;
        const int len = decode_one(window32_global(p.data, n_bytes, pos), tab, &idx);
        if (len == 0) {
            end = -1;
            break;
        }
        if (pos + len > p.n_bits) {
            end = p.n_bits;
            break;
        }
        const int off = pos - start;
        m[off >> 5] |= 1u << (off & 31);
        pos += len;
    }
    reinterpret_cast<uint4 *>(p.mask)[t] = make_uint4(m[0], m[1], m[2], m[3]);
    p.end[t] = end;
}

__global__ __launch_bounds__(kHuffThreads) void k_huff_fix(HuffParams p)
{
    __shared__ SharedTables s_tab;
    __shared__ int32_t s_any;
    __shared__ int32_t s_list[kHuffThreads];
    __shared__ int32_t s_nlist;
    if (threadIdx.x == 0)
        s_any = p.flags[0];
    load_tables(p, s_tab);
    __syncthreads();
    if (!s_any || !s_tab.valid)
        return;
    const Tables tab = tables_of(s_tab);
    const int nwords = ((p.nsub + 63) / 64) * 2;
    // Walk the bitmap in stream order, a slice of 256 words at a time: the
    // slice's nonzero words are collected in order, then one thread repairs.
    for (int base = 0; base < nwords; base += kHuffThreads) {
        if (threadIdx.x == 0)
            s_nlist = 0;
        __syncthreads();
        const int w = base + threadIdx.x;
        const uint32_t bits = w < nwords ? p.fail[w] : 0u;
        const uint64_t nz = __ballot(bits != 0u);
        __shared__ int32_t s_wn[kWaves];
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        if (lane == 0)
            s_wn[wave] = __popcll(nz);
        __syncthreads();
        int at = __popcll(nz & ((1ull << lane) - 1));
        for (int k = 0; k < wave; ++k)
            at += s_wn[k];
        if (bits)
            s_list[at] = w;
        if (threadIdx.x == 0)
            s_nlist = s_wn[0] + s_wn[1] + s_wn[2] + s_wn[3];
        __syncthreads();
        if (threadIdx.x == 0) {
            for (int k = 0; k < s_nlist; ++k) {
                const int wd = s_list[k];
                uint32_t b = p.fail[wd];
                while (b) {
                    int t = wd * 32 + __builtin_ctz(b);
                    b &= b - 1u;
                    // repair t, then its successors while they are out of step
                    while (t < p.nsub && !in_step(p, t, p.end[t - 1])) {
                        const int32_t from = p.end[t - 1];
                        if (from < 0)
                            break;            // a pattern that is no codeword upstream: corrupt stream
                        reparse(p, tab, t, from);
                        ++t;
                    }
                }
            }
        }
        __syncthreads();
    }
}

// Codewords of subsequence t from its true start (0 if none reaches it).
__device__ __forceinline__ int32_t count_from_start(const HuffParams &p, int t, int32_t *b_out)
{
    const int32_t b = t == 0 ? 0 : p.end[t - 1];
    *b_out = b;
    if (b < 0 || b >= p.n_bits)
        return 0;
    const uint4 mk = reinterpret_cast<const uint4 *>(p.mask)[t];
    const int off = b - t * kHuffSub;
    const uint32_t m[4] = {mk.x, mk.y, mk.z, mk.w};
    int32_t n = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int lo = k * 32;
        uint32_t v = m[k];
        if (off >= lo + 32)
            v = 0u;
        else if (off > lo)
            v &= ~0u << (off - lo);
        n += __popc(v);
    }
    return n;
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

__global__ __launch_bounds__(kHuffThreads) void k_huff_count(HuffParams p)
{
    __shared__ int32_t s_wsum[kWaves];
    __shared__ int32_t s_valid;
    if (threadIdx.x == 0)
        s_valid = p.tab[0];
    __syncthreads();
    if (!s_valid)
        return;
    const int t = blockIdx.x * kHuffThreads + threadIdx.x;
    int32_t n = 0, b = 0;
    if (t < p.nsub) {
        n = count_from_start(p, t, &b);
        // the true parse itself met a pattern that is no codeword: nothing
        // after it can be decoded (the smallest such subsequence is the true
        // one; later ones only look so because their start is not true)
        if (b >= 0 && b < p.n_bits && p.end[t] < 0) {
            atomicOr(p.status, PIC_HUFF_ERR_CODE);
            atomicMin(&p.flags[1], t);
        }
    }
    int32_t total;
    (void)block_sum_incl(n, s_wsum, &total);
    if (threadIdx.x == 0)
        p.blk[blockIdx.x] = total;
}

__global__ __launch_bounds__(kHuffThreads) void k_huff_write(HuffParams p)
{
    __shared__ SharedTables s_tab;
    __shared__ uint32_t s_words[kStageWords];
    __shared__ int32_t s_sorted[kHuffMaxTable];
    __shared__ int32_t s_wsum[kWaves];
    const int64_t w0 = (int64_t)blockIdx.x * kBlockWords;
    load_tables(p, s_tab);
    stage_words(p, s_words, w0);
    for (int i = threadIdx.x; i < p.n_table; i += kHuffThreads)
        s_sorted[i] = p.sorted[i];
    __syncthreads();
    if (!s_tab.valid)
        return;
    const Tables tab = tables_of(s_tab);
    // symbols before this block of subsequences: the earlier blocks' counts
    int32_t a[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int j = threadIdx.x; j < (int)blockIdx.x; j += 8 * kHuffThreads) {
#pragma unroll
        for (int u = 0; u < 8; ++u)
            a[u] += j + u * kHuffThreads < (int)blockIdx.x ? p.blk[j + u * kHuffThreads] : 0;
    }
    int32_t before;
    (void)block_sum_incl(((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7])), s_wsum, &before);
    const int t = blockIdx.x * kHuffThreads + threadIdx.x;
    int32_t n = 0, b = 0;
    if (t < p.nsub && t <= p.flags[1])
        n = count_from_start(p, t, &b);
    int32_t blk_total;
    const int32_t o = before + block_sum_incl(n, s_wsum, &blk_total) - n;
    // too few codewords: the bits ran out (unless a pattern that is no
    // codeword ended the decoding first, already reported)
    if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0 && (int64_t)before + blk_total < p.n_symbols &&
        !(*p.status & PIC_HUFF_ERR_CODE))
        atomicOr(p.status, PIC_HUFF_ERR_BITS);
    if (n == 0 || o >= p.n_symbols)
        return;
    const int32_t local0 = (int32_t)((int64_t)t * kHuffSub - w0 * 32);
    int32_t pos = b;
    const int32_t k_end = o + n < p.n_symbols ? n : p.n_symbols - o;
    for (int32_t k = 0; k < k_end; ++k) {
        int idx;
        const int len = decode_one(window32(s_words, local0 + (pos - t * kHuffSub)), tab, &idx);
        if (len == 0)
            break;                    // cannot happen: the count came from this parse
        p.out[o + k] = s_sorted[idx];
        pos += len;
    }
}

}  // namespace

hipError_t launch_huff(const HuffParams &p, hipStream_t s)
{
    if (p.nsub < 1)
        return hipErrorInvalidValue;
    const dim3 block(kHuffThreads);
    const dim3 grid((unsigned)((p.nsub + kHuffThreads - 1) / kHuffThreads));
    hipLaunchKernelGGL(k_huff_table, dim3(1), block, 0, s, p);
    hipLaunchKernelGGL(k_huff_parse, grid, block, 0, s, p);
    hipLaunchKernelGGL(k_huff_check, grid, block, 0, s, p);
    hipLaunchKernelGGL(k_huff_fix, dim3(1), block, 0, s, p);
    hipLaunchKernelGGL(k_huff_count, grid, block, 0, s, p);
    hipLaunchKernelGGL(k_huff_write, grid, block, 0, s, p);
    return hipGetLastError();
}

}  // namespace pic
