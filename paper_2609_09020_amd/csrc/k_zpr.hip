// Latent decoding from the ZpR symbol stream (PIC, Sec. 3.3 and Fig. 2;
// App. B, Alg. 1; Sec. 3.2 Eq. (6)-(7) for the patches and the DCT).
//
// Two kernels (three on very long streams).  The stream is partitioned into
// chunks of 256 symbols (one per thread) or, for streams of 2^18 symbols and
// more, 1024 (four per thread, so the per-workgroup set-up is spread over
// more blocks):
//
//   k_zpr_count   counts each chunk's end-of-block markers (and clears the
//                 status word).
//   k_zpr_scan    (one workgroup; only beyond 16384 chunks) turns the counts
//                 into their exclusive prefix.  Otherwise each workgroup of
//                 the next kernel sums the counts of the chunks before its
//                 own (L2-resident, a few loads per thread).  Either way the
//                 result is the index of the first block whose marker lies in
//                 the chunk; together the two replace the copy_if of marker
//                 offsets that Alg. 1 starts from: no offset array is built.
//   k_zpr_expand  stages its chunk (and the 256 symbols before it) in LDS
//                 and, with one workgroup scan, finds for every symbol the
//                 coefficients it produces, its block (the chunk's markers
//                 before it) and its offset in that block (a difference of
//                 two prefixes: Alg. 1's running offset without a serial
//                 walk); the chunk's marker positions are compacted.  A
//                 block's symbols start after the previous marker, found in
//                 the chunk or, for the first block, within the 65 staged
//                 symbols before it (a block of 64 symbols plus the preceding
//                 marker).  Each coefficient value's slot (its block and,
//                 through the zigzag table, its word of the block's 8x8
//                 tile) is found once.  Blocks are then decoded in windows
//                 of 32: the tiles are zeroed, every coefficient value of the
//                 window is written to its slot, and eight lanes per block
//                 run the separable inverse DCT (rows, an LDS transpose,
//                 columns; a factored 8-point transform with compile-time
//                 constants) and write the block's patch of its latent grid,
//                 cropped at the grid's edge.
//
// Memory traffic: the stream read by both kernels (plus the expand kernel's
// 256-symbol halos) and the pyramid written once; the HBM floor of the step
// is the stream read once and the pyramid written once.
#include "pic_internal.h"
#include "pic_zpr.h"

namespace pic {
namespace {

constexpr int kWaves = kZprThreads / 64;
constexpr int kHalo = kZprThreads;           // symbols staged before the chunk (>= 65)
constexpr int kGroups = kZprThreads / 8;     // blocks in flight per workgroup (8 lanes each)
constexpr int kTile = 64 + 8;                // LDS words per 8x8 tile: the pad puts the 8
                                             // groups' column reads on disjoint banks

// JPEG zigzag scan (ITU-T T.81, Fig. A.6): entry p is the row-major index of
// the p-th coefficient.
__constant__ uint8_t kZigzag[64] = {
    0,  1,  8,  16, 9,  2,  3,  10, 17, 24, 32, 25, 18, 11, 4,  5,
    12, 19, 26, 33, 40, 48, 41, 34, 27, 20, 13, 6,  7,  14, 21, 28,
    35, 42, 49, 56, 57, 50, 43, 36, 29, 22, 15, 23, 30, 37, 44, 51,
    58, 59, 52, 45, 38, 31, 39, 46, 53, 60, 61, 54, 47, 55, 62, 63};

// cos(k pi / 16) for k = 0 .. 8, each rounded to the nearest fp32 (cos(pi/2)
// is 0 exactly), and sqrt(1/8).
constexpr float kCos16[9] = {1.0f,           0x1.f6297cp-1f, 0x1.d906bcp-1f,
                             0x1.a9b662p-1f, 0x1.6a09e6p-1f, 0x1.1c73b4p-1f,
                             0x1.87de2ap-2f, 0x1.8f8b84p-3f, 0.0f};
constexpr float kSqrtEighth = 0x1.6a09e6p-2f;

// Entry (x, v) of the orthonormal 8-point inverse DCT: a(v) cos((2x + 1) v pi / 16)
// with a(0) = sqrt(1/8), a(v > 0) = 1/2, in fp32.  The angle is folded onto
// [0, pi/2] with cos(2 pi - t) = cos t and cos(pi - t) = -cos t; halving is exact.
// Called with constant arguments only, so every use is an instruction literal.
__host__ __device__ constexpr float dct_basis(int x, int v)
{
    if (v == 0)
        return kSqrtEighth;
    int k = ((2 * x + 1) * v) % 32;
    if (k > 16)
        k = 32 - k;
    return k > 8 ? -0.5f * kCos16[16 - k] : 0.5f * kCos16[k];
}

// Inclusive sum over the workgroup's threads of v (every thread calls it);
// also returns the workgroup total.  s_wsum holds kWaves ints.
__device__ __forceinline__ int32_t block_inclusive_sum(int32_t v, int32_t *s_wsum, int32_t *total)
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
    __syncthreads();   // s_wsum may be reused by the caller
    *total = tot;
    return off + incl;
}

template <int CH>
__global__ __launch_bounds__(kZprThreads) void k_zpr_count(ZprParams p)
{
    warm_kernel_args<sizeof(ZprParams)>();
    constexpr int SPT = CH / kZprThreads;
    __shared__ int32_t s_wsum[kWaves];
    const int t = threadIdx.x;
    const int64_t cs = (int64_t)blockIdx.x * CH;
    int32_t v[SPT];
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        const int64_t i = cs + j * kZprThreads + t;
        v[j] = i < p.n ? p.sym[i] : ~p.eob;
    }
    // each wave's markers: one ballot per row of symbols, counted on the
    // scalar unit
    int32_t mine = 0;
#pragma unroll
    for (int j = 0; j < SPT; ++j)
        mine += __popcll(__ballot(v[j] == p.eob));
    if ((t & 63) == 0)
        s_wsum[t >> 6] = mine;
    __syncthreads();
    if (t == 0) {
        int32_t tot = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w)
            tot += s_wsum[w];
        p.counts[blockIdx.x] = tot;
        if (blockIdx.x == 0)
            *p.status = 0;     // the decoding kernel ors its findings into it
    }
}

// One workgroup: counts[] -> exclusive prefix in place (long streams only).
// Segments of kScanSeg counts are staged in LDS with coalesced loads; each
// thread scans kScanPer consecutive entries, the workgroup scans the
// per-thread sums, and the segment is written back coalesced.
constexpr int kScanThreads = 1024;
constexpr int kScanPer = 16;
constexpr int kScanSeg = kScanThreads * kScanPer;

__global__ __launch_bounds__(kScanThreads) void k_zpr_scan(ZprParams p)
{
    warm_kernel_args<sizeof(ZprParams)>();
    __shared__ int32_t s_seg[kScanSeg];
    __shared__ int32_t s_wsum[kScanThreads / 64];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    int32_t carry = 0;
    for (int base = 0; base < p.nchunks; base += kScanSeg) {
        const int len = p.nchunks - base < kScanSeg ? p.nchunks - base : kScanSeg;
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) {
            const int i = j * kScanThreads + t;
            s_seg[i] = i < len ? p.counts[base + i] : 0;
        }
        __syncthreads();
        int32_t v[kScanPer], sum = 0;
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) {
            v[j] = s_seg[t * kScanPer + j];
            sum += v[j];
        }
        const int32_t incl = wave_inclusive_sum(sum);
        if (lane == 63)
            s_wsum[wave] = incl;
        __syncthreads();
        int32_t run = carry + incl - sum, seg_total = 0;
        for (int w = 0; w < kScanThreads / 64; ++w) {
            run += w < wave ? s_wsum[w] : 0;
            seg_total += s_wsum[w];
        }
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) {
            s_seg[t * kScanPer + j] = run;
            run += v[j];
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) {
            const int i = j * kScanThreads + t;
            if (i < len)
                p.counts[base + i] = s_seg[i];
        }
        carry += seg_total;
        __syncthreads();   // s_seg and s_wsum are rewritten by the next segment
    }
}

// Coefficients one symbol produces (Alg. 1): 1 for a coefficient value
// (s <= eob - 17), s - eob + 17 zeros for a run code (eob - 16 <= s < eob),
// none for the marker or a symbol above it.  Clamping s into
// [eob - 17, eob + 1] (one v_med3), d = clamped - (eob - 17) is 0 for a value, the run
// length for a run code, 17 for the marker and 18 above it (no overflow: the
// host keeps eob in [INT32_MIN + 17, INT32_MAX - 1]).
__device__ __forceinline__ int zpr_coeffs(int32_t s, int32_t eob)
{
    const int32_t lo = eob - 17, hi = eob + 1;
    const int d = (s < lo ? lo : (s > hi ? hi : s)) - lo;
    return d == 0 ? 1 : (d <= 16 ? d : 0);
}

// 8-point orthonormal inverse DCT, out[x] = sum_v in[v] a(v) cos((2x + 1) v pi / 16),
// factored by the symmetries of the basis: out[x] and out[7 - x] are the sum
// and difference of an even part (inputs v = 0, 2, 4, 6: a 4-point transform,
// itself split into v = 0, 4 and v = 2, 6) and an odd part (v = 1, 3, 5, 7:
// a 4 x 4 product).  35 operations instead of 64.
__device__ __forceinline__ void idct8(const float in[8], float out[8])
{
    constexpr float A0 = dct_basis(0, 0), C4 = dct_basis(0, 4);
    constexpr float C2 = dct_basis(0, 2), C6 = dct_basis(0, 6);
    const float dc = in[0] * A0;
    const float ee0 = __builtin_fmaf(in[4], C4, dc);     // rows x = 0, 3
    const float ee1 = __builtin_fmaf(in[4], -C4, dc);    // rows x = 1, 2
    const float eo0 = __builtin_fmaf(in[6], C6, in[2] * C2);
    const float eo1 = __builtin_fmaf(in[6], -C2, in[2] * C6);
    const float e[4] = {ee0 + eo0, ee1 + eo1, ee1 - eo1, ee0 - eo0};
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        float o = in[1] * dct_basis(x, 1);
        o = __builtin_fmaf(in[3], dct_basis(x, 3), o);
        o = __builtin_fmaf(in[5], dct_basis(x, 5), o);
        o = __builtin_fmaf(in[7], dct_basis(x, 7), o);
        out[x] = e[x] + o;
        out[7 - x] = e[x] - o;
    }
}

template <int CH, bool COEFF>
__global__ __launch_bounds__(kZprThreads) void k_zpr_expand(ZprParams p)
{
    warm_kernel_args<sizeof(ZprParams)>();
    constexpr int NS = kHalo + CH;                 // staged symbols
    constexpr int SPS = NS / kZprThreads;          // per thread, consecutive
    static_assert(NS % kZprThreads == 0, "staging must divide evenly");
    static_assert(NS * 16 < 32768, "coefficient prefixes and positions fit 16 bits");
    __shared__ int32_t s_sym[NS];
    __shared__ uint16_t s_cex[NS];                 // coefficients produced by the staged symbols before
                                                   // (at most 16 per symbol: < 2^15); once read, where
                                                   // a coefficient value goes: block * 64 + tile word
    uint16_t *const s_code = s_cex;
    __shared__ int16_t s_pos[CH + 1];              // [0]: marker before block 0; [1 + r]: block r's marker
    __shared__ __attribute__((aligned(16))) float s_blk[kGroups * kTile];   // tiles: S, then T in place
    __shared__ uint8_t s_zz[64];
    __shared__ int4 s_geo[PIC_MAX_LEVELS];         // stream level i: {h, w, pw | k << 16, ceil(2^k / pw)}
    __shared__ int32_t s_first[PIC_MAX_LEVELS];
    __shared__ float *s_lat[PIC_MAX_LEVELS];
    __shared__ int32_t s_wsum[kWaves];
    __shared__ int32_t s_err;

    const int t = threadIdx.x, lane = t & 63;
    const int64_t cs = (int64_t)blockIdx.x * CH;
    const int32_t eob = p.eob;
    // Stage [cs - kHalo, cs + CH).  Positions before the stream act as markers
    // (the first block starts at 0); positions past its end are never markers
    // and never inside a block.  The loads go out first and land in LDS after
    // the prefix below, so the two round trips overlap.
    int32_t staged[SPS];
#pragma unroll
    for (int u = 0; u < SPS; ++u) {
        const int64_t gi = cs - kHalo + t + u * kZprThreads;
        staged[u] = gi < 0 ? eob : (gi < p.n ? p.sym[gi] : 0);
    }

    // Blocks whose markers precede the chunk: the scan kernel's prefix, or the
    // sum of the earlier chunks' counts (L2-resident; eight independent loads
    // in flight per thread).
    int32_t g0;
    if (p.counts_are_prefix) {
        g0 = p.counts[blockIdx.x];
    } else {
        const int c = (int)blockIdx.x;
        int32_t a[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int j = t; j < c; j += 8 * kZprThreads) {
#pragma unroll
            for (int u = 0; u < 8; ++u)
                a[u] += j + u * kZprThreads < c ? p.counts[j + u * kZprThreads] : 0;
        }
        const int32_t part = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
        (void)block_inclusive_sum(part, s_wsum, &g0);
    }

#pragma unroll
    for (int u = 0; u < SPS; ++u)
        s_sym[t + u * kZprThreads] = staged[u];
    if (t < 64)
        s_zz[t] = kZigzag[t];
    if (!COEFF && t < p.L) {
        s_geo[t] = make_int4(p.hk[t], p.wk[t], p.pw[t] | p.pw_shift[t] << 16, p.pw_recip[t]);
        s_first[t] = p.first[t];
        s_lat[t] = p.lat[t];
    }
    if (t == 0)
        s_err = 0;
    __syncthreads();

    // Every staged symbol once: the coefficients it produces and whether it
    // is one of the chunk's markers.  One workgroup scan of both counts
    // (packed: coefficients in the high half, markers in the low) gives each
    // symbol its block (markers before it) and the coefficients produced
    // before it, so a symbol's place in its block is a difference of two
    // prefixes -- Alg. 1's running offset without a serial walk.
    int32_t sv[SPS], c[SPS], cp[SPS], rr[SPS];
    uint32_t mflags = 0;
    int32_t csum = 0, nm = 0;
#pragma unroll
    for (int j = 0; j < SPS; ++j) {
        const int i = t * SPS + j;
        sv[j] = s_sym[i];
        const int k = i - kHalo;
        const bool mk = k >= 0 && cs + k < p.n && sv[j] == eob;
        c[j] = zpr_coeffs(sv[j], eob);
        csum += c[j];
        nm += mk ? 1 : 0;
        mflags |= mk ? 1u << j : 0u;
    }
    int32_t total;
    const int32_t incl = block_inclusive_sum(csum << 16 | nm, s_wsum, &total);
    int32_t cpre = (incl >> 16) - csum, mpre = (incl & 0xffff) - nm;
    const int m = total & 0xffff;
#pragma unroll
    for (int j = 0; j < SPS; ++j) {
        const int i = t * SPS + j;
        s_cex[i] = (uint16_t)cpre;
        cp[j] = cpre;
        rr[j] = mpre;
        cpre += c[j];
        if (mflags >> j & 1u)
            s_pos[1 + mpre++] = (int16_t)i;
    }
    __syncthreads();
    if (t == 0 && blockIdx.x == (unsigned)p.nchunks - 1 &&
        ((int64_t)g0 + m != p.expected || (p.n > 0 && p.sym[p.n - 1] != eob)))
        atomicOr(p.status, PIC_ZPR_ERR_COUNT);   // marker count, or symbols after the last marker
    if (m == 0)
        return;   // uniform: no block ends in this chunk

    // The marker before the chunk's first block: the nearest of the 65
    // staged symbols before it; none means the block is too long (its last
    // 65 symbols are taken, which the length test below flags).
    if (t < 64) {
        const int f = s_pos[1];                              // >= kHalo
        const uint64_t hit = __ballot(s_sym[f - 1 - lane] == eob);
        int prev;
        if (hit)
            prev = f - 1 - (__ffsll((unsigned long long)hit) - 1);
        else
            prev = s_sym[f - 65] == eob ? f - 65 : f - 66;
        if (lane == 0)
            s_pos[0] = (int16_t)prev;
    }
    __syncthreads();

    // Each symbol's destination, once: block r (< m, one the stream has)
    // begins after s_pos[r], and a coefficient value lands at its place in
    // the block through the zigzag table.  Symbols outside the chunk's blocks
    // and markers get no slot; a symbol above the marker is flagged and
    // skipped, as Alg. 1 has no code for it; a block of more than 64 symbols
    // or coefficients is flagged once any of its symbols passes 64.  The
    // code fits 16 bits: a slot's block holds a symbol of the chunk, so it
    // is at most CH - 2.
    const int p0 = s_pos[0];
    int err = 0;
    uint32_t code[SPS];
#pragma unroll
    for (int j = 0; j < SPS; ++j) {
        const int i = t * SPS + j;
        const int r = rr[j];
        code[j] = 0xffffu;
        if (r < m && i > p0 && g0 + r < p.expected && sv[j] != eob) {
            if (sv[j] > eob) {
                err |= PIC_ZPR_ERR_SYMBOL;
            } else {
                const int begin = s_pos[r] + 1;
                const int pos = cp[j] - s_cex[begin];
                if (i - begin >= 64 || pos + c[j] > 64)
                    err |= PIC_ZPR_ERR_OVERFLOW;
                if (sv[j] <= eob - 17 && pos < 64)
                    code[j] = (uint32_t)r << 6 | s_zz[pos];
            }
        }
    }
    __syncthreads();   // every prefix is read: the slots take their place
#pragma unroll
    for (int j = 0; j < SPS; ++j)
        s_code[t * SPS + j] = (uint16_t)code[j];

    // Windows of kGroups blocks: zero the tiles, write the window's
    // coefficient values into their slots (any thread, any block), then
    // eight lanes per block transform and store it.
    const int grp = t >> 3, gl = t & 7;
    float *blk = s_blk + grp * kTile;
    const int32_t img0 = g0 / p.blocks_per_image;
    const int32_t j0 = g0 - img0 * p.blocks_per_image;
    for (int r0 = 0; r0 < m; r0 += kGroups) {
        reinterpret_cast<float4 *>(blk + gl * 8)[0] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        reinterpret_cast<float4 *>(blk + gl * 8)[1] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        __syncthreads();   // tiles zeroed (and the slots written, first round)
        const int rend = r0 + kGroups < m ? r0 + kGroups : m;
        const int lo = s_pos[r0] + 1, hi = s_pos[rend];
        for (int i = lo + t; i < hi; i += kZprThreads) {
            const uint32_t code = s_code[i];
            const int32_t s = s_sym[i];
            if (code != 0xffffu) {
                float *word = s_blk + ((int)(code >> 6) - r0) * kTile + (code & 63u);
                if (COEFF)
                    *reinterpret_cast<int32_t *>(word) = s;
                else
                    *word = (float)s;
            }
        }
        __syncthreads();   // the window's tiles are complete

        const int r = r0 + grp;
        const int32_t g = g0 + r;
        if (r < m && g < p.expected) {               // uniform over the 8 lanes of a block
            if (COEFF) {
                const int4 *src = reinterpret_cast<const int4 *>(blk + gl * 8);
                int4 *dst = reinterpret_cast<int4 *>(p.coeffs + (int64_t)g * 64 + gl * 8);
                dst[0] = src[0];
                dst[1] = src[1];
                continue;
            }
            // Rows: lane gl transforms row gl and stores it in place; then it
            // reads column gl (the LDS transpose) and transforms that.
            const float4 sa = reinterpret_cast<const float4 *>(blk + gl * 8)[0];
            const float4 sb = reinterpret_cast<const float4 *>(blk + gl * 8)[1];
            const float S[8] = {sa.x, sa.y, sa.z, sa.w, sb.x, sb.y, sb.z, sb.w};
            float T[8];
            idct8(S, T);
            reinterpret_cast<float4 *>(blk + gl * 8)[0] = make_float4(T[0], T[1], T[2], T[3]);
            reinterpret_cast<float4 *>(blk + gl * 8)[1] = make_float4(T[4], T[5], T[6], T[7]);
            asm volatile("" ::: "memory");
            float C[8], Z[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                C[u] = blk[u * 8 + gl];
            idct8(C, Z);
            asm volatile("" ::: "memory");

            // Un-patchify: image, level (stream order, found against the
            // uniform first-block table), patch; lane gl writes column gl.
            int32_t img = img0, j = j0 + r;
            if (j >= p.blocks_per_image) {
                const int32_t d = j / p.blocks_per_image;
                img += d;
                j -= d * p.blocks_per_image;
            }
            // The level: the table runs past the last level with blocks no
            // image has, so every entry can be compared.
            int lv = 0;
#pragma unroll
            for (int i = 1; i < PIC_MAX_LEVELS; ++i)
                lv += j >= p.first[i] ? 1 : 0;
            const int4 geo = s_geo[lv];
            float *base = s_lat[lv];
            // q / pw as (q * ceil(2^k / pw)) >> k, k = 24 + ceil(log2 pw): exact
            // for q < 2^24 (the handle refuses larger levels)
            const uint32_t q = (uint32_t)(j - s_first[lv]);
            const int32_t pwl = geo.z & 0xffff, sh = geo.z >> 16;
            const int32_t py = (int32_t)(((uint64_t)q * (uint32_t)geo.w) >> sh);
            const int32_t px = (int32_t)q - py * pwl;
            const int32_t col = px * 8 + gl;
            float *dst = base + ((int64_t)img * geo.x + py * 8) * geo.y + col;
            if (py * 8 + 8 <= geo.x && px * 8 + 8 <= geo.y) {      // whole patch inside the grid
#pragma unroll
                for (int y = 0; y < 8; ++y)
                    dst[(int64_t)y * geo.y] = Z[y];
            } else if (col < geo.y) {
#pragma unroll
                for (int y = 0; y < 8; ++y)
                    if (py * 8 + y < geo.x)
                        dst[(int64_t)y * geo.y] = Z[y];
            }
        }
    }

    if (err)
        atomicOr(&s_err, err);
    __syncthreads();
    if (t == 0 && s_err)
        atomicOr(p.status, s_err);
}

}  // namespace

template <int CH>
hipError_t launch_chunk(const ZprParams &p, bool coeff_only, hipStream_t s)
{
    const dim3 grid((unsigned)p.nchunks), block(kZprThreads);
    hipLaunchKernelGGL(k_zpr_count<CH>, grid, block, 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    if (p.counts_are_prefix) {
        hipLaunchKernelGGL(k_zpr_scan, dim3(1), dim3(kScanThreads), 0, s, p);
        e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    if (coeff_only)
        hipLaunchKernelGGL((k_zpr_expand<CH, true>), grid, block, 0, s, p);
    else
        hipLaunchKernelGGL((k_zpr_expand<CH, false>), grid, block, 0, s, p);
    return hipGetLastError();
}

hipError_t launch_zpr(const ZprParams &p, bool coeff_only, hipStream_t s)
{
    if (p.nchunks < 1)
        return hipErrorInvalidValue;
    if (p.chunk == kZprChunkSmall)
        return launch_chunk<kZprChunkSmall>(p, coeff_only, s);
    if (p.chunk == kZprChunkLarge)
        return launch_chunk<kZprChunkLarge>(p, coeff_only, s);
    return hipErrorInvalidValue;
}

}  // namespace pic
