// Latent decoding from the ZpR symbol stream (PIC, Sec. 3.3 and Fig. 2;
// App. B, Alg. 1; Sec. 3.2 Eq. (6)-(7) for the patches and the DCT).
//
// Three kernels.  The stream is partitioned into chunks of 256 symbols (one
// per thread) or, for streams of 2^18 symbols and more, 1024 (four per
// thread, so the per-workgroup set-up is spread over more blocks):
//
//   k_zpr_count   counts each chunk's end-of-block markers.
//   k_zpr_scan    (one workgroup) turns the counts into their exclusive
//                 prefix -- the index of the first block whose marker lies in
//                 each chunk -- and writes the run's status word.  Together
//                 the two replace the copy_if of marker offsets that Alg. 1
//                 starts from: no offset array is built.
//   k_zpr_expand  stages its chunk (and the 68 symbols before it) in LDS,
//                 compacts the positions of its markers, and decodes every
//                 block whose marker it holds.  A block's symbols start after
//                 the previous marker, found in the chunk or, for the first
//                 block, within the 65 staged symbols before it (a block of
//                 64 symbols plus the preceding marker).  Eight lanes decode
//                 one block: each takes eight consecutive symbols, the lanes
//                 scan how many coefficients their symbols produce (Alg. 1's
//                 running offset; a DPP scan inside the 8-lane segment), and
//                 every literal is scattered through the zigzag table into a
//                 zeroed 8x8 tile in LDS.  The tile then goes through the
//                 separable inverse DCT: each lane transforms one row, the
//                 rows go through LDS once to be read back as columns, and
//                 each lane transforms one column and writes it to the
//                 block's patch of the latent grid, cropped at the grid's
//                 edge.  The basis entries are compile-time constants.
//
// Memory traffic per block: its symbols (read by the count and the expand
// kernels) and its 64 samples written once; the HBM floor is the stream read
// once and the pyramid written once.
#include "pic_internal.h"
#include "pic_zpr.h"

namespace pic {
namespace {

constexpr int kWaves = kZprThreads / 64;
constexpr int kHalo = 68;                    // >= 65 symbols before the chunk
constexpr int kGroups = kZprThreads / 8;     // blocks in flight per workgroup (8 lanes each)
constexpr int kTile = 64 + 4;                // LDS words per 8x8 tile: the pad spreads the
                                             // groups' tiles over different banks

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
    __syncthreads();   // s_wsum may be reused by the caller
    *total = tot;
    return off + incl;
}

template <int CH>
__global__ __launch_bounds__(kZprThreads) void k_zpr_count(ZprParams p)
{
    constexpr int SPT = CH / kZprThreads;
    __shared__ int32_t s_wsum[kWaves];
    const int t = threadIdx.x;
    const int64_t cs = (int64_t)blockIdx.x * CH;
    int32_t mine = 0;
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        const int64_t i = cs + j * kZprThreads + t;
        mine += (i < p.n && p.sym[i] == p.eob) ? 1 : 0;
    }
    int32_t tot;
    (void)block_inclusive_sum(mine, s_wsum, &tot);
    if (t == 0)
        p.counts[blockIdx.x] = tot;
}

// One workgroup: counts[] -> exclusive prefix in place, and the status word.
// Segments of kScanSeg counts are staged in LDS with coalesced loads; each
// thread scans kScanPer consecutive entries, the workgroup scans the
// per-thread sums, and the segment is written back coalesced.
constexpr int kScanThreads = 1024;
constexpr int kScanPer = 16;
constexpr int kScanSeg = kScanThreads * kScanPer;

__global__ __launch_bounds__(kScanThreads) void k_zpr_scan(ZprParams p)
{
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
        int32_t incl = sum;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t o = __shfl_up(incl, d, 64);
            if (lane >= d)
                incl += o;
        }
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
    if (t == 0) {
        int32_t st = carry != p.expected ? PIC_ZPR_ERR_COUNT : 0;
        if (p.n > 0 && p.sym[p.n - 1] != p.eob)
            st |= PIC_ZPR_ERR_COUNT;
        *p.status = st;
    }
}

// Inclusive sum over the 8-lane segment of x (lane gl = threadIdx.x & 7 of
// its segment), with DPP row shifts: no LDS round trip.  row_shr:n reads the
// lane n below within the 16-lane row; the gl >= n test drops what crosses
// into the neighbouring segment.
__device__ __forceinline__ int seg8_inclusive_sum(int x, int gl)
{
    int y = __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
    x += gl >= 1 ? y : 0;
    y = __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);       // row_shr:2
    x += gl >= 2 ? y : 0;
    y = __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);       // row_shr:4
    x += gl >= 4 ? y : 0;
    return x;
}

template <int CH, bool COEFF>
__global__ __launch_bounds__(kZprThreads) void k_zpr_expand(ZprParams p)
{
    constexpr int SPT = CH / kZprThreads;
    __shared__ int32_t s_sym[kHalo + CH];
    __shared__ int32_t s_pos[CH + 1];             // [0]: marker before the first block; [1 + r]: r-th marker
    __shared__ __attribute__((aligned(16))) float s_blk[kGroups * kTile];   // S, then T in place
    __shared__ uint8_t s_zz[64];
    __shared__ int4 s_geo[PIC_MAX_LEVELS];        // stream level i: {h, w, patches per row, 0}
    __shared__ float *s_lat[PIC_MAX_LEVELS];
    __shared__ int32_t s_wsum[kWaves];
    __shared__ int32_t s_err;

    const int t = threadIdx.x, lane = t & 63;
    const int64_t cs = (int64_t)blockIdx.x * CH;
    const int32_t eob = p.eob;

    // Stage the chunk and the symbols before it.  Positions before the stream
    // act as markers (the first block starts at 0); positions past its end
    // are never markers and never inside a block.
    for (int i = t; i < kHalo + CH; i += kZprThreads) {
        const int64_t gi = cs - kHalo + i;
        s_sym[i] = gi < 0 ? eob : (gi < p.n ? p.sym[gi] : 0);
    }
    if (t < 64)
        s_zz[t] = kZigzag[t];
    if (!COEFF && t < p.L) {
        s_geo[t] = make_int4(p.hk[t], p.wk[t], p.pw[t], 0);
        s_lat[t] = p.lat[t];
    }
    if (t == 0)
        s_err = 0;
    __syncthreads();

    // Compact the chunk's marker positions (staged index) in stream order;
    // thread t looks at the SPT consecutive symbols from t * SPT.
    int32_t flags = 0, nm = 0;
#pragma unroll
    for (int j = 0; j < SPT; ++j) {
        const int k = t * SPT + j;
        const bool mk = cs + k < p.n && s_sym[kHalo + k] == eob;
        flags |= mk ? 1 << j : 0;
        nm += mk ? 1 : 0;
    }
    int32_t m;
    int32_t at = block_inclusive_sum(nm, s_wsum, &m) - nm;
#pragma unroll
    for (int j = 0; j < SPT; ++j)
        if (flags & (1 << j))
            s_pos[1 + at++] = kHalo + t * SPT + j;
    __syncthreads();
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
            s_pos[0] = prev;
    }
    __syncthreads();

    // Eight lanes per block: lane gl holds symbols 8 gl .. 8 gl + 7 of it and,
    // in the transform, row gl of the tile.
    const int grp = t >> 3, gl = t & 7;
    float *blk = s_blk + grp * kTile;
    float *tmp = blk;   // row gl of T replaces row gl of S, which only lane gl reads
    const int32_t g0 = p.counts[blockIdx.x];        // blocks whose markers precede the chunk
    const int32_t img0 = g0 / p.blocks_per_image;
    const int32_t j0 = g0 - img0 * p.blocks_per_image;
    int err = 0;
    for (int r0 = 0; r0 < m; r0 += kGroups) {
        const int r = r0 + grp;
        const int32_t g = g0 + r;
        if (r >= m || g >= p.expected)               // uniform over the 8 lanes of a block
            continue;
        const int end = s_pos[1 + r];
        int begin = s_pos[r] + 1;
        if (end - begin > 64) {
            err |= PIC_ZPR_ERR_OVERFLOW;
            begin = end - 64;
        }
        // Alg. 1 on this lane's eight symbols: coefficients each produces.
        int32_t sv[8];
        int cnt[8];
        int tot = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int idx = begin + 8 * gl + e;
            const bool in = idx < end;
            const int32_t s = in ? s_sym[idx] : 0;
            const bool over = in && s > eob;
            const bool run = in && !over && s >= eob - 16;
            const bool lit = in && s < eob - 16;
            cnt[e] = run ? s - eob + 17 : (lit ? 1 : 0);
            sv[e] = lit ? s : 0;                       // runs and padding write nothing
            err |= over ? PIC_ZPR_ERR_SYMBOL : 0;
            tot += cnt[e];
        }
        const int incl = seg8_inclusive_sum(tot, gl);
        if (gl == 7 && incl > 64)
            err |= PIC_ZPR_ERR_OVERFLOW;
        int pos = incl - tot;

        reinterpret_cast<float4 *>(blk)[2 * gl] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        reinterpret_cast<float4 *>(blk)[2 * gl + 1] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        asm volatile("" ::: "memory");
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if (sv[e] != 0 && pos < 64) {
                if (COEFF)
                    reinterpret_cast<int32_t *>(blk)[s_zz[pos]] = sv[e];
                else
                    blk[s_zz[pos]] = (float)sv[e];
            }
            pos += cnt[e];
        }
        asm volatile("" ::: "memory");

        if (COEFF) {
            const int4 *src = reinterpret_cast<const int4 *>(blk);
            int4 *dst = reinterpret_cast<int4 *>(p.coeffs + (int64_t)g * 64);
            dst[2 * gl] = src[2 * gl];
            dst[2 * gl + 1] = src[2 * gl + 1];
            continue;
        }

        // Rows: lane gl transforms row u = gl of S,
        //   T[u][x] = sum_v S[u][v] a(v) cos((2x + 1) v pi / 16),
        // and stores it; then it reads back column x = gl of T (the LDS
        // transpose) and transforms it,
        //   Z[y][x] = sum_u a(u) cos((2y + 1) u pi / 16) T[u][x].
        const float4 sa = reinterpret_cast<const float4 *>(blk + gl * 8)[0];
        const float4 sb = reinterpret_cast<const float4 *>(blk + gl * 8)[1];
        const float S[8] = {sa.x, sa.y, sa.z, sa.w, sb.x, sb.y, sb.z, sb.w};
        float T[8];
#pragma unroll
        for (int x = 0; x < 8; ++x) {
            float acc = S[0] * dct_basis(x, 0);
#pragma unroll
            for (int v = 1; v < 8; ++v)
                acc = __builtin_fmaf(S[v], dct_basis(x, v), acc);
            T[x] = acc;
        }
        reinterpret_cast<float4 *>(tmp + gl * 8)[0] = make_float4(T[0], T[1], T[2], T[3]);
        reinterpret_cast<float4 *>(tmp + gl * 8)[1] = make_float4(T[4], T[5], T[6], T[7]);
        asm volatile("" ::: "memory");
        float C[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            C[u] = tmp[u * 8 + gl];
        float Z[8];
#pragma unroll
        for (int y = 0; y < 8; ++y) {
            float acc = C[0] * dct_basis(y, 0);
#pragma unroll
            for (int u = 1; u < 8; ++u)
                acc = __builtin_fmaf(C[u], dct_basis(y, u), acc);
            Z[y] = acc;
        }
        asm volatile("" ::: "memory");

        // Un-patchify: image, level (stream order, found against the uniform
        // first-block table), patch; lane gl writes column gl of the patch.
        int32_t img = img0, j = j0 + r;
        if (j >= p.blocks_per_image) {
            const int32_t d = j / p.blocks_per_image;
            img += d;
            j -= d * p.blocks_per_image;
        }
        int lv = 0;
#pragma unroll
        for (int i = 1; i < PIC_MAX_LEVELS; ++i)
            lv += (i < p.L && j >= p.first[i]) ? 1 : 0;
        const int4 geo = s_geo[lv];               // {h, w, patches per row, -}
        float *base = s_lat[lv];
        int32_t fl = 0;
#pragma unroll
        for (int i = 0; i < PIC_MAX_LEVELS; ++i)
            fl = i == lv ? p.first[i] : fl;
        const int32_t q = j - fl;
        const int32_t py = q / geo.z, px = q - py * geo.z;
        const int32_t col = px * 8 + gl;
        if (col < geo.y) {
            float *dst = base + ((int64_t)img * geo.x + py * 8) * geo.y + col;
#pragma unroll
            for (int y = 0; y < 8; ++y)
                if (py * 8 + y < geo.x)
                    dst[(int64_t)y * geo.y] = Z[y];
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
    hipLaunchKernelGGL(k_zpr_scan, dim3(1), dim3(kScanThreads), 0, s, p);
    e = hipGetLastError();
    if (e != hipSuccess || p.n == 0)
        return e;
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
