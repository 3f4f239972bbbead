// Latent decoding from the ZpR symbol stream (PIC, Sec. 3.3 and Fig. 2;
// App. B, Alg. 1; Sec. 3.2 Eq. (6)-(7) for the patches and the DCT).
//
// Two kernels over the same partition of the stream into chunks of
// kZprChunk symbols, one symbol per thread:
//
//   k_zpr_count   counts each chunk's end-of-block markers.  The workgroup
//                 that finishes last (an arrival counter, no waiting) turns
//                 the counts into their exclusive prefix, i.e. the index of
//                 the first block whose marker lies in each chunk, and writes
//                 the run's status word.  This replaces the copy_if of marker
//                 offsets that Alg. 1 starts from: no offset array is built.
//   k_zpr_expand  stages its chunk (and the 68 symbols before it) in LDS,
//                 compacts the positions of its markers, and decodes every
//                 block whose marker it holds.  A block's symbols start after
//                 the previous marker, found in the chunk or, for the first
//                 block, within the 65 staged symbols before it (a block of
//                 64 symbols plus the preceding marker).  Sixteen lanes decode
//                 one block: each takes four consecutive symbols, the lanes
//                 scan how many coefficients their symbols produce (Alg. 1's
//                 running offset), and every literal is scattered through the
//                 zigzag table into a zeroed 8x8 tile in LDS.  The tile then
//                 goes through the separable inverse DCT (rows, then columns,
//                 four outputs per lane) and is written to its patch of the
//                 latent grid, cropped at the grid's edge.
//
// Memory traffic per block: its symbols (read twice, once per kernel) and its
// 64 samples written once; the HBM floor is the written pyramid.
#include "pic_internal.h"
#include "pic_zpr.h"

namespace pic {
namespace {

constexpr int kWaves = kZprThreads / 64;
constexpr int kHalo = 68;                    // >= 65 symbols before the chunk
constexpr int kGroups = kZprThreads / 16;    // blocks in flight per workgroup

// JPEG zigzag scan (ITU-T T.81, Fig. A.6): entry p is the row-major index of
// the p-th coefficient.
__constant__ uint8_t kZigzag[64] = {
    0,  1,  8,  16, 9,  2,  3,  10, 17, 24, 32, 25, 18, 11, 4,  5,
    12, 19, 26, 33, 40, 48, 41, 34, 27, 20, 13, 6,  7,  14, 21, 28,
    35, 42, 49, 56, 57, 50, 43, 36, 29, 22, 15, 23, 30, 37, 44, 51,
    58, 59, 52, 45, 38, 31, 39, 46, 53, 60, 61, 54, 47, 55, 62, 63};

__global__ __launch_bounds__(kZprThreads) void k_zpr_count(ZprParams p)
{
    __shared__ int32_t s_wcnt[kWaves];
    __shared__ int32_t s_last;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int c = blockIdx.x;
    const int64_t i = (int64_t)c * kZprChunk + t;

    const bool mark = i < p.n && p.sym[i] == p.eob;
    const uint64_t bal = __ballot(mark);
    if (lane == 0)
        s_wcnt[wave] = __popcll(bal);
    __syncthreads();
    if (t == 0) {
        int32_t tot = 0;
        for (int w = 0; w < kWaves; ++w)
            tot += s_wcnt[w];
        __hip_atomic_store(&p.counts[c], tot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint32_t before =
            __hip_atomic_fetch_add(p.ticket, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        s_last = before == (uint32_t)(p.nchunks - 1);
    }
    __syncthreads();
    if (!s_last)
        return;

    // Last workgroup: every count is published.  Exclusive prefix in place.
    __atomic_thread_fence(__ATOMIC_ACQUIRE);
    __shared__ int32_t s_wsum[kWaves];
    int32_t carry = 0;
    for (int base = 0; base < p.nchunks; base += kZprThreads) {
        const int j = base + t;
        const int32_t v =
            j < p.nchunks ? __hip_atomic_load(&p.counts[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
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
        int32_t off = carry, step = 0;
        for (int w = 0; w < kWaves; ++w) {
            off += w < wave ? s_wsum[w] : 0;
            step += s_wsum[w];
        }
        if (j < p.nchunks)
            __hip_atomic_store(&p.counts[j], off + incl - v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        carry += step;
        __syncthreads();   // s_wsum is rewritten by the next round
    }
    if (t == 0) {
        int32_t st = carry != p.expected ? PIC_ZPR_ERR_COUNT : 0;
        if (p.n > 0 && p.sym[p.n - 1] != p.eob)
            st |= PIC_ZPR_ERR_COUNT;
        *p.status = st;
        __hip_atomic_store(p.ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

template <bool COEFF>
__global__ __launch_bounds__(kZprThreads) void k_zpr_expand(ZprParams p)
{
    __shared__ int32_t s_sym[kHalo + kZprChunk];
    __shared__ int32_t s_pos[kZprChunk + 1];      // [0]: marker before the first block; [1 + r]: r-th marker
    __shared__ __attribute__((aligned(16))) float s_blk[kGroups * 64];
    __shared__ __attribute__((aligned(16))) float s_tmp[kGroups * 64];
    __shared__ float s_basis[64];                 // [a * 8 + b] = a(b) cos((2a + 1) b pi / 16)
    __shared__ uint8_t s_zz[64];
    __shared__ int32_t s_first[PIC_MAX_LEVELS + 1], s_hk[PIC_MAX_LEVELS], s_wk[PIC_MAX_LEVELS],
        s_pw[PIC_MAX_LEVELS];
    __shared__ float *s_lat[PIC_MAX_LEVELS];
    __shared__ int32_t s_wcnt[kWaves];
    __shared__ int32_t s_err;

    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int64_t cs = (int64_t)blockIdx.x * kZprChunk;
    const int32_t eob = p.eob;

    // Stage the chunk and the symbols before it.  Positions before the stream
    // act as markers (the first block starts at 0); positions past its end
    // are never markers and never inside a block.
    for (int i = t; i < kHalo + kZprChunk; i += kZprThreads) {
        const int64_t gi = cs - kHalo + i;
        s_sym[i] = gi < 0 ? eob : (gi < p.n ? p.sym[gi] : 0);
    }
    if (t < 64) {
        s_zz[t] = kZigzag[t];
        if (!COEFF) {
            const int a = t >> 3, b = t & 7;
            const double ab = b == 0 ? 0.35355339059327376220 : 0.5;   // sqrt(1/8), sqrt(2/8)
            s_basis[t] = (float)(ab * cos((double)((2 * a + 1) * b) * (3.14159265358979323846 / 16.0)));
        }
    }
    if (t == 0) {
        s_err = 0;
        if (!COEFF) {
            for (int i = 0; i < p.L; ++i) {
                s_first[i] = p.first[i];
                s_hk[i] = p.hk[i];
                s_wk[i] = p.wk[i];
                s_pw[i] = p.pw[i];
                s_lat[i] = p.lat[i];
            }
            s_first[p.L] = p.first[p.L];
        }
    }
    __syncthreads();

    // Compact the chunk's marker positions (staged index) in stream order.
    const bool mark = cs + t < p.n && s_sym[kHalo + t] == eob;
    const uint64_t bal = __ballot(mark);
    if (lane == 0)
        s_wcnt[wave] = __popcll(bal);
    __syncthreads();
    int before = 0, m = 0;
    for (int w = 0; w < kWaves; ++w) {
        before += w < wave ? s_wcnt[w] : 0;
        m += s_wcnt[w];
    }
    if (mark)
        s_pos[1 + before + __popcll(bal & ((1ull << lane) - 1))] = kHalo + t;
    __syncthreads();
    if (m == 0)
        return;   // uniform: no block ends in this chunk

    // The marker before the chunk's first block: the nearest of the 65
    // staged symbols before it; none means the block is too long (its last
    // 65 symbols are taken, which the length test below flags).
    if (wave == 0) {
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

    // Per-lane constants of the separable inverse DCT.
    const int grp = t >> 4, gl = t & 15;
    const int u = gl >> 1, x0 = (gl & 1) * 4;                 // tile row, first of 4 columns
    float b1[4][8], b2[8];
    __syncthreads();
    if (!COEFF) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int v = 0; v < 8; ++v)
                b1[e][v] = s_basis[(x0 + e) * 8 + v];
#pragma unroll
        for (int v = 0; v < 8; ++v)
            b2[v] = s_basis[u * 8 + v];
    }

    const int32_t g0 = p.counts[blockIdx.x];   // blocks whose markers precede the chunk
    float *blk = s_blk + grp * 64;
    float *tmp = s_tmp + grp * 64;
    int err = 0;
    for (int r0 = 0; r0 < m; r0 += kGroups) {
        const int r = r0 + grp;
        const int32_t g = g0 + r;
        if (r >= m || g >= p.expected)       // uniform over the 16 lanes of a block
            continue;
        const int end = s_pos[1 + r];
        int begin = s_pos[r] + 1;
        if (end - begin > 64) {
            err |= PIC_ZPR_ERR_OVERFLOW;
            begin = end - 64;
        }
        // Alg. 1 on this lane's four symbols: coefficients produced by each.
        int32_t sv[4];
        int cnt[4];
        bool lit[4];
        int tot = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int idx = begin + 4 * gl + e;
            const int32_t s = idx < end ? s_sym[idx] : 0;
            const bool in = idx < end;
            const bool over = in && s > eob;
            const bool run = in && !over && s >= eob - 16;
            lit[e] = in && s < eob - 16;
            cnt[e] = run ? s - eob + 17 : (lit[e] ? 1 : 0);
            sv[e] = s;
            err |= over ? PIC_ZPR_ERR_SYMBOL : 0;
            tot += cnt[e];
        }
        int incl = tot;
#pragma unroll
        for (int d = 1; d < 16; d <<= 1) {
            const int o = __shfl_up(incl, d, 16);
            if (gl >= d)
                incl += o;
        }
        if (__shfl(incl, 15, 16) > 64)
            err |= PIC_ZPR_ERR_OVERFLOW;
        int pos = incl - tot;

        reinterpret_cast<float4 *>(blk)[gl] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        asm volatile("" ::: "memory");
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (lit[e] && pos < 64) {
                if (COEFF)
                    reinterpret_cast<int32_t *>(blk)[s_zz[pos]] = sv[e];
                else
                    blk[s_zz[pos]] = (float)sv[e];
            }
            pos += cnt[e];
        }
        asm volatile("" ::: "memory");

        if (COEFF) {
            const int4 q = reinterpret_cast<const int4 *>(blk)[gl];
            reinterpret_cast<int4 *>(p.coeffs + (int64_t)g * 64)[gl] = q;
            continue;
        }

        // Rows: T[u][x] = sum_v S[u][v] a(v) cos((2x + 1) v pi / 16), x = x0 .. x0 + 3.
        const float4 sa = reinterpret_cast<const float4 *>(blk + u * 8)[0];
        const float4 sb = reinterpret_cast<const float4 *>(blk + u * 8)[1];
        const float S[8] = {sa.x, sa.y, sa.z, sa.w, sb.x, sb.y, sb.z, sb.w};
        float tv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float acc = 0.0f;
#pragma unroll
            for (int v = 0; v < 8; ++v)
                acc = __builtin_fmaf(S[v], b1[e][v], acc);
            tv[e] = acc;
        }
        reinterpret_cast<float4 *>(tmp + u * 8 + x0)[0] = make_float4(tv[0], tv[1], tv[2], tv[3]);
        asm volatile("" ::: "memory");
        // Columns: Z[y][x] = sum_u a(u) cos((2y + 1) u pi / 16) T[u][x], y = u (this lane's row).
        float z[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const float4 tt = reinterpret_cast<const float4 *>(tmp + k * 8 + x0)[0];
            z[0] = __builtin_fmaf(b2[k], tt.x, z[0]);
            z[1] = __builtin_fmaf(b2[k], tt.y, z[1]);
            z[2] = __builtin_fmaf(b2[k], tt.z, z[2]);
            z[3] = __builtin_fmaf(b2[k], tt.w, z[3]);
        }
        asm volatile("" ::: "memory");

        // Un-patchify: image, level (stream order), patch.
        const int32_t img = g / p.blocks_per_image;
        const int32_t j = g - img * p.blocks_per_image;
        int lv = 0;
        while (lv + 1 < p.L && j >= s_first[lv + 1])
            ++lv;
        const int32_t q = j - s_first[lv];
        const int32_t pwl = s_pw[lv];
        const int32_t py = q / pwl, px = q - py * pwl;
        const int32_t hk = s_hk[lv], wk = s_wk[lv];
        const int32_t row = py * 8 + u, col = px * 8 + x0;
        if (row < hk) {
            float *dst = s_lat[lv] + ((int64_t)img * hk + row) * wk + col;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (col + e < wk)
                    dst[e] = z[e];
        }
    }

    if (err)
        atomicOr(&s_err, err);
    __syncthreads();
    if (t == 0 && s_err)
        atomicOr(p.status, s_err);
}

}  // namespace

hipError_t launch_zpr(const ZprParams &p, bool coeff_only, hipStream_t s)
{
    if (p.nchunks < 1)
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)p.nchunks), block(kZprThreads);
    hipLaunchKernelGGL(k_zpr_count, grid, block, 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.n == 0)
        return e;
    if (coeff_only)
        hipLaunchKernelGGL(k_zpr_expand<true>, grid, block, 0, s, p);
    else
        hipLaunchKernelGGL(k_zpr_expand<false>, grid, block, 0, s, p);
    return hipGetLastError();
}

}  // namespace pic
