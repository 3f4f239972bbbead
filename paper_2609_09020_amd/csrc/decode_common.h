// Device pieces shared by the matrix-core decode kernels: tile geometry, the
// LDS latent boxes, the bilinear upsample from them, the cross-lane sums of
// the output layer and the epilogue.
//
// The upsample (PIC, Sec. 3.1): level k of an H x W image is a grid of
// ceil(H / 2^k) x ceil(W / 2^k) samples; output pixel (y, x) samples it at
// source coordinate max((y + 1/2) 2^-k - 1/2, 0) (and likewise for x), from
// the two neighbouring samples of each axis, the upper one clamped to the
// grid (edge replication).
#pragma once

#include <utility>

#include "pic_internal.h"

namespace pic {
namespace tile {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int TH = 8;    // tile rows (two per wavefront)
constexpr int TWG = 4;   // 16-pixel column groups per tile row
constexpr int TW = 16 * TWG;   // tile columns

// Latent box staged per level for one tile.  A tile's pixels o0 .. o1 along
// an axis sample source indices floor(src(o0)) .. floor(src(o1)) + 1, at most
// ceil((n - 1) / 2^k) + 2 of them; the box holds that many (rounded up by one)
// starting at floor(src(o0)).  Indices past the grid are staged as the grid's
// last sample, which is exactly the edge replication of the upsample, so every
// pixel's second tap is at +1 (column) and +pitch (row).
// THT: tile rows (TH, or 16 for the kernels that take taller tiles).
__host__ __device__ constexpr int box_dim(int n, int k) { return ((n - 1 + (1 << k) - 1) >> k) + 3; }
__host__ __device__ constexpr int box_pitch(int k) { return box_dim(TW, k); }
template <int THT = TH>
__host__ __device__ constexpr int box_rows(int k) { return box_dim(THT, k); }
template <int THT = TH>
__host__ __device__ constexpr int box_floats(int k) { return box_rows<THT>(k) * box_pitch(k); }
template <int THT = TH>
__host__ __device__ constexpr int box_offset(int k)
{
    return k == 0 ? 0 : box_offset<THT>(k - 1) + box_floats<THT>(k - 1);
}

__device__ __forceinline__ float pow2_neg(int k) { return __int_as_float((127 - k) << 23); }

// floor of the clamped source coordinate max((o + 1/2) 2^-k - 1/2, 0), which is
// (2 o + 1 - 2^k) / 2^(k+1): the arithmetic shift floors it, exactly.
__host__ __device__ constexpr int src_floor(int o, int k)
{
    return (2 * o + 1 - (1 << k)) >> (k + 1) > 0 ? (2 * o + 1 - (1 << k)) >> (k + 1) : 0;
}

// Image b's copy of latent level k: b hk wk texels past image 0's (hk wk <
// 2^31, so a 32 x 32-bit product)
__device__ __forceinline__ const float *level_base(const DecodeParams &p, int k, int b)
{
    return p.lat[k] + (uint64_t)(uint32_t)b * (uint32_t)(p.hk[k] * p.wk[k]);
}

// Image b's copy of layer l's parameters (wave-uniform pointers).
struct LayerParams {
    const void *w;    // [out][in], fp32 or bf16
    const float *b;   // [out]
    bool bf16;
    __device__ __forceinline__ float weight(int idx) const
    {
        if (bf16)
            return __uint_as_float((uint32_t) static_cast<const uint16_t *>(w)[idx] << 16);
        return static_cast<const float *>(w)[idx];
    }
    __device__ __forceinline__ unsigned bits(int idx) const { return static_cast<const uint16_t *>(w)[idx]; }
    // Entry min(idx, n - 1) (n >= 1) of the weights, known to be bf16 (BF16)
    // or fp32, and of the bias: a raw copy whose entries past n are never
    // read, loaded without a branch or a select, so that nothing waits for
    // the loads before they are stored
    template <bool BF16>
    __device__ __forceinline__ float weight_clamped(int idx, int n) const
    {
        const int i = idx < n ? idx : n - 1;
        return BF16 ? __uint_as_float((uint32_t) static_cast<const uint16_t *>(w)[i] << 16)
                    : static_cast<const float *>(w)[i];
    }
    __device__ __forceinline__ float bias_clamped(int idx, int n) const { return b[idx < n ? idx : n - 1]; }
};

__device__ __forceinline__ LayerParams layer_params(const DecodeParams &p, int l, int b)
{
    LayerParams lp;
    lp.w = p.wl[l];
    lp.b = p.bl[l];
    lp.bf16 = p.weights_bf16 != 0;
    if (b != 0) {   // (uniform) image 0, the one-image case, needs no offsets
        lp.w = static_cast<const char *>(lp.w) + (int64_t)b * p.wls[l] * (p.weights_bf16 ? 2 : 4);
        lp.b += (int64_t)b * p.bls[l];
    }
    return lp;
}

// Parameter staging in two phases, so that every global load of a workgroup's
// prologue is in flight before the first one is waited for: load_part reads
// entries threadIdx.x, + kThreads, ... of a COUNT-entry table into registers,
// store_part writes them to LDS.
template <int COUNT, class T>
struct Part {
    static constexpr int kPer = (COUNT + kThreads - 1) / kThreads;
    T v[kPer];
};

template <int COUNT, class T, class F>
__device__ __forceinline__ Part<COUNT, T> load_part(F value)
{
    Part<COUNT, T> r;
#pragma unroll
    for (int i = 0; i < Part<COUNT, T>::kPer; ++i) {
        const int s = (int)threadIdx.x + i * kThreads;
        // (in a last, partial round, threads past the table evaluate its last
        // entry, which store_part does not store: no branch, so nothing waits
        // for the round's loads here)
        r.v[i] = value(s < COUNT ? s : COUNT - 1);
    }
    return r;
}

// base[idx] if ok, else 0, without a branch: an entry that holds nothing
// reads base[0] and discards it, so that the LDS reads of every entry a
// thread gathers can be in flight together.
__device__ __forceinline__ float lds_or_zero(const float *base, bool ok, int idx)
{
    const float v = base[ok ? idx : 0];
    return ok ? v : 0.0f;
}

template <int COUNT, class T>
__device__ __forceinline__ void store_part(T *dst, const Part<COUNT, T> &r)
{
#pragma unroll
    for (int i = 0; i < Part<COUNT, T>::kPer; ++i) {
        const int s = (int)threadIdx.x + i * kThreads;
        if (s < COUNT)
            dst[s] = r.v[i];
    }
}

// Tile schedule of a workgroup.  Its first tile is static; when the grid has
// fewer workgroups than tiles, the others come from a counter: the next tile
// is base + (the counter's old value), while that is below end.
// Workgroups are dealt to the 8 XCDs in turn (workgroup i to XCD i mod 8),
// and each XCD has its own L2.  In a one-image grid (of a multiple of 8
// workgroups) XCD x therefore takes the contiguous tile range
// [x tiles / 8, (x + 1) tiles / 8) with a counter of its own, so that the halo
// rows and columns two neighbouring tiles share are read into one L2.
// Other grids keep the plain order and one counter per image (batches of a
// multiple of 8 images keep each image on one XCD anyway, since images
// interleave over the grid).
struct TileSchedule {
    int first;
    int *ctr;
    int base, end;
};

__device__ __forceinline__ TileSchedule tile_schedule(const DecodeParams &p, int block, int bpi, int tiles)
{
    TileSchedule ts;
    if (p.batch == 1 && (unsigned)bpi % kXcds == 0) {
        // unsigned 32-bit arithmetic (tiles < 2^23, so 8 tiles < 2^32)
        const unsigned x = (unsigned)block % kXcds, t = (unsigned)tiles;
        const int r0 = (int)(t * x / kXcds);
        ts.first = r0 + (int)((unsigned)block / kXcds);
        ts.ctr = p.tile_ctr + x;
        ts.base = r0 + (int)((unsigned)bpi / kXcds);
        ts.end = (int)(t * (x + 1) / kXcds);
    } else {
        const int b = block % p.batch;
        ts.first = block / p.batch;
        ts.ctr = p.tile_ctr + b;
        ts.base = bpi;
        ts.end = tiles;
    }
    return ts;
}

// max(x, 0) for a non-NaN float as one integer max: non-negative floats order
// like their bit patterns, negative ones (sign bit set) are negative integers.
__device__ __forceinline__ float relu(float x) { return __int_as_float(max(__float_as_int(x), 0)); }

// Sum of x over the four 16-lane rows of the wavefront, in every lane:
// permlane16_swap pairs rows (0,1) and (2,3), permlane32_swap pairs the halves;
// the two outputs of each swap hold both members of the pair.
__device__ __forceinline__ float row_sum(float x)
{
    const unsigned xi = __float_as_uint(x);
    const u32x2 a = __builtin_amdgcn_permlane16_swap(xi, xi, false, false);
    const float s = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const unsigned si = __float_as_uint(s);
    const u32x2 c = __builtin_amdgcn_permlane32_swap(si, si, false, false);
    return __uint_as_float(c[0]) + __uint_as_float(c[1]);
}

// Lane-group sums of three per-lane partials, transposed: lane group g (< 3)
// receives the sum over all four lane groups of partial g.  permlane16_swap
// exchanges the odd rows of its first operand with the even rows of its
// second; permlane32_swap exchanges the upper half of its first operand with
// the lower half of its second.
//   swap16(o0, o1), add  -> rows hold [o0 01, o1 01, o0 23, o1 23] (pair sums)
//   swap16(o2, 0), add   -> rows hold [o2 01, 0,     o2 23, 0    ]
//   swap32(first, second), add -> rows hold [o0, o1, o2, 0] (totals)
__device__ __forceinline__ float row_sum3(float o0, float o1, float o2)
{
    const u32x2 a = __builtin_amdgcn_permlane16_swap(__float_as_uint(o0), __float_as_uint(o1), false, false);
    const float s = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const u32x2 c = __builtin_amdgcn_permlane16_swap(__float_as_uint(o2), 0u, false, false);
    const float t = __uint_as_float(c[0]) + __uint_as_float(c[1]);
    const u32x2 e = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(t), false, false);
    return __uint_as_float(e[0]) + __uint_as_float(e[1]);
}

// A raw buffer over the n_bytes at p: the hardware's range check returns 0
// for a load at a byte offset past n_bytes.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_buffer(const void *p, unsigned n_bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)n_bytes, 0x00020000);
}

// Index of texel (r, c) in a level with wk columns.  Image sides are below
// 2^23 and images below 2^31 pixels (the descriptor's limits), so r and wk
// fit the unsigned 24-bit multiplier and r * wk + c < 2^31: one full-rate
// multiply-add and one 64-bit address add, where 64-bit index arithmetic
// takes a quarter-rate multiply and two adds.
__device__ __forceinline__ uint32_t texel(int r, int wk, int c)
{
    return __umul24((uint32_t)r, (uint32_t)wk) + (uint32_t)c;
}

// Row of tile t in a grid tiles_x tiles wide, t / tiles_x, as the high half of
// t m for the host's m = ceil(2^32 / tiles_x) = (2^32 + e) / tiles_x, 0 <= e <
// tiles_x: t m / 2^32 exceeds t / tiles_x by t e / (tiles_x 2^32), which stays
// below 1 / tiles_x, so the floor is the quotient, while t tiles_x < 2^32.  The
// host passes m = 0 where that does not hold for every tile of the launch (and
// for tiles_x = 1), and the division runs instead.
__device__ __forceinline__ int tile_row(int t, int tiles_x, uint32_t m)
{
    if (m)
        return (int)__umulhi((uint32_t)t, m);
    asm volatile("" : "+s"(tiles_x));   // (keeps the division's set-up on this path)
    return t / tiles_x;
}

// Box staging in a load phase (into registers) and a store phase, so that
// every load is in flight before the first is waited for (and, in the
// prologue, while the parameter loads are).  box_regs<KMAX>() registers per
// thread; levels past L load level 0 (into boxes no lane samples).
template <int THT>
__host__ __device__ constexpr int box_regs_from(int k, int kmax)
{
    return k >= kmax ? 0 : (box_floats<THT>(k) + kThreads - 1) / kThreads + box_regs_from<THT>(k + 1, kmax);
}
template <int KMAX, int THT = TH>
__host__ __device__ constexpr int box_regs() { return box_regs_from<THT>(0, KMAX); }

template <int KMAX, int THT = TH>
__device__ __forceinline__ void load_boxes(float (&v)[(box_regs<KMAX, THT>())], const DecodeParams &p, int b, int ty0,
                                           int tx0, int tid, int z = 0)
{
    // image b's copies of the levels (one uniform branch: image 0, the
    // one-image case, skips the offsets)
    const float *src0[KMAX];
#pragma unroll
    for (int k = 0; k < KMAX; ++k)
        src0[k] = p.lat[k + z];
    if (b != 0) {
#pragma unroll
        for (int k = 0; k < KMAX; ++k)
            src0[k] = level_base(p, k + z, b);
    }
    int idx = 0;
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
        // levels past L load level 0 (their slots repeat it; never stored)
        const int hk = p.hk[k + z], wk = p.wk[k + z];
        const int ry = src_floor(ty0, k), rx = src_floor(tx0, k);
        const float *src = src0[k];
        const int n = box_floats<THT>(k), pc = box_pitch(k);
#pragma unroll
        for (int i0 = 0; i0 < n; i0 += kThreads) {
            const int i = min(i0 + tid, n - 1);
            const int r = min(ry + i / pc, hk - 1), c = min(rx + i % pc, wk - 1);
            v[idx++] = src[texel(r, wk, c)];
        }
    }
}

// Every store is unconditional: levels past L (whose loads repeat level 0)
// go to boxes no lane samples, and the threads past a box's last entry,
// which loaded that entry, write it again with the value it holds.
template <int KMAX, int THT = TH>
__device__ __forceinline__ void store_boxes(float *lat, const float (&v)[(box_regs<KMAX, THT>())], int tid)
{
    int idx = 0;
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
        const int n = box_floats<THT>(k);
#pragma unroll
        for (int i0 = 0; i0 < n; i0 += kThreads) {
            const int i = i0 + kThreads <= n ? i0 + tid : min(i0 + tid, n - 1);
            lat[box_offset<THT>(k) + i] = v[idx++];
        }
    }
}

// Stage the boxes of levels 0 .. KMAX - 1 of image b for the tile at (ty0,
// tx0) into lat (box k at lat + box_offset(k); those past L repeat level 0
// and are not sampled); all threads take part.  Every load is issued before the first store, so a tile waits for one
// memory round trip, not one per level.  The thread's box indices and the
// levels' geometry are derived here, per tile.
template <int KMAX, int THT = TH>
__device__ __forceinline__ void stage_boxes(float *lat, const DecodeParams &p, int b, int ty0, int tx0, int tid)
{
    // (the levels are indexed with an opaque zero added, so that nothing
    // derived from their geometry is hoisted into the prologue either, which
    // one-tile launches would pay for without staging a second tile)
    int z = 0;
    asm volatile("" : "+s"(z), "+v"(tid));
    float v[box_regs<KMAX, THT>()];
    load_boxes<KMAX, THT>(v, p, b, ty0, tx0, tid, z);
    store_boxes<KMAX, THT>(lat, v, tid);
}

// One lane's view of one level for the current tile: where its box starts in
// LDS, its pitch, and the horizontal tap offsets / weights of the tile's four
// 16-pixel column groups.
struct LaneLevel {
    float inv;        // 2^-k
    int loff;         // LDS offset of the level's box (floats)
    int pitch;        // box row pitch (floats)
    int rbase;        // first source row of the box
    int coff[TWG];    // loff + first-tap column - first box column, per column group
    float clx[TWG];   // horizontal lerp weight, per column group
};

// Lane group g samples level K0 + KS g (level 0 where that level does not
// exist: its first-layer weights are zero).  The four lane groups' box
// offsets (16 bits each) and pitches (8 bits each) are packed into
// compile-time constants and picked by shifts: no loop over the levels
// below, no multiply, no branch.
template <int THT, int K0, int KS>
__device__ __forceinline__ void lane_level_init(LaneLevel &lv, int g, int L, int lat_base)
{
    constexpr int K3 = K0 + 3 * KS;
    static_assert(box_offset<THT>(K3) < 65536 && box_pitch(0) < 256, "packed box geometry");
    constexpr uint32_t off01 = (uint32_t)box_offset<THT>(K0) | (uint32_t)box_offset<THT>(K0 + KS) << 16;
    constexpr uint32_t off23 = (uint32_t)box_offset<THT>(K0 + 2 * KS) | (uint32_t)box_offset<THT>(K3) << 16;
    constexpr uint32_t pitches = (uint32_t)box_pitch(K0) | (uint32_t)box_pitch(K0 + KS) << 8 |
                                 (uint32_t)box_pitch(K0 + 2 * KS) << 16 | (uint32_t)box_pitch(K3) << 24;
    const int k = K0 + KS * g;
    const bool ok = k < L;
    const int off = (int)(((g < 2 ? off01 : off23) >> (16 * (g & 1))) & 0xffff);
    const int pitch = (int)((pitches >> (8 * g)) & 0xff);
    lv.inv = pow2_neg(ok ? k : 0);
    lv.loff = lat_base + (ok ? off : 0);
    lv.pitch = ok ? pitch : box_pitch(0);
}

// lv[s] for lane group g's level A s + KS g, s < N (N = sizeof...(S)).
template <int THT, int A, int KS, int... S>
__device__ __forceinline__ void lane_levels_init(LaneLevel (&lv)[sizeof...(S)], int g, int L, int lat_base,
                                                 std::integer_sequence<int, S...>)
{
    (lane_level_init<THT, A * S, KS>(lv[S], g, L, lat_base), ...);
}

__device__ __forceinline__ void lane_level_tile(LaneLevel &lv, int ty0, int tx0, int tx1, int col)
{
    const int k = 127 - (__float_as_int(lv.inv) >> 23);   // lv.inv = 2^-k
    const int rx = src_floor(tx0, k);
    lv.rbase = src_floor(ty0, k);
#pragma unroll
    for (int cg = 0; cg < TWG; ++cg) {
        const int x = min(tx0 + 16 * cg + col, tx1);
        const float sx = fmaxf(((float)x + 0.5f) * lv.inv - 0.5f, 0.0f);
        const int x0 = (int)sx;
        lv.clx[cg] = sx - (float)x0;
        lv.coff[cg] = lv.loff + x0 - rx;
    }
}

// Vertical part for output row y: box row offset of the first tap and weight.
__device__ __forceinline__ void lane_level_row(const LaneLevel &lv, int y, int &roff, float &ly)
{
    const float sy = fmaxf(((float)y + 0.5f) * lv.inv - 0.5f, 0.0f);
    const int y0 = (int)sy;
    ly = sy - (float)y0;
    roff = (y0 - lv.rbase) * lv.pitch;
}

// Bilinear sample from the box: taps at +0, +1, +pitch, +pitch+1.
__device__ __forceinline__ float lane_level_sample(const float *lds, const LaneLevel &lv, int roff, float ly, int cg)
{
    const float *q0 = lds + roff + lv.coff[cg];
    const float *q1 = q0 + lv.pitch;
    const float a = q0[0], b = q0[1], c = q1[0], d = q1[1];
    const float lx = lv.clx[cg];
    const float top = __builtin_fmaf(lx, b - a, a);
    const float bot = __builtin_fmaf(lx, d - c, c);
    return __builtin_fmaf(ly, bot - top, top);
}

// Write one output value (lane group g < 3 writes channel g).
__device__ __forceinline__ void store_out(const DecodeParams &p, int64_t o, float v)
{
    if (p.out_kind == OUT_RAW_F32) {
        static_cast<float *>(p.out)[o] = v;
    } else {
        const float cl = fminf(fmaxf(v, 0.0f), 1.0f);
        if (p.out_kind == OUT_CLAMPED_F32)
            static_cast<float *>(p.out)[o] = cl;
        else
            static_cast<uint8_t *>(p.out)[o] = (uint8_t)(int)floorf(__builtin_fmaf(cl, 255.0f, 0.5f));
    }
}

// m for tile_row: ceil(2^32 / tiles_x) when t tiles_x < 2^32 for every tile
// index t < tiles and tiles_x > 1, else 0 (tile_row divides).
inline uint32_t tile_row_recip(int tiles_x, int tiles)
{
    if (tiles_x < 2 || (uint64_t)tiles * (uint64_t)tiles_x >= (1ULL << 32))
        return 0;
    return (uint32_t)(((1ULL << 32) + (uint64_t)tiles_x - 1) / (uint64_t)tiles_x);
}

// Grid size for a persistent kernel: as many workgroups as fit at once,
// split evenly over the images (at least one, at most one per tile).
template <typename K>
int blocks_per_image(K kernel, const DecodeParams &p, int num_cus, int tiles, int &occ_cache)
{
    if (occ_cache == 0) {
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kThreads, 0) != hipSuccess || n < 1)
            n = 2;
        occ_cache = n;
    }
    int bpi = (occ_cache * num_cus + p.batch - 1) / p.batch;
    return bpi < 1 ? 1 : (bpi > tiles ? tiles : bpi);
}

}  // namespace tile
}  // namespace pic
