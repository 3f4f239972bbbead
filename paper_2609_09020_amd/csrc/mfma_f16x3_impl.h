// fp32 decode on the fp16 matrix cores (v_mfma_f32_16x16x32_f16), shared by
// the k_mfma_f16x3*.hip translation units that instantiate it.
//
// Same computation and tiling as the fp32 family (PIC, Sec. 3.1 and App. A;
// tiles, LDS boxes and upsample in decode_common.h): fp32 weights, fp32
// activations, binary32 accuracy.  Every product w * x that feeds a matrix
// core is formed from fp16 parts:
//
//   w = wh + wl + O(2^-22 |w|),  x = xh + xl + O(2^-22 |x|),
//   wh = fp16(w), wl = fp16(w - wh) (likewise x), all rounded to nearest,
//   w * x = wh * xh + wh * xl + wl * xh + O(2^-21 |w x|),
//
// with products of fp16 numbers exact in the fp32 accumulator.  The three
// partial products of one input are three K entries of the same dot product,
// so they cost K slots, not separate matrix operations.
//
// Scaling.  The low parts must stay normal fp16 numbers (the matrix cores
// drop subnormal inputs) and every part below the fp16 maximum.  So each
// layer's weights are scaled by the power of two that brings their largest
// magnitude into [2^14, 2^15), once per workgroup, and each pixel's inputs of
// a layer by the power of two that does the same for that pixel (a column of
// the B operand, so it scales only that pixel's column of the product).  The
// accumulator is then multiplied by the inverse powers of two and the bias
// added.  Scaling by powers of two is exact; an input smaller than the
// pixel's largest by more than 2^27 (a weight, than the layer's largest)
// loses low bits, an error below 2^-25 of the largest term.
//
// Matrix-core mapping (lane l, lane group g = l / 16, i = l % 16)
//   v_mfma_f32_16x16x32_f16 takes A[i][8g + j] and B[8g + j][i], j = 0..7,
//   from lane l and returns D[4g + r][i] in register r of lane l.  Row 4g + r
//   of output block ob holds neuron 16 ob + 4r + g, so lane group g holds the
//   neurons n = 4q + g, q = 4 ob + r: every lane group holds a quarter of any
//   width.  A lane group's next-layer K entries come from its own values
//   v_q, q < Q (Q = ceil(width / 4); for the first layer v_q is level 4q + g
//   of the lane's pixel): K slot pair p (two fp16 halves of one register) is
//     p < Q            (x_h, x_l) of v_p, against (w_h, w_h),
//     Q <= p < Q + T   (x_h of v_2t, x_h of v_2t+1), t = p - Q, against their w_l,
//   T = ceil(Q / 2); four pairs a K step, the rest zero.  The weights are
//   scaled, split and laid out to match once per workgroup.  The output
//   layer (3 neurons) runs in fp32 on the vector ALU.
#pragma once

#include "decode_common.h"

namespace pic {
namespace mfma_f16x3 {

using namespace tile;

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// K steps (32 entries) for Q values per lane group: Q (hi, lo) pairs and
// ceil(Q / 2) (hi, hi) pairs, four pairs a step.
__host__ __device__ constexpr int ksteps(int q) { return (q + (q + 1) / 2 + 3) / 4; }

template <int NB, int NH, int LS, int KSH, int THT>
struct Layout {
    static constexpr int S1 = ksteps(LS);                           // first-layer K steps
    static constexpr int SH = ksteps(KSH);                          // hidden-layer K steps
    static constexpr int W1A = 0;                                   // u32 [NB][S1][64][4]
    static constexpr int WHA = W1A + NB * S1 * 256;                 // u32 [NH][NB][SH][64][4]
    static constexpr int B1 = WHA + NH * NB * SH * 256;             // f32 [NB][64][4]
    static constexpr int BH = B1 + NB * 256;                        // f32 [NH][NB][64][4]
    static constexpr int W3 = BH + NH * NB * 256;                   // f32 [NB][4 r][4 g][4 c]
    static constexpr int WSC = W3 + NB * 64;                        // f32 [NH + 1][kWaves]: weight maxima
    static constexpr int LAT = WSC + (NH + 1) * kWaves;             // latent boxes
    static constexpr int SIZE = LAT + box_offset<THT>(4 * LS);
    // the parameters as the caller lays them out are first staged in the
    // regions their operand layouts then replace (each is large enough)
    static constexpr int N = 16 * NB;
    static_assert(N * 4 * LS <= NB * S1 * 256, "layer 1 fits its region");
    static_assert(N * N <= NB * SH * 256, "a hidden layer fits its region");
    static_assert(3 * N <= NB * 64, "output layer fits its region");
};

// Neuron on row `row` of an output block; the map is its own inverse.
__device__ __forceinline__ int row_neuron(int row) { return 4 * (row & 3) + (row >> 2); }

__device__ __forceinline__ unsigned pack_f16(float a, float b)
{
    return __builtin_bit_cast(unsigned, f16x2{(_Float16)a, (_Float16)b});
}


// The fp16 parts of w: (w_h, w_l).
__device__ __forceinline__ void split_weight(float w, float &h, float &l)
{
    const _Float16 wh = (_Float16)w;
    h = (float)wh;
    l = (float)(_Float16)(w - h);
}

// K entries of a layer's input: the lane group's values v_q, q < Q, times the
// power of two sc, as the B operand of ksteps(Q) matrix steps (slot pairs as
// in the header).  The scaling is exact, so h_q = fp16(sc v_q) and
// l_q = fp16(sc v_q - h_q), with sc v_q - h_q exact in fp32; each is one
// mixed-precision FMA (fp32 in, fp16 out).
template <int Q>
__device__ __forceinline__ void build_b(const float (&v)[Q], float sc, u32x4 (&b)[ksteps(Q)])
{
    constexpr int T = (Q + 1) / 2;
    unsigned reg[4 * ksteps(Q)];
#pragma unroll
    for (int q = 0; q < Q; ++q) {              // (hi, lo)
        const _Float16 hi = (_Float16)(v[q] * sc);
        const _Float16 lo = (_Float16)__builtin_fmaf(v[q], sc, -(float)hi);
        reg[q] = __builtin_bit_cast(unsigned, f16x2{hi, lo});
    }
#pragma unroll
    for (int t = 0; t < T; ++t)                // (hi, hi) pairs: the low halves of two (hi, lo) registers
        reg[Q + t] = __builtin_amdgcn_perm(2 * t + 1 < Q ? reg[2 * t + 1] : 0u, reg[2 * t], 0x05040100u);
#pragma unroll
    for (int k = Q + T; k < 4 * ksteps(Q); ++k)
        reg[k] = 0u;
#pragma unroll
    for (int s = 0; s < ksteps(Q); ++s)
        b[s] = u32x4{reg[4 * s], reg[4 * s + 1], reg[4 * s + 2], reg[4 * s + 3]};
}

// Register w of K step s of lane (g, i) of output block ob in the A layout:
// the packed fp16 weights that match build_b's slots.  `raw` is the layer's
// [out][in] matrix, Q the values per lane group (input neuron or level of
// value q: 4q + g).
template <int Q>
__device__ __forceinline__ unsigned a_entry(const float *raw, int fin, int fout, int ob, int s, int lane, int w,
                                            float wsc)
{
    // Branch-free, so that the reads of all entries a thread forms can be in
    // flight together: an entry that holds no weight reads raw[0] and
    // discards it.
    constexpr int T = (Q + 1) / 2;
    const int g = lane >> 4, out = 16 * ob + row_neuron(lane & 15);
    const int p = 4 * s + w;
    const bool pair = p >= Q;   // slots Q .. Q+T-1 hold the low parts of two inputs
    const int t = p - Q;
    const int in0 = pair ? 4 * (2 * t) + g : 4 * p + g;
    const int in1 = 4 * (2 * t + 1) + g;
    const bool live = out < fout && p < Q + T;
    const bool ok0 = live && in0 < fin;
    const bool ok1 = live && pair && 2 * t + 1 < Q && in1 < fin;
    const float x0 = raw[ok0 ? out * fin + in0 : 0] * wsc;
    const float x1 = raw[ok1 ? out * fin + in1 : 0] * wsc;
    float hi0, lo0, hi1, lo1;
    split_weight(x0, hi0, lo0);
    split_weight(x1, hi1, lo1);
    const float h0 = ok0 ? (pair ? lo0 : hi0) : 0.0f;
    const float h1 = pair ? (ok1 ? lo1 : 0.0f) : h0;
    return pack_f16(h0, h1);
}

__device__ __forceinline__ f16x8 as_f16x8(u32x4 v) { return __builtin_bit_cast(f16x8, v); }

// The power of two that brings m (>= 0) into [2^14, 2^15), at most 2^63 (so
// that products of two inverses stay normal and finite), and its inverse.
__device__ __forceinline__ float scale_for(float m, float &inv)
{
    const int e = (__float_as_int(m) >> 23) & 0xff;        // biased exponent
    const int se = min(268 - e, 190);                      // biased exponent of 2^(14 - (e - 127))
    inv = __int_as_float((254 - se) << 23);
    return __int_as_float(se << 23);
}

// Largest of x over the four lane groups of this lane's column.
__device__ __forceinline__ float column_max(float x)
{
    const unsigned xi = __float_as_uint(x);
    const u32x2 a = __builtin_amdgcn_permlane16_swap(xi, xi, false, false);
    const float m = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const unsigned mi = __float_as_uint(m);
    const u32x2 c = __builtin_amdgcn_permlane32_swap(mi, mi, false, false);
    return fmaxf(__uint_as_float(c[0]), __uint_as_float(c[1]));
}

// The power of two that brings this pixel's inputs of a layer (its values
// v_q in every lane group) into range, and its inverse.
template <int Q>
__device__ __forceinline__ float input_scale(const float (&v)[Q], float &inv)
{
    float m = 0.0f;
#pragma unroll
    for (int q = 0; q < Q; ++q)
        m = fmaxf(m, fabsf(v[q]));
    return scale_for(column_max(m), inv);
}

// Largest magnitude in a part (this thread's entries).
template <int COUNT>
__device__ __forceinline__ float part_max(const Part<COUNT, float> &r)
{
    float m = 0.0f;
#pragma unroll
    for (int i = 0; i < Part<COUNT, float>::kPer; ++i)
        m = fmaxf(m, fabsf(r.v[i]));
    return m;
}

// Largest of x over the wavefront.
__device__ __forceinline__ float wave_max(float x)
{
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1)
        x = fmaxf(x, __shfl_xor(x, d, 64));
    return x;
}

// NB: 16-neuron blocks of the hidden width; NH: hidden layers; LS: levels per
// lane group (ceil(L / 4)); KSH: values per lane group of the hidden layers'
// inputs (ceil(width / 4)); RPW: tile rows per wavefront (a tile is 4 RPW
// rows: 8, or 16 when the launch has tiles to spare).
template <int NB, int NH, int LS, int KSH, int RPW>
__global__ __launch_bounds__(kThreads) void k_mfma_f16x3(DecodeParams p, int blocks_per_image, int tiles_x,
                                                         int tiles)
{
    static_assert(KSH <= 4 * NB && KSH > 4 * (NB - 1), "KSH must end in the last block");
    constexpr int THT = kWaves * RPW;   // tile rows
    using LY = Layout<NB, NH, LS, KSH, THT>;
    constexpr int S1 = LY::S1, SH = LY::SH;
    __shared__ __attribute__((aligned(16))) float lds[LY::SIZE];
    unsigned *ldsu = reinterpret_cast<unsigned *>(lds);

    warm_kernel_args<sizeof(DecodeParams)>();
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, col = lane & 15;
    // images interleave over the grid, so that every image's workgroups are
    // spread over the dispatch order (older workgroups on a CU run ahead)
    const int b = blockIdx.x % p.batch;
    const TileSchedule ts = tile_schedule(p, blockIdx.x, blocks_per_image, tiles);
    const int blk = ts.first;
    const int L = p.L;
    // the output layer's bias, read now so its latency hides behind the
    // parameter loads
    const float *b3 = layer_params(p, NH + 1, b).b;
    const float b3_0 = b3[0], b3_1 = b3[1], b3_2 = b3[2];

    // ---- the first tile's latent loads go out first, so their latency
    // overlaps the parameter gather below
    float boxv[box_regs<4 * LS, THT>()];
    if (blk < tiles)
        load_boxes<4 * LS, THT>(boxv, p, b, (blk / tiles_x) * THT, (blk % tiles_x) * TW, tid);

    // ---- this image's parameters: contiguous loads (all in flight at once)
    // into LDS as the caller lays them out, then scaled, split into fp16
    // parts and permuted into the operand layouts through registers
    float wsc[NH + 1], winv[NH + 1];
    {
        // every layer's pointers and widths first (one batch of scalar
        // loads), then the raw copies, branch-free (entries past a layer's
        // size repeat its last entry: the maxima are unchanged and the
        // permutation reads only valid ones)
        LayerParams lp[NH + 2];
        int wd[NH + 3];
#pragma unroll
        for (int l = 0; l < NH + 2; ++l)
            lp[l] = layer_params(p, l, b);
#pragma unroll
        for (int l = 0; l < NH + 3; ++l)
            wd[l] = p.widths[l];
        const int N1 = wd[1], NL = wd[NH + 1];
        const auto r1 = load_part<LY::N * 4 * LS, float>([&](int s) { return lp[0].template weight_clamped<false>(s, N1 * L); });
        Part<LY::N * LY::N, float> rh[NH > 0 ? NH : 1];
#pragma unroll
        for (int h = 0; h < NH; ++h) {
            const int n = wd[1 + h] * wd[2 + h];
            rh[h] = load_part<LY::N * LY::N, float>([&](int s) { return lp[1 + h].template weight_clamped<false>(s, n); });
        }
        const auto r3 = load_part<3 * LY::N, float>([&](int s) { return lp[NH + 1].template weight_clamped<false>(s, 3 * NL); });
        Part<LY::N, float> rb[NH + 1];
#pragma unroll
        for (int h = 0; h <= NH; ++h) {
            const int fout = wd[1 + h];
            rb[h] = load_part<LY::N, float>([&](int s) { return lp[h].bias_clamped(s, fout); });
        }
        {
            const float m1 = wave_max(part_max(r1));
            float mh[NH > 0 ? NH : 1];
#pragma unroll
            for (int h = 0; h < NH; ++h)
                mh[h] = wave_max(part_max(rh[h]));
            if (lane == 0) {
                lds[LY::WSC + wave] = m1;
#pragma unroll
                for (int h = 0; h < NH; ++h)
                    lds[LY::WSC + (1 + h) * kWaves + wave] = mh[h];
            }
        }
        store_part(lds + LY::W1A, r1);
#pragma unroll
        for (int h = 0; h < NH; ++h)
            store_part(lds + LY::WHA + h * NB * SH * 256, rh[h]);
        store_part(lds + LY::W3, r3);
#pragma unroll
        for (int h = 0; h <= NH; ++h)
            store_part(lds + LY::B1 + h * NB * 256, rb[h]);
        __syncthreads();
        // each layer's weight scale and its inverse (wave-uniform)
#pragma unroll
        for (int h = 0; h <= NH; ++h) {
            const float *m = lds + LY::WSC + h * kWaves;
            wsc[h] = scale_for(fmaxf(fmaxf(m[0], m[1]), fmaxf(m[2], m[3])), winv[h]);
        }

        const auto w1a = load_part<NB * S1 * 256, unsigned>([&](int s) {      // layer 1, A layout
            const int w = s & 3, ln = (s >> 2) & 63, st = (s >> 8) % S1, ob = (s >> 8) / S1;
            return a_entry<LS>(lds + LY::W1A, L, N1, ob, st, ln, w, wsc[0]);
        });
        Part<NB * SH * 256, unsigned> wha[NH > 0 ? NH : 1];
#pragma unroll
        for (int h = 0; h < NH; ++h) {                                         // hidden layers, A layout
            const int fin = p.widths[1 + h], fout = p.widths[2 + h];
            wha[h] = load_part<NB * SH * 256, unsigned>([&](int s) {
                const int w = s & 3, ln = (s >> 2) & 63, st = (s >> 8) % SH, ob = (s >> 8) / SH;
                return a_entry<KSH>(lds + LY::WHA + h * NB * SH * 256, fin, fout, ob, st, ln, w, wsc[1 + h]);
            });
        }
        Part<NB * 256, float> bias[NH + 1];
#pragma unroll
        for (int h = 0; h <= NH; ++h) {                                        // biases, accumulator layout
            const int fout = p.widths[1 + h];
            bias[h] = load_part<NB * 256, float>([&](int s) {
                const int r = s & 3, ln = (s >> 2) & 63, ob = s >> 8;
                const int n = 16 * ob + 4 * r + (ln >> 4);
                return lds_or_zero(lds + LY::B1 + h * NB * 256, n < fout, n);
            });
        }
        const auto w3 = load_part<NB * 64, float>([&](int s) {                // output layer [ob][r][g][c]
            const int c = s & 3, gg = (s >> 2) & 3, r = (s >> 4) & 3, ob = s >> 6;
            const int n = 16 * ob + 4 * r + gg;
            return lds_or_zero(lds + LY::W3, c < 3 && n < NL, c * NL + n);
        });
        __syncthreads();                   // every raw value is read
        store_part(ldsu + LY::W1A, w1a);
#pragma unroll
        for (int h = 0; h < NH; ++h)
            store_part(ldsu + LY::WHA + h * NB * SH * 256, wha[h]);
#pragma unroll
        for (int h = 0; h <= NH; ++h)
            store_part(lds + LY::B1 + h * NB * 256, bias[h]);
        store_part(lds + LY::W3, w3);
    }
    if (blk < tiles)
        store_boxes<4 * LS, THT>(lds + LY::LAT, boxv, p, tid);
    __syncthreads();

    // ---- the level each lane samples as its value q of the first layer:
    // 4q + g (level 0 where that level does not exist; its weights are zero)
    LaneLevel lv[LS];
#pragma unroll
    for (int s = 0; s < LS; ++s) {
        const int k = 4 * s + g;
        lane_level_init<THT>(lv[s], k < L ? k : 0, LY::LAT);
    }

    const int H = p.H, W = p.W;
    const int64_t plane = (int64_t)H * W;
    // Lane group g (< 3) stores channel g; lane group 0 carries the output
    // biases in its partial sums.
    const int64_t obase = (int64_t)b * 3 * plane + (int64_t)min(g, 2) * plane;
    const float ob0 = g == 0 ? b3_0 : 0.0f, ob1 = g == 0 ? b3_1 : 0.0f, ob2 = g == 0 ? b3_2 : 0.0f;

    // Tiles: the workgroup's first is tile blk; the others come from its
    // schedule's counter (tile ts.base + ticket, while below ts.end), so that
    // workgroups that run faster take more of them.  The grid's first
    // workgroup clears the counters of the next run.
    __shared__ int s_next;
    const bool dynamic = blocks_per_image < tiles;
    if (blockIdx.x == 0)
        for (int i = tid; i < p.tile_ctr_len; i += kThreads)
            p.tile_ctr_next[i] = 0;
    for (int t = blk;;) {
        const int ty0 = (t / tiles_x) * THT, tx0 = (t % tiles_x) * TW;
        const int ty1 = min(ty0 + THT, H) - 1, tx1 = min(tx0 + TW, W) - 1;

        if (t != blk) {       // the first tile was staged with the parameters
            __syncthreads();   // every wavefront is done with the previous tile's boxes
            stage_boxes<4 * LS, THT>(lds + LY::LAT, p, b, ty0, tx0, tid);
            __syncthreads();
        }
        int ticket = 0;    // the tile after this one; its latency hides behind the tile
        if (dynamic && tid == 0)
            ticket = atomicAdd(ts.ctr, 1);
#pragma unroll
        for (int s = 0; s < LS; ++s)
            lane_level_tile(lv[s], ty0, tx0, tx1, col);

#pragma unroll 1
        for (int rr = 0; rr < RPW; ++rr) {
            const int y = ty0 + RPW * wave + rr;
            if (y > ty1)
                break;   // wave-uniform: the row lies below the image
            int roff[LS];
            float rly[LS];
#pragma unroll
            for (int s = 0; s < LS; ++s)
                lane_level_row(lv[s], y, roff[s], rly[s]);
            const int64_t orow = obase + (int64_t)y * W + tx0 + col;

#pragma unroll
            for (int cg = 0; cg < TWG; ++cg) {
                if (tx0 + 16 * cg > tx1)
                    break;   // wave-uniform: the column group lies right of the image
                // Re-read the LDS operands per group rather than letting the
                // compiler keep loop-invariant ones in VGPRs (occupancy).
                asm volatile("" ::: "memory");

                // layer 1: B operand = the upsampled pyramid in fp16 parts
                float u[LS];
#pragma unroll
                for (int s = 0; s < LS; ++s)
                    u[s] = lane_level_sample(lds, lv[s], roff[s], rly[s], cg);
                float inv1;
                const float sc1 = input_scale<LS>(u, inv1);
                const float un1 = inv1 * winv[0];
                u32x4 b1[S1];
                build_b<LS>(u, sc1, b1);
                f32x4 d[NB];
#pragma unroll
                for (int ob = 0; ob < NB; ++ob)
                    d[ob] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int s = 0; s < S1; ++s)
#pragma unroll
                    for (int ob = 0; ob < NB; ++ob) {
                        const u32x4 a = *reinterpret_cast<const u32x4 *>(&ldsu[LY::W1A + ((ob * S1 + s) * 64 + lane) * 4]);
                        d[ob] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_f16x8(a), as_f16x8(b1[s]), d[ob], 0, 0, 0);
                    }
                // unscale, add the bias, ReLU
                float v[KSH];
#pragma unroll
                for (int q = 0; q < KSH; ++q)
                    v[q] = relu(__builtin_fmaf(d[q >> 2][q & 3], un1,
                                               lds[LY::B1 + ((q >> 2) * 64 + lane) * 4 + (q & 3)]));

                // hidden layers
#pragma unroll
                for (int h = 0; h < NH; ++h) {
                    float invh;
                    const float sch = input_scale<KSH>(v, invh);
                    const float unh = invh * winv[1 + h];
                    u32x4 bh[SH];
                    build_b<KSH>(v, sch, bh);
                    f32x4 e[NB];
#pragma unroll
                    for (int ob = 0; ob < NB; ++ob)
                        e[ob] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                    for (int s = 0; s < SH; ++s)
#pragma unroll
                        for (int ob = 0; ob < NB; ++ob) {
                            const u32x4 a = *reinterpret_cast<const u32x4 *>(
                                &ldsu[LY::WHA + (((h * NB + ob) * SH + s) * 64 + lane) * 4]);
                            e[ob] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_f16x8(a), as_f16x8(bh[s]), e[ob], 0, 0,
                                                                          0);
                        }
#pragma unroll
                    for (int q = 0; q < KSH; ++q)
                        v[q] = relu(__builtin_fmaf(e[q >> 2][q & 3], unh,
                                                   lds[LY::BH + ((h * NB + (q >> 2)) * 64 + lane) * 4 + (q & 3)]));
                }

                // output layer on the vector ALU: partial sums over this lane's
                // values, then a sum over the four lane groups
                // (weights read six values at a time, all before their first
                // use, so one LDS round trip covers each chunk)
                float o0 = ob0, o1 = ob1, o2 = ob2;
                constexpr int W3CH = 6;
#pragma unroll
                for (int q0 = 0; q0 < KSH; q0 += W3CH) {
                    f32x4 w3[W3CH];
#pragma unroll
                    for (int j = 0; j < W3CH; ++j)
                        if (q0 + j < KSH)
                            w3[j] = *reinterpret_cast<const f32x4 *>(&lds[LY::W3 + ((q0 + j) * 4 + g) * 4]);
#pragma unroll
                    for (int j = 0; j < W3CH; ++j) {
                        if (q0 + j < KSH) {
                            o0 = __builtin_fmaf(w3[j][0], v[q0 + j], o0);
                            o1 = __builtin_fmaf(w3[j][1], v[q0 + j], o1);
                            o2 = __builtin_fmaf(w3[j][2], v[q0 + j], o2);
                        }
                    }
                }
                const float vo = row_sum3(o0, o1, o2);
                if (g < 3 && tx0 + 16 * cg + col <= tx1)
                    store_out(p, orow + 16 * cg, vo);
            }
        }
        if (!dynamic)
            break;    // uniform: one tile per workgroup
        if (tid == 0)
            s_next = ts.base + ticket;
        __syncthreads();
        t = s_next;
        if (t >= ts.end)
            break;    // uniform
    }
}

int hidden_blocks(int nl, const int32_t *widths);

// Values per lane group of the hidden activations: ceil(width / 4) of the
// widest hidden layer (the last one feeds the output layer, so it counts too).
int hidden_values(int nl, const int32_t *widths);

template <int NB, int NH, int LS, int KSH, int RPW>
hipError_t launch_rows(const DecodeParams &p, hipStream_t s, int tiles_x, int tiles, int bpi)
{
    const int64_t nblocks = (int64_t)bpi * p.batch;
    if (nblocks > 0x7fffffff)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_mfma_f16x3<NB, NH, LS, KSH, RPW>), dim3((unsigned)nblocks), dim3(kThreads), 0, s, p,
                       bpi, tiles_x, tiles);
    return hipGetLastError();
}

// 16-row tiles when every workgroup of the launch averages two or more and
// the taller boxes cost no occupancy (as in the fp32 family), else 8-row.
template <int NB, int NH, int LS, int KSH>
hipError_t launch(const DecodeParams &p, hipStream_t s, int num_cus)
{
    const int tiles_x = (p.W + TW - 1) / TW;
    const int tiles8 = tiles_x * ((p.H + TH - 1) / TH);
    const int tiles16 = tiles_x * ((p.H + 4 * kWaves - 1) / (4 * kWaves));
    static int occ8 = 0, occ16 = 0;   // workgroups per CU of each instance
    const int bpi8 = blocks_per_image(k_mfma_f16x3<NB, NH, LS, KSH, 2>, p, num_cus, tiles8, occ8);
    const int bpi16 = blocks_per_image(k_mfma_f16x3<NB, NH, LS, KSH, 4>, p, num_cus, tiles16, occ16);
    if (occ16 >= occ8 && tiles16 >= 2 * bpi16)
        return launch_rows<NB, NH, LS, KSH, 4>(p, s, tiles_x, tiles16, bpi16);
    return launch_rows<NB, NH, LS, KSH, 2>(p, s, tiles_x, tiles8, bpi8);
}

template <int NH>
hipError_t launch_nh(const DecodeParams &p, hipStream_t s, int num_cus)
{
    const int NB = hidden_blocks(p.nl, p.widths);
    const int LS = (p.L + 3) / 4;
    // Width 33..40 (three blocks, last one half used) gets its own value
    // count; every other width runs all 4 NB values over zero padding.
    const bool k10 = NH > 0 && NB == 3 && hidden_values(p.nl, p.widths) <= 10;
#define PIC_CASE(nb, ls, ksh) \
    if (NB == nb && LS == ls && (ksh != 4 * nb) == (nb == 3 && k10)) return launch<nb, NH, ls, ksh>(p, s, num_cus);
    PIC_CASE(1, 1, 4) PIC_CASE(1, 2, 4) PIC_CASE(1, 3, 4)
    PIC_CASE(2, 1, 8) PIC_CASE(2, 2, 8) PIC_CASE(2, 3, 8)
    PIC_CASE(3, 1, 12) PIC_CASE(3, 2, 12) PIC_CASE(3, 3, 12)
    PIC_CASE(4, 1, 16) PIC_CASE(4, 2, 16) PIC_CASE(4, 3, 16)
    if constexpr (NH > 0) {
        PIC_CASE(3, 1, 10) PIC_CASE(3, 2, 10) PIC_CASE(3, 3, 10)
    }
#undef PIC_CASE
    return hipErrorInvalidValue;
}

}  // namespace mfma_f16x3
}  // namespace pic
