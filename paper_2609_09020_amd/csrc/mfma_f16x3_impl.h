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
//   scaled, split and laid out to match once per workgroup, a pair of inputs
//   of one neuron at a time (AItems below).  A layer's biases sit in LDS
//   once per neuron, in the order that gives lane group g the four neurons
//   16 ob + 4 r + g of its registers as one 16-byte read.  The output layer
//   (3 neurons) runs in fp32 on the vector ALU.
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
    static constexpr int B1 = WHA + NH * NB * SH * 256;             // f32 [NH + 1][16 NB], swz order
    static constexpr int W3 = B1 + (NH + 1) * 16 * NB;              // f32 [NB][4 r][4 g][4 c]
    static constexpr int WSC = W3 + NB * 64;                        // f32 [NH + 1][kWaves]: weight maxima
    static constexpr int LAT = WSC + (NH + 1) * kWaves;             // latent boxes
    static constexpr int SIZE = LAT + box_offset<THT>(4 * LS);
    static constexpr int N = 16 * NB;
};

// Neuron on row `row` of an output block; the map is its own inverse.
__device__ __forceinline__ int row_neuron(int row) { return 4 * (row & 3) + (row >> 2); }

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

// Position (u32 index) of slot p of output neuron `out` in lane group g in a
// layer's A layout of S K steps: block out / 16, step p / 4, lane
// 16 g + (the row that holds out), word p % 4.
template <int S>
__device__ __forceinline__ int a_word(int out, int g, int p)
{
    return (((out >> 4) * S + (p >> 2)) * 64 + 16 * g + row_neuron(out & 15)) * 4 + (p & 3);
}

// A layer's weights in the A layout (slot pairs as in the header), formed a
// work item at a time: item (out, g, t) takes inputs 4 (2t) + g and
// 4 (2t + 1) + g of neuron `out` (zero past the layer's shape), scaled by
// the power of two wsc and split into fp16 parts once each, and gives three
// words: (w_h, w_h) of the first input for slot 2t, of the second for slot
// 2t + 1 (when 2t + 1 < Q), and the pair of their w_l for slot Q + t.  The
// slots from Q + T on are zero, so each word of the layout is written by
// exactly one item or by the zero fill.
//
// Three steps, so that nothing waits for a load before every load is out:
// load (the caller's [out][in] matrix straight from global memory, an input
// outside the shape reading entry 0, which is a weight of the same layer and
// so leaves the layer's maximum unchanged), max_abs, then split (once the
// layer's scale is known; the outside inputs become zero) and store.
template <int Q, int NB>
struct AItems {
    static constexpr int S = ksteps(Q);
    static constexpr int T = (Q + 1) / 2;
    static constexpr int ITEMS = 16 * NB * 4 * T;
    static constexpr int PER = (ITEMS + kThreads - 1) / kThreads;
    static constexpr int ZSLOTS = 4 * S - Q - T;   // zero slots per block and lane
    static constexpr int ZWORDS = NB * 64 * ZSLOTS;
    float x0[PER], x1[PER];                        // the two weights of each item, as loaded
    unsigned hh0[PER], hh1[PER], ll[PER];          // its three words

    // (out, g, t) of item it, and whether its two inputs lie in the shape
    __device__ static void decode(int it, int fin, int fout, int &out, int &g, int &t, bool &ok0, bool &ok1)
    {
        g = it & 3;
        t = (it >> 2) % T;
        out = (it >> 2) / T;
        ok0 = out < fout && 8 * t + g < fin;
        ok1 = out < fout && 2 * t + 1 < Q && 8 * t + 4 + g < fin;
    }

    // (a thread past the last item repeats it: its values count once more
    // in the maximum and are not stored)
    __device__ void load(const float *w, int fin, int fout)
    {
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int it0 = (int)threadIdx.x + k * kThreads;
            int out, g, t;
            bool ok0, ok1;
            decode(it0 < ITEMS ? it0 : ITEMS - 1, fin, fout, out, g, t, ok0, ok1);
            x0[k] = w[ok0 ? out * fin + 8 * t + g : 0];
            x1[k] = w[ok1 ? out * fin + 8 * t + 4 + g : 0];
        }
    }

    __device__ float max_abs() const
    {
        float m = 0.0f;
#pragma unroll
        for (int k = 0; k < PER; ++k)
            m = fmaxf(m, fmaxf(fabsf(x0[k]), fabsf(x1[k])));
        return m;
    }

    __device__ void split(int fin, int fout, float wsc)
    {
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int it0 = (int)threadIdx.x + k * kThreads;
            int out, g, t;
            bool ok0, ok1;
            decode(it0 < ITEMS ? it0 : ITEMS - 1, fin, fout, out, g, t, ok0, ok1);
            const float a = ok0 ? x0[k] * wsc : 0.0f, c = ok1 ? x1[k] * wsc : 0.0f;
            const _Float16 h0 = (_Float16)a, h1 = (_Float16)c;
            const _Float16 l0 = (_Float16)(a - (float)h0), l1 = (_Float16)(c - (float)h1);
            hh0[k] = __builtin_bit_cast(unsigned, f16x2{h0, h0});
            hh1[k] = __builtin_bit_cast(unsigned, f16x2{h1, h1});
            ll[k] = __builtin_bit_cast(unsigned, f16x2{l0, l1});
        }
    }

    __device__ void store(unsigned *dst) const
    {
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int it = (int)threadIdx.x + k * kThreads;
            if (it < ITEMS) {
                const int g = it & 3, t = (it >> 2) % T, out = (it >> 2) / T;
                dst[a_word<S>(out, g, 2 * t)] = hh0[k];
                if (2 * t + 1 < Q)
                    dst[a_word<S>(out, g, 2 * t + 1)] = hh1[k];
                dst[a_word<S>(out, g, Q + t)] = ll[k];
            }
        }
        if constexpr (ZSLOTS > 0) {
#pragma unroll
            for (int z0 = 0; z0 < ZWORDS; z0 += kThreads) {
                const int z = z0 + (int)threadIdx.x;
                if (z < ZWORDS) {
                    const int bl = z / ZSLOTS, p = Q + T + z % ZSLOTS;   // bl: block * 64 + lane
                    dst[(((bl >> 6) * S + (p >> 2)) * 64 + (bl & 63)) * 4 + (p & 3)] = 0u;
                }
            }
        }
    }
};

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

// Largest of x (>= 0, not NaN: such floats order like their bit patterns)
// over the wavefront, by data-parallel moves within the vector unit instead
// of exchanges through LDS: the maximum of each quad (two quad
// permutations), of each row of 16 (row shifts by 4 and 8 leave it in lane
// 15), then of rows 0-1 and 2-3 (lane 15 of the row before broadcast into
// rows 1 and 3) and of the wavefront (lane 31 broadcast into rows 2 and 3),
// read from lane 63.  Lanes a move does not write keep their own value.
__device__ __forceinline__ float wave_max(float x)
{
    int v = __float_as_int(x);
    v = max(v, __builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false));    // quad_perm [1, 0, 3, 2]
    v = max(v, __builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false));    // quad_perm [2, 3, 0, 1]
    v = max(v, __builtin_amdgcn_update_dpp(v, v, 0x114, 0xF, 0xF, false));   // row_shr:4
    v = max(v, __builtin_amdgcn_update_dpp(v, v, 0x118, 0xF, 0xF, false));   // row_shr:8
    v = max(v, __builtin_amdgcn_update_dpp(v, v, 0x142, 0xA, 0xF, false));   // row_bcast:15, rows 1 and 3
    v = max(v, __builtin_amdgcn_update_dpp(v, v, 0x143, 0xC, 0xF, false));   // row_bcast:31, rows 2 and 3
    return __int_as_float(__builtin_amdgcn_readlane(v, 63));
}

// NB: 16-neuron blocks of the hidden width; NH: hidden layers; LS: levels per
// lane group (ceil(L / 4)); KSH: values per lane group of the hidden layers'
// inputs (ceil(width / 4)); RPW: tile rows per wavefront (a tile is 4 RPW
// rows: 8, or 16 when the launch has tiles to spare).
template <int NB, int NH, int LS, int KSH, int RPW>
__global__ __launch_bounds__(kThreads) void k_mfma_f16x3(DecodeParams p, int blocks_per_image, int tiles_x,
                                                         int tiles, uint32_t tx_recip)
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
    int b = 0;
    if (p.batch > 1)
        b = blockIdx.x % p.batch;
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
    if (blk < tiles) {
        const int by = tile_row(blk, tiles_x, tx_recip);
        load_boxes<4 * LS, THT>(boxv, p, b, by * THT, (blk - by * tiles_x) * TW, tid);
    }

    // ---- this image's parameters, loaded straight into their operand
    // layouts' order (all loads in flight at once); each layer's largest
    // weight magnitude gives its scale, after one barrier the weights are
    // split into fp16 parts and stored
    float wsc[NH + 1], winv[NH + 1];
    {
        LayerParams lp[NH + 2];
        int wd[NH + 3];
#pragma unroll
        for (int l = 0; l < NH + 2; ++l)
            lp[l] = layer_params(p, l, b);
#pragma unroll
        for (int l = 0; l < NH + 3; ++l)
            wd[l] = p.widths[l];
        const int N1 = wd[1], NL = wd[NH + 1];
        AItems<LS, NB> w1a;                                                    // layer 1
        w1a.load(static_cast<const float *>(lp[0].w), L, N1);
        AItems<KSH, NB> wha[NH > 0 ? NH : 1];
#pragma unroll
        for (int h = 0; h < NH; ++h)                                            // hidden layers
            wha[h].load(static_cast<const float *>(lp[1 + h].w), wd[1 + h], wd[2 + h]);
        // biases in swz order (position s holds neuron swz(s)), the output
        // layer as [ob][r][g][c] (neuron 16 ob + 4 r + g, channel c): raw
        // loads (an entry outside the shape reads entry 0), zeroed when stored
        constexpr int BPER = (LY::N + kThreads - 1) / kThreads, WPER = (NB * 64 + kThreads - 1) / kThreads;
        float braw[NH + 1][BPER], w3raw[WPER];
#pragma unroll
        for (int h = 0; h <= NH; ++h)
#pragma unroll
            for (int k = 0; k < BPER; ++k) {
                const int s = min((int)threadIdx.x + k * kThreads, LY::N - 1);
                const int n = (s & ~15) | ((s & 3) << 2) | ((s >> 2) & 3);
                braw[h][k] = lp[h].b[n < wd[1 + h] ? n : 0];
            }
        const float *w3p = static_cast<const float *>(lp[NH + 1].w);
#pragma unroll
        for (int k = 0; k < WPER; ++k) {
            const int s = min((int)threadIdx.x + k * kThreads, NB * 64 - 1);
            const int c = s & 3, n = 16 * (s >> 6) + 4 * ((s >> 4) & 3) + ((s >> 2) & 3);
            w3raw[k] = w3p[c < 3 && n < NL ? c * NL + n : 0];
        }
        {
            const float m1 = wave_max(w1a.max_abs());
            float mh[NH > 0 ? NH : 1];
#pragma unroll
            for (int h = 0; h < NH; ++h)
                mh[h] = wave_max(wha[h].max_abs());
            if (lane == 0) {
                lds[LY::WSC + wave] = m1;
#pragma unroll
                for (int h = 0; h < NH; ++h)
                    lds[LY::WSC + (1 + h) * kWaves + wave] = mh[h];
            }
        }
#pragma unroll
        for (int h = 0; h <= NH; ++h)
#pragma unroll
            for (int k = 0; k < BPER; ++k) {
                const int s = (int)threadIdx.x + k * kThreads;
                const int n = (s & ~15) | ((s & 3) << 2) | ((s >> 2) & 3);
                if (s < LY::N)
                    lds[LY::B1 + h * LY::N + s] = n < wd[1 + h] ? braw[h][k] : 0.0f;
            }
#pragma unroll
        for (int k = 0; k < WPER; ++k) {
            const int s = (int)threadIdx.x + k * kThreads;
            const int c = s & 3, n = 16 * (s >> 6) + 4 * ((s >> 4) & 3) + ((s >> 2) & 3);
            if (s < NB * 64)
                lds[LY::W3 + s] = c < 3 && n < NL ? w3raw[k] : 0.0f;
        }
        if (blk < tiles)
            store_boxes<4 * LS, THT>(lds + LY::LAT, boxv, tid);
        __syncthreads();
        // each layer's weight scale and its inverse (wave-uniform)
#pragma unroll
        for (int h = 0; h <= NH; ++h) {
            const float *m = lds + LY::WSC + h * kWaves;
            wsc[h] = scale_for(fmaxf(fmaxf(m[0], m[1]), fmaxf(m[2], m[3])), winv[h]);
        }
        w1a.split(L, N1, wsc[0]);
        w1a.store(ldsu + LY::W1A);
#pragma unroll
        for (int h = 0; h < NH; ++h) {
            wha[h].split(wd[1 + h], wd[2 + h], wsc[1 + h]);
            wha[h].store(ldsu + LY::WHA + h * NB * SH * 256);
        }
    }
    __syncthreads();

    // ---- the level each lane samples as its value q of the first layer:
    // 4q + g (level 0 where that level does not exist; its weights are zero)
    LaneLevel lv[LS];
    lane_levels_init<THT, 4, 1>(lv, g, L, LY::LAT, std::make_integer_sequence<int, LS>{});

    const int H = p.H, W = p.W;
    const int64_t plane = (int64_t)H * W;
    // Lane group g (< 3) stores channel g; lane group 0 carries the output
    // biases in its partial sums.
    const int64_t obase = (int64_t)(uint64_t)(uint32_t)(3 * b + min(g, 2)) * plane;
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
        const int tr = tile_row(t, tiles_x, tx_recip);
        const int ty0 = tr * THT, tx0 = (t - tr * tiles_x) * TW;
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
            const int64_t orow = obase + (uint32_t)(y * W + tx0 + col);   // < H W + 64 <= 2^31 + 63

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
                // unscale, add the bias, ReLU (the biases of a block's four
                // registers: one 16-byte read, the same for the lane group)
                float v[KSH];
#pragma unroll
                for (int ob = 0; ob < (KSH + 3) / 4; ++ob) {
                    const f32x4 bb = *reinterpret_cast<const f32x4 *>(&lds[LY::B1 + 16 * ob + 4 * g]);
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (4 * ob + r < KSH)
                            v[4 * ob + r] = relu(__builtin_fmaf(d[ob][r], un1, bb[r]));
                }

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
                    for (int ob = 0; ob < (KSH + 3) / 4; ++ob) {
                        const f32x4 bb =
                            *reinterpret_cast<const f32x4 *>(&lds[LY::B1 + (1 + h) * LY::N + 16 * ob + 4 * g]);
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (4 * ob + r < KSH)
                                v[4 * ob + r] = relu(__builtin_fmaf(e[ob][r], unh, bb[r]));
                    }
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
                       bpi, tiles_x, tiles, tile_row_recip(tiles_x, tiles));
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
