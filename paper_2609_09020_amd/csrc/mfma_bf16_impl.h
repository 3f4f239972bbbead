// bf16-weight matrix-core decode kernel (v_mfma_f32_16x16x32_bf16), shared by
// the k_mfma_bf16*.hip translation units that instantiate it.
//
// Same computation and tiling as the fp32 family (PIC, Sec. 3.1 and App. A;
// tiles, LDS boxes and upsample in decode_common.h), with the MLP weights
// given in bfloat16.  The weights are used exactly; every activation h fed to
// a matrix core is split into two bfloat16 numbers, hi = h with the low 16
// mantissa bits cleared and lo = round-to-nearest-even(h - hi), and each
// product is formed as W * hi + W * lo (two MFMAs into one fp32
// accumulator).  |h - hi - lo| <= 2^-16 |h|, so the split costs about as
// much accuracy as binary32 rounding of a short dot product, not bfloat16's.
//
// Matrix-core mapping (lane l, lane group g = l / 16, i = l % 16)
//   v_mfma_f32_16x16x32_bf16 takes A[i][8g + j] and B[8g + j][i], j = 0..7,
//   from lane l and returns D[4g + r][i] in register r of lane l.  Row i of
//   output block ob holds neuron 16 ob + i, so lane (g, i) holds neurons
//   16 ob + 4g + r of pixel i.  K step s of the next layer covers input blocks
//   2s and 2s+1: K index 8g + j is neuron 16 (2s + j / 4) + 4g + j % 4, which
//   the lane already holds (registers j % 4 of blocks 2s + j / 4).  The
//   weights are laid out to match.  For the first layer, lane group g carries
//   levels LPG g + j (j < LPG = ceil(L / 4)) at K indices 8g + j.
//   Biases start the accumulators; the output layer (3 neurons) runs in fp32
//   on the vector ALU as in the fp32 family.
#pragma once

#include "decode_common.h"

namespace pic {
namespace mfma_bf16 {

using namespace tile;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

template <int NB, int NH, int LPG>
struct Layout {
    static constexpr int KS2 = (NB + 1) / 2;                        // hidden K steps (32 inputs each)
    static constexpr int W1A = 0;                                   // u32 [NB][64][4]
    static constexpr int WHA = W1A + NB * 64 * 4;                   // u32 [NH][NB][KS2][64][4]
    static constexpr int B1 = WHA + NH * NB * KS2 * 64 * 4;         // f32 [NB][64][4]
    static constexpr int BH = B1 + NB * 64 * 4;                     // f32 [NH][NB][64][4]
    static constexpr int W3 = BH + NH * NB * 64 * 4;                // f32 [NB][4 r][4 g][4 c]
    static constexpr int LAT = W3 + NB * 64;                        // latent boxes
    static constexpr int SIZE = LAT + box_offset(4 * LPG);
};

// (x0, x1) -> {hi, lo}: the packed bfloat16 pairs (hi0, hi1) and (lo0, lo1),
// low halves first.
__device__ __forceinline__ u32x2 split_pair(float x0, float x1)
{
    const unsigned b0 = __float_as_uint(x0), b1 = __float_as_uint(x1);
    // the high halves of b0 and b1, in one byte permute
    const unsigned hi = __builtin_amdgcn_perm(b1, b0, 0x07060302u);
    const float r0 = x0 - __uint_as_float(b0 & 0xffff0000u);
    const float r1 = x1 - __uint_as_float(b1 & 0xffff0000u);
    // both remainders rounded to bfloat16 by one packed conversion
    const bf16x2 l = __builtin_convertvector((f32x2{r0, r1}), bf16x2);
    return u32x2{hi, __builtin_bit_cast(unsigned, l)};
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// NB: 16-neuron blocks of the hidden width; NH: hidden layers; LPG: levels
// per lane group in the first layer (ceil(L / 4)).
template <int NB, int NH, int LPG>
__global__ __launch_bounds__(kThreads) void k_mfma_bf16(DecodeParams p, int blocks_per_image,
                                                        int tiles_x, int tiles)
{
    using LY = Layout<NB, NH, LPG>;
    constexpr int KS2 = LY::KS2;
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
    float boxv[box_regs<4 * LPG>()];
    if (blk < tiles)
        load_boxes<4 * LPG>(boxv, p, b, (blk / tiles_x) * TH, (blk % tiles_x) * TW, tid);

    // ---- stage this image's parameters into LDS in operand layouts (every
    // load in flight before the first store)
    {
        const int N1 = p.widths[1];
        const LayerParams l0 = layer_params(p, 0, b);
        const auto w1a = load_part<NB * 64 * 4, unsigned>([&](int s) {        // layer 1, A layout
            const int u = s & 3, ln = (s >> 2) & 63, ob = s >> 8;
            const int out = 16 * ob + (ln & 15), gg = ln >> 4;
            unsigned w = 0;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int j = 2 * u + h, lvl = LPG * gg + j;
                if (j < LPG && lvl < L && out < N1)
                    w |= l0.bits(out * L + lvl) << (16 * h);
            }
            return w;
        });
        Part<NB * KS2 * 64 * 4, unsigned> wha[NH > 0 ? NH : 1];
#pragma unroll
        for (int hl = 0; hl < NH; ++hl) {                                      // hidden layers, A layout
            const int fin = p.widths[1 + hl], fout = p.widths[2 + hl];
            const LayerParams lh = layer_params(p, 1 + hl, b);
            wha[hl] = load_part<NB * KS2 * 64 * 4, unsigned>([&](int s) {
                const int u = s & 3, ln = (s >> 2) & 63, rest = s >> 8;
                const int st = rest % KS2, ob = rest / KS2;
                const int out = 16 * ob + (ln & 15), gg = ln >> 4;
                unsigned w = 0;
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int j = 2 * u + h;
                    const int in = 16 * (2 * st + (j >> 2)) + 4 * gg + (j & 3);
                    if (out < fout && in < fin)
                        w |= lh.bits(out * fin + in) << (16 * h);
                }
                return w;
            });
        }
        Part<NB * 256, float> bias[NH + 1];
#pragma unroll
        for (int hl = 0; hl <= NH; ++hl) {                                     // biases, accumulator layout
            const int fout = p.widths[1 + hl];
            const float *bp = layer_params(p, hl, b).b;
            bias[hl] = load_part<NB * 256, float>([&](int s) {
                const int r = s & 3, ln = (s >> 2) & 63, ob = s >> 8;
                const int n = 16 * ob + 4 * (ln >> 4) + r;
                return n < fout ? bp[n] : 0.0f;
            });
        }
        const int NL = p.widths[NH + 1];
        const LayerParams lo = layer_params(p, NH + 1, b);
        const auto w3 = load_part<NB * 64, float>([&](int s) {                // output layer [ob][r][g][c]
            const int c = s & 3, gg = (s >> 2) & 3, r = (s >> 4) & 3, ob = s >> 6;
            const int n = 16 * ob + 4 * gg + r;
            return (c < 3 && n < NL) ? lo.weight(c * NL + n) : 0.0f;
        });
        store_part(ldsu + LY::W1A, w1a);
#pragma unroll
        for (int hl = 0; hl < NH; ++hl)
            store_part(ldsu + LY::WHA + hl * NB * KS2 * 256, wha[hl]);
#pragma unroll
        for (int hl = 0; hl <= NH; ++hl)
            store_part(lds + LY::B1 + hl * NB * 256, bias[hl]);
        store_part(lds + LY::W3, w3);
    }
    if (blk < tiles)
        store_boxes<4 * LPG>(lds + LY::LAT, boxv, p, tid);
    __syncthreads();

    u32x4 w1[NB];
#pragma unroll
    for (int ob = 0; ob < NB; ++ob)
        w1[ob] = *reinterpret_cast<const u32x4 *>(&ldsu[LY::W1A + (ob * 64 + lane) * 4]);
    u32x4 wh[NH > 0 ? NH : 1][NB][KS2];
#pragma unroll
    for (int hl = 0; hl < NH; ++hl)
#pragma unroll
        for (int ob = 0; ob < NB; ++ob)
#pragma unroll
            for (int st = 0; st < KS2; ++st)
                wh[hl][ob][st] = *reinterpret_cast<const u32x4 *>(&ldsu[LY::WHA + (((hl * NB + ob) * KS2 + st) * 64 + lane) * 4]);

    // ---- the levels this lane samples: LPG g + j, j < LPG (level 0 where the
    // level does not exist; its weights are zero).
    LaneLevel lv[LPG];
#pragma unroll
    for (int j = 0; j < LPG; ++j) {
        const int k = LPG * g + j;
        lane_level_init(lv[j], k < L ? k : 0, LY::LAT);
    }

    const int H = p.H, W = p.W;
    const int64_t plane = (int64_t)H * W;
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
        const int ty0 = (t / tiles_x) * TH, tx0 = (t % tiles_x) * TW;
        const int ty1 = min(ty0 + TH, H) - 1, tx1 = min(tx0 + TW, W) - 1;

        if (t != blk) {       // the first tile was staged with the parameters
            __syncthreads();   // every wavefront is done with the previous tile's boxes
            stage_boxes<4 * LPG>(lds + LY::LAT, p, b, ty0, tx0, tid);
            __syncthreads();
        }
        int ticket = 0;    // the tile after this one; its latency hides behind the tile
        if (dynamic && tid == 0)
            ticket = atomicAdd(ts.ctr, 1);
#pragma unroll
        for (int j = 0; j < LPG; ++j)
            lane_level_tile(lv[j], ty0, tx0, tx1, col);

#pragma unroll 1
        for (int rr = 0; rr < 2; ++rr) {
            const int y = ty0 + 2 * wave + rr;
            if (y > ty1)
                break;
            int roff[LPG];
            float rly[LPG];
#pragma unroll
            for (int j = 0; j < LPG; ++j)
                lane_level_row(lv[j], y, roff[j], rly[j]);
            const int64_t orow = obase + (int64_t)y * W + tx0 + col;

#pragma unroll
            for (int cg = 0; cg < TWG; ++cg) {
                if (tx0 + 16 * cg > tx1)
                    break;
                // Re-read the LDS operands per group rather than letting the
                // compiler keep loop-invariant ones in VGPRs (occupancy).
                asm volatile("" ::: "memory");

                // layer 1: B operand = the lane's LPG upsampled levels, split
                float u[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int j = 0; j < LPG; ++j)
                    u[j] = lane_level_sample(lds, lv[j], roff[j], rly[j], cg);
                u32x4 bh = {0u, 0u, 0u, 0u}, bl = {0u, 0u, 0u, 0u};
                {
                    const u32x2 q = split_pair(u[0], u[1]);
                    bh[0] = q[0];
                    bl[0] = q[1];
                }
                if (LPG > 2) {
                    const u32x2 q = split_pair(u[2], u[3]);
                    bh[1] = q[0];
                    bl[1] = q[1];
                }
                f32x4 d[NB];
#pragma unroll
                for (int ob = 0; ob < NB; ++ob) {
                    d[ob] = *reinterpret_cast<const f32x4 *>(&lds[LY::B1 + (ob * 64 + lane) * 4]);
                    d[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w1[ob]), as_bf16x8(bh), d[ob], 0, 0, 0);
                    d[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w1[ob]), as_bf16x8(bl), d[ob], 0, 0, 0);
                }
#pragma unroll
                for (int ob = 0; ob < NB; ++ob)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        d[ob][r] = relu(d[ob][r]);

                // hidden layers
#pragma unroll
                for (int hl = 0; hl < NH; ++hl) {
                    u32x4 xh[KS2], xl[KS2];
#pragma unroll
                    for (int st = 0; st < KS2; ++st) {
#pragma unroll
                        for (int w = 0; w < 4; ++w) {
                            const int nb = 2 * st + (w >> 1);
                            if (nb < NB) {
                                const u32x2 q = split_pair(d[nb][2 * (w & 1)], d[nb][2 * (w & 1) + 1]);
                                xh[st][w] = q[0];
                                xl[st][w] = q[1];
                            } else {
                                xh[st][w] = 0u;
                                xl[st][w] = 0u;
                            }
                        }
                    }
                    f32x4 e[NB];
#pragma unroll
                    for (int ob = 0; ob < NB; ++ob)
                        e[ob] = *reinterpret_cast<const f32x4 *>(&lds[LY::BH + ((hl * NB + ob) * 64 + lane) * 4]);
#pragma unroll
                    for (int st = 0; st < KS2; ++st)
#pragma unroll
                        for (int ob = 0; ob < NB; ++ob) {
                            e[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(wh[hl][ob][st]),
                                                                            as_bf16x8(xh[st]), e[ob], 0, 0, 0);
                            e[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(wh[hl][ob][st]),
                                                                            as_bf16x8(xl[st]), e[ob], 0, 0, 0);
                        }
#pragma unroll
                    for (int ob = 0; ob < NB; ++ob)
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            d[ob][r] = relu(e[ob][r]);
                }

                // output layer on the vector ALU (fp32); a block's four weight
                // reads are issued before their first use, so one LDS round
                // trip covers them
                float o0 = ob0, o1 = ob1, o2 = ob2;
#pragma unroll
                for (int ob = 0; ob < NB; ++ob) {
                    f32x4 w3[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        w3[r] = *reinterpret_cast<const f32x4 *>(&lds[LY::W3 + ((ob * 4 + r) * 4 + g) * 4]);
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        o0 = __builtin_fmaf(w3[r][0], d[ob][r], o0);
                        o1 = __builtin_fmaf(w3[r][1], d[ob][r], o1);
                        o2 = __builtin_fmaf(w3[r][2], d[ob][r], o2);
                    }
                }
                const float v = row_sum3(o0, o1, o2);
                if (g < 3 && tx0 + 16 * cg + col <= tx1)
                    store_out(p, orow + 16 * cg, v);
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

template <int NB, int NH, int LPG>
hipError_t launch(const DecodeParams &p, hipStream_t s, int num_cus)
{
    const int tiles_x = (p.W + TW - 1) / TW, tiles_y = (p.H + TH - 1) / TH;
    const int tiles = tiles_x * tiles_y;
    static int occ = 0;
    const int bpi = blocks_per_image(k_mfma_bf16<NB, NH, LPG>, p, num_cus, tiles, occ);
    const int64_t nblocks = (int64_t)bpi * p.batch;
    if (nblocks > 0x7fffffff)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_mfma_bf16<NB, NH, LPG>), dim3((unsigned)nblocks), dim3(kThreads), 0, s, p, bpi,
                       tiles_x, tiles);
    return hipGetLastError();
}

int hidden_blocks(int nl, const int32_t *widths);

template <int NH>
hipError_t launch_nh(const DecodeParams &p, hipStream_t s, int num_cus)
{
    const int NB = hidden_blocks(p.nl, p.widths);
    const int LPG = (p.L + 3) / 4;
#define PIC_CASE(nb, lpg) \
    if (NB == nb && LPG == lpg) return launch<nb, NH, lpg>(p, s, num_cus);
    PIC_CASE(1, 1) PIC_CASE(1, 2) PIC_CASE(1, 3)
    PIC_CASE(2, 1) PIC_CASE(2, 2) PIC_CASE(2, 3)
    PIC_CASE(3, 1) PIC_CASE(3, 2) PIC_CASE(3, 3)
    PIC_CASE(4, 1) PIC_CASE(4, 2) PIC_CASE(4, 3)
#undef PIC_CASE
    return hipErrorInvalidValue;
}

}  // namespace mfma_bf16
}  // namespace pic
