// bf16-weight matrix-core decode kernel (v_mfma_f32_16x16x32_bf16), shared by
// the k_mfma_bf16*.hip translation units that instantiate it.
//
// Same computation and tiling as the fp32 family (PIC, Sec. 3.1 and App. A;
// tiles, LDS boxes and upsample in decode_common.h), with the MLP weights
// given in bfloat16.  The weights are used exactly; every activation h fed to
// a matrix core is split into two bfloat16 numbers, hi = RNE_bf16(h) and
// lo = RNE_bf16(h - hi), and each product is formed as W * hi + W * lo (two
// MFMAs into one fp32 accumulator).  |h - hi| <= 2^-8 |h| and
// |h - hi - lo| <= 2^-8 |h - hi| <= 2^-16 |h|, so the split costs about as
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
//   levels LPG g + j (j < LPG = ceil(L / 4)), hi and lo parts both, in one K
//   step: K word w (indices 8g + 2w, 8g + 2w + 1) holds the hi parts of
//   levels 2p, 2p + 1 for w = 2p, their lo parts for w = 2p + 1, and for odd
//   LPG the last level's (hi, lo) in word LPG - 1; the weights repeat to
//   match, so one MFMA per block forms W * hi + W * lo.
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

template <int NB, int NH, int LPG, int THT>
struct Layout {
    static constexpr int KS2 = (NB + 1) / 2;                        // hidden K steps (32 inputs each)
    static constexpr int W1A = 0;                                   // u32 [NB][64][4]
    static constexpr int WHA = W1A + NB * 64 * 4;                   // u32 [NH][NB][KS2][64][4]
    static constexpr int B1 = WHA + NH * NB * KS2 * 64 * 4;         // f32 [NB][64][4]
    static constexpr int BH = B1 + NB * 64 * 4;                     // f32 [NH][NB][64][4]
    static constexpr int W3 = BH + NH * NB * 64 * 4;                // f32 [NB][4 r][4 g][4 c]
    static constexpr int LAT = W3 + NB * 64;                        // latent boxes
    static constexpr int SIZE = LAT + box_offset<THT>(4 * LPG);
};

// (x0, x1) -> {hi, lo}: the packed bfloat16 pairs (hi0, hi1) and (lo0, lo1),
// low halves first.  hi = RNE_bf16(x); the remainder x - hi is formed by one
// dot product per value, hi . (-1, -0) + x0 and hi . (-0, -1) + x1 (exact:
// the products are exact and the result is representable in binary32), and
// rounded by one packed conversion: 4 instructions per pair.
__device__ __forceinline__ u32x2 split_pair(float x0, float x1)
{
    const bf16x2 hi = __builtin_convertvector((f32x2{x0, x1}), bf16x2);
    // (-1, -0) and (-0, -1), not (-1, 0): the compiler would encode (-1, 0)
    // as the inline constant -1.0, which the instruction does not read as
    // that bf16 pair; these two stay 32-bit literals.  -0 * hi adds nothing.
    const bf16x2 neg_lo = {(__bf16)-1.0f, (__bf16)-0.0f}, neg_hi = {(__bf16)-0.0f, (__bf16)-1.0f};
    const float r0 = __builtin_amdgcn_fdot2_f32_bf16(hi, neg_lo, x0, false);
    const float r1 = __builtin_amdgcn_fdot2_f32_bf16(hi, neg_hi, x1, false);
    const bf16x2 lo = __builtin_convertvector((f32x2{r0, r1}), bf16x2);
    return u32x2{__builtin_bit_cast(unsigned, hi), __builtin_bit_cast(unsigned, lo)};
}

// x -> the packed pair (hi, lo) of one value, as split_pair computes them.
__device__ __forceinline__ unsigned split_one(float x)
{
    const bf16x2 h = __builtin_convertvector((f32x2{x, 0.0f}), bf16x2);
    const bf16x2 neg_lo = {(__bf16)-1.0f, (__bf16)-0.0f};
    const float r = __builtin_amdgcn_fdot2_f32_bf16(h, neg_lo, x, false);
    return __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2{x, r}), bf16x2));
}

// Level j (< LPG) of a lane group behind half h of first-layer K word w, or
// -1 for an empty slot (the word order of the hi/lo packing above).
template <int LPG>
__host__ __device__ constexpr int l1_level(int w, int h)
{
    return w < 2 * (LPG / 2) ? 2 * (w / 2) + h : (w == LPG - 1 && (LPG & 1) ? LPG - 1 : -1);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// NB: 16-neuron blocks of the hidden width; NH: hidden layers; LPG: levels
// per lane group in the first layer (ceil(L / 4)); RPW: tile rows per
// wavefront (a tile is 4 RPW rows: 8, or 16 or 32 when the launch has tiles
// to spare).
template <int NB, int NH, int LPG, int RPW>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(LPG <= 2 ? 4 : 1)))
void k_mfma_bf16(DecodeParams p, int blocks_per_image, int tiles_x, int tiles, uint32_t tx_recip)
{
    constexpr int THT = kWaves * RPW;   // tile rows
    using LY = Layout<NB, NH, LPG, THT>;
    constexpr int KS2 = LY::KS2;
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
    float boxv[box_regs<4 * LPG, THT>()];
    if (blk < tiles) {
        const int by = tile_row(blk, tiles_x, tx_recip);
        load_boxes<4 * LPG, THT>(boxv, p, b, by * THT, (blk - by * tiles_x) * TW, tid);
    }

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
                const int j = l1_level<LPG>(u, h), lvl = LPG * gg + j;
                if (j >= 0 && lvl < L && out < N1)
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
        store_boxes<4 * LPG, THT>(lds + LY::LAT, boxv, tid);
    __syncthreads();


    // ---- the levels this lane samples: LPG g + j, j < LPG (level 0 where the
    // level does not exist; its weights are zero).
    LaneLevel lv[LPG];
    lane_levels_init<THT, 1, LPG>(lv, g, L, LY::LAT, std::make_integer_sequence<int, LPG>{});

    const int H = p.H, W = p.W;
    const int64_t plane = (int64_t)H * W;
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
            stage_boxes<4 * LPG, THT>(lds + LY::LAT, p, b, ty0, tx0, tid);
            __syncthreads();
        }
        int ticket = 0;    // the tile after this one; its latency hides behind the tile
        if (dynamic && tid == 0)
            ticket = atomicAdd(ts.ctr, 1);
#pragma unroll
        for (int j = 0; j < LPG; ++j)
            lane_level_tile(lv[j], ty0, tx0, tx1, col);

#pragma unroll 1
        for (int rr = 0; rr < RPW; ++rr) {
            const int y = ty0 + RPW * wave + rr;
            if (y > ty1)
                break;
            int roff[LPG];
            float rly[LPG];
#pragma unroll
            for (int j = 0; j < LPG; ++j)
                lane_level_row(lv[j], y, roff[j], rly[j]);
            const int64_t orow = obase + (uint32_t)(y * W + tx0 + col);   // < H W + 64 <= 2^31 + 63

#pragma unroll
            for (int cg = 0; cg < TWG; ++cg) {
                if (tx0 + 16 * cg > tx1)
                    break;
                // Re-read the LDS operands per group rather than letting the
                // compiler keep loop-invariant ones in VGPRs (occupancy).
                asm volatile("" ::: "memory");

                // layer 1: B operand = the lane's LPG upsampled levels, split
                // and packed hi and lo into one K step
                float u[LPG];
#pragma unroll
                for (int j = 0; j < LPG; ++j)
                    u[j] = lane_level_sample(lds, lv[j], roff[j], rly[j], cg);
                u32x4 bx = {0u, 0u, 0u, 0u};
#pragma unroll
                for (int j = 0; j + 1 < LPG; j += 2) {
                    const u32x2 q = split_pair(u[j], u[j + 1]);
                    bx[j] = q[0];
                    bx[j + 1] = q[1];
                }
                if (LPG & 1)
                    bx[LPG - 1] = split_one(u[LPG - 1]);
                f32x4 d[NB];
#pragma unroll
                for (int ob = 0; ob < NB; ++ob) {
                    // (A operands read from LDS per group, like the hidden layers')
                    const u32x4 w1 = *reinterpret_cast<const u32x4 *>(&ldsu[LY::W1A + (ob * 64 + lane) * 4]);
                    d[ob] = *reinterpret_cast<const f32x4 *>(&lds[LY::B1 + (ob * 64 + lane) * 4]);
                    d[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w1), as_bf16x8(bx), d[ob], 0, 0, 0);
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
                    // A operands from LDS (16 bytes per lane per block and K
                    // step), read per group: held in VGPRs they would cost a
                    // wavefront per SIMD
#pragma unroll
                    for (int st = 0; st < KS2; ++st) {
                        u32x4 wa[NB];
#pragma unroll
                        for (int ob = 0; ob < NB; ++ob)
                            wa[ob] = *reinterpret_cast<const u32x4 *>(
                                &ldsu[LY::WHA + (((hl * NB + ob) * KS2 + st) * 64 + lane) * 4]);
#pragma unroll
                        for (int ob = 0; ob < NB; ++ob) {
                            e[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(wa[ob]), as_bf16x8(xh[st]), e[ob],
                                                                            0, 0, 0);
                            e[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(wa[ob]), as_bf16x8(xl[st]), e[ob],
                                                                            0, 0, 0);
                        }
                    }
#pragma unroll
                    for (int ob = 0; ob < NB; ++ob)
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            d[ob][r] = relu(e[ob][r]);
                }

                // output layer on the vector ALU (fp32); weight reads are issued
                // two at a time before their first use (four at a time cost
                // the wider shapes a wavefront per SIMD)
                float o0 = ob0, o1 = ob1, o2 = ob2;
#pragma unroll
                for (int ob = 0; ob < NB; ++ob) {
#pragma unroll
                    for (int r0 = 0; r0 < 4; r0 += 2) {
                        f32x4 w3[2];
#pragma unroll
                        for (int r = 0; r < 2; ++r)
                            w3[r] = *reinterpret_cast<const f32x4 *>(&lds[LY::W3 + ((ob * 4 + r0 + r) * 4 + g) * 4]);
#pragma unroll
                        for (int r = 0; r < 2; ++r) {
                            o0 = __builtin_fmaf(w3[r][0], d[ob][r0 + r], o0);
                            o1 = __builtin_fmaf(w3[r][1], d[ob][r0 + r], o1);
                            o2 = __builtin_fmaf(w3[r][2], d[ob][r0 + r], o2);
                        }
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

template <int NB, int NH, int LPG, int RPW>
hipError_t launch_rows(const DecodeParams &p, hipStream_t s, int tiles_x, int tiles, int bpi)
{
    const int64_t nblocks = (int64_t)bpi * p.batch;
    if (nblocks > 0x7fffffff)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_mfma_bf16<NB, NH, LPG, RPW>), dim3((unsigned)nblocks), dim3(kThreads), 0, s, p, bpi,
                       tiles_x, tiles, tile_row_recip(tiles_x, tiles));
    return hipGetLastError();
}

// 32- or 16-row tiles when every workgroup of the launch averages two or
// more of them and the taller boxes keep 4 wavefronts per SIMD (or the
// 8-row instance's occupancy, if lower), else 8-row.
template <int NB, int NH, int LPG>
hipError_t launch(const DecodeParams &p, hipStream_t s, int num_cus)
{
    const int tiles_x = (p.W + TW - 1) / TW;
    const int tiles8 = tiles_x * ((p.H + TH - 1) / TH);
    const int tiles16 = tiles_x * ((p.H + 4 * kWaves - 1) / (4 * kWaves));
    static int occ8 = 0, occ16 = 0;   // workgroups per CU of each instance
    const int bpi8 = blocks_per_image(k_mfma_bf16<NB, NH, LPG, 2>, p, num_cus, tiles8, occ8);
    const int bpi16 = blocks_per_image(k_mfma_bf16<NB, NH, LPG, 4>, p, num_cus, tiles16, occ16);
    const int tiles32 = tiles_x * ((p.H + 8 * kWaves - 1) / (8 * kWaves));
    static int occ32 = 0;
    const int bpi32 = blocks_per_image(k_mfma_bf16<NB, NH, LPG, 8>, p, num_cus, tiles32, occ32);
    // (4 wavefronts per SIMD hide the tile loop's latencies: the 32-row
    // tiles' smaller share of per-tile work outweighs a fifth)
    const int occ_need = occ8 < 4 ? occ8 : 4;
    if (occ32 >= occ_need && tiles32 >= 2 * bpi32)
        return launch_rows<NB, NH, LPG, 8>(p, s, tiles_x, tiles32, bpi32);
    if (occ16 >= occ_need && tiles16 >= 2 * bpi16)
        return launch_rows<NB, NH, LPG, 4>(p, s, tiles_x, tiles16, bpi16);
    return launch_rows<NB, NH, LPG, 2>(p, s, tiles_x, tiles8, bpi8);
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
