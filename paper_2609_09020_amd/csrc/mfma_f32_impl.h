// fp32 matrix-core decode kernel (v_mfma_f32_16x16x4_f32), shared by the
// k_mfma_f32_nh*.hip translation units that instantiate it.
//
// What it computes (PIC, Sec. 3.1 and App. A): per pixel, every latent level
// upsampled bilinearly (half-pixel centres, edge replication, scale 2^k) into
// an L-vector, then the synthesis MLP (ReLU between layers, none after the
// last), clamp to [0, 1], optional 8-bit quantisation.
//
// Work decomposition
//   A workgroup (4 wavefronts) owns one image and walks tiles of 8 rows x 64
//   columns of it.  Per tile it stages, for every level, the box of latent
//   texels the tile's pixels sample into LDS with coalesced loads
//   (decode_common.h); each wavefront then evaluates two rows of the tile,
//   16 consecutive pixels at a time.
//
// Matrix-core mapping (lane l, lane group g = l / 16, i = l % 16)
//   v_mfma_f32_16x16x4_f32 takes A[i][g] and B[g][i] from lane l and returns
//   D[4g + r][i] in register r of lane l.  A layer is D = W * H^T + bias with
//   16 output neurons on the rows of a block and the 16 pixels on the columns.
//   Row 4g + r of output block ob holds neuron 16 ob + 4 r + g, so register r
//   of block nb, read across the lane groups, holds neurons 16 nb + 4 r + g:
//   exactly the B operand of K step (nb, r) of the next layer, with K index g.
//   Layers therefore chain through the accumulators with no data movement.
//   K steps run in increasing input order (inputs 4j .. 4j+3 at step j), and a
//   partially filled last block keeps its n valid inputs on steps < ceil(n/4)
//   so steps over padding are skipped.  Lane group g of the first layer's B
//   operand supplies level 4 s + g of the lane's pixel at K step s.
//
//   Weights are gathered once per workgroup into LDS in that operand layout
//   (zero padded).  The first layer's operands are then held in VGPRs; the
//   hidden layers' are read from LDS as needed (16 bytes per lane cover four
//   K steps), which keeps VGPR use low enough for 3-5 wavefronts per SIMD;
//   biases (accumulator layout) and the output layer's weights are read from
//   LDS per 16-pixel group too.  The output layer (3 neurons) runs on the vector ALU: each
//   lane forms partial sums over the hidden values it holds and two cross-lane
//   swaps add the four lane groups.
//
//   fp32 matrix and vector instructions share a SIMD's issue capacity, so the
//   per-group vector work is kept small: fixed-offset bilinear taps, ReLU as
//   one integer max, no padding registers touched.
#pragma once

#include <type_traits>

#include "decode_common.h"

namespace pic {
namespace mfma_f32 {

using namespace tile;

template <int NB, int NH, int LS, int KSH>
struct Layout {
    static constexpr int W1A = 0;                                   // [NB][LS][64]
    static constexpr int KSH4 = (KSH + 3) / 4;                      // quads of hidden K steps
    static constexpr int WHA = W1A + NB * LS * 64;                  // [NH][NB][KSH4][64][4 steps]
    static constexpr int B1 = WHA + NH * NB * KSH4 * 256;           // [NB][64][4]
    static constexpr int BH = B1 + NB * 64 * 4;                     // [NH][NB][64][4]
    static constexpr int W3 = BH + NH * NB * 64 * 4;                // [NB][4 r][4 g][4 c]
    static constexpr int LAT = W3 + NB * 4 * 4 * 4;                 // latent boxes
    static constexpr int SIZE = LAT + box_offset(4 * LS);
    // the parameters as the caller lays them out are first staged in the
    // regions their operand layouts then replace (each is at least as large)
    static constexpr int N = 16 * NB;
    static_assert(N * 4 * LS <= NB * LS * 64, "layer 1 fits its region");
    static_assert(N * N <= NB * KSH4 * 256 || KSH < 4 * NB, "hidden layers fit their regions");
    static_assert(3 * N <= NB * 64, "output layer fits its region");
};

// Neuron on row `row` of an output block; the map is its own inverse.
__device__ __forceinline__ int row_neuron(int row) { return 4 * (row & 3) + (row >> 2); }

// NB: 16-neuron blocks of the hidden width; NH: hidden layers; LS: K steps of
// the first layer (ceil(L / 4)); KSH: K steps of the hidden layers (inputs
// 4 KSH and up are padding and skipped).
template <int NB, int NH, int LS, int KSH>
__global__ __launch_bounds__(kThreads) void k_mfma_f32(DecodeParams p, int blocks_per_image, int tiles_x, int tiles)
{
    static_assert(KSH <= 4 * NB && KSH > 4 * (NB - 1), "KSH must end in the last block");
    using LY = Layout<NB, NH, LS, KSH>;
    __shared__ __attribute__((aligned(16))) float lds[LY::SIZE];

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

    float boxv[box_regs<4 * LS>()];

    // ---- stage this image's parameters into LDS in operand layouts: first
    // as the caller lays them out, with contiguous loads all in flight at
    // once, then permuted through registers
    {
        // every layer's pointers and widths first (one batch of scalar
        // loads), then the loads themselves: raw copies whose entries past
        // the layer's size hold anything (the permutation reads only valid
        // ones), so no load is waited for before the latents' go out
        LayerParams lp[NH + 2];
        int wd[NH + 3];
#pragma unroll
        for (int l = 0; l < NH + 2; ++l)
            lp[l] = layer_params(p, l, b);
#pragma unroll
        for (int l = 0; l < NH + 3; ++l)
            wd[l] = p.widths[l];
        const int N1 = wd[1], NL = wd[NH + 1];
        constexpr int KSH4 = LY::KSH4;
        // raw copies: layer 1 in W1A, hidden layer h in its WHA block (or, when
        // the last K steps are skipped and the block is smaller, in the box
        // area), the output layer in W3, biases in B1 / BH
        constexpr int RAW_H = LY::N * LY::N <= NB * KSH4 * 256 ? 0 : 1;
        static_assert(!RAW_H || NH * LY::N * LY::N <= box_offset(4 * LS), "hidden layers fit the box area");
        auto raw_h = [&](int h) { return RAW_H ? LY::LAT + h * LY::N * LY::N : LY::WHA + h * NB * KSH4 * 256; };
        Part<LY::N, float> rb[NH + 1];
#pragma unroll
        for (int h = 0; h <= NH; ++h) {
            const int fout = wd[1 + h];
            rb[h] = load_part<LY::N, float>([&](int s) { return lp[h].bias_clamped(s, fout); });
        }
        Part<LY::N * 4 * LS, float> r1;
        Part<LY::N * LY::N, float> rh[NH > 0 ? NH : 1];
        Part<3 * LY::N, float> r3;
        // one straight run of loads per weight type (uniform branch)
        auto load_weights = [&](auto bf16) {
            constexpr bool BF = decltype(bf16)::value;
            r1 = load_part<LY::N * 4 * LS, float>([&](int s) { return lp[0].template weight_clamped<BF>(s, N1 * L); });
#pragma unroll
            for (int h = 0; h < NH; ++h) {
                const int n = wd[1 + h] * wd[2 + h];
                rh[h] = load_part<LY::N * LY::N, float>([&](int s) { return lp[1 + h].template weight_clamped<BF>(s, n); });
            }
            r3 = load_part<3 * LY::N, float>([&](int s) { return lp[NH + 1].template weight_clamped<BF>(s, 3 * NL); });
        };
        if (lp[0].bf16)
            load_weights(std::true_type{});
        else
            load_weights(std::false_type{});
        // the first tile's latent loads go out behind the parameters: loads
        // complete in order, so the permutation below need not wait for them
        if (blk < tiles)
            load_boxes<4 * LS>(boxv, p, b, (blk / tiles_x) * TH, (blk % tiles_x) * TW, tid);
        store_part(lds + LY::W1A, r1);
#pragma unroll
        for (int h = 0; h < NH; ++h)
            store_part(lds + raw_h(h), rh[h]);
        store_part(lds + LY::W3, r3);
#pragma unroll
        for (int h = 0; h <= NH; ++h)
            store_part(lds + LY::B1 + h * NB * 256, rb[h]);
        __syncthreads();

        const auto w1a = load_part<NB * LS * 64, float>([&](int s) {          // layer 1, A layout
            const int ln = s & 63, step = (s >> 6) % LS, ob = (s >> 6) / LS;
            const int out = 16 * ob + row_neuron(ln & 15), in = 4 * step + (ln >> 4);
            return (out < N1 && in < L) ? lds[LY::W1A + out * L + in] : 0.0f;
        });
        Part<NB * KSH4 * 256, float> wha[NH > 0 ? NH : 1];
#pragma unroll
        for (int h = 0; h < NH; ++h) {                                         // hidden layers, A layout
            const int fin = p.widths[1 + h], fout = p.widths[2 + h];
            wha[h] = load_part<NB * KSH4 * 256, float>([&](int s) {
                const int j = s & 3, ln = (s >> 2) & 63, q = (s >> 8) % KSH4, ob = (s >> 8) / KSH4;
                const int ks = 4 * q + j;
                const int out = 16 * ob + row_neuron(ln & 15);
                const int in = 16 * (ks >> 2) + 4 * (ks & 3) + (ln >> 4);
                return (ks < KSH && out < fout && in < fin) ? lds[raw_h(h) + out * fin + in] : 0.0f;
            });
        }
        Part<NB * 256, float> bias[NH + 1];
#pragma unroll
        for (int h = 0; h <= NH; ++h) {                                        // biases, accumulator layout
            const int fout = p.widths[1 + h];
            bias[h] = load_part<NB * 256, float>([&](int s) {
                const int r = s & 3, ln = (s >> 2) & 63, ob = s >> 8;
                const int n = 16 * ob + 4 * r + (ln >> 4);
                return n < fout ? lds[LY::B1 + h * NB * 256 + n] : 0.0f;
            });
        }
        const auto w3 = load_part<NB * 64, float>([&](int s) {                // output layer [ob][r][g][c]
            const int c = s & 3, gg = (s >> 2) & 3, r = (s >> 4) & 3, ob = s >> 6;
            const int n = 16 * ob + 4 * r + gg;
            return (c < 3 && n < NL) ? lds[LY::W3 + c * NL + n] : 0.0f;
        });
        __syncthreads();                   // every raw value is read
        store_part(lds + LY::W1A, w1a);
#pragma unroll
        for (int h = 0; h < NH; ++h)
            store_part(lds + LY::WHA + h * NB * KSH4 * 256, wha[h]);
#pragma unroll
        for (int h = 0; h <= NH; ++h)
            store_part(lds + LY::B1 + h * NB * 256, bias[h]);
        store_part(lds + LY::W3, w3);
    }
    if (blk < tiles)
        store_boxes<4 * LS>(lds + LY::LAT, boxv, p, tid);
    __syncthreads();

    float w1[NB][LS];
#pragma unroll
    for (int ob = 0; ob < NB; ++ob)
#pragma unroll
        for (int s = 0; s < LS; ++s)
            w1[ob][s] = lds[LY::W1A + (ob * LS + s) * 64 + lane];

    // ---- the level each lane samples for K step s of the first layer.  Lanes
    // whose level 4 s + g does not exist sample level 0 instead: their
    // first-layer weights are zero, so the (finite) value is ignored.
    LaneLevel lv[LS];
#pragma unroll
    for (int s = 0; s < LS; ++s) {
        const int k = 4 * s + g;
        lane_level_init(lv[s], k < L ? k : 0, LY::LAT);
    }

    const int H = p.H, W = p.W;
    const int64_t plane = (int64_t)H * W;
    // Lane group g (< 3) stores channel g; lane group 0 carries the output
    // biases in its partial sums.
    const int64_t obase = (int64_t)b * 3 * plane + (int64_t)min(g, 2) * plane;
    const float ob0 = g == 0 ? b3_0 : 0.0f, ob1 = g == 0 ? b3_1 : 0.0f, ob2 = g == 0 ? b3_2 : 0.0f;
    constexpr int KS1 = KSH;   // live registers of a hidden activation
    constexpr int W3CH = 6;   // (larger chunks raise the VGPR count of the wider shapes)

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
            stage_boxes<4 * LS>(lds + LY::LAT, p, b, ty0, tx0, tid);
            __syncthreads();
        }
        int ticket = 0;    // the tile after this one; its latency hides behind the tile
        if (dynamic && tid == 0)
            ticket = atomicAdd(ts.ctr, 1);
#pragma unroll
        for (int s = 0; s < LS; ++s)
            lane_level_tile(lv[s], ty0, tx0, tx1, col);

        // A wavefront's priority is raised for the first row of each tile and
        // dropped after it, so that the wavefronts of a SIMD progress together
        // instead of oldest first, and none is left to run alone at the end.
        __builtin_amdgcn_s_setprio(1);
#pragma unroll 1
        for (int rr = 0; rr < 2; ++rr) {
            const int y = ty0 + 2 * wave + rr;
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

                // layer 1: K = levels, B operand = upsampled pyramid
                f32x4 d[NB];
#pragma unroll
                for (int ob = 0; ob < NB; ++ob)
                    d[ob] = *reinterpret_cast<const f32x4 *>(&lds[LY::B1 + (ob * 64 + lane) * 4]);
#pragma unroll
                for (int s = 0; s < LS; ++s) {
                    const float u = lane_level_sample(lds, lv[s], roff[s], rly[s], cg);
#pragma unroll
                    for (int ob = 0; ob < NB; ++ob)
                        d[ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(w1[ob][s], u, d[ob], 0, 0, 0);
                }
#pragma unroll
                for (int ks = 0; ks < KS1; ++ks)
                    d[ks >> 2][ks & 3] = relu(d[ks >> 2][ks & 3]);

                // hidden layers
#pragma unroll
                for (int h = 0; h < NH; ++h) {
                    f32x4 e[NB];
#pragma unroll
                    for (int ob = 0; ob < NB; ++ob)
                        e[ob] = *reinterpret_cast<const f32x4 *>(&lds[LY::BH + ((h * NB + ob) * 64 + lane) * 4]);
                    // A operands of K steps 4q .. 4q+3 come from LDS, one 16-byte
                    // read per output block; step 4q + j pairs with register j
                    // of input block q.
#pragma unroll
                    for (int q = 0; q < LY::KSH4; ++q) {
                        f32x4 wq[NB];
#pragma unroll
                        for (int ob = 0; ob < NB; ++ob)
                            wq[ob] = *reinterpret_cast<const f32x4 *>(
                                &lds[LY::WHA + ((h * NB + ob) * LY::KSH4 + q) * 256 + lane * 4]);
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            if (4 * q + j < KSH) {
#pragma unroll
                                for (int ob = 0; ob < NB; ++ob)
                                    e[ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(wq[ob][j], d[q][j], e[ob], 0, 0, 0);
                            }
                        }
                    }
#pragma unroll
                    for (int ks = 0; ks < KS1; ++ks)
                        d[ks >> 2][ks & 3] = relu(e[ks >> 2][ks & 3]);
                }

                // output layer on the vector ALU: partial sums over this lane's
                // live hidden values, then a sum over the four lane groups
                // (weights are read W3CH at a time, all before their first use,
                // so one LDS round trip covers each chunk)
                float o0 = ob0, o1 = ob1, o2 = ob2;
#pragma unroll
                for (int k0 = 0; k0 < KS1; k0 += W3CH) {
                    f32x4 w3[W3CH];
#pragma unroll
                    for (int j = 0; j < W3CH; ++j)
                        if (k0 + j < KS1)
                            w3[j] = *reinterpret_cast<const f32x4 *>(&lds[LY::W3 + ((k0 + j) * 4 + g) * 4]);
#pragma unroll
                    for (int j = 0; j < W3CH; ++j) {
                        if (k0 + j < KS1) {
                            const float hv = d[(k0 + j) >> 2][(k0 + j) & 3];
                            o0 = __builtin_fmaf(w3[j][0], hv, o0);
                            o1 = __builtin_fmaf(w3[j][1], hv, o1);
                            o2 = __builtin_fmaf(w3[j][2], hv, o2);
                        }
                    }
                }
                const float v = row_sum3(o0, o1, o2);
                if (g < 3 && tx0 + 16 * cg + col <= tx1)
                    store_out(p, orow + 16 * cg, v);
            }
            __builtin_amdgcn_s_setprio(0);
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

// Hidden K steps the shape needs: ceil(width / 4) of the widest hidden input.
int hidden_ksteps(int nl, const int32_t *widths);

template <int NB, int NH, int LS, int KSH>
hipError_t launch(const DecodeParams &p, hipStream_t s, int num_cus)
{
    const int tiles_x = (p.W + TW - 1) / TW, tiles_y = (p.H + TH - 1) / TH;
    const int tiles = tiles_x * tiles_y;
    static int occ = 0;
    const int bpi = blocks_per_image(k_mfma_f32<NB, NH, LS, KSH>, p, num_cus, tiles, occ);
    const int64_t nblocks = (int64_t)bpi * p.batch;
    if (nblocks > 0x7fffffff)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_mfma_f32<NB, NH, LS, KSH>), dim3((unsigned)nblocks), dim3(kThreads), 0, s, p, bpi,
                       tiles_x, tiles);
    return hipGetLastError();
}

template <int NH>
hipError_t launch_nh(const DecodeParams &p, hipStream_t s, int num_cus)
{
    const int NB = hidden_blocks(p.nl, p.widths);
    const int LS = (p.L + 3) / 4;
    // Width 33..40 (three blocks, last one half used) gets its own K-step
    // count; every other width runs all 4 NB steps over zero padding.
    const bool k10 = NH > 0 && NB == 3 && hidden_ksteps(p.nl, p.widths) <= 10;
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

}  // namespace mfma_f32
}  // namespace pic
