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
//   The first layer's operands are loaded once per workgroup straight into
//   VGPRs.  The hidden matrices, the biases and the output layer's weights
//   are copied once per workgroup into LDS, zero padded, at positions that
//   make every operand a contiguous 16-byte read (see swz below), and read
//   from there per 16-pixel group, which keeps VGPR use low enough for 3-5
//   wavefronts per SIMD.  The output layer (3 neurons) runs on the vector
//   ALU: each lane forms partial sums over the hidden values it holds and two
//   cross-lane swaps add the four lane groups.
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

// Operand placement.  Output neuron 16 ob + 4 r + g sits on accumulator row
// 4 g + r of block ob (lane group g, register r), and a hidden layer's K step
// (q, r) takes inputs 16 q + 4 r + g.  In LDS each 16-neuron group is stored
// with the two 2-bit halves of its index swapped, swz(n), for both the rows
// (output neurons) and the columns (inputs) of a matrix and for the bias and
// output-layer vectors.  A lane's four K steps of a quad are then one
// contiguous 16-byte read: row swz(16 ob + rn(i)) = 16 ob + i holds, at
// columns 16 q + 4 g .. + 3, inputs 16 q + 4 r + g for r = 0 .. 3; its
// accumulator-layout bias is the 16 bytes at 16 ob + 4 g, and so are its
// output-layer weights.  The staging needs no index arithmetic either: a
// wavefront copies whole matrix rows, one column per lane, so the row part
// of every address is uniform and the column part is the lane's own.
__host__ __device__ constexpr int swz(int n) { return (n & ~15) | ((n & 3) << 2) | ((n >> 2) & 3); }

template <int NB, int NH, int LS, int KSH, int THT>
struct Layout {
    static constexpr int N = 16 * NB;                               // padded hidden width
    static constexpr int KSH4 = (KSH + 3) / 4;                      // quads of hidden K steps
    // row pitch of a staged hidden matrix: a multiple of 4 floats (16-byte
    // reads) with pitch / 4 odd, so the 16 rows one lane group reads fall in
    // distinct 16-byte bank groups
    static constexpr int PITCH = N + 4;
    static constexpr int WH = 0;                                    // [NH][N rows][PITCH]
    static constexpr int BIAS = WH + NH * N * PITCH;                // [NH + 1][N]
    static constexpr int W3 = BIAS + (NH + 1) * N;                  // [3][N]
    static constexpr int LAT = W3 + 3 * N;                          // latent boxes
    static constexpr int SIZE = LAT + box_offset<THT>(4 * LS);
};

// Neuron on row `row` of an output block; the map is its own inverse.
__device__ __forceinline__ int row_neuron(int row) { return 4 * (row & 3) + (row >> 2); }

// s_setprio with a run-time level in 0 .. 3 (the instruction takes an
// immediate)
__device__ __forceinline__ void set_priority(int level)
{
    switch (level) {
    case 3: __builtin_amdgcn_s_setprio(3); break;
    case 2: __builtin_amdgcn_s_setprio(2); break;
    case 1: __builtin_amdgcn_s_setprio(1); break;
    default: __builtin_amdgcn_s_setprio(0); break;
    }
}

// NB: 16-neuron blocks of the hidden width; NH: hidden layers; LS: K steps of
// the first layer (ceil(L / 4)); KSH: K steps of the hidden layers (inputs
// 4 KSH and up are padding and skipped); RPW: tile rows per wavefront (a tile
// is 4 RPW rows: 8, or 16 when the launch has tiles to spare).  The 64-wide
// 16-row instances are held to 128 VGPRs (4 wavefronts per SIMD, as their
// 8-row ones; unconstrained they take 145); held there, the 40- and 48-wide
// ones measured slower at the same register count, so they are not.
template <int NB, int NH, int LS, int KSH, int RPW>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(RPW == 4 && NB == 4 && LS <= 2 ? 4 : 1)))
void k_mfma_f32(DecodeParams p, int blocks_per_image, int tiles_x, int tiles, uint32_t tx_recip)
{
    static_assert(KSH <= 4 * NB && KSH > 4 * (NB - 1), "KSH must end in the last block");
    constexpr int THT = kWaves * RPW;   // tile rows
    using LY = Layout<NB, NH, LS, KSH, THT>;
    constexpr int N = LY::N, PITCH = LY::PITCH;
    __shared__ __attribute__((aligned(16))) float lds[LY::SIZE];

    warm_kernel_args<sizeof(DecodeParams)>();
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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

    float boxv[box_regs<4 * LS, THT>()];
    float w1[NB][LS];

    // ---- parameters.  Every load is issued before the first is waited for:
    // the first tile's latent boxes, then the first layer's operands
    // straight into registers and the hidden matrices' rows, biases and
    // output weights into registers; after that everything is stored to LDS.
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
        constexpr int RW = N / 4;                  // matrix rows per wavefront
        float hrow[NH > 0 ? NH : 1][RW];
        float bv, w3v;
        // The parameters are read through raw buffers whose range check
        // returns 0 past each array's end, so no index is clamped to stay in
        // bounds: rows past a layer's outputs read 0, and entries of a row
        // past the layer's inputs (which read the next row) are zeroed when
        // stored.  No load sits behind a branch or feeds a select before the
        // last load is issued, so no wait is placed between them.  A hidden
        // matrix row's offset is the lane's plus a constant per row.
        const int lw = min(wave, NH), l3 = min(wave, 2);    // bias layer / output row of this wavefront
        auto load_all = [&](auto bf16) {
            constexpr bool BF = decltype(bf16)::value;
            constexpr unsigned ES = BF ? 2 : 4;
            auto ld = [](__amdgpu_buffer_rsrc_t r, unsigned byte_off) {
                if constexpr (BF)
                    return __uint_as_float((uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, byte_off, 0, 0) << 16);
                else
                    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0));
            };
            // layer 1, A operand: lane (g, i) holds W1[16 ob + rn(i)][4 s + g]
            const auto w1b = raw_buffer(lp[0].w, (unsigned)(N1 * L) * ES);
            const unsigned w1o = (unsigned)(row_neuron(col) * L + g) * ES;
#pragma unroll
            for (int ob = 0; ob < NB; ++ob)
#pragma unroll
                for (int s = 0; s < LS; ++s)
                    w1[ob][s] = ld(w1b, w1o + (unsigned)(16 * ob * L + 4 * s) * ES);
            // hidden layer h: wavefront w copies rows w, w + 4, ..., lane c column c
#pragma unroll
            for (int h = 0; h < NH; ++h) {
                const int fin = wd[1 + h], fout = wd[2 + h];
                const auto hb = raw_buffer(lp[1 + h].w, (unsigned)(fout * fin) * ES);
                const unsigned o0 = (unsigned)(wave * fin + lane) * ES, step = (unsigned)(4 * fin) * ES;
#pragma unroll
                for (int t = 0; t < RW; ++t)
                    hrow[h][t] = ld(hb, o0 + t * step);
            }
            // the bias of layer min(w, NH); row min(w, 2) of the output layer
            const LayerParams lb = layer_params(p, lw, b);
            bv = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                raw_buffer(lb.b, (unsigned)p.widths[1 + lw] * 4), (unsigned)lane * 4, 0, 0));
            w3v = ld(raw_buffer(lp[NH + 1].w, (unsigned)(3 * NL) * ES), (unsigned)(l3 * NL + lane) * ES);
        };
        // the first tile's latent loads go out first: every workgroup reads
        // texels of its own, while the parameters are shared and sit in the
        // L2 (the parameter stores below then wait for the boxes as well,
        // which measured cheaper than starting the boxes later)
        if (blk < tiles) {
            const int by = tile_row(blk, tiles_x, tx_recip);
            load_boxes<4 * LS, THT>(boxv, p, b, by * THT, (blk - by * tiles_x) * TW, tid);
        }
        if (lp[0].bf16)
            load_all(std::true_type{});
        else
            load_all(std::false_type{});
        // zero what lies outside each layer's shape.  The first layer's rows
        // past its outputs read 0; of its inputs only the last K step's can
        // lie past L (4 (LS - 1) < L), and those read the next row.
        {
            const bool in_l = 4 * (LS - 1) + g < L;
#pragma unroll
            for (int ob = 0; ob < NB; ++ob)
                w1[ob][LS - 1] = in_l ? w1[ob][LS - 1] : 0.0f;
        }
        if (lane < N) {
            // row wave + 4 t goes to swz(wave + 4 t) = 16 (t / 4) + 4 wave + t % 4
            // (wave < 4): a per-lane base plus a constant per row
            const int sc = swz(lane);
            float *wrow = lds + LY::WH + 4 * wave * PITCH + sc;
#pragma unroll
            for (int h = 0; h < NH; ++h) {
                const bool cin = lane < wd[1 + h];
#pragma unroll
                for (int t = 0; t < RW; ++t)
                    wrow[(h * N + 16 * (t >> 2) + (t & 3)) * PITCH] = cin ? hrow[h][t] : 0.0f;
            }
            if (wave <= NH)
                lds[LY::BIAS + wave * N + sc] = bv;
            if (wave < 3)
                lds[LY::W3 + wave * N + sc] = lane < NL ? w3v : 0.0f;
        }
    }
    if (blk < tiles)
        store_boxes<4 * LS, THT>(lds + LY::LAT, boxv, tid);
    __syncthreads();

    // ---- the level each lane samples for K step s of the first layer.  Lanes
    // whose level 4 s + g does not exist sample level 0 instead: their
    // first-layer weights are zero, so the (finite) value is ignored.
    LaneLevel lv[LS];
    lane_levels_init<THT, 4, 1>(lv, g, L, LY::LAT, std::make_integer_sequence<int, LS>{});

    const int H = p.H, W = p.W;
    const int64_t plane = (int64_t)H * W;
    // Lane group g (< 3) stores channel g; lane group 0 carries the output
    // biases in its partial sums.
    const int64_t obase = (int64_t)(uint64_t)(uint32_t)(3 * b + min(g, 2)) * plane;
    const float ob0 = g == 0 ? b3_0 : 0.0f, ob1 = g == 0 ? b3_1 : 0.0f, ob2 = g == 0 ? b3_2 : 0.0f;
    constexpr int KS1 = KSH;   // live registers of a hidden activation
    constexpr int W3NB = 2;   // (larger chunks raise the VGPR count of the wider shapes)

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

        // A wavefront's priority is raised for the first row of each tile and
        // dropped after it, so that the wavefronts of a SIMD progress together
        // instead of oldest first, and none is left to run alone at the end.
        // 8-row tiles (one tile per workgroup in small launches) step it
        // down per pair of 16-pixel groups instead: 3, 2 over the first
        // row, 1, 0 over the second.
        __builtin_amdgcn_s_setprio(1);
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

            // 8-row tiles (small launches, mostly one tile per workgroup)
            // evaluate two 16-pixel groups per pass: their matrix chains
            // interleave and share every weight read.  (The second group of a
            // pair may lie right of the image: its taps read clamped box
            // entries and its store is skipped.)  16-row tiles keep one group
            // per pass, for occupancy; the paired code instantiated with one
            // group compiled to more VGPRs, so they keep their own loop.
            constexpr bool PAIRS = RPW == 2;
            if constexpr (PAIRS) {
                constexpr int G = 2;
#pragma unroll
                for (int cg = 0; cg < TWG; cg += G) {
                    if (tx0 + 16 * cg > tx1)
                        break;   // wave-uniform: the column group lies right of the image
                    // Re-read the LDS operands per pass rather than letting the
                    // compiler keep loop-invariant ones in VGPRs (occupancy).
                    asm volatile("" ::: "memory");
                    set_priority((rr == 0 ? 3 : 1) - cg / 2);

                    // layer 1: K = levels, B operand = upsampled pyramid
                    f32x4 d[G][NB];
#pragma unroll
                    for (int ob = 0; ob < NB; ++ob) {
                        const f32x4 bias = *reinterpret_cast<const f32x4 *>(&lds[LY::BIAS + 16 * ob + 4 * g]);
#pragma unroll
                        for (int gi = 0; gi < G; ++gi)
                            d[gi][ob] = bias;
                    }
#pragma unroll
                    for (int s = 0; s < LS; ++s) {
                        float u[G];
#pragma unroll
                        for (int gi = 0; gi < G; ++gi)
                            u[gi] = lane_level_sample(lds, lv[s], roff[s], rly[s], cg + gi);
#pragma unroll
                        for (int ob = 0; ob < NB; ++ob)
#pragma unroll
                            for (int gi = 0; gi < G; ++gi)
                                d[gi][ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(w1[ob][s], u[gi], d[gi][ob], 0, 0, 0);
                    }
#pragma unroll
                    for (int gi = 0; gi < G; ++gi)
#pragma unroll
                        for (int ks = 0; ks < KS1; ++ks)
                            d[gi][ks >> 2][ks & 3] = relu(d[gi][ks >> 2][ks & 3]);

                    // hidden layers
#pragma unroll
                    for (int h = 0; h < NH; ++h) {
                        f32x4 e[G][NB];
#pragma unroll
                        for (int ob = 0; ob < NB; ++ob) {
                            const f32x4 bias =
                                *reinterpret_cast<const f32x4 *>(&lds[LY::BIAS + (1 + h) * N + 16 * ob + 4 * g]);
#pragma unroll
                            for (int gi = 0; gi < G; ++gi)
                                e[gi][ob] = bias;
                        }
                        // A operands of K steps 4q .. 4q+3 come from LDS, one 16-byte
                        // read per output block; step 4q + j pairs with register j
                        // of input block q.
#pragma unroll
                        for (int q = 0; q < LY::KSH4; ++q) {
                            f32x4 wq[NB];
#pragma unroll
                            for (int ob = 0; ob < NB; ++ob)
                                wq[ob] = *reinterpret_cast<const f32x4 *>(
                                    &lds[LY::WH + (h * N + 16 * ob + col) * PITCH + 16 * q + 4 * g]);
#pragma unroll
                            for (int j = 0; j < 4; ++j) {
                                if (4 * q + j < KSH) {
#pragma unroll
                                    for (int ob = 0; ob < NB; ++ob)
#pragma unroll
                                        for (int gi = 0; gi < G; ++gi)
                                            e[gi][ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(wq[ob][j], d[gi][q][j],
                                                                                             e[gi][ob], 0, 0, 0);
                                }
                            }
                        }
#pragma unroll
                        for (int gi = 0; gi < G; ++gi)
#pragma unroll
                            for (int ks = 0; ks < KS1; ++ks)
                                d[gi][ks >> 2][ks & 3] = relu(e[gi][ks >> 2][ks & 3]);
                    }

                    // output layer on the vector ALU: partial sums over this lane's
                    // live hidden values, then a sum over the four lane groups
                    // (weights of W3NB blocks are read at a time, all before their
                    // first use, so one LDS round trip covers each chunk)
                    float o[G][3];
#pragma unroll
                    for (int gi = 0; gi < G; ++gi) {
                        o[gi][0] = ob0;
                        o[gi][1] = ob1;
                        o[gi][2] = ob2;
                    }
#pragma unroll
                    for (int nb0 = 0; nb0 < NB; nb0 += W3NB) {
                        f32x4 w3[W3NB][3];
#pragma unroll
                        for (int j = 0; j < W3NB; ++j)
                            if (nb0 + j < NB)
#pragma unroll
                                for (int c = 0; c < 3; ++c)
                                    w3[j][c] = *reinterpret_cast<const f32x4 *>(&lds[LY::W3 + c * N + 16 * (nb0 + j) + 4 * g]);
#pragma unroll
                        for (int j = 0; j < W3NB; ++j) {
#pragma unroll
                            for (int r = 0; r < 4; ++r) {
                                if (nb0 + j < NB && 4 * (nb0 + j) + r < KS1) {
#pragma unroll
                                    for (int gi = 0; gi < G; ++gi) {
                                        const float hv = d[gi][nb0 + j][r];
                                        o[gi][0] = __builtin_fmaf(w3[j][0][r], hv, o[gi][0]);
                                        o[gi][1] = __builtin_fmaf(w3[j][1][r], hv, o[gi][1]);
                                        o[gi][2] = __builtin_fmaf(w3[j][2][r], hv, o[gi][2]);
                                    }
                                }
                            }
                        }
                    }
#pragma unroll
                    for (int gi = 0; gi < G; ++gi) {
                        const float v = row_sum3(o[gi][0], o[gi][1], o[gi][2]);
                        if (g < 3 && tx0 + 16 * (cg + gi) + col <= tx1)
                            store_out(p, orow + 16 * (cg + gi), v);
                    }
                }
            } else {
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
                        d[ob] = *reinterpret_cast<const f32x4 *>(&lds[LY::BIAS + 16 * ob + 4 * g]);
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
                            e[ob] = *reinterpret_cast<const f32x4 *>(&lds[LY::BIAS + (1 + h) * N + 16 * ob + 4 * g]);
                        // A operands of K steps 4q .. 4q+3 come from LDS, one 16-byte
                        // read per output block; step 4q + j pairs with register j
                        // of input block q.
#pragma unroll
                        for (int q = 0; q < LY::KSH4; ++q) {
                            f32x4 wq[NB];
#pragma unroll
                            for (int ob = 0; ob < NB; ++ob)
                                wq[ob] = *reinterpret_cast<const f32x4 *>(
                                    &lds[LY::WH + (h * N + 16 * ob + col) * PITCH + 16 * q + 4 * g]);
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
                    // (weights of W3NB blocks are read at a time, all before their
                    // first use, so one LDS round trip covers each chunk)
                    float o0 = ob0, o1 = ob1, o2 = ob2;
#pragma unroll
                    for (int nb0 = 0; nb0 < NB; nb0 += W3NB) {
                        f32x4 w3[W3NB][3];
#pragma unroll
                        for (int j = 0; j < W3NB; ++j)
                            if (nb0 + j < NB)
#pragma unroll
                                for (int c = 0; c < 3; ++c)
                                    w3[j][c] = *reinterpret_cast<const f32x4 *>(&lds[LY::W3 + c * N + 16 * (nb0 + j) + 4 * g]);
#pragma unroll
                        for (int j = 0; j < W3NB; ++j) {
#pragma unroll
                            for (int r = 0; r < 4; ++r) {
                                if (nb0 + j < NB && 4 * (nb0 + j) + r < KS1) {
                                    const float hv = d[nb0 + j][r];
                                    o0 = __builtin_fmaf(w3[j][0][r], hv, o0);
                                    o1 = __builtin_fmaf(w3[j][1][r], hv, o1);
                                    o2 = __builtin_fmaf(w3[j][2][r], hv, o2);
                                }
                            }
                        }
                    }
                    const float v = row_sum3(o0, o1, o2);
                    if (g < 3 && tx0 + 16 * cg + col <= tx1)
                        store_out(p, orow + 16 * cg, v);
                }
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

// Hidden K steps the shape needs: ceil(width / 4) of the widest hidden layer.
// Every hidden activation is the input of a later layer (the next hidden
// layer or the output layer), and the K-step count also bounds the ReLU and
// the output layer's sums, so the last hidden width counts as well.
int hidden_ksteps(int nl, const int32_t *widths);

template <int NB, int NH, int LS, int KSH, int RPW>
hipError_t launch_rows(const DecodeParams &p, hipStream_t s, int tiles_x, int tiles, int bpi)
{
    const int64_t nblocks = (int64_t)bpi * p.batch;
    if (nblocks > 0x7fffffff)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_mfma_f32<NB, NH, LS, KSH, RPW>), dim3((unsigned)nblocks), dim3(kThreads), 0, s, p, bpi,
                       tiles_x, tiles, tile_row_recip(tiles_x, tiles));
    return hipGetLastError();
}

// 16-row tiles (4 rows per wavefront) when every workgroup of the launch
// averages two or more of them and the taller boxes cost no occupancy: the
// per-tile work (box staging, its two barriers, the tile's level geometry)
// then spreads over twice the pixels.  Else 8-row tiles, so that a single
// small image still fills the device.
template <int NB, int NH, int LS, int KSH>
hipError_t launch(const DecodeParams &p, hipStream_t s, int num_cus)
{
    const int tiles_x = (p.W + TW - 1) / TW;
    const int tiles8 = tiles_x * ((p.H + TH - 1) / TH);
    const int tiles16 = tiles_x * ((p.H + 4 * kWaves - 1) / (4 * kWaves));
    static int occ8 = 0, occ16 = 0;   // workgroups per CU of each instance
    const int bpi8 = blocks_per_image(k_mfma_f32<NB, NH, LS, KSH, 2>, p, num_cus, tiles8, occ8);
    const int bpi16 = blocks_per_image(k_mfma_f32<NB, NH, LS, KSH, 4>, p, num_cus, tiles16, occ16);
    if (occ16 >= occ8 && tiles16 >= 2 * bpi16)
        return launch_rows<NB, NH, LS, KSH, 4>(p, s, tiles_x, tiles16, bpi16);
    return launch_rows<NB, NH, LS, KSH, 2>(p, s, tiles_x, tiles8, bpi8);
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
