// Fast fp32 kernel family: the synthesis MLP on the fp32 matrix cores
// (v_mfma_f32_16x16x4_f32), upsample and output layer on the vector ALU.
//
// Work unit: a wavefront evaluates 16 pixels at a time.  For every layer it
// computes D = W * H^T + bias with the output neurons on the 16 rows of a
// 16x16 block (one block per 16 neurons) and the 16 pixels on the columns.
//
// Operand layouts of v_mfma_f32_16x16x4_f32 (lane l, g = l / 16, i = l % 16):
//   A (16x4): lane l holds A[i][g];  B (4x16): lane l holds B[g][i];
//   D (16x16): lane l, register r holds D[4g + r][i].
// Row 4g + r of output block ob is neuron 16 ob + 4 r + g.  With that mapping
// register r of block nb, read across the four lane groups, holds neurons
// 16 nb + 4 r + g -- exactly a B operand with K index g.  A layer's output
// therefore feeds the next layer's MFMA directly, with no data movement; the
// next layer's weights are laid out to match (A[i][g] = W[row i's neuron]
// [16 nb + 4 r + g]).  A partially filled last block puts its n valid
// neurons on registers r < ceil(n / 4), so K steps over padding are skipped.
//
// Weights and biases of the image are loaded once per wavefront into VGPRs
// (zero padded) and stay there while the wavefront walks its pixels.  The
// first layer's B operand is the upsampled pyramid: lane group g computes
// level 4 s + g of the lane's pixel for K step s.  The output layer (3
// neurons) is done on the vector ALU: each lane multiplies the 4 NB hidden
// values it holds, then two cross-lane butterflies sum the four lane groups.
#include "pic_internal.h"

namespace pic {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxLS = 3;            // K steps of the first layer: ceil(L / 4) <= 3

__device__ __forceinline__ float weight_at(const DecodeParams &p, int64_t base, int idx)
{
    if (p.weights_bf16) {
        const uint16_t bits = static_cast<const uint16_t *>(p.weights)[base + idx];
        return __uint_as_float((uint32_t)bits << 16);
    }
    return static_cast<const float *>(p.weights)[base + idx];
}

// Neuron held on row `row` (0..15) of an output block.
__device__ __forceinline__ int row_neuron(int row) { return 4 * (row & 3) + (row >> 2); }

__device__ __forceinline__ float pow2_neg(int k) { return __int_as_float((127 - k) << 23); }

struct LevelLane {
    const float *base;   // this image's grid of the level
    int hk, wk;
    float inv;           // 2^-k
    bool valid;
};

__device__ __forceinline__ float sample(const LevelLane &lv, int y, int x)
{
    float sy = ((float)y + 0.5f) * lv.inv - 0.5f;
    float sx = ((float)x + 0.5f) * lv.inv - 0.5f;
    sy = fmaxf(sy, 0.0f);
    sx = fmaxf(sx, 0.0f);
    const int y0 = (int)sy, x0 = (int)sx;            // sy, sx >= 0: truncation is floor
    const int y1 = min(y0 + 1, lv.hk - 1), x1 = min(x0 + 1, lv.wk - 1);
    const float ly = sy - (float)y0, lx = sx - (float)x0;
    const float *r0 = lv.base + y0 * lv.wk, *r1 = lv.base + y1 * lv.wk;
    const float a = r0[x0], b = r0[x1], c = r1[x0], d = r1[x1];
    const float top = __builtin_fmaf(lx, b - a, a);
    const float bot = __builtin_fmaf(lx, d - c, c);
    return __builtin_fmaf(ly, bot - top, top);
}

template <int NB, int NH>
__global__ __launch_bounds__(kThreads) void k_mfma_f32(DecodeParams p, int blocks_per_image)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;
    const int b = blockIdx.x / blocks_per_image;
    const int blk = blockIdx.x - b * blocks_per_image;
    if (b >= p.batch)
        return;

    const int L = p.L;
    const int LS = (L + 3) >> 2;
    const int64_t wbase = (int64_t)b * p.w_stride;
    const int64_t bbase = (int64_t)b * p.b_stride;

    // ---- per-lane level descriptors for the first layer's B operand
    LevelLane lv[kMaxLS];
#pragma unroll
    for (int s = 0; s < kMaxLS; ++s) {
        const int k = 4 * s + g;
        lv[s].valid = k < L;
        const int kk = k < L ? k : 0;
        lv[s].hk = p.hk[kk];
        lv[s].wk = p.wk[kk];
        lv[s].inv = pow2_neg(kk);
        lv[s].base = p.lat[kk] + (int64_t)b * p.hk[kk] * p.wk[kk];
    }

    // ---- weights as A operands, biases as initial accumulators
    const int N1 = p.widths[1];
    float w1[NB][kMaxLS];
    f32x4 b1[NB];
#pragma unroll
    for (int ob = 0; ob < NB; ++ob) {
        const int out = 16 * ob + row_neuron(col);
#pragma unroll
        for (int s = 0; s < kMaxLS; ++s) {
            const int in = 4 * s + g;
            w1[ob][s] = (out < N1 && in < L) ? weight_at(p, wbase + p.woff[0], out * L + in) : 0.0f;
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int n = 16 * ob + 4 * r + g;
            b1[ob][r] = n < N1 ? p.biases[bbase + p.boff[0] + n] : 0.0f;
        }
    }
    float wh[NH > 0 ? NH : 1][NB][4 * NB];
    f32x4 bh[NH > 0 ? NH : 1][NB];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
        const int fin = p.widths[1 + h], fout = p.widths[2 + h];
#pragma unroll
        for (int ob = 0; ob < NB; ++ob) {
            const int out = 16 * ob + row_neuron(col);
#pragma unroll
            for (int ks = 0; ks < 4 * NB; ++ks) {
                const int in = 16 * (ks >> 2) + 4 * (ks & 3) + g;
                wh[h][ob][ks] = (out < fout && in < fin)
                                    ? weight_at(p, wbase + p.woff[1 + h], out * fin + in) : 0.0f;
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int n = 16 * ob + 4 * r + g;
                bh[h][ob][r] = n < fout ? p.biases[bbase + p.boff[1 + h] + n] : 0.0f;
            }
        }
    }
    const int NL = p.widths[NH + 1];           // width feeding the output layer
    float w3[3][NB][4];
#pragma unroll
    for (int c = 0; c < 3; ++c)
#pragma unroll
        for (int ob = 0; ob < NB; ++ob)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int n = 16 * ob + 4 * r + g;
                w3[c][ob][r] = n < NL ? weight_at(p, wbase + p.woff[NH + 1], c * NL + n) : 0.0f;
            }
    const float b3_0 = p.biases[bbase + p.boff[NH + 1] + 0];
    const float b3_1 = p.biases[bbase + p.boff[NH + 1] + 1];
    const float b3_2 = p.biases[bbase + p.boff[NH + 1] + 2];

    // ---- walk this block's share of the image's 16-pixel groups
    const int64_t npix = (int64_t)p.H * p.W;
    const int G = p.groups_per_image;
    const int per_blk = (G + blocks_per_image - 1) / blocks_per_image;
    const int g_begin = blk * per_blk;
    const int g_end = min(G, g_begin + per_blk);
    const int64_t plane = npix;
    const int64_t obase = (int64_t)b * 3 * plane;

    for (int grp = g_begin + wave; grp < g_end; grp += kWaves) {
        const int64_t pix = (int64_t)grp * 16 + col;
        const int64_t pc = pix < npix ? pix : npix - 1;
        const int y = (int)(pc / p.W);
        const int x = (int)(pc - (int64_t)y * p.W);

        // layer 1: K = levels
        f32x4 d[NB];
#pragma unroll
        for (int ob = 0; ob < NB; ++ob)
            d[ob] = b1[ob];
#pragma unroll
        for (int s = 0; s < kMaxLS; ++s) {
            if (s < LS) {
                const float u = lv[s].valid ? sample(lv[s], y, x) : 0.0f;
#pragma unroll
                for (int ob = 0; ob < NB; ++ob)
                    d[ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(w1[ob][s], u, d[ob], 0, 0, 0);
            }
        }
#pragma unroll
        for (int ob = 0; ob < NB; ++ob)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                d[ob][r] = fmaxf(d[ob][r], 0.0f);

        // hidden layers
#pragma unroll
        for (int h = 0; h < NH; ++h) {
            const int fin = p.widths[1 + h];
            f32x4 e[NB];
#pragma unroll
            for (int ob = 0; ob < NB; ++ob)
                e[ob] = bh[h][ob];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if (16 * nb + 4 * r < fin) {
#pragma unroll
                        for (int ob = 0; ob < NB; ++ob)
                            e[ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(wh[h][ob][4 * nb + r], d[nb][r],
                                                                         e[ob], 0, 0, 0);
                    }
                }
#pragma unroll
            for (int ob = 0; ob < NB; ++ob)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    d[ob][r] = fmaxf(e[ob][r], 0.0f);
        }

        // output layer on the vector ALU, then sum over the four lane groups
        float o0 = 0.0f, o1 = 0.0f, o2 = 0.0f;
#pragma unroll
        for (int ob = 0; ob < NB; ++ob)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                o0 = __builtin_fmaf(w3[0][ob][r], d[ob][r], o0);
                o1 = __builtin_fmaf(w3[1][ob][r], d[ob][r], o1);
                o2 = __builtin_fmaf(w3[2][ob][r], d[ob][r], o2);
            }
        o0 += __shfl_xor(o0, 16);
        o1 += __shfl_xor(o1, 16);
        o2 += __shfl_xor(o2, 16);
        o0 += __shfl_xor(o0, 32);
        o1 += __shfl_xor(o1, 32);
        o2 += __shfl_xor(o2, 32);

        if (g < 3 && pix < npix) {
            const float v = g == 0 ? o0 + b3_0 : (g == 1 ? o1 + b3_1 : o2 + b3_2);
            const int64_t o = obase + (int64_t)g * plane + pix;
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
    }
}

int hidden_blocks(int nl, const int32_t *widths)
{
    int m = 1;
    for (int l = 1; l < nl; ++l)
        m = widths[l] > m ? widths[l] : m;
    return (m + 15) / 16;
}

template <int NB, int NH>
hipError_t launch_t(const DecodeParams &p, hipStream_t s, int num_cus)
{
    // Enough blocks to give every SIMD two wavefronts, split evenly over images.
    const int target = 2 * num_cus;
    int bpi = (target + p.batch - 1) / p.batch;
    const int max_bpi = (p.groups_per_image + kWaves - 1) / kWaves;
    bpi = bpi < 1 ? 1 : (bpi > max_bpi ? max_bpi : bpi);
    const int64_t nblocks = (int64_t)bpi * p.batch;
    if (nblocks > 0x7fffffff)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_mfma_f32<NB, NH>), dim3((unsigned)nblocks), dim3(kThreads), 0, s, p, bpi);
    return hipGetLastError();
}

template <int NH>
hipError_t launch_nb(int NB, const DecodeParams &p, hipStream_t s, int num_cus)
{
    switch (NB) {
    case 1: return launch_t<1, NH>(p, s, num_cus);
    case 2: return launch_t<2, NH>(p, s, num_cus);
    case 3: return launch_t<3, NH>(p, s, num_cus);
    case 4: return launch_t<4, NH>(p, s, num_cus);
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool mfma_f32_supports(int L, int nl, const int32_t *widths)
{
    return L >= 1 && L <= 4 * kMaxLS && nl >= 2 && nl <= 4 && hidden_blocks(nl, widths) <= 4;
}

hipError_t launch_mfma_f32(const DecodeParams &p, hipStream_t s, const char **name, int *px_per_step,
                           int num_cus)
{
    if (!mfma_f32_supports(p.L, p.nl, p.widths))
        return hipErrorInvalidValue;
    const int NB = hidden_blocks(p.nl, p.widths);
    *name = "k_mfma_f32";
    *px_per_step = 16;
    switch (p.nl - 2) {
    case 0: return launch_nb<0>(NB, p, s, num_cus);
    case 1: return launch_nb<1>(NB, p, s, num_cus);
    case 2: return launch_nb<2>(NB, p, s, num_cus);
    }
    return hipErrorInvalidValue;
}

}  // namespace pic
