// Reference kernel family: the synthesis step in plain binary32 vector-ALU
// arithmetic with a fixed operation order, one pixel per lane.
//
// Per pixel (PIC, Sec. 3.1 and App. A): the L levels are upsampled bilinearly
// (half-pixel centres, edge replication, scale 2^k) into the MLP's input, then
// every layer computes out_j = b_j + sum_i W[j][i] h_i as a chain of fused
// multiply-adds started from the bias, inputs in increasing index, ReLU after
// every layer but the last; the epilogue clamps to [0, 1] and quantises to
// floor(fma(c, 255, 1/2)).  The upsample's products and sums are each rounded
// once, in the order (1-lx)*a + lx*b per row and (1-ly)*top + ly*bot across
// rows (this file is compiled without floating-point contraction).
//
// Layer weights are staged, zero-padded, into LDS one layer at a time; all
// lanes read the same address, which LDS serves as a broadcast.  Activations
// stay in VGPRs, padded to a multiple of 8 so the zero padding only appends
// exact no-op terms (fma(0, h, acc) == acc) to every chain.
#include "pic_internal.h"

namespace pic {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float pow2_neg(int k)
{
    return __int_as_float((127 - k) << 23);   // 2^-k, exact for k < 127
}

// Element idx of image b's layer-l matrix, as fp32 (bf16 widened exactly).
__device__ __forceinline__ float load_weight(const DecodeParams &p, int l, int b, int idx)
{
    const int64_t i = (int64_t)b * p.wls[l] + idx;
    if (p.weights_bf16) {
        const uint16_t bits = static_cast<const uint16_t *>(p.wl[l])[i];
        return __uint_as_float((uint32_t)bits << 16);
    }
    return static_cast<const float *>(p.wl[l])[i];
}

// Level k of image b sampled at output pixel (y, x).
__device__ __forceinline__ float upsample_level(const DecodeParams &p, int b, int k, int y, int x)
{
    const int hk = p.hk[k], wk = p.wk[k];
    const float *g = p.lat[k] + (int64_t)b * hk * wk;
    if (k == 0)
        return g[(int64_t)y * wk + x];
    const float inv = pow2_neg(k);
    float sy = ((float)y + 0.5f) * inv - 0.5f;
    float sx = ((float)x + 0.5f) * inv - 0.5f;
    sy = sy < 0.0f ? 0.0f : sy;
    sx = sx < 0.0f ? 0.0f : sx;
    const int y0 = (int)floorf(sy), x0 = (int)floorf(sx);
    const int y1 = y0 + 1 < hk ? y0 + 1 : hk - 1;
    const int x1 = x0 + 1 < wk ? x0 + 1 : wk - 1;
    const float ly = sy - (float)y0, lx = sx - (float)x0;
    const float a = g[(int64_t)y0 * wk + x0], bb = g[(int64_t)y0 * wk + x1];
    const float c = g[(int64_t)y1 * wk + x0], d = g[(int64_t)y1 * wk + x1];
    const float top = (1.0f - lx) * a + lx * bb;
    const float bot = (1.0f - lx) * c + lx * d;
    return (1.0f - ly) * top + ly * bot;
}

// Stage layer l of image b into LDS as a zero-padded [KOUT][KIN] matrix and
// a zero-padded bias vector of KOUT entries.
template <int KIN, int KOUT>
__device__ __forceinline__ void stage_layer(float *sW, float *sB, const DecodeParams &p, int b, int l)
{
    const int fin = p.widths[l], fout = p.widths[l + 1];
    for (int i = threadIdx.x; i < KOUT * KIN; i += kThreads) {
        const int r = i / KIN, c = i - (i / KIN) * KIN;
        sW[i] = (r < fout && c < fin) ? load_weight(p, l, b, r * fin + c) : 0.0f;
    }
    const float *bias = p.bl[l] + (int64_t)b * p.bls[l];
    for (int i = threadIdx.x; i < KOUT; i += kThreads)
        sB[i] = i < fout ? bias[i] : 0.0f;
}

// g[j] = act(sB[j] + sum_i sW[j][i] * h[i]) for j < N, canonical order.
template <int K, int N, bool RELU>
__device__ __forceinline__ void dense(const float *h, float *g, const float *sW, const float *sB)
{
    static_assert(K % 4 == 0, "K must be a multiple of 4");
#pragma unroll
    for (int j = 0; j < N; ++j) {
        float acc = sB[j];
#pragma unroll
        for (int i = 0; i < K; i += 4) {
            const float4 w = *reinterpret_cast<const float4 *>(&sW[j * K + i]);
            acc = __builtin_fmaf(w.x, h[i + 0], acc);
            acc = __builtin_fmaf(w.y, h[i + 1], acc);
            acc = __builtin_fmaf(w.z, h[i + 2], acc);
            acc = __builtin_fmaf(w.w, h[i + 3], acc);
        }
        g[j] = RELU ? fmaxf(acc, 0.0f) : acc;
    }
}

template <int PL, int PW>
__global__ __launch_bounds__(kThreads) void k_valu(DecodeParams p)
{
    warm_kernel_args<sizeof(DecodeParams)>();
    constexpr int PA = PL > PW ? PL : PW;
    __shared__ __attribute__((aligned(16))) float sW[PA * PA > 4 * PA ? PA * PA : 4 * PA];
    __shared__ __attribute__((aligned(16))) float sB[PA];

    const int b = blockIdx.y;
    const int64_t npix = (int64_t)p.H * p.W;
    const int64_t pix = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const bool active = pix < npix;
    const int y = active ? (int)(pix / p.W) : 0;
    const int x = active ? (int)(pix - (pix / p.W) * p.W) : 0;

    float h[PA];
#pragma unroll
    for (int k = 0; k < PA; ++k)
        h[k] = 0.0f;
#pragma unroll
    for (int k = 0; k < PL; ++k)
        if (k < p.L)
            h[k] = upsample_level(p, b, k, y, x);

    for (int l = 0; l < p.nl; ++l) {
        const bool last = l == p.nl - 1;
        __syncthreads();   // previous layer's weights are no longer read
        if (l == 0) {
            if (last) stage_layer<PL, 4>(sW, sB, p, b, l);
            else stage_layer<PL, PW>(sW, sB, p, b, l);
        } else {
            if (last) stage_layer<PW, 4>(sW, sB, p, b, l);
            else stage_layer<PW, PW>(sW, sB, p, b, l);
        }
        __syncthreads();
        float g[PA];
#pragma unroll
        for (int k = 0; k < PA; ++k)
            g[k] = 0.0f;
        if (l == 0) {
            if (last) dense<PL, 4, false>(h, g, sW, sB);
            else dense<PL, PW, true>(h, g, sW, sB);
        } else {
            if (last) dense<PW, 4, false>(h, g, sW, sB);
            else dense<PW, PW, true>(h, g, sW, sB);
        }
#pragma unroll
        for (int k = 0; k < PA; ++k)
            h[k] = g[k];
    }

    if (!active)
        return;
    const int64_t plane = npix;
    const int64_t o = (int64_t)b * 3 * plane + pix;
#pragma unroll
    for (int c = 0; c < 3; ++c) {
        const float v = h[c];
        if (p.out_kind == OUT_RAW_F32) {
            static_cast<float *>(p.out)[o + c * plane] = v;
        } else {
            const float cl = fminf(fmaxf(v, 0.0f), 1.0f);
            if (p.out_kind == OUT_CLAMPED_F32)
                static_cast<float *>(p.out)[o + c * plane] = cl;
            else
                static_cast<uint8_t *>(p.out)[o + c * plane] =
                    (uint8_t)(int)floorf(__builtin_fmaf(cl, 255.0f, 0.5f));
        }
    }
}

int padded_levels(int L) { return ((L + 3) / 4) * 4; }

int padded_hidden(int nl, const int32_t *widths)
{
    int m = 8;
    for (int l = 1; l < nl; ++l)
        m = widths[l] > m ? widths[l] : m;
    return ((m + 7) / 8) * 8;
}

template <int PL, int PW>
hipError_t launch_t(const DecodeParams &p, hipStream_t s)
{
    const int64_t npix = (int64_t)p.H * p.W;
    dim3 grid((unsigned)((npix + kThreads - 1) / kThreads), (unsigned)p.batch);
    hipLaunchKernelGGL((k_valu<PL, PW>), grid, dim3(kThreads), 0, s, p);
    return hipGetLastError();
}

template <int PL>
hipError_t launch_pw(int PW, const DecodeParams &p, hipStream_t s)
{
    switch (PW) {
    case 8: return launch_t<PL, 8>(p, s);
    case 16: return launch_t<PL, 16>(p, s);
    case 24: return launch_t<PL, 24>(p, s);
    case 32: return launch_t<PL, 32>(p, s);
    case 40: return launch_t<PL, 40>(p, s);
    case 48: return launch_t<PL, 48>(p, s);
    case 56: return launch_t<PL, 56>(p, s);
    case 64: return launch_t<PL, 64>(p, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool valu_supports(int L, int nl, const int32_t *widths)
{
    return L >= 1 && L <= 12 && nl >= 1 && padded_hidden(nl, widths) <= 64;
}

hipError_t launch_valu(const DecodeParams &p, hipStream_t s, const char **name, int *px_per_step)
{
    if (!valu_supports(p.L, p.nl, p.widths))
        return hipErrorInvalidValue;
    const int PL = padded_levels(p.L), PW = padded_hidden(p.nl, p.widths);
    *name = "k_valu";
    *px_per_step = 64;
    switch (PL) {
    case 4: return launch_pw<4>(PW, p, s);
    case 8: return launch_pw<8>(PW, p, s);
    case 12: return launch_pw<12>(PW, p, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace pic
