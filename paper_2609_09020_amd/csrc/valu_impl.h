// Reference kernel family, device code: the synthesis step in plain binary32
// vector-ALU arithmetic with a fixed operation order, one pixel per lane.
// Included by k_valu.hip (hidden widths up to 64) and k_valu_w{96,128}.hip
// (the wide instances, one translation unit each: they are large).
//
// Per pixel (PIC, Sec. 3.1 and App. A): the L levels are upsampled bilinearly
// (half-pixel centres, edge replication, scale 2^k) into the MLP's input, then
// every layer computes out_j = b_j + sum_i W[j][i] h_i as a chain of fused
// multiply-adds started from the bias, inputs in increasing index, ReLU after
// every layer but the last; the epilogue clamps to [0, 1] and quantises to
// floor(fma(c, 255, 1/2)).  The upsample's products and sums are each rounded
// once, in the order (1-lx)*a + lx*b per row and (1-ly)*top + ly*bot across
// rows (the library is compiled without floating-point contraction).
//
// Layer weights are staged, zero-padded, into LDS one layer at a time; all
// lanes read the same address, which LDS serves as a broadcast.  Activations
// stay in VGPRs, padded to a multiple of 8 (to 96 or 128 above 64) so the
// zero padding only appends exact no-op terms (fma(0, h, acc) == acc) to
// every chain.
#pragma once

#include "pic_internal.h"

namespace pic {
namespace valu {

constexpr int kThreads = 256;
constexpr int kNarrow = 64;    // widest hidden layer of the k_valu instances

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

// g[j] = act(sB[j] + sum_i sW[j][i] * h[i]) for J0 <= j < J1, canonical
// order.  The outputs are expanded at compile time (halving the range), so
// every index into h and g is a constant however wide the layer: an output
// loop the compiler declined to unroll would index g at run time and move it
// to scratch memory.
template <int K, int J0, int J1, bool RELU>
__device__ __forceinline__ void dense_rows(const float *h, float *g, const float *sW, const float *sB)
{
    if constexpr (J1 - J0 == 1) {
        float acc = sB[J0];
#pragma unroll
        for (int i = 0; i < K; i += 4) {
            const float4 w = *reinterpret_cast<const float4 *>(&sW[J0 * K + i]);
            acc = __builtin_fmaf(w.x, h[i + 0], acc);
            acc = __builtin_fmaf(w.y, h[i + 1], acc);
            acc = __builtin_fmaf(w.z, h[i + 2], acc);
            acc = __builtin_fmaf(w.w, h[i + 3], acc);
        }
        g[J0] = RELU ? fmaxf(acc, 0.0f) : acc;
    } else {
        constexpr int JM = (J0 + J1) / 2;
        dense_rows<K, J0, JM, RELU>(h, g, sW, sB);
        dense_rows<K, JM, J1, RELU>(h, g, sW, sB);
    }
}

template <int K, int N, bool RELU>
__device__ __forceinline__ void dense(const float *h, float *g, const float *sW, const float *sB)
{
    static_assert(K % 4 == 0, "K must be a multiple of 4");
    dense_rows<K, 0, N, RELU>(h, g, sW, sB);
}

template <int PL, int PW>
__device__ __forceinline__ void valu_decode(const DecodeParams &p)
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

// Hidden widths up to 64: two or more wavefronts per SIMD.
template <int PL, int PW>
__global__ __launch_bounds__(kThreads) void k_valu(DecodeParams p)
{
    static_assert(PW <= kNarrow, "narrow kernel");
    valu_decode<PL, PW>(p);
}

// Hidden widths 65 .. 128: a pixel's input and output activations of a layer
// (2 x 128 values) stay in registers, which takes the whole register file of
// a SIMD (VGPRs plus AGPRs) for one wavefront.  This is the reference family;
// the matrix-core families are the fast path.
template <int PL, int PW>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_valu_wide(DecodeParams p)
{
    static_assert(PW > kNarrow && PW <= PIC_MAX_WIDTH, "wide kernel");
    valu_decode<PL, PW>(p);
}

template <int PL, int PW>
hipError_t launch_t(const DecodeParams &p, hipStream_t s)
{
    const int64_t npix = (int64_t)p.H * p.W;
    dim3 grid((unsigned)((npix + kThreads - 1) / kThreads), (unsigned)p.batch);
    if constexpr (PW <= kNarrow)
        hipLaunchKernelGGL((k_valu<PL, PW>), grid, dim3(kThreads), 0, s, p);
    else
        hipLaunchKernelGGL((k_valu_wide<PL, PW>), grid, dim3(kThreads), 0, s, p);
    return hipGetLastError();
}

// The wide instances (levels padded to 12: the first layer is a small part of
// a wide net's work), defined in k_valu_w96.hip and k_valu_w128.hip.
hipError_t launch_wide96(const DecodeParams &p, hipStream_t s);
hipError_t launch_wide128(const DecodeParams &p, hipStream_t s);

}  // namespace valu
}  // namespace pic
