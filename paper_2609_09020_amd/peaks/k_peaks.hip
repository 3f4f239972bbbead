// Peak-rate microbenchmarks of one gfx950 SIMD's issue paths, measured by
// `bench.py --peaks`: the rates the decode kernels' design rests on.  Not part
// of the decoder; built into its own library (libpic_peaks.so).
//
// Every kernel runs `iters` iterations of a fixed instruction mix per
// wavefront on independent accumulators (no dependency between consecutive
// instructions of one chain), then folds the accumulators into one value per
// lane and stores it, so that nothing is removed by the compiler.
//
//   kind 0  fp32 matrix:  8 x v_mfma_f32_16x16x4_f32        (2048 FLOP each)
//   kind 1  bf16 matrix:  8 x v_mfma_f32_16x16x32_bf16      (16384 FLOP each)
//   kind 2  fp16 matrix:  8 x v_mfma_f32_16x16x32_f16       (16384 FLOP each)
//   kind 3  fp32 vector: 32 x v_fma_f32 on 8 chains          (128 FLOP each)
//   kind 4  kinds 0 and 3 interleaved in every wavefront (8 + 32 per iteration)
//   kind 5  kinds 1 and 3 interleaved in every wavefront (8 + 32 per iteration)
//
// The vector FMAs are built with packed fp32 disabled, like the decoder, so
// they are single v_fma_f32 instructions (64 lanes x 2 FLOP).
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int kAcc = 8;

template <int KIND>
__global__ __launch_bounds__(kThreads) void k_peak(int iters, float seed, float *out)
{
    const int lane = threadIdx.x & 63;
    f32x4 acc[kAcc];
#pragma unroll
    for (int i = 0; i < kAcc; ++i)
        acc[i] = f32x4{seed * i, 0.f, 0.f, 0.f};
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
        v[i] = seed * (lane + i);
    const float a = seed + 1.0f, b = seed * 0.5f;
    bf16x8 ab, bb;
    f16x8 ah, bh;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        ab[i] = (__bf16)(a * i);
        bb[i] = (__bf16)(b + i);
        ah[i] = (_Float16)(a * i);
        bh[i] = (_Float16)(b + i);
    }
    for (int it = 0; it < iters; ++it) {
        if constexpr (KIND == 0 || KIND == 4) {
#pragma unroll
            for (int i = 0; i < kAcc; ++i)
                acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[i], 0, 0, 0);
        }
        if constexpr (KIND == 1 || KIND == 5) {
#pragma unroll
            for (int i = 0; i < kAcc; ++i)
                acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ab, bb, acc[i], 0, 0, 0);
        }
        if constexpr (KIND == 2) {
#pragma unroll
            for (int i = 0; i < kAcc; ++i)
                acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bh, acc[i], 0, 0, 0);
        }
        if constexpr (KIND >= 3) {
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    v[i] = __builtin_fmaf(v[i], a, b);
        }
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < kAcc; ++i)
        s += acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3];
#pragma unroll
    for (int i = 0; i < 8; ++i)
        s += v[i];
    out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = s;
}

}  // namespace

extern "C" __attribute__((visibility("default")))
int pic_peaks_launch(int kind, int blocks, int iters, float *out, void *stream)
{
    if (blocks < 1 || iters < 1 || !out)
        return 1;
    hipStream_t s = (hipStream_t)stream;
    const dim3 g((unsigned)blocks), t(kThreads);
    switch (kind) {
    case 0: hipLaunchKernelGGL(k_peak<0>, g, t, 0, s, iters, 1e-3f, out); break;
    case 1: hipLaunchKernelGGL(k_peak<1>, g, t, 0, s, iters, 1e-3f, out); break;
    case 2: hipLaunchKernelGGL(k_peak<2>, g, t, 0, s, iters, 1e-3f, out); break;
    case 3: hipLaunchKernelGGL(k_peak<3>, g, t, 0, s, iters, 1e-3f, out); break;
    case 4: hipLaunchKernelGGL(k_peak<4>, g, t, 0, s, iters, 1e-3f, out); break;
    case 5: hipLaunchKernelGGL(k_peak<5>, g, t, 0, s, iters, 1e-3f, out); break;
    default: return 1;
    }
    return hipGetLastError() == hipSuccess ? 0 : 2;
}
