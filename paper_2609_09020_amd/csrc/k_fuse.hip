// Folding instance normalisation + channel modulation into the next linear
// layer (PIC, App. A): W' = W diag(gamma / sigma),
// b' = b + W (beta - gamma * mu / sigma).  One workgroup per image, one
// thread per output neuron; double precision, rounded once to fp32.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "pic_decode.h"

namespace {

constexpr int kThreads = 64;

__global__ __launch_bounds__(kThreads) void k_fuse(int in, int out, const float *w, int64_t w_stride,
                                                   const float *b, int64_t b_stride, const float *gamma,
                                                   const float *beta, const float *mu, const float *sigma,
                                                   int64_t stat_stride, float *w_fused, float *b_fused)
{
    const int img = blockIdx.x;
    const float *W = w + (int64_t)img * w_stride;
    const float *g = gamma + (int64_t)img * stat_stride;
    const float *be = beta + (int64_t)img * stat_stride;
    const float *m = mu + (int64_t)img * stat_stride;
    const float *sg = sigma + (int64_t)img * stat_stride;
    float *Wf = w_fused + (int64_t)img * in * out;
    for (int o = threadIdx.x; o < out; o += kThreads) {
        double acc = (double)b[(int64_t)img * b_stride + o];
        for (int c = 0; c < in; ++c) {
            const double wc = (double)W[(int64_t)o * in + c];
            const double scale = (double)g[c] / (double)sg[c];
            Wf[(int64_t)o * in + c] = (float)(wc * scale);
            acc += wc * ((double)be[c] - scale * (double)m[c]);
        }
        b_fused[(int64_t)img * out + o] = (float)acc;
    }
}

}  // namespace

extern "C" pic_status pic_fuse_modulation(int32_t in, int32_t out, int32_t batch, const float *w,
                                          int64_t w_stride, const float *b, int64_t b_stride,
                                          const float *gamma, const float *beta, const float *mu,
                                          const float *sigma, int64_t stat_stride, float *w_fused,
                                          float *b_fused, void *stream)
{
    if (in < 1 || in > PIC_MAX_WIDTH || out < 1 || out > PIC_MAX_WIDTH || batch < 0 || batch > PIC_MAX_BATCH)
        return PIC_E_INVALID;
    if (w_stride < 0 || b_stride < 0 || stat_stride < 0)
        return PIC_E_INVALID;
    if ((w_stride != 0 && w_stride < (int64_t)in * out) || (b_stride != 0 && b_stride < out) ||
        (stat_stride != 0 && stat_stride < in))
        return PIC_E_INVALID;
    if (batch == 0)
        return PIC_OK;
    const void *ptrs[] = {w, b, gamma, beta, mu, sigma, w_fused, b_fused};
    for (const void *q : ptrs)
        if (!q || ((uintptr_t)q % 4))
            return PIC_E_INVALID;
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
        (void)hipGetLastError();
        return PIC_E_NODEVICE;
    }
    hipLaunchKernelGGL(k_fuse, dim3((unsigned)batch), dim3(kThreads), 0, (hipStream_t)stream, in, out, w, w_stride,
                       b, b_stride, gamma, beta, mu, sigma, stat_stride, w_fused, b_fused);
    if (hipGetLastError() != hipSuccess)
        return PIC_E_HIP;
    return PIC_OK;
}
