// Glue between quantized layers on the device (Sec. 4.2: the post-processing
// stage after a convolution, "MP&ReLU", and the pooled features that feed the
// classifier), so that a network's forward pass runs only library kernels:
//
//  * k_maxpool: NHWC fp32 max pooling, padding never selected (every window
//    holds an input element when pad < window); a NaN in a window gives NaN.
//    One thread per output pixel and four channels (16-byte loads, the 16
//    threads of a 64-channel pixel read 256 contiguous bytes), HBM bound.
//  * k_avgpool: the global average over the H x W positions of each image and
//    channel, summed in fp64 in position order and divided in fp64, rounded to
//    fp32 once; optionally raising a running max |out|.
//  * k_absmax: max |x| over a tensor into a device scalar (the scale of a DDA
//    candidate grid), as the unsigned maximum of fp32 bit patterns with the
//    sign cleared, so that a NaN wins over every number; two workgroups per CU,
//    one atomic maximum per workgroup.
#include "esb_internal.h"

namespace esb {

namespace {

__device__ __forceinline__ float max_nan(float m, float v) {
    return (v > m || v != v) ? v : m;   // once m is NaN it stays NaN
}

template <int VEC>
__global__ __launch_bounds__(256) void k_maxpool(const float* __restrict__ x, PoolGeom g,
                                                 float* __restrict__ out) {
    const int CV = g.C / VEC;
    const int64_t total = (int64_t)g.N * g.P * g.Q * CV;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int cv = (int)(t % CV);
        const int64_t pix = t / CV;
        const int q = (int)(pix % g.Q);
        const int64_t np = pix / g.Q;
        const int p = (int)(np % g.P);
        const int n = (int)(np / g.P);
        const int ih0 = p * g.sh - g.ph, iw0 = q * g.sw - g.pw;
        float m[VEC];
#pragma unroll
        for (int c = 0; c < VEC; c++) m[c] = -__builtin_inff();
        for (int r = 0; r < g.R; r++) {
            const int ih = ih0 + r;
            if ((unsigned)ih >= (unsigned)g.H) continue;
            const float* row = x + (((int64_t)n * g.H + ih) * g.W) * g.C + VEC * cv;
            for (int s = 0; s < g.S; s++) {
                const int iw = iw0 + s;
                if ((unsigned)iw >= (unsigned)g.W) continue;
                if (VEC == 4) {
                    const f32x4 v = *(const f32x4*)(row + (int64_t)iw * g.C);
#pragma unroll
                    for (int c = 0; c < VEC; c++) m[c] = max_nan(m[c], v[c]);
                } else {
                    m[0] = max_nan(m[0], row[(int64_t)iw * g.C]);
                }
            }
        }
        float* o = out + pix * g.C + VEC * cv;
        if (VEC == 4) {
            *(f32x4*)o = f32x4{m[0], m[1], m[2], m[3]};
        } else {
            o[0] = m[0];
        }
    }
}

// Bit pattern of |v| ordered as an unsigned integer (NaN above +Inf).
__device__ __forceinline__ uint32_t abs_bits(float v) { return __float_as_uint(v) & 0x7fffffffu; }

constexpr int kAvgAhead = 64;
__global__ __launch_bounds__(256) void k_avgpool(const float* __restrict__ x, int N, int HW, int C,
                                                 float* __restrict__ out, uint32_t* absmax) {
    const int64_t total = (int64_t)N * C;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    uint32_t m = 0;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int64_t n = t / C, c = t - n * C;
        const float* p = x + n * HW * C + c;
        double sum = 0.0;
        // positions kAvgAhead at a time, every load in flight before the first add
        // (indices clamped, so the loads carry no branch); the adds in position order
        for (int i0 = 0; i0 < HW; i0 += kAvgAhead) {
            float v[kAvgAhead];
#pragma unroll
            for (int u = 0; u < kAvgAhead; u++) v[u] = p[(int64_t)min(i0 + u, HW - 1) * C];
#pragma unroll
            for (int u = 0; u < kAvgAhead; u++)
                if (i0 + u < HW) sum += (double)v[u];
        }
        const float v = (float)(sum / (double)HW);
        out[t] = v;
        m = max(m, abs_bits(v));
    }
    if (absmax) absmax_flush_block(absmax, m);
}

// Four 16-byte loads in flight per thread and iteration; one atomic per workgroup.
__global__ __launch_bounds__(256) void k_absmax(const float* __restrict__ x, int64_t len,
                                                uint32_t* absmax) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t m = 0;
    // x is 16-byte aligned (checked by the caller for the vector path)
    const f32x4* x4 = (const f32x4*)x;
    const int64_t n4 = len / 4;
    int64_t t = t0;
    for (; t + 3 * stride < n4; t += 4 * stride) {
        f32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; u++) v[u] = x4[t + u * stride];
#pragma unroll
        for (int u = 0; u < 4; u++)
            m = max(m, max(max(abs_bits(v[u][0]), abs_bits(v[u][1])),
                           max(abs_bits(v[u][2]), abs_bits(v[u][3]))));
    }
    for (; t < n4; t += stride) {
        const f32x4 v = x4[t];
        m = max(m, max(max(abs_bits(v[0]), abs_bits(v[1])), max(abs_bits(v[2]), abs_bits(v[3]))));
    }
    for (int64_t e = 4 * n4 + t0; e < len; e += stride) m = max(m, abs_bits(x[e]));
    absmax_flush_block(absmax, m);
}

__global__ __launch_bounds__(256) void k_absmax_scalar(const float* __restrict__ x, int64_t len,
                                                       uint32_t* absmax) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    uint32_t m = 0;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < len; t += stride)
        m = max(m, abs_bits(x[t]));
    absmax_flush_block(absmax, m);
}

unsigned grid_of(int64_t items, int per_cu) {
    int64_t b = (items + 255) / 256;
    const int64_t cap = (int64_t)num_cus() * per_cu;
    if (b > cap) b = cap;
    return (unsigned)(b < 1 ? 1 : b);
}

}  // namespace

hipError_t launch_maxpool(const float* x, const PoolGeom& g, float* out, hipStream_t s) {
    const bool vec = g.C % 4 == 0 && (uintptr_t)x % 16 == 0 && (uintptr_t)out % 16 == 0;
    const int64_t items = (int64_t)g.N * g.P * g.Q * (vec ? g.C / 4 : g.C);
    if (items == 0) return hipSuccess;
    if (vec) k_maxpool<4><<<grid_of(items, 16), 256, 0, s>>>(x, g, out);
    else k_maxpool<1><<<grid_of(items, 16), 256, 0, s>>>(x, g, out);
    return hipGetLastError();
}

hipError_t launch_avgpool(const float* x, int N, int HW, int C, float* out, float* absmax,
                          hipStream_t s) {
    const int64_t items = (int64_t)N * C;
    if (items == 0) return hipSuccess;
    k_avgpool<<<grid_of(items, 4), 256, 0, s>>>(x, N, HW, C, out, (uint32_t*)absmax);
    return hipGetLastError();
}

hipError_t launch_absmax(const float* x, int64_t len, float* absmax, hipStream_t s) {
    if (len == 0) return hipSuccess;
    // two workgroups per CU: few atomics on the one address, enough loads in flight
    if ((uintptr_t)x % 16 == 0) k_absmax<<<grid_of(len / 16 + 1, 2), 256, 0, s>>>(x, len, (uint32_t*)absmax);
    else k_absmax_scalar<<<grid_of(len, 2), 256, 0, s>>>(x, len, (uint32_t*)absmax);
    return hipGetLastError();
}

}  // namespace esb
