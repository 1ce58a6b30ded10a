// Projection onto the ESB value set (eq. (6)-(8)) and dequantization, gfx950.
//
// Each element: v = fl32(x / alpha) with the IEEE binary32 division, then the
// shift-round of eq. (7) done on the bit pattern of |v|:
//   |v| >= 1: keep the leading 1 and k fraction bits, adding half an ulp of the
//             kept precision before truncating (ties go to the larger magnitude);
//             the carry into the exponent field is the round-up to the next binade;
//   |v| <  1: the step is fixed at 2^-k (the subnormal binade, eq. (5)), so the
//             significand is shifted right by 150 - E - k with the same rounding;
//   |v| >= C: clip to C (eq. (8)); NaN gives +0.
// The rounded bit pattern is the code itself: for |v| >= 1 the biased fp32
// exponent minus 127 is the ESB exponent field and the kept fraction bits are
// the ESB fraction field.  HBM bound: 4 B read + 1 B written per element.
#include "esb_internal.h"

namespace esb {

ProjParams proj_params(const Fmt& f) {
    ProjParams p;
    p.k = (uint32_t)f.k;
    p.zero_code = f.zero_code;
    p.c_code = f.c_code;
    p.c_bits = f.c_bits;
    p.sign_bit = f.sign_bit;
    p.one = 1u << f.k;
    return p;
}

__device__ __forceinline__ uint32_t esb_code(float x, float alpha, const ProjParams& p) {
    const float v = x / alpha;   // correctly rounded binary32 division
    const uint32_t vb = __float_as_uint(v);
    const uint32_t ab = vb & 0x7fffffffu;
    const uint32_t ef = ab >> 23;
    // |v| in [1, C): round to k fraction bits; the result is (e+127) << k | f.
    const uint32_t shA = 23u - p.k;
    const uint32_t codeA = ((ab + (1u << (shA - 1u))) >> shA) - (127u << p.k);
    // |v| < 1: m = round(|v| * 2^k) in [0, 2^k]; m == 2^k is the value 1 (code 0).
    const uint32_t mant = (ab & 0x7fffffu) | (ef ? 0x800000u : 0u);
    const uint32_t sB = min(150u - max(ef, 1u) - p.k, 25u);   // >= 17 for |v| < 1
    const uint32_t m = (mant + (1u << (sB - 1u))) >> sB;       // sB == 25 gives 0
    const uint32_t codeB = (m >= p.one) ? 0u : (p.zero_code | m);
    uint32_t code = (ef >= 127u) ? codeA : codeB;
    code = (ab >= p.c_bits) ? p.c_code : code;            // clip (covers +-Inf)
    code = (ab > 0x7f800000u) ? p.zero_code : code;       // NaN
    code |= ((vb >> 31) && code != p.zero_code) ? p.sign_bit : 0u;
    return code;
}

__device__ __forceinline__ bool alpha_valid(float a) { return a > 0.0f && a < __builtin_inff(); }

// Vector path: 4 elements per 16-byte load, 4 codes per 4-byte store.
__global__ __launch_bounds__(256) void k_project_vec(const f32x4* __restrict__ x4, int64_t n4,
                                                     const float* __restrict__ alpha_p,
                                                     ProjParams p, uint32_t* __restrict__ out4) {
    const float alpha = *alpha_p;
    const bool ok = alpha_valid(alpha);
    const uint32_t z4 = p.zero_code * 0x01010101u;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n4; i += 4 * stride) {
        f32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; u++) v[u] = __builtin_nontemporal_load(&x4[i + u * stride]);
#pragma unroll
        for (int u = 0; u < 4; u++) {
            uint32_t c = z4;
            if (ok)
                c = esb_code(v[u].x, alpha, p) | (esb_code(v[u].y, alpha, p) << 8) |
                    (esb_code(v[u].z, alpha, p) << 16) | (esb_code(v[u].w, alpha, p) << 24);
            __builtin_nontemporal_store(c, &out4[i + u * stride]);
        }
    }
    for (; i < n4; i += stride) {
        const f32x4 v = x4[i];
        uint32_t c = z4;
        if (ok)
            c = esb_code(v.x, alpha, p) | (esb_code(v.y, alpha, p) << 8) |
                (esb_code(v.z, alpha, p) << 16) | (esb_code(v.w, alpha, p) << 24);
        out4[i] = c;
    }
}

// Scalar path: unaligned pointers and the tail of the vector path.
__global__ __launch_bounds__(256) void k_project_scalar(const float* __restrict__ x, int64_t len,
                                                        const float* __restrict__ alpha_p,
                                                        ProjParams p, uint8_t* __restrict__ out) {
    const float alpha = *alpha_p;
    const bool ok = alpha_valid(alpha);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < len; i += stride)
        out[i] = (uint8_t)(ok ? esb_code(x[i], alpha, p) : p.zero_code);
}

static int grid_for(int64_t work, int per_block) {
    int64_t blocks = (work + per_block - 1) / per_block;
    int64_t cap = (int64_t)num_cus() * 8;
    if (blocks > cap) blocks = cap;
    return (int)(blocks < 1 ? 1 : blocks);
}

hipError_t launch_project(const float* x, int64_t len, const float* alpha, const Fmt& f,
                          uint8_t* codes, hipStream_t s) {
    if (len <= 0) return hipSuccess;
    const ProjParams p = proj_params(f);
    const bool aligned = ((uintptr_t)x % 16 == 0) && ((uintptr_t)codes % 4 == 0);
    int64_t head = 0;
    if (aligned && len >= 4) {
        const int64_t n4 = len / 4;
        k_project_vec<<<grid_for(n4, 256), 256, 0, s>>>((const f32x4*)x, n4, alpha, p,
                                                        (uint32_t*)codes);
        head = n4 * 4;
    }
    if (head < len)
        k_project_scalar<<<grid_for(len - head, 256), 256, 0, s>>>(x + head, len - head, alpha,
                                                                   p, codes + head);
    return hipGetLastError();
}

// Dequantization: fl32(alpha * q(code)); q is exact in fp32 for every format.
struct DeqTable { float q[256]; };

__global__ __launch_bounds__(256) void k_dequantize(const uint8_t* __restrict__ codes, int64_t len,
                                                    const float* __restrict__ alpha_p,
                                                    DeqTable t, float* __restrict__ out) {
    __shared__ float q[256];
    q[threadIdx.x] = t.q[threadIdx.x];
    __syncthreads();
    const float alpha = *alpha_p;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < len; i += stride)
        out[i] = alpha * q[codes[i]];
}

hipError_t launch_dequantize(const uint8_t* codes, int64_t len, const float* alpha, const Fmt& f,
                             float* out, hipStream_t s) {
    if (len <= 0) return hipSuccess;
    DeqTable t;
    for (int c = 0; c < 256; c++) t.q[c] = (float)decode_value(f, (uint32_t)c);
    k_dequantize<<<grid_for(len, 256), 256, 0, s>>>(codes, len, alpha, t, out);
    return hipGetLastError();
}

}  // namespace esb
