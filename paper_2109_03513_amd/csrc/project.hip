// Projection onto the ESB value set (eq. (6)-(8)) and dequantization, gfx950.
//
// Reference semantics (esb_code): v = fl32(x / alpha) with the IEEE binary32
// division, then the shift-round of eq. (7) on the bit pattern of |v|:
//   |v| >= 1: keep the leading 1 and k fraction bits, adding half an ulp of the
//             kept precision before truncating (ties go to the larger magnitude);
//             the carry into the exponent field is the round-up to the next binade;
//   |v| <  1: the step is fixed at 2^-k (the subnormal binade, eq. (5));
//   |v| >= C: clip to C (eq. (8)); NaN gives +0.
// The rounded bit pattern is the code itself: for |v| >= 1 the biased fp32
// exponent minus 127 is the ESB exponent field and the kept fraction bits are
// the ESB fraction field.
//
// Fast path: esb_code_fast / code4 in the internal header (shared with the
// fused contraction epilogue), the exact esb_code near cell midpoints.
// HBM bound: 4 B read + 1 B written per element.
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

// One contiguous tile of kTile4 = 4 x 256 float4 (16 KB in, 4 KB out) per
// workgroup, the four loads of a thread in flight together.  Measured on MI355X
// with the same access pattern and trivial arithmetic: contiguous tiles stream
// at ~6.1 TB/s where a grid-stride loop stays at ~5.1.
constexpr int kTile4 = 4 * 256;

// Data normalization of Alg. 1 (DN before ESB): fl32(fl32(x - mean) / den),
// den = fl32(std + 1e-7), the IEEE binary32 division.  Fast form: with
// rd = fl32(1 / den), q = fl32(a rd), the residual a - den q is exact in one
// fma and fl32(q + residual rd) is the correctly rounded a / den (Markstein,
// IBM J. Res. Develop. 34(1), 1990: rd correctly rounded, q within an ulp),
// provided nothing underflows or overflows: den in [2^-24, 2^24] and
// |a| in [2^-100, 2^100] (zero, Inf and NaN excluded); other elements take the
// IEEE division.
struct DnArgs {
    float mean, den, rd;
    bool fast;
};
__device__ __forceinline__ DnArgs dn_args(const float* dn) {
    DnArgs a;
    a.mean = dn[0];
    a.den = dn[1] + 1e-7f;
    a.rd = 1.0f / a.den;
    a.fast = a.den >= 0x1p-24f && a.den <= 0x1p24f;
    return a;
}
__device__ __forceinline__ bool dn_in_range(float a) {
    const uint32_t e = __float_as_uint(a) & 0x7fffffffu;
    return e - 0x0d800000u <= 0x71800000u - 0x0d800000u;   // 2^-100 <= |a| <= 2^100
}
__device__ __forceinline__ float dn_fast(float a, const DnArgs& d) {
    const float q = a * d.rd;
    const float r = __builtin_fmaf(-q, d.den, a);
    return __builtin_fmaf(r, d.rd, q);
}
__device__ __forceinline__ f32x4 dn4(f32x4 v, const DnArgs& a) {
    const f32x4 c{v.x - a.mean, v.y - a.mean, v.z - a.mean, v.w - a.mean};
    if (a.fast && dn_in_range(c.x) && dn_in_range(c.y) && dn_in_range(c.z) && dn_in_range(c.w))
        return f32x4{dn_fast(c.x, a), dn_fast(c.y, a), dn_fast(c.z, a), dn_fast(c.w, a)};
    return f32x4{c.x / a.den, c.y / a.den, c.z / a.den, c.w / a.den};
}

template <int DN>
__device__ __forceinline__ void project_tile(const f32x4* __restrict__ x4, int64_t n4,
                                             const float* __restrict__ alpha_p, const ProjParams& p,
                                             uint32_t* __restrict__ out4, const float* __restrict__ dn,
                                             int64_t tile) {
    const float alpha = *alpha_p;
    DnArgs da{0.0f, 1.0f, 1.0f, false};
    if (DN) da = dn_args(dn);
    const bool ok = alpha_valid(alpha);
    const bool fast = fast_scale(alpha);
    const float r = 1.0f / alpha;
    const uint32_t z4 = p.zero_code * 0x01010101u;
    const int64_t i0 = tile * kTile4 + threadIdx.x;
    if (i0 + 3 * 256 < n4) {
        f32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; u++) v[u] = __builtin_nontemporal_load(&x4[i0 + u * 256]);
        if (DN) {
#pragma unroll
            for (int u = 0; u < 4; u++) v[u] = dn4(v[u], da);
        }
#pragma unroll
        for (int u = 0; u < 4; u++)
            __builtin_nontemporal_store(ok ? code4(v[u], alpha, r, fast, p) : z4, &out4[i0 + u * 256]);
    } else {
#pragma unroll
        for (int u = 0; u < 4; u++) {
            const int64_t i = i0 + u * 256;
            if (i < n4) out4[i] = ok ? code4(DN ? dn4(x4[i], da) : x4[i], alpha, r, fast, p) : z4;
        }
    }
}

template <int DN>
__global__ __launch_bounds__(256) void k_project_vec(const f32x4* __restrict__ x4, int64_t n4,
                                                     const float* __restrict__ alpha_p,
                                                     ProjParams p, uint32_t* __restrict__ out4,
                                                     const float* __restrict__ dn) {
    project_tile<DN>(x4, n4, alpha_p, p, out4, dn, (int64_t)blockIdx.x);
}

// Several tensors in one launch: tiles tile0 .. of the grid belong to job i
// (the vector part of each tensor; tails go to k_project_scalar).
constexpr int kProjMaxJobs = 8;
struct ProjJob {
    const f32x4* x4;
    int64_t n4;
    const float* alpha;
    uint32_t* out4;
    int64_t tile0;
    ProjParams p;
};
struct ProjBatch {
    ProjJob job[kProjMaxJobs];
    int count;
};

__global__ __launch_bounds__(256) void k_project_batch(ProjBatch B) {
    int j = 0;
    for (int i = 1; i < B.count; i++)
        if (B.job[i].tile0 <= (int64_t)blockIdx.x) j = i;
    const ProjJob& J = B.job[j];
    project_tile<0>(J.x4, J.n4, J.alpha, J.p, J.out4, nullptr, (int64_t)blockIdx.x - J.tile0);
}

// Scalar path: unaligned pointers and the tail of the vector path.
template <int DN>
__global__ __launch_bounds__(256) void k_project_scalar(const float* __restrict__ x, int64_t len,
                                                        const float* __restrict__ alpha_p,
                                                        ProjParams p, uint8_t* __restrict__ out,
                                                        const float* __restrict__ dn) {
    const float alpha = *alpha_p;
    const bool ok = alpha_valid(alpha);
    DnArgs da{0.0f, 1.0f, 1.0f, false};
    if (DN) da = dn_args(dn);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < len; i += stride) {
        const float xi = DN ? (x[i] - da.mean) / da.den : x[i];
        out[i] = (uint8_t)(ok ? esb_code(xi, alpha, p) : p.zero_code);
    }
}

static int grid_for(int64_t work, int per_block) {
    int64_t blocks = (work + per_block - 1) / per_block;
    int64_t cap = (int64_t)num_cus() * 8;
    if (blocks > cap) blocks = cap;
    return (int)(blocks < 1 ? 1 : blocks);
}

hipError_t launch_project(const float* x, int64_t len, const float* alpha, const Fmt& f,
                          uint8_t* codes, const float* dn, hipStream_t s) {
    if (len <= 0) return hipSuccess;
    const ProjParams p = proj_params(f);
    const bool aligned = ((uintptr_t)x % 16 == 0) && ((uintptr_t)codes % 4 == 0);
    int64_t head = 0;
    if (aligned && len >= 4) {
        const int64_t n4 = len / 4;
        const int64_t tiles = (n4 + kTile4 - 1) / kTile4;
        if (tiles > 0x7fffffff) return hipErrorInvalidValue;
        if (dn) k_project_vec<1><<<(unsigned)tiles, 256, 0, s>>>((const f32x4*)x, n4, alpha, p,
                                                                 (uint32_t*)codes, dn);
        else k_project_vec<0><<<(unsigned)tiles, 256, 0, s>>>((const f32x4*)x, n4, alpha, p,
                                                              (uint32_t*)codes, dn);
        head = n4 * 4;
    }
    if (head < len) {
        if (dn) k_project_scalar<1><<<grid_for(len - head, 256), 256, 0, s>>>(
                    x + head, len - head, alpha, p, codes + head, dn);
        else k_project_scalar<0><<<grid_for(len - head, 256), 256, 0, s>>>(
                    x + head, len - head, alpha, p, codes + head, dn);
    }
    return hipGetLastError();
}

hipError_t launch_project_batch(const ProjJobDesc* jobs, int count, hipStream_t s) {
    for (int c0 = 0; c0 < count; c0 += kProjMaxJobs) {
        ProjBatch B;
        B.count = 0;
        int64_t tiles = 0;
        for (int i = c0; i < count && i < c0 + kProjMaxJobs; i++) {
            const ProjJobDesc& d = jobs[i];
            if (d.len <= 0) continue;
            const ProjParams p = proj_params(d.f);
            const bool aligned = ((uintptr_t)d.x % 16 == 0) && ((uintptr_t)d.codes % 4 == 0);
            int64_t head = 0;
            if (aligned && d.len >= 4) {
                ProjJob& J = B.job[B.count++];
                J.x4 = (const f32x4*)d.x;
                J.n4 = d.len / 4;
                J.alpha = d.alpha;
                J.out4 = (uint32_t*)d.codes;
                J.tile0 = tiles;
                J.p = p;
                tiles += (J.n4 + kTile4 - 1) / kTile4;
                head = J.n4 * 4;
            }
            if (head < d.len)
                k_project_scalar<0><<<grid_for(d.len - head, 256), 256, 0, s>>>(
                    d.x + head, d.len - head, d.alpha, p, d.codes + head, nullptr);
        }
        if (B.count > 0) {
            if (tiles > 0x7fffffff) return hipErrorInvalidValue;
            k_project_batch<<<(unsigned)tiles, 256, 0, s>>>(B);
        }
    }
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
