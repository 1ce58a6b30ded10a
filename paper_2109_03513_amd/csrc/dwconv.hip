// Depthwise convolution over ESB codes (groups == C == K, one filter per
// channel), gfx950.  R*S multiply-adds per output: far below the MFMA ridge, so
// these are VALU kernels (codes in, int32 / fp32 out); at MobileNet sizes the
// byte extraction, table lookups and multiply-adds bound them, not HBM.
// k_dwconv16: sixteen channels of one output pixel per thread (C % 16 == 0);
// k_dwconv: four channels (C % 4 == 0) or one.  Decoded filter taps live in
// LDS as int16, activation codes are decoded through a 256-entry LDS table of
// exact integers.
#include "esb_internal.h"

namespace esb {

struct DwParams {
    ConvGeom g;
    const uint8_t* x;
    const uint8_t* w;
    const float* alphaX;
    const float* alphaW;
    int32_t* acc;
    float* y;
    int kx, kw;
    Post post;         // fused post-processing of the outputs (post.on == 0: none)
    int16_t tx[256];   // exact integer of every activation code
    int16_t tw[256];   // exact integer of every filter code
};

constexpr int kDwThreads = 256;
constexpr int kDwMaxTaps = 16384;   // C * R * S held in LDS

template <bool VEC>
__global__ __launch_bounds__(kDwThreads) void k_dwconv(DwParams p) {
    __shared__ int16_t wt[kDwMaxTaps];
    __shared__ int tx[256];
    const ConvGeom& g = p.g;
    const int C = g.C, RS = g.R * g.S;
    for (int i = threadIdx.x; i < C * RS; i += blockDim.x) wt[i] = p.tw[p.w[i]];
    tx[threadIdx.x] = p.tx[threadIdx.x];
    __syncthreads();
    float s = 0.0f;
    if (p.y || p.post.on) s = ldexpf(p.alphaX[0] * p.alphaW[0], -(p.kx + p.kw));
    const float qa = p.post.on ? post_alpha(p.post) : 0.0f;
    const int CV = VEC ? C / 4 : C;                 // channel groups per pixel
    const int64_t total = (int64_t)g.Nb * g.P * g.Q * CV;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    uint32_t amax = 0;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int cv = (int)(t % CV);
        const int64_t pix = t / CV;
        const int q = (int)(pix % g.Q);
        const int p_ = (int)((pix / g.Q) % g.P);
        const int n = (int)(pix / ((int64_t)g.Q * g.P));
        const int c0 = VEC ? 4 * cv : cv;
        int a0 = 0, a1 = 0, a2 = 0, a3 = 0;
        for (int r = 0; r < g.R; r++) {
            const int ih = p_ * g.sh - g.ph + r;
            if (ih < 0 || ih >= g.H) continue;
            for (int s2 = 0; s2 < g.S; s2++) {
                const int iw = q * g.sw - g.pw + s2;
                if (iw < 0 || iw >= g.W) continue;
                const int64_t base = (((int64_t)n * g.H + ih) * g.W + iw) * C + c0;
                const int tap = r * g.S + s2;
                if (VEC) {
                    const uint32_t w4 = *(const uint32_t*)(p.x + base);
                    a0 += tx[w4 & 0xff] * wt[(c0 + 0) * RS + tap];
                    a1 += tx[(w4 >> 8) & 0xff] * wt[(c0 + 1) * RS + tap];
                    a2 += tx[(w4 >> 16) & 0xff] * wt[(c0 + 2) * RS + tap];
                    a3 += tx[w4 >> 24] * wt[(c0 + 3) * RS + tap];
                } else {
                    a0 += tx[p.x[base]] * wt[c0 * RS + tap];
                }
            }
        }
        const int64_t o = pix * C + c0;
        if (VEC) {
            if (p.acc) *(int4*)(p.acc + o) = make_int4(a0, a1, a2, a3);
            if (p.post.on) {
                amax = max(amax, post_store(p.post, p.y, o, c0, s * (float)a0, qa));
                amax = max(amax, post_store(p.post, p.y, o + 1, c0 + 1, s * (float)a1, qa));
                amax = max(amax, post_store(p.post, p.y, o + 2, c0 + 2, s * (float)a2, qa));
                amax = max(amax, post_store(p.post, p.y, o + 3, c0 + 3, s * (float)a3, qa));
            } else if (p.y) {
                *(float4*)(p.y + o) = make_float4(s * (float)a0, s * (float)a1, s * (float)a2,
                                                  s * (float)a3);
            }
        } else {
            if (p.acc) p.acc[o] = a0;
            amax = max(amax, out_store(p.post, p.y, o, c0, s * (float)a0, qa));
        }
    }
    post_absmax_flush(p.post, amax);
}

// Sixteen channels per thread (C % 16 == 0, at most 16 filter taps): one 16-byte
// load of codes per tap, the taps' weights read as 32-byte rows of an LDS table
// laid out [tap][channel], four 16-byte stores per output.  The grid is sized so
// that the grid-stride step is a multiple of C / 16: every thread keeps one
// channel group and walks output pixels.
constexpr int kDw16MaxTaps = 16;
__global__ __launch_bounds__(kDwThreads) void k_dwconv16(DwParams p, int pix_step) {
    __shared__ __align__(16) int16_t wt[kDwMaxTaps];   // [tap][channel]
    __shared__ int tx[256];
    const ConvGeom& g = p.g;
    const int C = g.C, RS = g.R * g.S, CV = C / 16;
    for (int i = threadIdx.x; i < C * RS; i += blockDim.x) {
        const int c = i / RS, tap = i - c * RS;                  // KRSC: channel-major source
        wt[tap * C + c] = p.tw[p.w[i]];
    }
    tx[threadIdx.x] = p.tx[threadIdx.x];
    __syncthreads();
    float s = 0.0f;
    if (p.y || p.post.on) s = ldexpf(p.alphaX[0] * p.alphaW[0], -(p.kx + p.kw));
    const float qa = p.post.on ? post_alpha(p.post) : 0.0f;
    const int64_t gt = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int cv = (int)(gt % CV), c0 = 16 * cv;
    const int64_t npix = (int64_t)g.Nb * g.P * g.Q;
    uint32_t amax = 0;
    for (int64_t pix = gt / CV; pix < npix; pix += pix_step) {
        const int q = (int)(pix % g.Q);
        const int p_ = (int)((pix / g.Q) % g.P);
        const int n = (int)(pix / ((int64_t)g.Q * g.P));
        int a[16];
#pragma unroll
        for (int e = 0; e < 16; e++) a[e] = 0;
        for (int r = 0; r < g.R; r++) {
            const int ih = p_ * g.sh - g.ph + r;
            if (ih < 0 || ih >= g.H) continue;
            for (int s2 = 0; s2 < g.S; s2++) {
                const int iw = q * g.sw - g.pw + s2;
                if (iw < 0 || iw >= g.W) continue;
                const uint4 cx = *(const uint4*)(p.x + (((int64_t)n * g.H + ih) * g.W + iw) * C + c0);
                const int tap = r * g.S + s2;
                const int4* wr = (const int4*)(wt + tap * C + c0);
                const int4 w0 = wr[0], w1 = wr[1];
                const uint32_t cw[4] = {cx.x, cx.y, cx.z, cx.w};
                const uint32_t ww[8] = {(uint32_t)w0.x, (uint32_t)w0.y, (uint32_t)w0.z, (uint32_t)w0.w,
                                        (uint32_t)w1.x, (uint32_t)w1.y, (uint32_t)w1.z, (uint32_t)w1.w};
#pragma unroll
                for (int e = 0; e < 16; e++) {
                    const int xv = tx[(cw[e >> 2] >> (8 * (e & 3))) & 0xffu];
                    const int wv = (int)(int16_t)(ww[e >> 1] >> (16 * (e & 1)));
                    a[e] += xv * wv;
                }
            }
        }
        const int64_t o = pix * C + c0;
        if (p.acc) {
#pragma unroll
            for (int k = 0; k < 4; k++)
                *(int4*)(p.acc + o + 4 * k) = make_int4(a[4 * k], a[4 * k + 1], a[4 * k + 2], a[4 * k + 3]);
        }
        if (p.post.on) {
#pragma unroll
            for (int k = 0; k < 4; k++) {
                const f32x4 v{s * (float)a[4 * k], s * (float)a[4 * k + 1], s * (float)a[4 * k + 2],
                              s * (float)a[4 * k + 3]};
                amax = max(amax, post_store4(p.post, p.y, o + 4 * k, c0 + 4 * k, v, 4, qa));
            }
        } else if (p.y) {
#pragma unroll
            for (int k = 0; k < 4; k++)
                *(float4*)(p.y + o + 4 * k) = make_float4(s * (float)a[4 * k], s * (float)a[4 * k + 1],
                                                          s * (float)a[4 * k + 2], s * (float)a[4 * k + 3]);
        }
    }
    post_absmax_flush(p.post, amax);
}

hipError_t launch_dwconv(const ConvGeom& g, const uint8_t* x, const Fmt& fx, const float* alphaX,
                         const uint8_t* w, const Fmt& fw, const float* alphaW, int32_t* acc,
                         float* y, hipStream_t s, const Post* post) {
    DwParams p;
    p.g = g; p.x = x; p.w = w; p.alphaX = alphaX; p.alphaW = alphaW; p.acc = acc; p.y = y;
    p.post = post ? *post : Post{};
    p.kx = fx.k; p.kw = fw.k;
    for (int c = 0; c < 256; c++) {
        p.tx[c] = (int16_t)decode_int(fx, (uint32_t)c);
        p.tw[c] = (int16_t)decode_int(fw, (uint32_t)c);
    }
    const bool vec = (g.C % 4 == 0) && ((uintptr_t)x % 4 == 0) && (!acc || (uintptr_t)acc % 16 == 0) &&
                     (!y || (uintptr_t)y % 16 == 0);
    if (g.C % 16 == 0 && g.C * g.R * g.S <= kDwMaxTaps && g.R * g.S <= kDw16MaxTaps &&
        (uintptr_t)x % 16 == 0 &&
        (!acc || (uintptr_t)acc % 16 == 0) && (!y || (uintptr_t)y % 16 == 0)) {
        const int CV = g.C / 16;
        const int64_t npix = (int64_t)g.Nb * g.P * g.Q;
        // blocks: a multiple of CV / gcd(CV, 256), so that the thread count is a multiple of CV
        int unit = CV;
        for (int d = 256; d > 1; d /= 2)
            if (unit % 2 == 0 && d > 1) unit /= 2; else break;
        int64_t want = (npix * CV + kDwThreads - 1) / kDwThreads;
        const int64_t cap = (int64_t)num_cus() * 4;
        if (want > cap) want = cap;
        int64_t blocks = (want + unit - 1) / unit * unit;
        if (blocks < unit) blocks = unit;
        const int pix_step = (int)(blocks * kDwThreads / CV);
        k_dwconv16<<<(int)blocks, kDwThreads, 0, s>>>(p, pix_step);
        return hipGetLastError();
    }
    const int64_t total = (int64_t)g.Nb * g.P * g.Q * (vec ? g.C / 4 : g.C);
    int64_t blocks = (total + kDwThreads - 1) / kDwThreads;
    // each block decodes the filters into LDS first: few blocks, each over many outputs
    const int64_t cap = (int64_t)num_cus() * 4;
    if (blocks > cap) blocks = cap;
    if (blocks < 1) blocks = 1;
    if (vec) k_dwconv<true><<<(int)blocks, kDwThreads, 0, s>>>(p);
    else k_dwconv<false><<<(int)blocks, kDwThreads, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace esb
