// Depthwise convolution over ESB codes (groups == C == K, one filter per
// channel), gfx950.  R*S multiply-adds per output: far below the MFMA ridge, so
// this is a VALU kernel bound by HBM (codes in, int32 / fp32 out).  Each thread
// produces four consecutive channels of one output pixel; decoded filter taps
// live in LDS as int16, activation codes are decoded through a 256-entry LDS
// table of exact integers.
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
    const int64_t total = (int64_t)g.Nb * g.P * g.Q * (vec ? g.C / 4 : g.C);
    int64_t blocks = (total + kDwThreads - 1) / kDwThreads;
    const int64_t cap = (int64_t)num_cus() * 16;
    if (blocks > cap) blocks = cap;
    if (blocks < 1) blocks = 1;
    if (vec) k_dwconv<true><<<(int)blocks, kDwThreads, 0, s>>>(p);
    else k_dwconv<false><<<(int)blocks, kDwThreads, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace esb
