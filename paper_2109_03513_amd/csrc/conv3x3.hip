// Direct 3x3 / pad-1 convolution, stride 1 or 2, over ESB codes on the fp8 MFMA
// of gfx950 (Sec. 4.2: the convolution stage; products of codes by eq. (15),
// exact as in the implicit-GEMM path), for input and output channels that are
// multiples of 64.
//
// The implicit-GEMM kernels fetch and decode every input element once per
// filter tap it meets, nine times for a 3x3 filter.  Here a workgroup owns TM
// consecutive output pixels (flattened over the batch) and 64 output channels,
// and runs over the input channels in chunks of 64:
//  * per chunk, the input rows under the tile are decoded to E4M3 once into an
//    LDS patch, one 64-byte row per input pixel.  Every image is seen with a
//    zero row above and below it and a zero column left and right (the
//    padding), so a tile may cross images: output pixel (n, p, q) and tap
//    (r, s) read padded row n (H + 2) + st p + r - R0 (R0 the first padded row of
//    the tile) and padded column st q + s.  With stride 2 a patch row holds the
//    even padded columns first, then the odd ones, so that a tap over 32
//    consecutive output pixels still reads consecutive patch pixels.  The four 16-byte chunks of a patch pixel are
//    stored in the order chunk ^ ((pixel / 4) % 4), so that 16 consecutive
//    pixels read at one chunk (a quarter-wave of a fragment load) hit 16
//    different bank groups;
//  * per chunk the filter slice (64 outputs x 9 taps x 64 channels) is decoded
//    into LDS; with one chunk (64 input channels) it is decoded once per
//    workgroup and stays (workgroups are persistent over their tiles);
//  * the codes of the next chunk (or tile) are loaded into registers while the
//    current chunk's MFMAs run;
//  * per tap one v_mfma_scale_f32_32x32x64_f8f6f4 per 32 x 32 block;
//  * the epilogue is the contraction's: acc = the fp32 sum times 2^shift
//    (an exact integer), y0 = fl32(s fl32(acc)) and the fused post-processing,
//    four consecutive channels per lane after a round trip through LDS.
// The fp32 sums are exact under the same admission rule as the implicit-GEMM
// fp8 path (every product at most 2^12, 9 C x the largest product < 2^24), so
// the results equal that path's bit for bit.
#include "esb_internal.h"

namespace esb {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;           // four waves
constexpr int NT = 64;                  // output channels per workgroup
constexpr int CK = 64;                  // input channels per chunk
constexpr int TAPS = 9;
constexpr int WST = TAPS * CK + 16;     // LDS bytes per output channel of the filter slice:
                                        // 148 dwords, so the 16 lanes of a quarter-wave
                                        // (16 channels) take 16 different bank groups
constexpr int kPatchMax = 40 * 1024;    // bytes of the input patch
constexpr int kMaxCols = kThreads / 4;  // Q + 2: one thread per 16-byte chunk of a patch row
constexpr int SLAB = 72;                // fp32 row stride of the epilogue slabs
constexpr int kMaxFill = 10;            // patch chunks per thread and chunk of channels
constexpr int kWPer = NT * TAPS * 4 / kThreads;   // filter chunks per thread (9)
static_assert(4 * 32 * SLAB * 4 <= kPatchMax, "epilogue slabs fit the patch");
static_assert(kWPer * kThreads == NT * TAPS * 4, "whole filter chunks per thread");
constexpr int64_t kMultiMaxPixels = 16384;   // several chunks: at most this many output pixels

struct Conv3Params {
    const uint8_t* x;          // [N, H, W, C] codes (H = P, W = Q)
    const uint8_t* w;          // [K, 3, 3, C] codes
    const float* alphaX;
    const float* alphaW;
    int32_t* acc;              // [M, K] or NULL
    float* y;                  // [M, K] or NULL
    MmaDecode dx, dw;
    Post post;
    int N, P, Q, M;            // M = N P Q output pixels
    int H, W, st;              // input height and width, stride (1, or 2 in k_conv3x3)
    int half;                  // stride 2: padded columns of even index, (W + 3) / 2
    int C, K;                  // channels in and out (multiples of 64)
    int ntm, ntn;              // pixel tiles, channel tiles
    int out_shift;             // acc = fl32 sum * 2^out_shift
    int kX, kW;
};

__device__ __forceinline__ uint32_t dec8(uint32_t c, const MmaDecode& d) {
    const uint32_t t = (((c & d.lm) << d.shf) + d.inc) & d.lmf;   // exponent + 1 (mod 2^ebits)
    return ((c << d.shs) & 0x80808080u) | t;                       // sign to bit 7
}

__device__ __forceinline__ uint4 dec16(uint4 v, const MmaDecode& d) {
    return make_uint4(dec8(v.x, d), dec8(v.y, d), dec8(v.z, d), dec8(v.w, d));
}

// LDS byte offset of chunk c (0..3) of patch pixel pix.
__device__ __forceinline__ int patch_off(int pix, int c) {
    return (pix << 6) | ((c ^ ((pix >> 2) & 3)) << 4);
}

// The outputs of one 32-pixel block from a wave's slab (row stride sl floats,
// WCOLS channels from channel c0): four consecutive channels per lane.  AHEAD:
// the residual loads four at a time in flight before they are used (for kernels
// with one block per wave: with two, the registers do not fit); else one output
// group after the other.  Returns the lane's max |z| bit pattern.
template <int WCOLS, bool AHEAD>
__device__ __forceinline__ uint32_t store_block(const Conv3Params& p, const float* slab, int sl,
                                                int mrow, int c0, int lane, float qa) {
    constexpr int NIT = 32 * WCOLS / 256;
    uint32_t amax = 0;
    // Post-processing without a per-channel affine and without codes (ReLU /
    // residual / max|z| only) takes lean code instead of the general
    // post-processing; the unrolled form also takes the plain output (the rolled
    // form keeps its own plain loop, which issues no global load between the
    // stores).  z = v + 0 is the affine step of the general path with a = 1, b = 0
    // (one rounding: it turns -0 into +0), so both agree bit for bit.
    const bool lean = p.post.on ? (!p.post.a && !p.post.b && !p.post.codes) : AHEAD;
    const bool on = p.post.on != 0;
    const float* res = on ? p.post.res : nullptr;
    const bool relu = on && p.post.relu;
    const bool am = on && p.post.absmax;
    auto lean4 = [&](int64_t o, f32x4 z, f32x4 r) {
        if (on) {
#pragma unroll
            for (int c = 0; c < 4; c++) z[c] = z[c] + 0.0f;
        }
        if (res) {
#pragma unroll
            for (int c = 0; c < 4; c++) z[c] = z[c] + r[c];
        }
        if (relu) {
#pragma unroll
            for (int c = 0; c < 4; c++) z[c] = z[c] > 0.0f ? z[c] : 0.0f;
        }
        if (p.y) {
            float* d = p.y + o;
            if (((uintptr_t)d & 15) == 0) {
                *(f32x4*)d = z;
            } else {
#pragma unroll
                for (int c = 0; c < 4; c++) d[c] = z[c];
            }
        }
        uint32_t mz = 0;
        if (am) {
#pragma unroll
            for (int c = 0; c < 4; c++) mz = max(mz, __float_as_uint(z[c]) & 0x7fffffffu);
        }
        return mz;
    };
    auto res4 = [&](int64_t o) {
        f32x4 r = {0.0f, 0.0f, 0.0f, 0.0f};
        if (res) {
            const float* q = res + o;
            if (((uintptr_t)q & 15) == 0) {
                r = *(const f32x4*)q;
            } else {
#pragma unroll
                for (int c = 0; c < 4; c++) r[c] = q[c];
            }
        }
        return r;
    };
    if (AHEAD && lean) {   // unrolled, the residual loads four at a time ahead of use
#pragma unroll
        for (int k0 = 0; k0 < NIT; k0 += 4) {
            f32x4 rr[4];
#pragma unroll
            for (int k = 0; k < 4; k++) {
                const int e = 4 * lane + 256 * (k0 + k), row = e / WCOLS, col = e - row * WCOLS;
                const int m = mrow + row;
                rr[k] = (k0 + k < NIT && m < p.M) ? res4((int64_t)m * p.K + c0 + col)
                                                  : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            }
#pragma unroll
            for (int k = 0; k < 4; k++) {
                const int e = 4 * lane + 256 * (k0 + k), row = e / WCOLS, col = e - row * WCOLS;
                const int m = mrow + row;
                if (k0 + k < NIT && m < p.M) {
                    const int64_t o = (int64_t)m * p.K + c0 + col;
                    const f32x4 v = *(const f32x4*)(slab + row * sl + col);
                    amax = max(amax, lean4(o, v, rr[k]));
                }
            }
        }
        return amax;
    }
    if (!AHEAD) {
#pragma unroll 1
        for (int e = 4 * lane; e < 32 * WCOLS; e += 256) {
            const int row = e / WCOLS, col = e - row * WCOLS;
            const int m = mrow + row;
            if (m < p.M) {
                const int ch = c0 + col;
                const int64_t o = (int64_t)m * p.K + ch;
                const f32x4 v = *(const f32x4*)(slab + row * sl + col);
                if (lean) {
                    amax = max(amax, lean4(o, v, res4(o)));
                } else if (p.post.on) {
                    amax = max(amax, post_store4(p.post, p.y, o, ch, v, 4, qa));
                } else if (p.y) {
                    if (((uintptr_t)(p.y + o) & 15) == 0) {
                        *(f32x4*)(p.y + o) = v;
                    } else {
#pragma unroll
                        for (int c = 0; c < 4; c++) p.y[o + c] = v[c];
                    }
                }
            }
        }
        return amax;
    }
    if (p.post.on) {
#pragma unroll
        for (int k0 = 0; k0 < NIT; k0 += 4) {   // four residual loads in flight at a time
            f32x4 rr[4];
#pragma unroll
            for (int k = 0; k < 4; k++) {
                const int e = 4 * lane + 256 * (k0 + k), row = e / WCOLS, col = e - row * WCOLS;
                const int m = mrow + row;
                rr[k] = (k0 + k < NIT && m < p.M) ? post_res4(p.post, (int64_t)m * p.K + c0 + col)
                                                  : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            }
#pragma unroll
            for (int k = 0; k < 4; k++) {
                const int e = 4 * lane + 256 * (k0 + k), row = e / WCOLS, col = e - row * WCOLS;
                const int m = mrow + row;
                if (k0 + k < NIT && m < p.M) {
                    const int ch = c0 + col;
                    const f32x4 v = *(const f32x4*)(slab + row * sl + col);
                    amax = max(amax, post_apply4(p.post, p.y, (int64_t)m * p.K + ch, ch, v, rr[k], qa));
                }
            }
        }
    } else if (p.y) {
#pragma unroll
        for (int k = 0; k < NIT; k++) {
            const int e = 4 * lane + 256 * k, row = e / WCOLS, col = e - row * WCOLS;
            const int m = mrow + row;
            if (m < p.M) {
                const int64_t o = (int64_t)m * p.K + c0 + col;
                const f32x4 v = *(const f32x4*)(slab + row * sl + col);
                if (((uintptr_t)(p.y + o) & 15) == 0) {
                    *(f32x4*)(p.y + o) = v;
                } else {
#pragma unroll
                    for (int c = 0; c < 4; c++) p.y[o + c] = v[c];
                }
            }
        }
    }
    return amax;
}

// Two waves per SIMD: two workgroups share a CU (LDS 2 x 78 KB).  TMB: 32-pixel
// blocks per tile (8, 4 or 2; four waves take TMB x 2 blocks of 32 x 32).
// MULTI: more than one chunk of input channels (the filter slices then travel
// per chunk; at most 4 blocks per tile, for the registers).  ACC: the int32
// sums are written too (a separate instance: keeping both outputs live costs
// registers).
template <int TMB, bool MULTI, bool ACC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_conv3x3(Conv3Params p) {
    constexpr int TM = 32 * TMB;
    constexpr int NMB = TMB >= 8 ? 2 : 1;    // output blocks of a wave: NMB x NNB
    constexpr int NNB = TMB >= 4 ? 2 : 1;
    static_assert(4 * NMB * NNB == 2 * TMB, "four waves cover the tile");
    static_assert(!MULTI || TMB <= 4, "several chunks: at most 4 pixel blocks");
    __shared__ __align__(16) uint8_t wlds[NT * WST];
    __shared__ __align__(16) uint8_t patch[kPatchMax];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lr = lane & 31, lg = lane >> 5;
    // this wave's blocks: pixel blocks mbw + i (i < NMB), channel blocks nbw + j (j < NNB)
    const int mbw = TMB == 8 ? 2 * wave : (TMB == 4 ? wave : wave >> 1);
    const int nbw = TMB == 2 ? (wave & 1) : 0;

    const int nt = (int)blockIdx.x % p.ntn;          // this workgroup's output channels
    const int n0 = nt * NT;
    const int wg = (int)blockIdx.x / p.ntn, nwg = (int)gridDim.x / p.ntn;
    const int nchunks = MULTI ? p.C / CK : 1;

    const float s = ldexpf(p.alphaX[0] * p.alphaW[0], -(p.kX + p.kW));
    const float qa = post_alpha(p.post);
    uint32_t amax = 0;
    constexpr int FILL = kMaxFill;
    const int st = p.st;
    const int cols = p.W + 2, PP2 = p.H + 2, PQ = p.P * p.Q;
    // patch fill: thread t takes chunk t % (4 cols) of rows t / (4 cols), + rstep, ...
    const int cpr = 4 * cols;
    const int fci = tid % cpr, fri = tid / cpr, rstep = kThreads / cpr;
    const int fcol = fci >> 2, fc = fci & 3, iw = fcol - 1;
    const bool col_in = (unsigned)iw < (unsigned)p.W;
    // where padded column fcol sits in a patch row: stride 1 in order; stride 2 the
    // even columns first, then the odd ones, so that the taps of consecutive output
    // pixels (columns 2q + s) read consecutive patch pixels
    const int dcol = st == 1 ? fcol : ((fcol & 1) ? p.half + (fcol >> 1) : (fcol >> 1));
    const int tcol1 = st == 1 ? 1 : p.half, tcol2 = st == 1 ? 2 : 1;   // taps s = 1, 2
    // B fragments: channel 32 j + lr, bytes 32 lg .. + 31 of tap t
    const int boff = lr * WST + 32 * lg;
    const int64_t wrow = (int64_t)TAPS * p.C;        // filter bytes per output channel

    // The patch rows of a tile: padded rows R0 .. R0 + nrows - 1.
    auto rows_of = [&](int tile, int& R0, int& nrows) {
        const int m0 = tile * TM;
        const int i0 = m0 / PQ, p0 = (m0 - i0 * PQ) / p.Q;
        R0 = i0 * PP2 + st * p0;
        const int m1 = min(m0 + TM, p.M) - 1;
        const int i1 = m1 / PQ, p1 = (m1 - i1 * PQ) / p.Q;
        nrows = i1 * PP2 + st * p1 + 3 - R0;
    };
    // The codes of one (tile, chunk): this thread's patch chunks (chunk u is row
    // fri + u rstep; bit u of vmask: inside the input) and, with several chunks,
    // its filter chunks; every load in flight at once.
    uint4 raw[FILL], wraw[kWPer];
    uint32_t vmask = 0;
    auto fetch = [&](int tile, int ch) {
        int R0, nrows;
        rows_of(tile, R0, nrows);
        const int pr = R0 + fri;
        int n = pr / PP2, hp = pr - n * PP2;             // padded row hp of image n
        vmask = 0;
        const uint8_t* xc = p.x + CK * ch + 16 * fc;
#pragma unroll
        for (int u = 0; u < FILL; u++) {
            const int ih = hp - 1;
            const bool ok = fri < rstep && fri + u * rstep < nrows && col_in && n < p.N &&
                            (unsigned)ih < (unsigned)p.H;
            const int64_t pix = ok ? ((int64_t)n * p.H + ih) * p.W + iw : 0;
            raw[u] = *(const uint4*)(xc + pix * p.C);
            vmask |= ok ? (1u << u) : 0u;
            hp += rstep;
            while (hp >= PP2) { hp -= PP2; n++; }
        }
        if (MULTI) {
#pragma unroll
            for (int u = 0; u < kWPer; u++) {
                const int it = tid + u * kThreads;
                const int k = it / (TAPS * 4), rem = it - k * (TAPS * 4);
                const int t = rem >> 2, c16 = rem & 3;
                wraw[u] = *(const uint4*)(p.w + (n0 + k) * wrow + t * p.C + CK * ch + 16 * c16);
            }
        }
    };
    auto store_filter = [&]() {
#pragma unroll
        for (int u = 0; u < kWPer; u++) {
            const int it = tid + u * kThreads;
            const int k = it / (TAPS * 4), rem = it - k * (TAPS * 4);
            *(uint4*)&wlds[k * WST + 16 * rem] = dec16(wraw[u], p.dw);
        }
    };

    // ---- one chunk of channels: the filter once per workgroup, already in LDS
    if (!MULTI) {
#pragma unroll
        for (int u = 0; u < kWPer; u++) {
            const int it = tid + u * kThreads;
            const int k = it / (TAPS * 4), rem = it - k * (TAPS * 4);
            wraw[u] = *(const uint4*)(p.w + (n0 + k) * wrow + 16 * rem);
        }
        store_filter();
    }
    if (wg < p.ntm) fetch(wg, 0);

    for (int tile = wg; tile < p.ntm; tile += nwg) {
        const int m0 = tile * TM;
        int R0, nrows;
        rows_of(tile, R0, nrows);

        // ---- per lane and output block: the patch pixel of tap (0, 0)
        int pb[NMB];
#pragma unroll
        for (int i = 0; i < NMB; i++) {
            const int m = min(m0 + 32 * (mbw + i) + lr, p.M - 1);   // rows past M: any pixel
            const int n = m / PQ, rem = m - n * PQ;
            const int pp = rem / p.Q, q = rem - pp * p.Q;
            pb[i] = (n * PP2 + st * pp - R0) * cols + q;
        }
        v16f acc[NMB][NNB];
#pragma unroll
        for (int i = 0; i < NMB; i++)
#pragma unroll
            for (int j = 0; j < NNB; j++)
#pragma unroll
                for (int r = 0; r < 16; r++) acc[i][j][r] = 0.0f;

        for (int ch = 0; ch < nchunks; ch++) {
            __syncthreads();   // the previous chunk's (or tile's) reads of the LDS are done
            if (fri < rstep) {
#pragma unroll
                for (int u = 0; u < FILL; u++) {
                    const int i = fri + u * rstep;
                    if (i < nrows) {
                        const uint4 v = ((vmask >> u) & 1u) ? dec16(raw[u], p.dx)
                                                            : make_uint4(0u, 0u, 0u, 0u);   // E4M3 +0
                        *(uint4*)&patch[patch_off(i * cols + dcol, fc)] = v;
                    }
                }
            }
            if (MULTI) store_filter();
            __syncthreads();
            // the next chunk's codes, in flight during this chunk's MFMAs
            if (ch + 1 < nchunks) fetch(tile, ch + 1);
            else if (tile + nwg < p.ntm) fetch(tile + nwg, 0);

            // fragments of tap t (B: channel 32 j + lr; A: the patch pixel of tap t)
            auto frags = [&](int t, v8i (&fa)[NMB], v8i (&fb)[NNB]) {
                const int tr = t / 3, ts = t - 3 * tr;
#pragma unroll
                for (int j = 0; j < NNB; j++) {
                    const uint8_t* b = &wlds[boff + 32 * (nbw + j) * WST + 64 * t];
                    const v4i lo = *(const v4i*)b, hi = *(const v4i*)(b + 16);
                    fb[j] = v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                }
#pragma unroll
                for (int i = 0; i < NMB; i++) {
                    const int pix = pb[i] + tr * cols + (ts == 0 ? 0 : (ts == 1 ? tcol1 : tcol2));
                    const int a0 = patch_off(pix, 2 * lg);
                    const v4i lo = *(const v4i*)&patch[a0], hi = *(const v4i*)&patch[a0 ^ 16];
                    fa[i] = v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                }
            };
            // the next tap's fragments are read before this tap's MFMAs are issued, so
            // their LDS latency overlaps the MFMAs (two taps' fragments live at a time)
            v8i fa[NMB], fb[NNB];
            frags(0, fa, fb);
#pragma unroll
            for (int t = 0; t < TAPS; t++) {
                v8i na[NMB], nb[NNB];
                if (t + 1 < TAPS) frags(t + 1, na, nb);
#pragma unroll
                for (int i = 0; i < NMB; i++)
#pragma unroll
                    for (int j = 0; j < NNB; j++)
                        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                            fa[i], fb[j], acc[i][j], 0, 0, 0, 127, 0, 127);
                __builtin_amdgcn_sched_barrier(0);
                if (t + 1 < TAPS) {
#pragma unroll
                    for (int i = 0; i < NMB; i++) fa[i] = na[i];
#pragma unroll
                    for (int j = 0; j < NNB; j++) fb[j] = nb[j];
                }
            }
        }

        // ---- epilogue, one pixel block of each wave at a time: register r of
        //      block (i, j) is pixel m0 + 32 (mbw + i) + 8 (r / 4) + 4 lg + r % 4,
        //      channel n0 + 32 (nbw + j) + lr.  The scaled values go through the
        //      wave's LDS slab (row stride 72 floats: the two lane halves of a
        //      write are 32 banks apart) and come back as four consecutive
        //      channels per lane.
        __syncthreads();   // every read of the patch is done: the slabs reuse it
        float* slab = (float*)patch + wave * (32 * SLAB);
        constexpr int WCOLS = 32 * NNB;              // channels of a wave's blocks
        const int c0 = 32 * nbw;                      // their first column in the tile
#pragma unroll
        for (int i = 0; i < NMB; i++) {
            const int mrow = m0 + 32 * (mbw + i);
            if (ACC) {   // the exact integer sums, through the slab as well
#pragma unroll
                for (int j = 0; j < NNB; j++)
#pragma unroll
                    for (int r = 0; r < 16; r++)
                        ((int32_t*)slab)[(8 * (r >> 2) + 4 * lg + (r & 3)) * SLAB + 32 * j + lr] =
                            (int32_t)ldexpf(acc[i][j][r], p.out_shift);
                __syncthreads();
#pragma unroll 1
                for (int e = 4 * lane; e < 32 * WCOLS; e += 256) {
                    const int row = e / WCOLS, col = e - row * WCOLS;
                    const int m = mrow + row;
                    if (m < p.M) {
                        const int4 v = *(const int4*)((const int32_t*)slab + row * SLAB + col);
                        int32_t* d = p.acc + (int64_t)m * p.K + n0 + c0 + col;
                        if (((uintptr_t)d & 15) == 0) {
                            *(int4*)d = v;
                        } else {
                            d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
                        }
                    }
                }
                __syncthreads();
            }
#pragma unroll
            for (int j = 0; j < NNB; j++)
#pragma unroll
                for (int r = 0; r < 16; r++)
                    slab[(8 * (r >> 2) + 4 * lg + (r & 3)) * SLAB + 32 * j + lr] =
                        s * ldexpf(acc[i][j][r], p.out_shift);
            __syncthreads();
            amax = max(amax, store_block<WCOLS, NMB == 1>(p, slab, SLAB, mrow, n0 + c0, lane, qa));
            __syncthreads();
        }
    }
    post_absmax_flush(p.post, amax);
}

// ---------------------------------------------------------------------------
// Resident filter: for more than one chunk of input channels, one workgroup of
// eight waves per CU keeps the filter rows of its output channels (NTR = 64 or
// 32 of them, all 9 C bytes each) decoded in LDS for all of its tiles, so only
// the patch rows travel per chunk.  Tiles of 256 pixels, one 32-pixel block per
// wave; a row of the filter copy is 9 C + 16 bytes (an odd number of 16-byte
// groups: the 16 lanes of a quarter-wave take 16 different bank groups).
constexpr int kResThreads = 512;
constexpr int kResFilterMax = 76 * 1024;   // bytes of the resident filter copy
constexpr int kResFill = 10;               // filter chunks and patch chunks per thread

template <int NNB, bool ACC>
__global__ __launch_bounds__(kResThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_conv3x3_res(Conv3Params p) {
    constexpr int NTR = 32 * NNB;              // output channels per workgroup
    constexpr int TM = 256;                    // pixels per tile: block `wave` of 8
    constexpr int SL = NTR + 8;                // slab row stride (floats): two lane halves
                                               // 4 rows apart are 32 banks apart
    static_assert(4 * 32 * SL * 4 <= kPatchMax, "epilogue slabs fit");
    __shared__ __align__(16) uint8_t wres[kResFilterMax];
    __shared__ __align__(16) uint8_t patch[kPatchMax];
    __shared__ __align__(16) uint8_t spare[kPatchMax];   // the slabs of waves 4..7
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lr = lane & 31, lg = lane >> 5;

    const int nt = (int)blockIdx.x % p.ntn;
    const int n0 = nt * NTR;
    const int wg = (int)blockIdx.x / p.ntn, nwg = (int)gridDim.x / p.ntn;
    const int nchunks = p.C / CK;
    const int wst = TAPS * p.C + 16;                      // LDS bytes per filter row
    const int row16 = TAPS * p.C / 16;                    // 16-byte chunks of a filter row

    // ---- the filter rows n0 .. n0 + NTR - 1, once, every load in flight
    {
        uint4 wv[kResFill];
#pragma unroll
        for (int u = 0; u < kResFill; u++) {
            const int it = tid + u * kResThreads;
            const int k = it / row16, rem = it - k * row16;
            wv[u] = k < NTR ? *(const uint4*)(p.w + (int64_t)(n0 + k) * (TAPS * p.C) + 16 * rem)
                            : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int u = 0; u < kResFill; u++) {
            const int it = tid + u * kResThreads;
            const int k = it / row16, rem = it - k * row16;
            if (k < NTR) *(uint4*)&wres[k * wst + 16 * rem] = dec16(wv[u], p.dw);
        }
    }

    const float s = ldexpf(p.alphaX[0] * p.alphaW[0], -(p.kX + p.kW));
    const float qa = post_alpha(p.post);
    uint32_t amax = 0;
    const int cols = p.Q + 2, PP2 = p.P + 2, PQ = p.P * p.Q;
    const int cpr = 4 * cols;
    const int fci = tid % cpr, fri = tid / cpr, rstep = kResThreads / cpr;
    const int fcol = fci >> 2, fc = fci & 3, iw = fcol - 1;
    const bool col_in = (unsigned)iw < (unsigned)p.Q;
    // B fragments: output channel 32 j + lr, bytes 32 lg .. + 31 of (tap t, chunk ch)
    const int boff = lr * wst + 32 * lg;

    auto rows_of = [&](int tile, int& R0, int& nrows) {
        const int m0 = tile * TM;
        const int i0 = m0 / PQ, p0 = (m0 - i0 * PQ) / p.Q;
        R0 = i0 * PP2 + p0;
        const int m1 = min(m0 + TM, p.M) - 1;
        const int i1 = m1 / PQ, p1 = (m1 - i1 * PQ) / p.Q;
        nrows = i1 * PP2 + p1 + 3 - R0;
    };
    uint4 raw[kResFill];
    uint32_t vmask = 0;
    auto fetch = [&](int tile, int ch) {
        int R0, nrows;
        rows_of(tile, R0, nrows);
        const int pr = R0 + fri;
        int n = pr / PP2, hp = pr - n * PP2;
        vmask = 0;
        const uint8_t* xc = p.x + CK * ch + 16 * fc;
#pragma unroll
        for (int u = 0; u < kResFill; u++) {
            const int ih = hp - 1;
            const bool ok = fri < rstep && fri + u * rstep < nrows && col_in && n < p.N &&
                            (unsigned)ih < (unsigned)p.P;
            const int64_t pix = ok ? ((int64_t)n * p.P + ih) * p.Q + iw : 0;
            raw[u] = *(const uint4*)(xc + pix * p.C);
            vmask |= ok ? (1u << u) : 0u;
            hp += rstep;
            while (hp >= PP2) { hp -= PP2; n++; }
        }
    };
    if (wg < p.ntm) fetch(wg, 0);

    for (int tile = wg; tile < p.ntm; tile += nwg) {
        const int m0 = tile * TM;
        int R0, nrows;
        rows_of(tile, R0, nrows);
        int pb;
        {
            const int m = min(m0 + 32 * wave + lr, p.M - 1);   // rows past M: any pixel
            const int n = m / PQ, rem = m - n * PQ;
            const int pp = rem / p.Q, q = rem - pp * p.Q;
            pb = (n * PP2 + pp - R0) * cols + q;
        }
        v16f acc[NNB];
#pragma unroll
        for (int j = 0; j < NNB; j++)
#pragma unroll
            for (int r = 0; r < 16; r++) acc[j][r] = 0.0f;

        for (int ch = 0; ch < nchunks; ch++) {
            __syncthreads();   // the previous chunk's (or tile's) reads of the patch are done
            if (fri < rstep) {
#pragma unroll
                for (int u = 0; u < kResFill; u++) {
                    const int i = fri + u * rstep;
                    if (i < nrows) {
                        const uint4 v = ((vmask >> u) & 1u) ? dec16(raw[u], p.dx)
                                                            : make_uint4(0u, 0u, 0u, 0u);   // E4M3 +0
                        *(uint4*)&patch[patch_off(i * cols + fcol, fc)] = v;
                    }
                }
            }
            __syncthreads();
            if (ch + 1 < nchunks) fetch(tile, ch + 1);
            else if (tile + nwg < p.ntm) fetch(tile + nwg, 0);

            const uint8_t* wb = &wres[boff + CK * ch];
            auto frags = [&](int t, v8i& fa, v8i (&fb)[NNB]) {
                const int tr = t / 3, ts = t - 3 * tr;
#pragma unroll
                for (int j = 0; j < NNB; j++) {
                    const uint8_t* b = wb + 32 * j * wst + t * p.C;
                    const v4i lo = *(const v4i*)b, hi = *(const v4i*)(b + 16);
                    fb[j] = v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                }
                const int pix = pb + tr * cols + ts;
                const int a0 = patch_off(pix, 2 * lg);
                const v4i lo = *(const v4i*)&patch[a0], hi = *(const v4i*)&patch[a0 ^ 16];
                fa = v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            };
            v8i fa, fb[NNB];   // the next tap's fragments read before this tap's MFMAs
            frags(0, fa, fb);
#pragma unroll
            for (int t = 0; t < TAPS; t++) {
                v8i na, nb[NNB];
                if (t + 1 < TAPS) frags(t + 1, na, nb);
#pragma unroll
                for (int j = 0; j < NNB; j++)
                    acc[j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                        fa, fb[j], acc[j], 0, 0, 0, 127, 0, 127);
                __builtin_amdgcn_sched_barrier(0);
                if (t + 1 < TAPS) {
                    fa = na;
#pragma unroll
                    for (int j = 0; j < NNB; j++) fb[j] = nb[j];
                }
            }
        }

        // ---- epilogue: block `wave` (pixels m0 + 32 wave ..), register r of
        //      channel block j is pixel + 8 (r / 4) + 4 lg + r % 4, channel
        //      n0 + 32 j + lr; through the wave's slab, four channels per lane
        __syncthreads();   // every read of the patch is done: the slabs reuse it
        float* slab = (float*)(wave < 4 ? patch : spare) + (wave & 3) * (32 * SL);
        const int mrow = m0 + 32 * wave;
        if (ACC) {
#pragma unroll
            for (int j = 0; j < NNB; j++)
#pragma unroll
                for (int r = 0; r < 16; r++)
                    ((int32_t*)slab)[(8 * (r >> 2) + 4 * lg + (r & 3)) * SL + 32 * j + lr] =
                        (int32_t)ldexpf(acc[j][r], p.out_shift);
            __syncthreads();
#pragma unroll 1
            for (int e = 4 * lane; e < 32 * NTR; e += 256) {
                const int row = e / NTR, col = e - row * NTR;
                const int m = mrow + row;
                if (m < p.M) {
                    const int4 v = *(const int4*)((const int32_t*)slab + row * SL + col);
                    int32_t* d = p.acc + (int64_t)m * p.K + n0 + col;
                    if (((uintptr_t)d & 15) == 0) {
                        *(int4*)d = v;
                    } else {
                        d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
                    }
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int j = 0; j < NNB; j++)
#pragma unroll
            for (int r = 0; r < 16; r++)
                slab[(8 * (r >> 2) + 4 * lg + (r & 3)) * SL + 32 * j + lr] =
                    s * ldexpf(acc[j][r], p.out_shift);
        __syncthreads();
        amax = max(amax, store_block<NTR, true>(p, slab, SL, mrow, n0, lane, qa));
    }
    post_absmax_flush(p.post, amax);
}

// Output channels per workgroup of the resident-filter kernel (64, else 32), 0
// when neither copy fits.
int res_ntr(int C, int K) {
    for (int ntr = 64; ntr >= 32; ntr >>= 1)
        if (K % ntr == 0 && (int64_t)ntr * (TAPS * C + 16) <= kResFilterMax &&
            (int64_t)ntr * TAPS * C <= (int64_t)kResFill * 16 * kResThreads)
            return ntr;
    return 0;
}

bool res_tile_fits(int P, int Q) {
    if (4 * (Q + 2) > kResThreads) return false;
    const int rstep = kResThreads / (4 * (Q + 2));
    const int dg = (Q - 1 + 256 - 1) / Q, cross = (P - 1 + dg) / P;
    const int rows = dg + 2 * cross + 3;
    return (rows + rstep - 1) / rstep <= kResFill && (int64_t)rows * (Q + 2) * 64 <= kPatchMax;
}

// Rows of the patch of a tile of TM pixels: the padded rows from the first
// pixel's to two past the last pixel's, at most dg + 2 (images crossed) + 3
// rows with dg the output rows a tile spans beyond its first.
// With stride st the tile's output rows span st dg + 3 padded input rows, and each
// image boundary crossed adds the H + 2 - st P padded rows past the last output row's.
int patch_rows_max(int P, int Q, int TM, int H, int st) {
    const int dg = (Q - 1 + TM - 1) / Q;
    const int cross = (P - 1 + dg) / P;
    return st * dg + cross * (H + 2 - st * P) + 3;
}

bool tile_fits(int P, int Q, int TM, int H, int W, int st) {
    if (W + 2 > kMaxCols) return false;
    const int rstep = kThreads / (4 * (W + 2));
    const int rows = patch_rows_max(P, Q, TM, H, st);
    return (rows + rstep - 1) / rstep <= kMaxFill && (int64_t)rows * (W + 2) * 64 <= kPatchMax;
}

// 32-pixel blocks per tile: the largest of 8, 4, 2 (4, 2 with several chunks of
// input channels) whose tiles fit the patch and give at least one workgroup per
// CU (half a workgroup per CU with several chunks: every tile streams the filter
// slices again, so larger tiles halve that traffic per pixel; ResNet18 l4 at batch
// 64, 200 tiles of 128 pixels against 392 of 64: 33.9 against 35.5 us), else the
// largest that fits.
int choose_tmb(int64_t M, int ntn, int P, int Q, int H, int W, int st, bool multi) {
    const int cus = num_cus();
    int fit = 0;
    for (int tmb = multi ? 4 : 8; tmb >= 2; tmb >>= 1) {
        if (!tile_fits(P, Q, 32 * tmb, H, W, st)) continue;
        if (!fit) fit = tmb;
        if ((M + 32 * tmb - 1) / (32 * tmb) * ntn >= (multi ? cus / 2 : cus)) return tmb;
    }
    return fit;
}

}  // namespace

bool conv3x3_fits(const ConvGeom& g, int K, int groups, int op, const uint8_t* x,
                  const uint8_t* w) {
    if (!(groups == 1 && op == 1 && K % NT == 0 && K >= NT && g.C % CK == 0 && g.C >= CK &&
          g.Cg == g.C && g.pitch == g.C && g.R == 3 && g.S == 3 && g.ph == 1 && g.pw == 1 &&
          g.P >= 1 && g.Q >= 1))
        return false;
    const bool s1 = g.sh == 1 && g.sw == 1 && g.P == g.H && g.Q == g.W;
    const bool s2 = g.sh == 2 && g.sw == 2 && g.P == (g.H - 1) / 2 + 1 && g.Q == (g.W - 1) / 2 + 1;
    if (!s1 && !s2) return false;
    // Stride 2 takes tiles of 64 output pixels (the patch holds four times the input
    // of stride 1 per pixel), whose fill, repeated by every tile of 64 output channels,
    // outweighs the MFMAs unless the input channels run to several chunks: measured
    // at batch 64 against the implicit-GEMM path, 256 -> 512 at 14 x 14 24.1 against
    // 28.4 us, but 64 -> 128 at 56 x 56 25.3 against 21.0 and 128 -> 256 at 28 x 28
    // 28.5 against 19.6.
    if (s2 && g.C < 4 * CK) return false;
    if ((uintptr_t)x % 16 || (uintptr_t)w % 16) return false;
    const int64_t M = (int64_t)g.Nb * g.P * g.Q;
    if ((M + 256) * K >= ((int64_t)1 << 31) || (int64_t)K * TAPS * g.C >= ((int64_t)1 << 31))
        return false;
    // With several chunks every workgroup decodes its 64 filter rows per chunk and tile:
    // measured faster than the implicit-GEMM kernels only for few output pixels (ResNet18
    // 3x3 at batch 64: 256 channels at 14 x 14 and 512 at 7 x 7 faster, 128 at 28 x 28
    // with 50176 pixels slower).
    if (g.C > CK && M > kMultiMaxPixels)   // several chunks and many pixels: resident filter
        return s1 && res_ntr(g.C, K) != 0 && res_tile_fits(g.P, g.Q);
    return choose_tmb(M, K / NT, g.P, g.Q, g.H, g.W, g.sh, g.C > CK) != 0;
}

hipError_t launch_conv3x3(const ConvGeom& g, int K, const uint8_t* x, const Fmt& fx,
                          const float* alphaX, const uint8_t* w, const Fmt& fw,
                          const float* alphaW, int32_t* acc, float* y, hipStream_t s,
                          const Post* post) {
    Conv3Params p{};
    p.x = x;
    p.w = w;
    p.alphaX = alphaX;
    p.alphaW = alphaW;
    p.acc = acc;
    p.y = y;
    p.dx = mma_decode(fx, 1);
    p.dw = mma_decode(fw, 1);
    if (post) p.post = *post;
    p.N = g.Nb;
    p.P = g.P;
    p.Q = g.Q;
    p.H = g.H;
    p.W = g.W;
    p.st = g.sh;
    p.half = (g.W + 3) / 2;
    p.M = g.Nb * g.P * g.Q;
    p.C = g.C;
    p.K = K;
    if (p.M == 0) return hipSuccess;
    p.out_shift = fx.k + fw.k + 12;
    p.kX = fx.k;
    p.kW = fw.k;
    if (g.C > CK && p.M > kMultiMaxPixels) {   // the resident-filter kernel, one workgroup per CU
        if (p.st != 1) return hipErrorInvalidValue;
        const int ntr = res_ntr(g.C, K);
        if (ntr == 0 || !res_tile_fits(g.P, g.Q)) return hipErrorInvalidValue;
        p.ntn = K / ntr;
        p.ntm = (p.M + 255) / 256;
        int per = num_cus() / p.ntn;
        if (per < 1) per = 1;
        if (per > p.ntm) per = p.ntm;
        const unsigned blocks = (unsigned)(per * p.ntn);
        if (ntr == 64) {
            if (acc) k_conv3x3_res<2, true><<<blocks, kResThreads, 0, s>>>(p);
            else k_conv3x3_res<2, false><<<blocks, kResThreads, 0, s>>>(p);
        } else {
            if (acc) k_conv3x3_res<1, true><<<blocks, kResThreads, 0, s>>>(p);
            else k_conv3x3_res<1, false><<<blocks, kResThreads, 0, s>>>(p);
        }
        return hipGetLastError();
    }
    p.ntn = K / NT;
    const bool multi = g.C > CK;
    const int tmb = choose_tmb(p.M, p.ntn, g.P, g.Q, g.H, g.W, p.st, multi);
    if (tmb == 0) return hipErrorInvalidValue;
    p.ntm = (p.M + 32 * tmb - 1) / (32 * tmb);
    // persistent workgroups, a whole number per channel tile, two per CU
    int per = (num_cus() * 2) / p.ntn;
    if (per < 1) per = 1;
    if (per > p.ntm) per = p.ntm;
    const unsigned blocks = (unsigned)(per * p.ntn);
#define ESB_CONV3_LAUNCH(TMB, MULTI)                                                 \
    do {                                                                             \
        if (acc) k_conv3x3<TMB, MULTI, true><<<blocks, kThreads, 0, s>>>(p);         \
        else k_conv3x3<TMB, MULTI, false><<<blocks, kThreads, 0, s>>>(p);            \
    } while (0)
    if (!multi && tmb == 8) ESB_CONV3_LAUNCH(8, false);
    else if (!multi && tmb == 4) ESB_CONV3_LAUNCH(4, false);
    else if (!multi) ESB_CONV3_LAUNCH(2, false);
    else if (tmb == 4) ESB_CONV3_LAUNCH(4, true);
    else ESB_CONV3_LAUNCH(2, true);
#undef ESB_CONV3_LAUNCH
    return hipGetLastError();
}

}  // namespace esb
