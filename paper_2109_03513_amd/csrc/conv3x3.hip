// Direct 3x3 / stride-1 / pad-1 convolution over ESB codes with 64 input and
// 64 output channels, on the fp8 MFMA of gfx950 (Sec. 4.2: the convolution
// stage; products of codes by eq. (15), exact as in the implicit-GEMM path).
//
// The implicit-GEMM kernels fetch and decode every input element once per
// filter tap it meets, nine times for a 3x3 filter.  Here a workgroup owns 256
// consecutive output pixels (flattened over the batch) and all 64 channels:
//  * the filter (64 x 9 x 64 codes) is decoded to E4M3 once per workgroup and
//    stays in LDS (workgroups are persistent over the tiles);
//  * the input rows under a tile are decoded to E4M3 once into an LDS patch,
//    one 64-byte row per input pixel.  Every image is seen with a zero row
//    above and below it and a zero column left and right (the padding), so a
//    tile may cross images: output pixel (n, p, q) and tap (r, s) read patch
//    pixel (n (P + 2) + p + r - R0, q + s), R0 the padded row of the tile's
//    first pixel.  The four 16-byte chunks of a patch pixel are stored in the
//    order chunk ^ ((pixel / 4) % 4), so that 16 consecutive pixels read at one
//    chunk (a quarter-wave of a fragment load) hit 16 different bank groups;
//  * per tap one v_mfma_scale_f32_32x32x64_f8f6f4 per 32 x 32 block; wave w
//    takes output blocks 2w, 2w + 1 and both halves of the channels;
//  * the epilogue is the contraction's: acc = the fp32 sum times 2^shift
//    (an exact integer), y0 = fl32(s fl32(acc)) and the fused post-processing,
//    four consecutive channels per lane after a round trip through LDS.
// The fp32 sums are exact under the same admission rule as the implicit-GEMM
// fp8 path (every product at most 2^12, 576 x the largest product < 2^24), so
// the results equal that path's bit for bit.
#include "esb_internal.h"

namespace esb {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;           // four waves
constexpr int TM = 256;                 // output pixels per tile (8 blocks of 32)
constexpr int CH = 64;                  // input = output channels
constexpr int TAPS = 9;
constexpr int WST = TAPS * CH + 16;     // LDS bytes per output channel of the filter: 148
                                        // dwords, so the 16 lanes of a quarter-wave
                                        // (16 channels) take 16 different bank groups
constexpr int kPatchMax = 40 * 1024;    // bytes of the input patch
constexpr int kMaxCols = kThreads / 4;  // Q + 2: one thread per 16-byte chunk of a patch row
constexpr int SLAB = 72;                // fp32 row stride of the epilogue slabs
constexpr int kMaxFill = 12;            // patch chunks per thread and tile
static_assert(4 * 32 * SLAB * 4 <= kPatchMax, "epilogue slabs fit the patch");

struct Conv3Params {
    const uint8_t* x;          // [N, H, W, 64] codes (H = P, W = Q)
    const uint8_t* w;          // [64, 3, 3, 64] codes
    const float* alphaX;
    const float* alphaW;
    int32_t* acc;              // [M, 64] or NULL
    float* y;                  // [M, 64] or NULL
    MmaDecode dx, dw;
    Post post;
    int N, P, Q, M;            // M = N P Q output pixels
    int ntiles;
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

// Two waves per SIMD: two workgroups share a CU (LDS 2 x 78 KB).  ACC: the
// int32 sums are written too (a separate instance: keeping both outputs live
// costs registers).
template <bool ACC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_conv3x3(Conv3Params p) {
    __shared__ __align__(16) uint8_t wlds[CH * WST];
    __shared__ __align__(16) uint8_t patch[kPatchMax];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lr = lane & 31, lg = lane >> 5;

    // ---- the filter, once: channel k, tap t, chunk c at k * WST + 64 t + 16 c;
    //      the nine loads of a thread in flight together
    {
        constexpr int kPer = CH * TAPS * 4 / kThreads;
        static_assert(kPer * kThreads == CH * TAPS * 4, "whole chunks per thread");
        uint4 wv[kPer];
#pragma unroll
        for (int u = 0; u < kPer; u++) wv[u] = *(const uint4*)(p.w + 16 * (tid + u * kThreads));
#pragma unroll
        for (int u = 0; u < kPer; u++) {
            const int it = tid + u * kThreads;
            const int k = it / (TAPS * 4), rem = it - k * (TAPS * 4);
            *(uint4*)&wlds[k * WST + 16 * rem] = dec16(wv[u], p.dw);
        }
    }

    const float s = ldexpf(p.alphaX[0] * p.alphaW[0], -(p.kX + p.kW));
    const float qa = post_alpha(p.post);
    uint32_t amax = 0;
    const int cols = p.Q + 2, PP2 = p.P + 2, PQ = p.P * p.Q;
    // patch fill: thread t takes chunk t % (4 cols) of rows t / (4 cols), + rstep, ...
    const int cpr = 4 * cols;
    const int fci = tid % cpr, fri = tid / cpr, rstep = kThreads / cpr;
    const int fcol = fci >> 2, fc = fci & 3, iw = fcol - 1;
    const bool col_in = (unsigned)iw < (unsigned)p.Q;
    // B fragments: channel 32 j + lr, bytes 32 lg .. + 31 of tap t
    const int boff = lr * WST + 32 * lg;

    // The patch rows of a tile: padded rows R0 .. R0 + nrows - 1.
    auto rows_of = [&](int tile, int& R0, int& nrows) {
        const int m0 = tile * TM;
        const int n0 = m0 / PQ, p0 = (m0 - n0 * PQ) / p.Q;
        R0 = n0 * PP2 + p0;
        const int m1 = min(m0 + TM, p.M) - 1;
        const int n1 = m1 / PQ, p1 = (m1 - n1 * PQ) / p.Q;
        nrows = n1 * PP2 + p1 + 3 - R0;
    };
    // This thread's chunks of a tile's patch, all loads in flight at once: chunk u
    // is row fri + u rstep; bit u of vmask tells whether it lies inside the input.
    uint4 raw[kMaxFill];
    uint32_t vmask = 0;
    auto fetch = [&](int tile) {
        int R0, nrows;
        rows_of(tile, R0, nrows);
        const int pr = R0 + fri;
        int n = pr / PP2, hp = pr - n * PP2;             // padded row hp of image n
        vmask = 0;
#pragma unroll
        for (int u = 0; u < kMaxFill; u++) {
            const int ih = hp - 1;
            const bool ok = fri < rstep && fri + u * rstep < nrows && col_in && n < p.N &&
                            (unsigned)ih < (unsigned)p.P;
            const int64_t pix = ok ? ((int64_t)n * p.P + ih) * p.Q + iw : 0;
            raw[u] = *(const uint4*)(p.x + (pix << 6) + 16 * fc);
            vmask |= ok ? (1u << u) : 0u;
            hp += rstep;
            while (hp >= PP2) { hp -= PP2; n++; }
        }
    };
    if (blockIdx.x < p.ntiles) fetch(blockIdx.x);

    for (int tile = blockIdx.x; tile < p.ntiles; tile += gridDim.x) {
        const int m0 = tile * TM;
        int R0, nrows;
        rows_of(tile, R0, nrows);

        __syncthreads();   // the previous tile's reads of the patch are done
        if (fri < rstep) {
#pragma unroll
            for (int u = 0; u < kMaxFill; u++) {
                const int i = fri + u * rstep;
                if (i < nrows) {
                    const uint4 v = ((vmask >> u) & 1u) ? dec16(raw[u], p.dx)
                                                        : make_uint4(0u, 0u, 0u, 0u);   // E4M3 +0
                    *(uint4*)&patch[patch_off(i * cols + fcol, fc)] = v;
                }
            }
        }
        __syncthreads();
        if (tile + (int)gridDim.x < p.ntiles) fetch(tile + gridDim.x);   // in flight below

        // ---- per lane and output block: the patch pixel of tap (0, 0)
        int pb[2];
#pragma unroll
        for (int i = 0; i < 2; i++) {
            const int m = min(m0 + 32 * (2 * wave + i) + lr, p.M - 1);   // rows past M: any pixel
            const int n = m / PQ, rem = m - n * PQ;
            const int pp = rem / p.Q, q = rem - pp * p.Q;
            pb[i] = (n * PP2 + pp - R0) * cols + q;
        }
        v16f acc[2][2];
#pragma unroll
        for (int i = 0; i < 2; i++)
#pragma unroll
            for (int j = 0; j < 2; j++)
#pragma unroll
                for (int r = 0; r < 16; r++) acc[i][j][r] = 0.0f;
#pragma unroll
        for (int t = 0; t < TAPS; t++) {
            const int tr = t / 3, ts = t - 3 * tr;
            v8i fb[2], fa[2];
#pragma unroll
            for (int j = 0; j < 2; j++) {
                const uint8_t* b = &wlds[boff + 32 * j * WST + 64 * t];
                const v4i lo = *(const v4i*)b, hi = *(const v4i*)(b + 16);
                fb[j] = v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            }
#pragma unroll
            for (int i = 0; i < 2; i++) {
                const int pix = pb[i] + tr * cols + ts;
                const int a0 = patch_off(pix, 2 * lg);
                const v4i lo = *(const v4i*)&patch[a0], hi = *(const v4i*)&patch[a0 ^ 16];
                fa[i] = v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            }
#pragma unroll
            for (int i = 0; i < 2; i++)
#pragma unroll
                for (int j = 0; j < 2; j++)
                    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                        fa[i], fb[j], acc[i][j], 0, 0, 0, 127, 0, 127);
            __builtin_amdgcn_sched_barrier(0);   // one tap's fragments live at a time
        }

        // ---- epilogue, one output block of each wave at a time: register r of
        //      block (i, j) is pixel m0 + 32 (2 wave + i) + 8 (r / 4) + 4 lg + r % 4,
        //      channel 32 j + lr.  The scaled values go through the wave's LDS slab
        //      (row stride 72 floats: the two lane halves of a write are 32 banks
        //      apart) and come back as four consecutive channels per lane.
        __syncthreads();   // every read of the patch is done: the slabs reuse it
        float* slab = (float*)patch + wave * (32 * SLAB);
#pragma unroll
        for (int i = 0; i < 2; i++) {
            const int mrow = m0 + 32 * (2 * wave + i);
            if (ACC) {   // the exact integer sums, through the slab as well
#pragma unroll
                for (int j = 0; j < 2; j++)
#pragma unroll
                    for (int r = 0; r < 16; r++)
                        ((int32_t*)slab)[(8 * (r >> 2) + 4 * lg + (r & 3)) * SLAB + 32 * j + lr] =
                            (int32_t)ldexpf(acc[i][j][r], p.out_shift);
                __syncthreads();
#pragma unroll 1
                for (int e = 4 * lane; e < 32 * CH; e += 256) {
                    const int row = e / CH, col = e - row * CH;
                    const int m = mrow + row;
                    if (m < p.M) {
                        const int4 v = *(const int4*)((const int32_t*)slab + row * SLAB + col);
                        int32_t* d = p.acc + (int64_t)m * CH + col;
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
            for (int j = 0; j < 2; j++)
#pragma unroll
                for (int r = 0; r < 16; r++)
                    slab[(8 * (r >> 2) + 4 * lg + (r & 3)) * SLAB + 32 * j + lr] =
                        s * ldexpf(acc[i][j][r], p.out_shift);
            __syncthreads();
#pragma unroll 1
            for (int e = 4 * lane; e < 32 * CH; e += 256) {
                const int row = e / CH, col = e - row * CH;
                const int m = mrow + row;
                if (m < p.M) {
                    const int64_t o = (int64_t)m * CH + col;
                    const f32x4 v = *(const f32x4*)(slab + row * SLAB + col);
                    if (p.post.on) {
                        amax = max(amax, post_store4(p.post, p.y, o, col, v, 4, qa));
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
            __syncthreads();
        }
    }
    post_absmax_flush(p.post, amax);
}

// Rows of the patch of a tile: the padded rows from the first pixel's to two
// past the last pixel's, at most dg + 2 (images crossed) + 3 rows with dg the
// output rows a tile spans beyond its first.
int patch_rows_max(int P, int Q) {
    const int dg = (Q - 1 + TM - 1) / Q;
    const int cross = (P - 1 + dg) / P;
    return dg + 2 * cross + 3;
}

}  // namespace

bool conv3x3_fits(const ConvGeom& g, int K, int groups, int op, const uint8_t* x,
                  const uint8_t* w) {
    if (!(groups == 1 && op == 1 && K == CH && g.C == CH && g.Cg == CH && g.pitch == CH &&
          g.R == 3 && g.S == 3 && g.sh == 1 && g.sw == 1 && g.ph == 1 && g.pw == 1 &&
          g.P == g.H && g.Q == g.W && g.P >= 1 && g.Q >= 1))
        return false;
    if ((uintptr_t)x % 16 || (uintptr_t)w % 16) return false;
    if (g.Q + 2 > kMaxCols) return false;
    const int rstep = kThreads / (4 * (g.Q + 2));
    if ((patch_rows_max(g.P, g.Q) + rstep - 1) / rstep > kMaxFill) return false;
    const int64_t M = (int64_t)g.Nb * g.P * g.Q;
    if (M + TM >= ((int64_t)1 << 31) / CH) return false;
    return (int64_t)patch_rows_max(g.P, g.Q) * (g.Q + 2) * 64 <= kPatchMax;
}

hipError_t launch_conv3x3(const ConvGeom& g, const uint8_t* x, const Fmt& fx, const float* alphaX,
                          const uint8_t* w, const Fmt& fw, const float* alphaW, int32_t* acc,
                          float* y, hipStream_t s, const Post* post) {
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
    p.M = g.Nb * g.P * g.Q;
    if (p.M == 0) return hipSuccess;
    p.ntiles = (p.M + TM - 1) / TM;
    p.out_shift = fx.k + fw.k + 12;
    p.kX = fx.k;
    p.kW = fw.k;
    int blocks = num_cus() * 2;
    if (blocks > p.ntiles) blocks = p.ntiles;
    if (acc) k_conv3x3<true><<<blocks, kThreads, 0, s>>>(p);
    else k_conv3x3<false><<<blocks, kThreads, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace esb
