// Stem of a convolutional network on ESB codes: a convolution with few input
// channels and stride 2, the post-processing of eq. (16) with a ReLU, and the
// 3x3 / stride-2 max pool that follows it (Sec. 4.2: the convolution stage,
// then "MP&ReLU"), in one kernel that writes only the pooled outputs.
//
// The generic implicit-GEMM kernels gather the reduction of a 3-channel input
// byte by byte and write the full-resolution output (for the ResNet stem at
// batch 64: 205 MB of fp32) that the pool reads back.  Here a workgroup owns
// an 8 x 8 tile of pooled outputs and all 64 output channels:
//   * the input patch under the tile's 17 x 17 convolution outputs (39 x 39
//     pixels for a 7 x 7 filter; fetched while the previous tile's MFMAs run,
//     positions outside the image as the +0 code) is decoded to exact int8
//     integers m = q 2^k and kept in LDS in eight copies shifted by 0, 2, ...,
//     14 bytes, so that every 16-byte piece of a filter row, which starts at
//     an even byte, is one aligned LDS read;
//   * the reduction runs in the order (filter row r, then the S*C <= 32
//     contiguous bytes of that row), padded to 32 per row: one
//     v_mfma_i32_32x32x32_i8 per filter row and 32 x 32 output block, with the
//     filter's padding bytes zero so that the bytes read past a row's end add
//     nothing;
//   * the int32 sums are scaled (fl32(s fl32(acc))), post-processed and
//     rectified into an LDS tile, pooled (conv positions outside the output
//     are left out: every value is >= 0 and every window holds one inside),
//     and written once as fp32 and / or as the next layer's codes.
// The filter (64 x R x 32 bytes) is decoded once per workgroup into LDS;
// workgroups are persistent over the tiles.
#include "esb_internal.h"

namespace esb {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kThreads = 512;             // eight waves: two channel halves x four row groups
constexpr int TP = 8, TQ = 8;            // pooled outputs per tile
constexpr int CR = 2 * TP + 1;           // convolution outputs per tile: 17 x 17
constexpr int CC = 2 * TQ + 1;
constexpr int NPIX = CR * CC;            // 289
constexpr int MB = (NPIX + 31) / 32;     // 10 blocks of 32 rows
constexpr int WGR = kThreads / 128;      // waves per channel half (4)
constexpr int MBW = (MB + WGR - 1) / WGR;   // M blocks per wave (3)
constexpr int KO = 64;                   // output channels
constexpr int RMAX = 8;                  // filter rows
constexpr int PROWS = 2 * (CR - 1) + RMAX;   // input rows of a patch (<= 40)
constexpr int ROWB = 128;                // bytes of one stored patch row (one copy)
constexpr int CSTR = ROWB + 16;          // LDS stride of the copies: 9 bank groups of 16 bytes,
                                         // so that the lanes of an MFMA read (pixels at
                                         // different copies) spread over the banks
constexpr int NCOPY = 8;                 // copies shifted by 2 v bytes, v = 0..7
constexpr int STAGE_DW = ROWB / 4 + 4;   // a decoded patch row (+ spare dwords, zero)
constexpr int WST = RMAX * 32 + 16;      // LDS bytes per output channel of the filter: 68
                                         // dwords, so that the 16 lanes of a 16-byte read
                                         // (16 channels) take 16 different groups of 4 banks
constexpr int CTS = 40;                  // fp32 stride of an output row in the LDS tile: the
                                         // two lane halves of a write (rows 4 apart) are 160
                                         // dwords = 32 banks apart
constexpr int PATCH_BYTES = PROWS * NCOPY * CSTR;
constexpr int CT_BYTES = 32 * MB * CTS * 4;
constexpr int TILE_BYTES = PATCH_BYTES > CT_BYTES ? PATCH_BYTES : CT_BYTES;
constexpr int kFetch = PROWS * ROWB / 512;   // patch bytes fetched per thread (10 at 512 threads)

struct StemParams {
    const uint8_t* x;          // input codes [N, H, W, C]
    const uint8_t* w;          // filter codes [64, R, S, C]
    float* y;                  // pooled fp32 [N, PP, QQ, 64], or NULL
    const float* alphaX;
    const float* alphaW;
    DecodeInfo dx, dw;
    Post post;                 // a, b, codes / alpha / pp, absmax (ReLU always)
    int N, H, W, R, S, ph, pw, P, Q, PP, QQ;
    int tiles_p, tiles_q, ntiles;
    int kX, kW;
    uint32_t zero_code;        // the +0 code of the input format (outside the image)
};

__device__ __forceinline__ int decode_byte(uint32_t c, const DecodeInfo& d) {
    c &= (1u << d.n) - 1u;
    const uint32_t sg = (c >> (d.n - 1)) & 1u;
    const uint32_t e = (c >> d.k) & (uint32_t)d.emax;
    const uint32_t f = c & ((1u << d.k) - 1u);
    const int m = (e == (uint32_t)d.emax) ? (int)f : (int)(((1u << d.k) | f) << e);
    return sg ? -m : m;
}

// Four waves per SIMD: two workgroups share a CU (LDS and registers fit).
template <int C>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4, 4)))
void k_stem(StemParams p) {
    // patch: [PROWS][NCOPY][CSTR] int8; after the MFMAs the same bytes hold the
    // rectified outputs of one channel half, [32 MB][CTS] fp32
    __shared__ __align__(16) uint8_t patch[TILE_BYTES];
    __shared__ __align__(16) uint32_t stage[PROWS * STAGE_DW];
    __shared__ __align__(16) uint8_t wlds[KO * WST];          // the decoded filter
    __shared__ int8_t xlut[256];                             // code -> m of the input format
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = wave & 1;                 // output channels 32 half .. 32 half + 31
    const int mb0 = wave >> 1;                 // M blocks mb0, mb0 + WGR, ...
    const int R = p.R, SC = p.S * C;

    // decode tables and the filter, once: the filter as 64 x RMAX rows of 32 bytes
    // (zero past S*C and for rows past R); lane l later reads the B fragment of
    // channel 32 half + l % 32, bytes 16 (l / 32) .. + 15 of the row of filter row r
    if (tid < 256) xlut[tid] = (int8_t)decode_byte((uint32_t)tid, p.dx);
    for (int it = tid; it < KO * RMAX * 32; it += kThreads) {
        const int n = it / (RMAX * 32), r = (it / 32) % RMAX, j = it % 32;
        int m = 0;
        if (r < R && j < SC) m = decode_byte(p.w[((int64_t)n * R + r) * SC + j], p.dw);
        wlds[n * WST + r * 32 + j] = (uint8_t)m;
    }
    const int boff = (32 * half + (lane & 31)) * WST + 16 * (lane >> 5);
    for (int it = tid; it < PROWS * STAGE_DW; it += kThreads) stage[it] = 0u;
    const float s = ldexpf(p.alphaX[0] * p.alphaW[0], -(p.kX + p.kW));
    const float qa = post_alpha(p.post);
    const bool qok = alpha_valid(qa), qfast = fast_scale(qa);
    const float qr = 1.0f / qa;
    // 16-byte stores of y, 4-byte stores of the codes where the pointers allow
    const bool vec_out = (uintptr_t)p.y % 16 == 0 && (uintptr_t)p.post.codes % 4 == 0;
    uint32_t amax = 0;
    const int lr = lane & 31, lg = lane >> 5;

    // per lane and M block: the patch offset of its row's first 16-byte piece
    int aoff[MBW];
#pragma unroll
    for (int i = 0; i < MBW; i++) {
        const int mb = mb0 + WGR * i;
        const int pix = 32 * mb + lr;
        int off = 0;
        if (mb < MB && pix < NPIX) {
            const int tr = pix / CC, tc = pix - tr * CC;
            const int o = 2 * tc * C + 16 * lg;
            off = (2 * tr * NCOPY + ((o & 15) >> 1)) * CSTR + (o & ~15);
        }
        aoff[i] = off;
    }

    // The patch of a tile: byte bb of row pr is input row ih0 + pr, column
    // iw0 + bb / C, channel bb % C; bytes outside the image are the +0 code.
    // Thread t fetches byte bb = t % 128 of rows t / 128 + 4 u (512 threads); the
    // bytes of the next tile are in flight while the current tile's MFMAs run.
    static_assert(kThreads == 4 * ROWB && PROWS % 4 == 0, "fetch layout");
    const int tiles_img = p.tiles_p * p.tiles_q;
    const int fbb = tid & (ROWB - 1), fpr = tid >> 7;
    const int fcol = fbb / C, fch = fbb - fcol * C;
    const int rowstride = 4 * p.W * C;          // bytes between rows fpr + 4 u and + 4 (u + 1)
    const int imgbytes = p.H * p.W * C;         // < 2^31 (checked by the launcher)
    uint32_t raw[kFetch];
    auto fetch = [&](int tile) {
        const int img = tile / tiles_img, rem = tile - img * tiles_img;
        const int tp = rem / p.tiles_q, tq = rem - tp * p.tiles_q;
        const int ih = 2 * (2 * tp * TP - 1) - p.ph + fpr;
        const int iw = 2 * (2 * tq * TQ - 1) - p.pw + fcol;
        const bool colin = (unsigned)iw < (unsigned)p.W;
        const uint8_t* xi = p.x + (int64_t)img * imgbytes;
        int off = (ih * p.W + (colin ? iw : 0)) * C + fch;
#pragma unroll
        for (int u = 0; u < kFetch; u++) {
            const bool in = colin && (unsigned)(ih + 4 * u) < (unsigned)p.H;
            const uint32_t c = xi[in ? off : 0];
            raw[u] = in ? c : p.zero_code;
            off += rowstride;
        }
    };
    if (blockIdx.x < p.ntiles) fetch(blockIdx.x);
    __syncthreads();   // the decode table, filter and zeroed stage are in place

    for (int tile = blockIdx.x; tile < p.ntiles; tile += gridDim.x) {
        const int img = tile / tiles_img, rem = tile - img * tiles_img;
        const int tp = rem / p.tiles_q, tq = rem - tp * p.tiles_q;
        const int pp0 = tp * TP, qq0 = tq * TQ;
        const int cr0 = 2 * pp0 - 1, cc0 = 2 * qq0 - 1;     // conv position of tile row 0

        // ---- decode into the stage, then the eight shifted copies
        uint8_t* stage8 = (uint8_t*)stage;
#pragma unroll
        for (int u = 0; u < kFetch; u++)
            stage8[(fpr + 4 * u) * (STAGE_DW * 4) + fbb] = (uint8_t)xlut[raw[u] & 0xffu];
        __syncthreads();
        // copy v, dword d: patch bytes 4 d + 2 v .. + 3 = stage dword d + v / 2,
        // shifted by 2 bytes for odd v; one thread per (row, dword), all copies
        for (int it = tid; it < PROWS * (ROWB / 4); it += kThreads) {
            const int d = it % (ROWB / 4), pr = it / (ROWB / 4);
            uint32_t sw[5];
#pragma unroll
            for (int u = 0; u < 5; u++) sw[u] = stage[pr * STAGE_DW + d + u];
#pragma unroll
            for (int v = 0; v < NCOPY; v++) {
                const uint32_t val = (v & 1) ? __builtin_amdgcn_alignbyte(sw[(v >> 1) + 1], sw[v >> 1], 2u)
                                             : sw[v >> 1];
                *(uint32_t*)&patch[(pr * NCOPY + v) * CSTR + 4 * d] = val;
            }
        }
        __syncthreads();
        if (tile + (int)gridDim.x < p.ntiles) fetch(tile + gridDim.x);   // in flight below

        // ---- the contraction: one 32x32x32 int8 MFMA per filter row and block;
        //      the A fragments of filter row r + 1 are read while those of r run
        v16i acc[MBW];
#pragma unroll
        for (int i = 0; i < MBW; i++)
#pragma unroll
            for (int r = 0; r < 16; r++) acc[i][r] = 0;
        v4i fa[2][MBW];
#pragma unroll
        for (int i = 0; i < MBW; i++) fa[0][i] = *(const v4i*)&patch[aoff[i]];
        // all RMAX filter rows: the rows past R are zero in the filter copy, and
        // the patch rows they read (2 * 16 + 7 at most) are inside the patch
#pragma unroll
        for (int r = 0; r < RMAX; r++) {
            if (r + 1 < RMAX) {
#pragma unroll
                for (int i = 0; i < MBW; i++)
                    fa[(r + 1) & 1][i] = *(const v4i*)&patch[aoff[i] + (r + 1) * NCOPY * CSTR];
            }
            const v4i bf = *(const v4i*)&wlds[boff + 32 * r];
#pragma unroll
            for (int i = 0; i < MBW; i++)
                if (mb0 + WGR * i < MB)
                    acc[i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[r & 1][i], bf, acc[i], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
        __syncthreads();   // every read of the patch is done

        // ---- per channel half: the post-processed, rectified outputs into LDS,
        //      then the pool (tiles at the image border leave out the conv
        //      positions outside the output: every value is >= 0 and every window
        //      holds a position inside)
        const bool interior = cr0 >= 0 && cr0 + CR <= p.P && cc0 >= 0 && cc0 + CC <= p.Q;
        float* ct = (float*)patch;                  // [32 MB][CTS]
#pragma unroll 1
        for (int hh = 0; hh < 2; hh++) {
            if (half == hh) {
                const int ch = 32 * hh + lr;
                const float pa = p.post.a ? p.post.a[ch] : 1.0f;
                const float pb = p.post.b ? p.post.b[ch] : 0.0f;
                // register r of block mb is row 32 mb + 8 (r / 4) + 4 lg + r % 4: one base
                // address per block, the rest immediate offsets
#pragma unroll
                for (int i = 0; i < MBW; i++) {
                    const int mb = mb0 + WGR * i;
                    float* base = ct + (32 * mb + 4 * lg) * CTS + lr;
                    if (mb < MB) {
#pragma unroll
                        for (int r = 0; r < 16; r++) {
                            // rows NPIX .. 32 MB - 1 are written too and never read
                            const float z = __builtin_fmaf(pa, s * (float)acc[i][r], pb);
                            base[(8 * (r >> 2) + (r & 3)) * CTS] = z > 0.0f ? z : 0.0f;
                        }
                    }
                }
            }
            __syncthreads();
            // four channels of one pooled output per thread: lanes 8 apart take pooled
            // columns 2 apart (conv outputs 4 apart, 160 dwords), so each 16-lane
            // group of a 16-byte read covers the 64 banks once
            {
                const int quad = tid & 7, j = tid >> 3;
                const int pr = j >> 3, pc = 2 * (j & 1) + ((j >> 1) & 1) + 4 * ((j >> 2) & 1);
                const float* t = ct + ((2 * pr) * CC + 2 * pc) * CTS + 4 * quad;
                // rectified values are >= 0 and never NaN: their bit patterns order
                // as unsigned integers
                uint32_t m0 = 0, m1 = 0, m2 = 0, m3 = 0;
#pragma unroll
                for (int dr = 0; dr < 3; dr++) {
                    const bool rin = interior || (unsigned)(cr0 + 2 * pr + dr) < (unsigned)p.P;
#pragma unroll
                    for (int dc = 0; dc < 3; dc++) {
                        const bool in = rin && (interior || (unsigned)(cc0 + 2 * pc + dc) < (unsigned)p.Q);
                        const f32x4 v = *(const f32x4*)(t + (dr * CC + dc) * CTS);
                        if (in) {
                            m0 = max(m0, __float_as_uint(v.x));
                            m1 = max(m1, __float_as_uint(v.y));
                            m2 = max(m2, __float_as_uint(v.z));
                            m3 = max(m3, __float_as_uint(v.w));
                        }
                    }
                }
                const int pp = pp0 + pr, qq = qq0 + pc;
                if (pp < p.PP && qq < p.QQ) {
                    const int64_t o = (((int64_t)img * p.PP + pp) * p.QQ + qq) * KO + 32 * hh + 4 * quad;
                    const f32x4 v = {__uint_as_float(m0), __uint_as_float(m1), __uint_as_float(m2),
                                     __uint_as_float(m3)};
                    const uint32_t c4 = p.post.codes == nullptr ? 0u
                                        : qok ? code4(v, qa, qr, qfast, p.post.pp)
                                              : p.post.pp.zero_code * 0x01010101u;
                    if (vec_out) {
                        if (p.y) *(f32x4*)(p.y + o) = v;
                        if (p.post.codes) *(uint32_t*)(p.post.codes + o) = c4;
                    } else {
#pragma unroll
                        for (int c = 0; c < 4; c++) {
                            if (p.y) p.y[o + c] = v[c];
                            if (p.post.codes) p.post.codes[o + c] = (uint8_t)(c4 >> (8 * c));
                        }
                    }
                    amax = max(amax, max(max(m0, m1), max(m2, m3)));
                }
            }
            __syncthreads();
        }
    }
    post_absmax_flush(p.post, amax);
}

}  // namespace

bool stem_fits(const ConvGeom& g, int K, int groups, const Fmt& fx, const Fmt& fw, int pool_r,
               int pool_stride, int pool_pad) {
    return groups == 1 && K == KO && g.sh == 2 && g.sw == 2 && g.C >= 1 && g.C <= 3 &&
           g.S * g.C <= 32 && g.R >= 1 && g.R <= RMAX && g.S >= 1 && pool_r == 3 &&
           pool_stride == 2 && pool_pad == 1 && fx.max_int <= 127 && fw.max_int <= 127 &&
           g.P >= 1 && g.Q >= 1 && (int64_t)g.H * g.W * g.C < ((int64_t)1 << 31) &&
           (int64_t)g.R * g.S * g.C * fx.max_int * fw.max_int <= 0x7fffffff;
}

hipError_t launch_stem(const ConvGeom& g, const uint8_t* x, const Fmt& fx, const float* alphaX,
                       const uint8_t* w, const Fmt& fw, const float* alphaW, float* y, int PP,
                       int QQ, const Post& post, hipStream_t s) {
    StemParams p;
    p.N = g.Nb; p.H = g.H; p.W = g.W; p.R = g.R; p.S = g.S; p.ph = g.ph; p.pw = g.pw;
    p.P = g.P; p.Q = g.Q;
    p.PP = PP;
    p.QQ = QQ;
    p.tiles_p = (PP + TP - 1) / TP;
    p.tiles_q = (QQ + TQ - 1) / TQ;
    const int64_t nt = (int64_t)g.Nb * p.tiles_p * p.tiles_q;
    if (nt == 0) return hipSuccess;
    if (nt > 0x7fffffff) return hipErrorInvalidValue;
    p.ntiles = (int)nt;
    p.x = x;
    p.w = w;
    p.dx = decode_info(fx);
    p.dw = decode_info(fw);
    p.zero_code = fx.zero_code;
    p.alphaX = alphaX;
    p.alphaW = alphaW;
    p.kX = fx.k;
    p.kW = fw.k;
    p.y = y;
    p.post = post;
    int64_t blocks = (int64_t)num_cus() * 2;   // two workgroups fit a CU (LDS, registers)
    if (blocks > nt) blocks = nt;
    if (g.C == 1) k_stem<1><<<(unsigned)blocks, kThreads, 0, s>>>(p);
    else if (g.C == 2) k_stem<2><<<(unsigned)blocks, kThreads, 0, s>>>(p);
    else k_stem<3><<<(unsigned)blocks, kThreads, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace esb
