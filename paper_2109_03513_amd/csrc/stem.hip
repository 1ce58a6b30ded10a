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
//     pixels for a 7 x 7 filter) is loaded once, decoded to exact int8
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
constexpr int NCOPY = 8;                 // copies shifted by 2 v bytes, v = 0..7
constexpr int STAGE_DW = ROWB / 4 + 2;   // decoded row as fetched (dword aligned), + 2 spare

struct StemParams {
    ConvGeom g;                // input N, H, W, C; filter R, S; stride 2; pads; P x Q outputs
    int PP, QQ;                // pooled outputs
    int tiles_p, tiles_q, ntiles;
    const uint8_t* x;
    const uint8_t* w;
    DecodeInfo dx, dw;
    const float* alphaX;
    const float* alphaW;
    int kX, kW;
    float* y;                  // pooled fp32 [N, PP, QQ, 64], or NULL
    Post post;                 // a, b, relu (on), codes / alpha / pp, absmax
};

__device__ __forceinline__ uint32_t decode4x(uint32_t w, const DecodeInfo& d) {
    if (d.mode == 0) {
        uint32_t r = 0;
#pragma unroll
        for (int b = 0; b < 4; b++) {
            uint32_t c = (w >> (8 * b)) & ((1u << d.n) - 1u);
            const uint32_t s = (c >> (d.n - 1)) & 1u;
            const uint32_t e = (c >> d.k) & (uint32_t)d.emax;
            const uint32_t f = c & ((1u << d.k) - 1u);
            const int m = (e == (uint32_t)d.emax) ? (int)f : (int)(((1u << d.k) | f) << e);
            r |= ((uint32_t)(s ? -m : m) & 0xffu) << (8 * b);
        }
        return r;
    }
    const uint32_t sel = w & 0x07070707u;
    const uint32_t r0 = __builtin_amdgcn_perm(d.lut[1], d.lut[0], sel);
    if (d.mode == 3) return r0;
    const uint32_t r1 = __builtin_amdgcn_perm(d.lut[3], d.lut[2], sel);
    const uint32_t m3 = ((w >> 3) & 0x01010101u) * 0xffu;
    const uint32_t r01 = (r1 & m3) | (r0 & ~m3);
    if (d.mode == 4) return r01;
    const uint32_t r2 = __builtin_amdgcn_perm(d.lut[5], d.lut[4], sel);
    const uint32_t r3 = __builtin_amdgcn_perm(d.lut[7], d.lut[6], sel);
    const uint32_t r23 = (r3 & m3) | (r2 & ~m3);
    const uint32_t m4 = ((w >> 4) & 0x01010101u) * 0xffu;
    return (r23 & m4) | (r01 & ~m4);
}

__global__ __launch_bounds__(kThreads) void k_stem(StemParams p) {
    // patch: [PROWS][NCOPY][ROWB] int8; after the MFMAs the same bytes hold the
    // rectified outputs of one channel half, [NPIX][32] fp32
    __shared__ __align__(16) uint8_t patch[PROWS * NCOPY * ROWB];
    __shared__ __align__(16) uint32_t stage[PROWS * STAGE_DW];
    __shared__ __align__(16) uint8_t wlds[KO * RMAX * 32];   // the decoded filter
    const ConvGeom& g = p.g;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = wave & 1;                 // output channels 32 half .. 32 half + 31
    const int mb0 = wave >> 1;                 // M blocks mb0, mb0 + WGR, ...
    const int R = g.R, C = g.C, SC = g.S * g.C;
    const int prow_n = 2 * (CR - 1) + R;       // patch rows used
    const int pbytes = (2 * (CC - 1) + g.S) * C;   // bytes of a patch row used

    // the filter, decoded once into LDS as 64 x R rows of 32 bytes (zero past
    // S*C); lane l reads the B fragment of channel 32 half + l % 32, bytes
    // 16 (l / 32) .. + 15 of the row of filter row r
    for (int it = tid; it < KO * R * 8; it += kThreads) {
        const int n = it / (R * 8), r = (it / 8) % R, t4 = it % 8;
        uint32_t v = 0u;
#pragma unroll
        for (int b = 0; b < 4; b++) {
            const int j = 4 * t4 + b;
            if (j < SC) {
                const uint32_t code = p.w[((int64_t)n * R + r) * SC + j];
                v |= (decode4x(code, p.dw) & 0xffu) << (8 * b);
            }
        }
        *(uint32_t*)&wlds[(n * R + r) * 32 + 4 * t4] = v;
    }
    const int boff = ((32 * half + (lane & 31)) * R) * 32 + 16 * (lane >> 5);
    const float s = ldexpf(p.alphaX[0] * p.alphaW[0], -(p.kX + p.kW));
    const float qa = post_alpha(p.post);
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
            off = (2 * tr * NCOPY + ((o & 15) >> 1)) * ROWB + (o & ~15);
        }
        aoff[i] = off;
    }

    for (int tile = blockIdx.x; tile < p.ntiles; tile += gridDim.x) {
        const int img = tile / (p.tiles_p * p.tiles_q);
        const int rem = tile - img * p.tiles_p * p.tiles_q;
        const int pp0 = (rem / p.tiles_q) * TP, qq0 = (rem % p.tiles_q) * TQ;
        const int cr0 = 2 * pp0 - 1, cc0 = 2 * qq0 - 1;     // conv position of tile row 0
        const int ih0 = 2 * cr0 - g.ph, iw0 = 2 * cc0 - g.pw;  // input position of patch (0, 0)

        // ---- the patch: fetch whole dwords of each row, decode, zero what lies
        //      outside the image; then the eight shifted copies.  Row pr of the
        //      patch starts `lead` bytes into the dword it is fetched with.
        const int64_t gb0 = ((int64_t)iw0) * C;                  // byte of column iw0 in a row
        auto row_base = [&](int pr) {                            // byte of the input row
            return ((int64_t)img * g.H + (ih0 + pr)) * g.W * C;
        };
        auto row_lead = [&](int pr) {
            return (int)((((row_base(pr) + gb0) % 4) + 4) % 4);
        };
        const int ndw = (3 + pbytes + 3) / 4;                    // dwords fetched per row
        for (int it = tid; it < prow_n * ndw; it += kThreads) {
            const int pr = it / ndw, q = it - pr * ndw;
            const int ih = ih0 + pr;
            uint32_t v = 0u;
            if ((unsigned)ih < (unsigned)g.H) {
                const int64_t rowb = row_base(pr);
                const int64_t rowe = rowb + (int64_t)g.W * C;
                const int64_t a = rowb + gb0 - row_lead(pr) + 4 * q;   // first byte of the dword
                uint32_t raw = 0u, keep = 0u;
                if (a >= rowb && a + 4 <= rowe) {
                    raw = *(const uint32_t*)(p.x + a);
                    keep = 0xffffffffu;
                } else {
#pragma unroll
                    for (int b = 0; b < 4; b++)
                        if (a + b >= rowb && a + b < rowe) {
                            raw |= (uint32_t)p.x[a + b] << (8 * b);
                            keep |= 0xffu << (8 * b);
                        }
                }
                v = decode4x(raw, p.dx) & keep;
            }
            stage[pr * STAGE_DW + q] = v;
        }
        for (int it = tid; it < prow_n * STAGE_DW; it += kThreads) {   // dwords past ndw: zero
            const int pr = it / STAGE_DW, q = it - pr * STAGE_DW;
            if (q >= ndw) stage[it] = 0u;
        }
        __syncthreads();
        // copy v, dword d: patch bytes 4 d + 2 v .. + 3, i.e. stage bytes from lead + 4 d + 2 v
        for (int it = tid; it < prow_n * NCOPY * (ROWB / 4); it += kThreads) {
            const int d = it % (ROWB / 4);
            const int rv = it / (ROWB / 4);
            const int v = rv % NCOPY, pr = rv / NCOPY;
            const int sb = row_lead(pr) + 4 * d + 2 * v;          // stage byte
            const int sq = sb >> 2, sh = sb & 3;
            const uint32_t lo = sq < STAGE_DW ? stage[pr * STAGE_DW + sq] : 0u;
            const uint32_t hi = sq + 1 < STAGE_DW ? stage[pr * STAGE_DW + sq + 1] : 0u;
            const uint32_t val = sh ? __builtin_amdgcn_alignbyte(hi, lo, (uint32_t)sh) : lo;
            *(uint32_t*)&patch[(pr * NCOPY + v) * ROWB + 4 * d] = val;
        }
        __syncthreads();

        // ---- the contraction: one 32x32x32 int8 MFMA per filter row and block
        v16i acc[MBW];
#pragma unroll
        for (int i = 0; i < MBW; i++)
#pragma unroll
            for (int r = 0; r < 16; r++) acc[i][r] = 0;
        // A fragments of filter row r + 1 are read while the MFMAs of row r run
        v4i fa[2][MBW];
#pragma unroll
        for (int i = 0; i < MBW; i++) fa[0][i] = *(const v4i*)&patch[aoff[i]];
#pragma unroll
        for (int r = 0; r < RMAX; r++) {
            if (r < R) {
                if (r + 1 < R) {
#pragma unroll
                    for (int i = 0; i < MBW; i++)
                        fa[(r + 1) & 1][i] = *(const v4i*)&patch[aoff[i] + (r + 1) * NCOPY * ROWB];
                }
                const v4i bf = *(const v4i*)&wlds[boff + 32 * r];
#pragma unroll
                for (int i = 0; i < MBW; i++)
                    if (mb0 + WGR * i < MB)
                        acc[i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[r & 1][i], bf, acc[i], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        __syncthreads();   // every read of the patch is done

        // ---- per channel half: the scaled sums into LDS, then the post-processing,
        //      the ReLU and the pool (conv positions outside the output left out)
        float* ct = (float*)patch;                  // [NPIX][32]
#pragma unroll 1
        for (int hh = 0; hh < 2; hh++) {
            if (half == hh) {
                // register r of block mb is row 32 mb + 8 (r / 4) + 4 lg + r % 4: one base
                // address per block, the rest immediate offsets
#pragma unroll
                for (int i = 0; i < MBW; i++) {
                    const int mb = mb0 + WGR * i;
                    float* base = ct + (32 * mb + 4 * lg) * 32 + lr;
                    if (32 * mb + 31 < NPIX) {
#pragma unroll
                        for (int r = 0; r < 16; r++)
                            base[(8 * (r >> 2) + (r & 3)) * 32] = s * (float)acc[i][r];
                    } else if (mb < MB) {
#pragma unroll
                        for (int r = 0; r < 16; r++)
                            if (32 * mb + 8 * (r >> 2) + 4 * lg + (r & 3) < NPIX)
                                base[(8 * (r >> 2) + (r & 3)) * 32] = s * (float)acc[i][r];
                    }
                }
            }
            __syncthreads();
            const int c = tid & 31, ch = 32 * hh + c;
            const float pa = p.post.a ? p.post.a[ch] : 1.0f;
            const float pb = p.post.b ? p.post.b[ch] : 0.0f;
#pragma unroll 2
            for (int k = 0; k < (TP * TQ * 32) / kThreads; k++) {
                const int pi = (tid >> 5) + k * (kThreads / 32);
                const int pr = pi / TQ, pc = pi - pr * TQ;
                const int pp = pp0 + pr, qq = qq0 + pc;
                float m = 0.0f;
#pragma unroll
                for (int dr = 0; dr < 3; dr++) {
                    const bool rin = (unsigned)(cr0 + 2 * pr + dr) < (unsigned)g.P;
#pragma unroll
                    for (int dc = 0; dc < 3; dc++) {
                        const bool in = rin && (unsigned)(cc0 + 2 * pc + dc) < (unsigned)g.Q;
                        float z = __builtin_fmaf(pa, ct[((2 * pr + dr) * CC + 2 * pc + dc) * 32 + c], pb);
                        z = z > 0.0f ? z : 0.0f;
                        m = in ? fmaxf(m, z) : m;
                    }
                }
                if (pp < p.PP && qq < p.QQ) {
                    const int64_t o = (((int64_t)img * p.PP + pp) * p.QQ + qq) * KO + ch;
                    if (p.y) p.y[o] = m;
                    if (p.post.codes)
                        p.post.codes[o] = (uint8_t)(alpha_valid(qa) ? esb_code(m, qa, p.post.pp)
                                                                    : p.post.pp.zero_code);
                    amax = max(amax, __float_as_uint(m) & 0x7fffffffu);
                }
            }
            __syncthreads();
        }
    }
    post_absmax_flush(p.post, amax);
}

}  // namespace

bool stem_fits(const ConvGeom& g, int K, int groups, const Fmt& fx, const Fmt& fw, int pool_r,
               int pool_stride, int pool_pad, const uint8_t* x) {
    return groups == 1 && K == KO && g.sh == 2 && g.sw == 2 && g.C >= 1 && g.C <= 3 &&
           (uintptr_t)x % 4 == 0 &&
           g.S * g.C <= 32 && g.R >= 1 && g.R <= RMAX && g.S >= 1 && pool_r == 3 &&
           pool_stride == 2 && pool_pad == 1 && fx.max_int <= 127 && fw.max_int <= 127 &&
           g.P >= 1 && g.Q >= 1 && (int64_t)g.R * g.S * g.C * fx.max_int * fw.max_int <= 0x7fffffff;
}

hipError_t launch_stem(const ConvGeom& g, const uint8_t* x, const Fmt& fx, const float* alphaX,
                       const uint8_t* w, const Fmt& fw, const float* alphaW, float* y, int PP,
                       int QQ, const Post& post, hipStream_t s) {
    StemParams p;
    p.g = g;
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
    p.alphaX = alphaX;
    p.alphaW = alphaW;
    p.kX = fx.k;
    p.kW = fw.k;
    p.y = y;
    p.post = post;
    int64_t blocks = (int64_t)num_cus() * 2;   // two workgroups fit a CU (LDS, registers)
    if (blocks > nt) blocks = nt;
    k_stem<<<(unsigned)blocks, kThreads, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace esb
