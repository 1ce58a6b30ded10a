// Contraction over ESB codes (Sec. 4.2; multiplication eq. (15)) on int8 MFMA, gfx950.
//
// Codes are decoded to their exact integers m = q * 2^k while a tile moves from
// HBM to LDS: eq. (15) says a product of two ESB values is a (k+1)-bit by
// (k+1)-bit fraction product shifted by the exponents, so m_A * m_B is exactly
// 2^(kA+kB) * q_A * q_B and an integer dot product over m is exact.  When
// every |m| <= 127 the decoded tile feeds v_mfma_i32_16x16x64_i8 directly;
// otherwise each m is split as 256*hi + lo with int8 hi, lo, and the partial
// products are combined with weights 1, 256, 65536 (int32, wrap-around exact
// because the final sum fits int32).
//
// Tiles: BM x BN per workgroup (256 threads, 4 waves of WM x WN), BK = 64 bytes
// of reduction per step, LDS double buffer.  LDS rows are 64 bytes; the four
// 16-byte chunks of a row are XOR-swizzled by (row >> 1) & 3 so that the
// ds_read_b128 of 8 consecutive rows at one chunk covers all 32 banks.
// A is addressed as an implicit im2col of an NHWC tensor (a dense row-major
// matrix is the special case H = W = R = S = 1 with pixel pitch lda).
#include "esb_internal.h"

namespace esb {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int BK = 64;
constexpr int NT = 256;

struct GemmParams {
    int M, N, K;            // per-group GEMM sizes (K = R*S*Cg)
    ConvGeom ga;
    const uint8_t* A;
    const uint8_t* B;
    int64_t ldb;
    DecodeInfo da, db;
    const float* alphaA;
    const float* alphaB;
    int32_t* acc;
    float* y;
    int64_t ldc;
    uint32_t zeroA, zeroB;  // the +0 code of each operand (padding / out of range)
    Post post;              // fused post-processing of the outputs (post.on == 0: none)
};

// ------------------------------------------------------------------ decode
__device__ __forceinline__ int decode_one(uint32_t c, const DecodeInfo& d) {
    c &= (1u << d.n) - 1u;
    const uint32_t s = (c >> (d.n - 1)) & 1u;
    const uint32_t e = (c >> d.k) & (uint32_t)d.emax;
    const uint32_t f = c & ((1u << d.k) - 1u);
    const int m = (e == (uint32_t)d.emax) ? (int)f : (int)(((1u << d.k) | f) << e);
    return s ? -m : m;
}

// Four codes (one per byte) to four int8 integers.
__device__ __forceinline__ uint32_t decode4(uint32_t w, const DecodeInfo& d) {
    if (d.mode == 0) {
        uint32_t r = 0;
#pragma unroll
        for (int b = 0; b < 4; b++) r |= ((uint32_t)decode_one((w >> (8 * b)) & 0xffu, d) & 0xffu) << (8 * b);
        return r;
    }
    // v_perm_b32 as an 8-entry byte table: selector bytes 0-3 pick bytes of the
    // second source, 4-7 bytes of the first.
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

// Four codes to the high and low int8 planes of m = 256 * hi + lo.
__device__ __forceinline__ void decode4_split(uint32_t w, const DecodeInfo& d, uint32_t& hi,
                                              uint32_t& lo) {
    hi = 0;
    lo = 0;
#pragma unroll
    for (int b = 0; b < 4; b++) {
        const int m = decode_one((w >> (8 * b)) & 0xffu, d);
        const int l = (int)(int8_t)(m & 0xff);
        const int h = (m - l) >> 8;
        lo |= ((uint32_t)l & 0xffu) << (8 * b);
        hi |= ((uint32_t)h & 0xffu) << (8 * b);
    }
}

__device__ __forceinline__ int swz(int row, int chunk) {
    return row * BK + ((chunk ^ ((row >> 1) & 3)) << 4);
}

template <int P>
__device__ __forceinline__ void store_tile(int8_t* base, int plane_stride, int row, int chunk,
                                           uint4 codes, const DecodeInfo& d) {
    const int off = swz(row, chunk);
    if (P == 1) {
        uint4 v;
        v.x = decode4(codes.x, d); v.y = decode4(codes.y, d);
        v.z = decode4(codes.z, d); v.w = decode4(codes.w, d);
        *(uint4*)(base + off) = v;
    } else {
        uint4 h, l;
        decode4_split(codes.x, d, h.x, l.x); decode4_split(codes.y, d, h.y, l.y);
        decode4_split(codes.z, d, h.z, l.z); decode4_split(codes.w, d, h.w, l.w);
        *(uint4*)(base + off) = l;                 // plane 0: low
        *(uint4*)(base + plane_stride + off) = h;  // plane 1: high
    }
}

// ----------------------------------------------------------------- loaders
// A slot: one 16-byte chunk (row, chunk) of the BM x 64 tile, fixed per thread.
struct ASlot {
    int valid;     // row inside M
    int nimg, ih0, iw0;
    int r, s, cc;  // (r, s, c) of the chunk's first reduction index (VEC16 path)
};

__device__ __forceinline__ void a_slot_init(ASlot& sl, const GemmParams& g, int m, int chunk) {
    const ConvGeom& c = g.ga;
    sl.valid = m < g.M;
    const int mm = sl.valid ? m : 0;
    const int pq = c.P * c.Q;
    sl.nimg = mm / pq;
    const int rem = mm - sl.nimg * pq;
    const int p = rem / c.Q, q = rem - (rem / c.Q) * c.Q;
    sl.ih0 = p * c.sh - c.ph;
    sl.iw0 = q * c.sw - c.pw;
    const int kk = 16 * chunk;
    const int cg = max(c.Cg, 1);
    const int rs = kk / cg;
    sl.cc = kk - rs * cg;
    sl.r = rs / c.S;
    sl.s = rs - sl.r * c.S;
}

// Requires Cg >= 16 (the 16-byte path is only chosen for K > 0 with Cg % 16 == 0).
__device__ __forceinline__ void a_slot_advance(ASlot& sl, const ConvGeom& c) {
    if (c.Cg <= 0) return;
    sl.cc += BK;
    while (sl.cc >= c.Cg) {
        sl.cc -= c.Cg;
        if (++sl.s == c.S) { sl.s = 0; ++sl.r; }
    }
}

// VEC16: C/groups % 16 == 0, pitch % 16 == 0, 16-byte aligned base.
__device__ __forceinline__ uint4 a_load16(const ASlot& sl, const GemmParams& g, int k_start,
                                          int goff) {
    const ConvGeom& c = g.ga;
    const uint32_t z4 = g.zeroA * 0x01010101u;
    uint4 v = make_uint4(z4, z4, z4, z4);
    if (sl.valid && k_start < g.K) {
        const int ih = sl.ih0 + sl.r, iw = sl.iw0 + sl.s;
        if (ih >= 0 && ih < c.H && iw >= 0 && iw < c.W) {
            const uint8_t* p = g.A + (((int64_t)sl.nimg * c.H + ih) * c.W + iw) * c.pitch + goff + sl.cc;
            v = *(const uint4*)p;
        }
    }
    return v;
}

// Byte path for any geometry.  With a table (kt != nullptr) the reduction index
// kk maps to {address offset from the pixel at (ih0, iw0), r << 16 | s}, built
// once per workgroup; without it (long reductions) the division chain is used.
constexpr int kKtabMax = 2048;

__device__ __forceinline__ uint4 a_load1(const ASlot& sl, const GemmParams& g, int k_start,
                                         int goff, const int2* kt) {
    const ConvGeom& c = g.ga;
    uint32_t w[4];
    const int64_t pix = (((int64_t)sl.nimg * c.H + sl.ih0) * c.W + sl.iw0) * c.pitch + goff;
#pragma unroll
    for (int q4 = 0; q4 < 4; q4++) {
        uint32_t acc = 0;
#pragma unroll
        for (int b = 0; b < 4; b++) {
            const int kk = k_start + 4 * q4 + b;
            uint32_t code = g.zeroA;
            if (sl.valid && kk < g.K) {
                int r, s;
                int64_t off;
                if (kt) {
                    const int2 e = kt[kk];
                    off = e.x;
                    r = e.y >> 16;
                    s = e.y & 0xffff;
                } else {
                    const int rs = kk / c.Cg;
                    const int ch = kk - rs * c.Cg;
                    r = rs / c.S;
                    s = rs - r * c.S;
                    off = ((int64_t)r * c.W + s) * c.pitch + ch;
                }
                const int ih = sl.ih0 + r, iw = sl.iw0 + s;
                if ((unsigned)ih < (unsigned)c.H && (unsigned)iw < (unsigned)c.W) code = g.A[pix + off];
            }
            acc |= code << (8 * b);
        }
        w[q4] = acc;
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// B: output-channel row n (within the group), chunk of 16 reduction indices.
template <int BV>   // 16: NK vector, 1: NK bytes, 2: KN (strided bytes)
__device__ __forceinline__ uint4 b_load(const GemmParams& g, int n, int k_start, int64_t brow0) {
    const uint32_t z4 = g.zeroB * 0x01010101u;
    uint4 v = make_uint4(z4, z4, z4, z4);
    if (n >= g.N || k_start >= g.K) return v;
    if (BV == 16) {
        return *(const uint4*)(g.B + (brow0 + n) * g.ldb + k_start);
    }
    uint32_t w[4];
#pragma unroll
    for (int q4 = 0; q4 < 4; q4++) {
        uint32_t acc = 0;
#pragma unroll
        for (int b = 0; b < 4; b++) {
            const int kk = k_start + 4 * q4 + b;
            uint32_t code = g.zeroB;
            if (kk < g.K)
                code = (BV == 1) ? g.B[(brow0 + n) * g.ldb + kk] : g.B[(int64_t)kk * g.ldb + brow0 + n];
            acc |= code << (8 * b);
        }
        w[q4] = acc;
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// ------------------------------------------------------------------ kernel
// POST: the fused post-processing epilogue (a separate instantiation, so that
// the plain kernel keeps its register budget).
template <int BM, int BN, int WM, int WN, int PA, int PB, int AV, int BV, bool POST>
__global__ __launch_bounds__(NT) void k_contract(GemmParams g) {
    static_assert((BM / WM) * (BN / WN) == NT / 64, "4 waves per workgroup");
    constexpr int CA = (BM * 4 + NT - 1) / NT;   // A chunks per thread per stage
    constexpr int CB = (BN * 4 + NT - 1) / NT;
    constexpr int TI = WM / 16, TJ = WN / 16;
    constexpr int NACC = PA + PB - 1;
    __shared__ __align__(16) int8_t sA[2][PA][BM * BK];
    __shared__ __align__(16) int8_t sB[2][PB][BN * BK];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int grp = blockIdx.z;
    const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
    const int wr = (wave / (BN / WN)) * WM, wc = (wave % (BN / WN)) * WN;
    const int goffA = grp * g.ga.Cg;
    const int64_t brow0 = (int64_t)grp * g.N;

    // byte path: the reduction-index table (short reductions)
    __shared__ int2 s_ktab[AV == 1 ? kKtabMax : 1];
    const int2* ktab = nullptr;
    if (AV == 1 && g.K <= kKtabMax &&
        (int64_t)g.ga.R * g.ga.W * g.ga.pitch + g.ga.pitch < 0x7fffffff) {
        for (int kk = threadIdx.x; kk < g.K; kk += NT) {
            const int cg = max(g.ga.Cg, 1);
            const int rs = kk / cg;
            const int ch = kk - rs * cg;
            const int r = rs / g.ga.S, s = rs - r * g.ga.S;
            s_ktab[kk] = make_int2((r * g.ga.W + s) * g.ga.pitch + ch, (r << 16) | s);
        }
        __syncthreads();
        ktab = s_ktab;
    }
    ASlot as[CA];
#pragma unroll
    for (int i = 0; i < CA; i++) {
        const int c = tid + i * NT;
        a_slot_init(as[i], g, m0 + c / 4, c % 4);
        if (c >= BM * 4) as[i].valid = 0;
    }

    v4i acc[NACC][TI][TJ];
#pragma unroll
    for (int a = 0; a < NACC; a++)
#pragma unroll
        for (int i = 0; i < TI; i++)
#pragma unroll
            for (int j = 0; j < TJ; j++) acc[a][i][j] = v4i{0, 0, 0, 0};

    uint4 ra[CA], rb[CB];
    auto load_stage = [&](int k0) {
#pragma unroll
        for (int i = 0; i < CA; i++) {
            const int c = tid + i * NT;
            const int kst = k0 + 16 * (c % 4);
            ra[i] = (AV == 16) ? a_load16(as[i], g, kst, goffA) : a_load1(as[i], g, kst, goffA, ktab);
        }
#pragma unroll
        for (int i = 0; i < CB; i++) {
            const int c = tid + i * NT;
            rb[i] = b_load<BV>(g, n0 + c / 4, k0 + 16 * (c % 4), brow0);
        }
    };
    auto store_stage = [&](int buf) {
#pragma unroll
        for (int i = 0; i < CA; i++) {
            const int c = tid + i * NT;
            if (c < BM * 4) store_tile<PA>(&sA[buf][0][0], BM * BK, c / 4, c % 4, ra[i], g.da);
        }
#pragma unroll
        for (int i = 0; i < CB; i++) {
            const int c = tid + i * NT;
            if (c < BN * 4) store_tile<PB>(&sB[buf][0][0], BN * BK, c / 4, c % 4, rb[i], g.db);
        }
    };
    auto advance = [&]() {
        if (AV == 16) {
#pragma unroll
            for (int i = 0; i < CA; i++) a_slot_advance(as[i], g.ga);
        }
    };

    const int KT = (g.K + BK - 1) / BK;
    load_stage(0);
    advance();
    store_stage(0);
    __syncthreads();
    for (int kt = 0; kt < KT; kt++) {
        const int buf = kt & 1;
        if (kt + 1 < KT) { load_stage((kt + 1) * BK); advance(); }
        v4i fa[PA][TI], fb[PB][TJ];
#pragma unroll
        for (int p = 0; p < PA; p++)
#pragma unroll
            for (int i = 0; i < TI; i++)
                fa[p][i] = *(const v4i*)&sA[buf][p][swz(wr + 16 * i + (lane & 15), lane >> 4)];
#pragma unroll
        for (int p = 0; p < PB; p++)
#pragma unroll
            for (int j = 0; j < TJ; j++)
                fb[p][j] = *(const v4i*)&sB[buf][p][swz(wc + 16 * j + (lane & 15), lane >> 4)];
#pragma unroll
        for (int i = 0; i < TI; i++)
#pragma unroll
            for (int j = 0; j < TJ; j++)
#pragma unroll
                for (int pa = 0; pa < PA; pa++)
#pragma unroll
                    for (int pb = 0; pb < PB; pb++)
                        acc[pa + pb][i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                            fa[pa][i], fb[pb][j], acc[pa + pb][i][j], 0, 0, 0);
        if (kt + 1 < KT) store_stage(buf ^ 1);
        __syncthreads();
    }

    // epilogue: lane holds rows 4*(lane>>4) + r, column lane & 15 of each 16x16 block
    float s = 0.0f;
    if (g.y || POST) s = ldexpf(g.alphaA[0] * g.alphaB[0], -(g.da.k + g.db.k));
    auto ival = [&](int i, int j, int r) {
        uint32_t v = (uint32_t)acc[0][i][j][r];
        if (NACC > 1) v += (uint32_t)acc[NACC > 1 ? 1 : 0][i][j][r] << 8;
        if (NACC > 2) v += (uint32_t)acc[NACC > 2 ? 2 : 0][i][j][r] << 16;
        return (int32_t)v;
    };
    if constexpr (POST) {
        // fused post-processing through LDS, one row of 16x16 blocks at a time: each
        // wave's 16 x WN slab of scaled values is read back four outputs per lane, so
        // the post-processing code stays outside the unrolled register loops
        static_assert(NT / 64 * 16 * WN * 4 <= sizeof(sA), "post slabs fit the A buffers");
        float* slab = (float*)&sA[0][0][0] + wave * 16 * WN;
        const float qa = post_alpha(g.post);
        uint32_t amax = 0;
#pragma unroll
        for (int i = 0; i < TI; i++) {
            __syncthreads();
#pragma unroll
            for (int j = 0; j < TJ; j++)
#pragma unroll
                for (int r = 0; r < 4; r++) {
                    const int rl = 4 * (lane >> 4) + r, cl = 16 * j + (lane & 15);
                    const int row = m0 + wr + 16 * i + rl, col = n0 + wc + cl;
                    const int32_t iv = ival(i, j, r);
                    if (g.acc && row < g.M && col < g.N)
                        g.acc[(int64_t)row * g.ldc + (int64_t)grp * g.N + col] = iv;
                    slab[rl * WN + cl] = s * (float)iv;
                }
            __syncthreads();
#pragma unroll 1
            for (int e = 4 * lane; e < 16 * WN; e += 256) {
                const int rl = e / WN, cl = e - rl * WN;
                const int row = m0 + wr + 16 * i + rl, col = n0 + wc + cl;
                if (row < g.M && col < g.N) {
                    const int64_t ch = (int64_t)grp * g.N + col;
                    amax = max(amax, post_store4(g.post, g.y, (int64_t)row * g.ldc + ch, ch,
                                                 *(const f32x4*)(slab + e), min(4, g.N - col), qa));
                }
            }
        }
        post_absmax_flush(g.post, amax);
        return;
    }
#pragma unroll
    for (int i = 0; i < TI; i++)
#pragma unroll
        for (int j = 0; j < TJ; j++)
#pragma unroll
            for (int r = 0; r < 4; r++) {
                const int row = m0 + wr + 16 * i + 4 * (lane >> 4) + r;
                const int col = n0 + wc + 16 * j + (lane & 15);
                if (row < g.M && col < g.N) {
                    const int32_t iv = ival(i, j, r);
                    const int64_t o = (int64_t)row * g.ldc + (int64_t)grp * g.N + col;
                    if (g.acc) g.acc[o] = iv;
                    if (g.y) g.y[o] = s * (float)iv;
                }
            }
}

// ------------------------------------------------------------------ launch
DecodeInfo decode_info(const Fmt& f) {
    DecodeInfo d;
    d.n = f.n;
    d.k = f.k;
    d.emax = f.N;
    d.split = f.max_int > 127;
    d.mode = d.split ? 0 : (f.n <= 3 ? 3 : (f.n == 4 ? 4 : (f.n == 5 ? 5 : 0)));
    for (int w = 0; w < 8; w++) {
        uint32_t v = 0;
        for (int b = 0; b < 4; b++) {
            const uint32_t c = (uint32_t)(4 * w + b) & ((1u << f.n) - 1u);
            const int m = d.split ? 0 : decode_int(f, c);
            v |= ((uint32_t)m & 0xffu) << (8 * b);
        }
        d.lut[w] = v;
    }
    return d;
}

template <int BM, int BN, int WM, int WN, int PA, int PB, int AV, int BV>
static void launch_t(const GemmParams& g, int groups, hipStream_t s) {
    dim3 grid((g.M + BM - 1) / BM, (g.N + BN - 1) / BN, groups);
    if (g.post.on) k_contract<BM, BN, WM, WN, PA, PB, AV, BV, true><<<grid, NT, 0, s>>>(g);
    else k_contract<BM, BN, WM, WN, PA, PB, AV, BV, false><<<grid, NT, 0, s>>>(g);
}

template <int BM, int BN, int WM, int WN>
static void launch_fast(const GemmParams& g, int groups, int av, int bv, hipStream_t s) {
    if (av == 16) {
        if (bv == 16) launch_t<BM, BN, WM, WN, 1, 1, 16, 16>(g, groups, s);
        else if (bv == 1) launch_t<BM, BN, WM, WN, 1, 1, 16, 1>(g, groups, s);
        else launch_t<BM, BN, WM, WN, 1, 1, 16, 2>(g, groups, s);
    } else {
        if (bv == 16) launch_t<BM, BN, WM, WN, 1, 1, 1, 16>(g, groups, s);
        else if (bv == 1) launch_t<BM, BN, WM, WN, 1, 1, 1, 1>(g, groups, s);
        else launch_t<BM, BN, WM, WN, 1, 1, 1, 2>(g, groups, s);
    }
}

template <int PA, int PB>
static void launch_split(const GemmParams& g, int groups, int bv, hipStream_t s) {
    if (bv == 2) launch_t<64, 64, 32, 32, PA, PB, 1, 2>(g, groups, s);
    else launch_t<64, 64, 32, 32, PA, PB, 1, 1>(g, groups, s);
}

hipError_t launch_contraction(int M, int N, int K, int groups, const ConvGeom& ga,
                              const uint8_t* A, const DecodeInfo& da, const float* alphaA,
                              const uint8_t* B, int64_t ldb, int b_layout, const DecodeInfo& db,
                              const float* alphaB, int32_t* acc, float* y, int64_t ldc,
                              int /*out_col_per_group*/, hipStream_t s, const Post* post) {
    if (M <= 0 || N <= 0) return hipSuccess;
    GemmParams g;
    g.M = M; g.N = N; g.K = K; g.ga = ga;
    g.A = A; g.B = B; g.ldb = ldb; g.da = da; g.db = db;
    g.alphaA = alphaA; g.alphaB = alphaB; g.acc = acc; g.y = y; g.ldc = ldc;
    g.post = post ? *post : Post{};
    g.zeroA = (uint32_t)da.emax << da.k;
    g.zeroB = (uint32_t)db.emax << db.k;
    const bool a16 = (K > 0) && (ga.Cg >= 16) && (ga.Cg % 16 == 0) && (ga.pitch % 16 == 0) &&
                     ((uintptr_t)A % 16 == 0) &&
                     ((int64_t)groups * ga.Cg <= ga.pitch);
    int bv;
    if (b_layout == 1) bv = 2;
    else bv = ((K > 0) && (K % 16 == 0) && (ldb % 16 == 0) && ((uintptr_t)B % 16 == 0)) ? 16 : 1;
    const int av = a16 ? 16 : 1;
    if (da.split || db.split) {
        if (da.split && db.split) launch_split<2, 2>(g, groups, bv, s);
        else if (da.split) launch_split<2, 1>(g, groups, bv, s);
        else launch_split<1, 2>(g, groups, bv, s);
        return hipGetLastError();
    }
    // tile choice: the largest tile that still gives every CU a workgroup
    const int64_t cus = num_cus();
    auto tiles = [&](int bm, int bn) {
        return (int64_t)((M + bm - 1) / bm) * ((N + bn - 1) / bn) * groups;
    };
    if (N > 64 && tiles(128, 128) >= cus) launch_fast<128, 128, 64, 64>(g, groups, av, bv, s);
    else if (tiles(64, 64) >= cus) launch_fast<64, 64, 32, 32>(g, groups, av, bv, s);
    else launch_fast<64, 32, 32, 16>(g, groups, av, bv, s);
    return hipGetLastError();
}

}  // namespace esb
