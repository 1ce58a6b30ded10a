// Internal declarations of libesb (gfx950).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace esb {

// Native clang vectors (HIP's float4 is a struct, not usable with the
// nontemporal builtins).
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Parameters of one ESB(b, k) format, k = fraction bits (paper notation),
// derived on the host from (n, k_sig) by make_fmt().
struct Fmt {
    int n;            // total bits b
    int k;            // fraction bits, k = k_sig - 1
    int ebits;        // exponent bits, b - k - 1
    int N;            // 2^ebits - 1: the all-ones exponent is the subnormal binade
    uint32_t zero_code;   // +0: exponent all ones, fraction 0, sign 0
    uint32_t c_code;      // largest value C = 2^(N-1) * (2 - 2^-k)
    uint32_t sign_bit;    // 1 << (b-1)
    uint32_t c_bits;      // fp32 bit pattern of C
    float C;
    int max_int;          // largest |m|, m = q * 2^k the exact integer of a code
};

// Non-negative set value number c (ascending, c = 0 .. 2^(n-1)-1) of ESB(n, k):
// binade j = c >> k, fraction f; j = 0 is the subnormal binade f * 2^-k, else
// 2^(j-1) * (1 + f 2^-k) (eq. (4)-(5)).  Exact in fp32.
__host__ __device__ inline float set_value(int c, int k) {
    const int j = c >> k, f = c & ((1 << k) - 1);
    return j == 0 ? ldexpf((float)f, -k) : ldexpf((float)((1 << k) + f), j - 1 - k);
}
// Midpoint between values c-1 and c (k+2 significant bits: exact in fp32).
__host__ __device__ inline float set_mid(int c, int k) {
    return 0.5f * (set_value(c - 1, k) + set_value(c, k));
}

bool valid_fmt(int n, int k_sig);
Fmt make_fmt(int n, int k_sig);
int decode_int(const Fmt& f, uint32_t code);   // m = q * 2^k (host)
double decode_value(const Fmt& f, uint32_t code);
int num_cus();

// ----------------------------------------------------------------- projection
// dn (device, two fp32: mean, standard deviation, or NULL): project the
// normalized values fl32(fl32(x - mean) / fl32(std + 1e-7)) instead of x.
struct ProjParams {
    uint32_t k, zero_code, c_code, c_bits, sign_bit, one;   // one = 2^k
};
ProjParams proj_params(const Fmt& f);

// Code of x under scale alpha (eq. (6)-(8)): v = fl32(x / alpha) with the IEEE
// binary32 division, then the shift-round of eq. (7) on the bit pattern of |v|:
//   |v| >= 1: keep the leading 1 and k fraction bits, adding half an ulp of the
//             kept precision before truncating (ties go to the larger magnitude);
//             the carry into the exponent field is the round-up to the next binade;
//   |v| <  1: the step is fixed at 2^-k (the subnormal binade, eq. (5));
//   |v| >= C: clip to C (eq. (8)); NaN gives +0.
// For |v| >= 1 the rounded bit pattern is the code itself: the biased fp32
// exponent minus 127 is the ESB exponent field, the kept fraction bits the
// ESB fraction field.
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

// Fast projection: the IEEE division costs ~10 VALU operations per element and
// makes a projection ALU bound, so the quotient is approximated by
// q0 = fl32(x * r), r = fl32(1 / alpha).  |q0 - x/alpha| <= 2^-23 |q0| < 2
// ulp(q0), and fl32(x/alpha) is within another half ulp, so the two round to
// the same set value unless q0 lies within 3 ulps of a cell midpoint
// (midpoints sit at least 2^-(k+2) of a binade away from binade edges, so the
// check is on the bits the rounding discards).  Below 1 the rounding to the
// fixed step 2^-k is done on w = |q0| + 1 (one more half ulp).  Groups with an
// element within 4 ulps of a midpoint take the exact esb_code; this happens
// with probability ~2^(k-20) per element.  Used only for scales with alpha and
// 1/alpha normal (alpha in [2^-125, 2^125]).
// Fast code of x given r = fl32(1/alpha); sets `risky` if q0 is within 4 ulps
// of a midpoint (the caller then recomputes with esb_code).
__device__ __forceinline__ uint32_t esb_code_fast(float x, float r, const ProjParams& p,
                                                  uint32_t& risky) {
    const float q0 = x * r;
    const uint32_t qb = __float_as_uint(q0);
    const uint32_t ab = qb & 0x7fffffffu;
    const bool small = ab < 0x3f800000u;                       // |q0| < 1
    const float w = small ? __uint_as_float(ab) + 1.0f : __uint_as_float(ab);
    const uint32_t wb = __float_as_uint(w);
    const uint32_t shA = 23u - p.k;
    const uint32_t half = 1u << (shA - 1u);
    const uint32_t c = ((wb + half) >> shA) - (127u << p.k);   // (e << k) | f, or m for small
    const uint32_t d = wb & ((half << 1) - 1u);                  // discarded bits
    risky |= (d - half + 4u) <= 8u;
    // small: m = round((w - 1) * 2^k) in [0, 2^k]; zero + m wraps m == 2^k (the value 1) to 0
    uint32_t code = small ? ((p.zero_code + c) & (p.sign_bit - 1u)) : c;
    code = (ab >= p.c_bits) ? p.c_code : code;
    code = (ab > 0x7f800000u) ? p.zero_code : code;
    code |= (code != p.zero_code) ? ((qb >> 31) << (31u - __builtin_clz(p.sign_bit))) : 0u;
    return code;
}

__device__ __forceinline__ bool fast_scale(float alpha) {
    return alpha >= 0x1p-125f && alpha <= 0x1p125f;
}

// Vector path: 4 elements per 16-byte load, 4 codes per 4-byte store.
__device__ __forceinline__ uint32_t code4(const f32x4 v, float alpha, float r, bool fast,
                                          const ProjParams& p) {
    if (fast) {
        uint32_t risky = 0;
        const uint32_t c0 = esb_code_fast(v.x, r, p, risky);
        const uint32_t c1 = esb_code_fast(v.y, r, p, risky);
        const uint32_t c2 = esb_code_fast(v.z, r, p, risky);
        const uint32_t c3 = esb_code_fast(v.w, r, p, risky);
        if (!risky) return c0 | (c1 << 8) | (c2 << 16) | (c3 << 24);
    }
    return esb_code(v.x, alpha, p) | (esb_code(v.y, alpha, p) << 8) |
           (esb_code(v.z, alpha, p) << 16) | (esb_code(v.w, alpha, p) << 24);
}


// Fused post-processing of a contraction output (Sec. 4.2: the "BN and DN"
// step of eq. (16) folded into a per-channel a x + b, then the "ESB
// quantization" step), applied to the scaled output y0 = fl32(s fl32(acc)):
//   z = fma(a_ch, y0, b_ch)   (a_ch = 1, b_ch = 0 when absent; one rounding)
//   z = fl32(z + res_o)       (when a residual is given)
//   z = z > 0 ? z : 0         (relu; NaN gives 0)
// z goes to y (when given) and its code under *alpha to codes (when given);
// res, y and codes share the output indexing.  absmax (when given): the
// largest |z| over the call, as the fp32 bit pattern (a NaN wins over every
// number), combined into *absmax with an unsigned atomic maximum (the caller
// clears it).  on == 0: the plain epilogue.
struct Post {
    const float* a;
    const float* b;
    const float* res;
    const float* alpha;
    uint8_t* codes;
    uint32_t* absmax;
    ProjParams pp;
    int relu;
    int on;
};

__device__ __forceinline__ float post_alpha(const Post& P) { return P.codes ? *P.alpha : 0.0f; }

// Returns the bit pattern of |z| (0 when absmax is not requested).
__device__ __forceinline__ uint32_t post_store(const Post& P, float* y, int64_t o, int64_t ch,
                                               float y0, float qa) {
    float z = __builtin_fmaf(P.a ? P.a[ch] : 1.0f, y0, P.b ? P.b[ch] : 0.0f);
    if (P.res) z = z + P.res[o];
    if (P.relu) z = z > 0.0f ? z : 0.0f;
    if (y) y[o] = z;
    if (P.codes) P.codes[o] = (uint8_t)(alpha_valid(qa) ? esb_code(z, qa, P.pp) : P.pp.zero_code);
    return P.absmax ? (__float_as_uint(z) & 0x7fffffffu) : 0u;
}

// The residual of outputs o .. o+3 (16-byte load where the address allows), or
// zeros without a residual: callers may load it ahead of post_apply4.
__device__ __forceinline__ f32x4 post_res4(const Post& P, int64_t o) {
    f32x4 r = {0.0f, 0.0f, 0.0f, 0.0f};
    if (P.res) {
        if (((uintptr_t)(P.res + o) & 15) == 0) {
            r = *(const f32x4*)(P.res + o);
        } else {
#pragma unroll
            for (int c = 0; c < 4; c++) r[c] = P.res[o + c];
        }
    }
    return r;
}

// Four consecutive outputs o .. o+3 (channels ch .. ch+3, all inside the
// output) through the fused post-processing, their residual r already loaded
// (post_res4); 16-byte y stores and one 4-byte code store where the addresses
// allow.
__device__ __forceinline__ uint32_t post_apply4(const Post& P, float* y, int64_t o, int64_t ch,
                                                f32x4 v, f32x4 r, float qa) {
    f32x4 z;
#pragma unroll
    for (int c = 0; c < 4; c++)
        z[c] = __builtin_fmaf(P.a ? P.a[ch + c] : 1.0f, v[c], P.b ? P.b[ch + c] : 0.0f);
    if (P.res) {
#pragma unroll
        for (int c = 0; c < 4; c++) z[c] = z[c] + r[c];
    }
    if (P.relu) {
#pragma unroll
        for (int c = 0; c < 4; c++) z[c] = z[c] > 0.0f ? z[c] : 0.0f;
    }
    if (y) {
        if (((uintptr_t)(y + o) & 15) == 0) {
            *(f32x4*)(y + o) = z;
        } else {
#pragma unroll
            for (int c = 0; c < 4; c++) y[o + c] = z[c];
        }
    }
    if (P.codes) {
        const uint32_t q4 = alpha_valid(qa)
                                ? code4(z, qa, 1.0f / qa, fast_scale(qa), P.pp)
                                : P.pp.zero_code * 0x01010101u;
        if (((uintptr_t)(P.codes + o) & 3) == 0) {
            *(uint32_t*)(P.codes + o) = q4;
        } else {
#pragma unroll
            for (int c = 0; c < 4; c++) P.codes[o + c] = (uint8_t)(q4 >> (8 * c));
        }
    }
    uint32_t m = 0;
    if (P.absmax) {
#pragma unroll
        for (int c = 0; c < 4; c++) m = max(m, __float_as_uint(z[c]) & 0x7fffffffu);
    }
    return m;
}

// Four consecutive outputs o .. o+3 (channels ch .. ch+3; nv of them inside the
// output) through the fused post-processing; 16-byte residual / y accesses and
// one 4-byte code store where the addresses allow.
__device__ __forceinline__ uint32_t post_store4(const Post& P, float* y, int64_t o, int64_t ch,
                                                f32x4 v, int nv, float qa) {
    if (nv < 4) {
        uint32_t m = 0;
        for (int c = 0; c < nv; c++) m = max(m, post_store(P, y, o + c, ch + c, v[c], qa));
        return m;
    }
    return post_apply4(P, y, o, ch, v, post_res4(P, o), qa);
}

// The running |z| maxima of a workgroup into *absmax.  Every thread of the
// workgroup calls this (it holds a barrier).  Thousands of workgroups meet on
// one address, so the waves' maxima first meet in LDS, and the one thread
// that holds the workgroup's maximum reads the current value (an atomic load)
// and issues its atomic maximum only when its own is larger: a stale read
// costs one unneeded atomic, never a wrong result.
__device__ __forceinline__ void absmax_flush_block(uint32_t* absmax, uint32_t m) {
    __shared__ uint32_t s_amax[16];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
    const int wave = threadIdx.x >> 6, nwaves = (blockDim.x + 63) >> 6;
    if ((threadIdx.x & 63) == 0) s_amax[wave] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < nwaves; w++) m = max(m, s_amax[w]);
        const uint32_t cur = __hip_atomic_load(absmax, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (m > cur) atomicMax(absmax, m);
    }
}
__device__ __forceinline__ void post_absmax_flush(const Post& P, uint32_t m) {
    if (P.absmax) absmax_flush_block(P.absmax, m);   // uniform: every thread takes the same branch
}

// The epilogue store of one output: the plain scaled value, or the fused post-processing.
__device__ __forceinline__ uint32_t out_store(const Post& P, float* y, int64_t o, int64_t ch,
                                              float y0, float qa) {
    if (P.on) return post_store(P, y, o, ch, y0, qa);
    if (y) y[o] = y0;
    return 0u;
}

hipError_t launch_project(const float* x, int64_t len, const float* alpha, const Fmt& f,
                          uint8_t* codes, const float* dn, hipStream_t s);
struct ProjJobDesc {
    const float* x;
    int64_t len;
    const float* alpha;
    Fmt f;
    uint8_t* codes;
};
hipError_t launch_project_batch(const ProjJobDesc* jobs, int count, hipStream_t s);

// ------------------------------------------------------ normalization, analytic DDA
size_t dn_workspace(int64_t len);
hipError_t launch_dn_stats(const float* x, int64_t len, float* stats, void* ws, hipStream_t s);
hipError_t launch_dda_normal(const Fmt& f, const float* grid, int G, float* alpha_out,
                             double* D_out, double* dD_out, hipStream_t s);
hipError_t launch_dequantize(const uint8_t* codes, int64_t len, const float* alpha, const Fmt& f,
                             float* out, hipStream_t s);

// ----------------------------------------------------------------------- DDA
constexpr int kDdaMaxThresholds = 8192;   // G * (2^(b-1) - 1)
constexpr int kDdaMaxG = 1024;
constexpr int kDdaBins = 4096;
constexpr int kDdaMaxBlocks = 256;

struct DdaLayout {
    int G, M, A;            // candidates, midpoints per candidate, thresholds (G*M)
    int nblk;               // blocks of the one-pass histogram kernel
    size_t off_part, off_group, total;   // block and group partial objectives; bytes
};
bool dda_layout(int64_t len, const Fmt& f, int G, DdaLayout* L);
hipError_t launch_dda(const float* x, int64_t len, const Fmt& f, const float* grid, int G,
                      float* alpha_out, double* D_out, void* ws, const DdaLayout& L,
                      hipStream_t s);
// Several independent problems; each job's workspace ws holds L.total bytes.
struct DdaJobDesc {
    const float* x;
    int64_t len;
    Fmt f;
    const float* grid;
    int G;
    float* alpha_out;
    double* D_out;
    void* ws;
    DdaLayout L;
    const float* gscale;   // NULL, or a device scalar: candidate j is fl32(*gscale * grid[j])
    const uint8_t* plan;   // NULL, or a plan (grid unused): candidate j is 2^E factor_j,
                           // E the binary exponent of |*gscale|
};
hipError_t launch_dda_batch(const DdaJobDesc* jobs, int count, hipStream_t s);
// One job, then the projection of its tensor onto the chosen scale: the finishing
// step fused into the projection where it fits one block (codes: len bytes).
hipError_t launch_dda_quantize(const DdaJobDesc& d, uint8_t* codes, hipStream_t s);
// Plans: the grid-only set-up of the DDA for candidates factors[j], built once.
size_t dda_plan_bytes(const Fmt& f, int G);
hipError_t launch_dda_plan(const Fmt& f, const float* factors, int G, void* plan, hipStream_t s);

// ---------------------------------------------------------------- contraction
// Decoding of one operand's codes to exact integers.
struct DecodeInfo {
    uint32_t lut[8];   // int8 m for codes 0..31 (perm modes), 4 per dword
    int mode;          // 3, 4, 5: v_perm table for n <= 3, n == 4, n == 5; 0: arithmetic
    int n, k, emax;
    int split;         // 1: m needs the high/low int8 split
};
DecodeInfo decode_info(const Fmt& f);

struct ConvGeom {   // implicit-GEMM view; a dense row-major A is N=M, H=W=1, R=S=1
    int Nb, H, W, C, pitch, Cg, R, S, sh, sw, ph, pw, P, Q;
};

hipError_t launch_contraction(int M, int N, int K, int groups, const ConvGeom& ga,
                              const uint8_t* A, const DecodeInfo& da, const float* alphaA,
                              const uint8_t* B, int64_t ldb, int b_layout, const DecodeInfo& db,
                              const float* alphaB, int32_t* acc, float* y, int64_t ldc,
                              int out_col_per_group, hipStream_t s, const Post* post = nullptr);

// Large-tile path on the 32x32 MFMA shapes.  op 1: codes decoded to E4M3,
// fp32 accumulation; op 0: codes of n <= 3 bits decoded to int8 by one
// v_perm_b32 lookup, int32 accumulation.
struct MmaDecode {
    uint32_t lm, inc, lmf, sel, t0, t1;   // four-byte masks / tables
    int shf, shs;                         // fraction and sign shifts
};
MmaDecode mma_decode(const Fmt& f, int op);
// 1 (E4M3), 0 (int8 table) or -1 (not eligible) for this pair of formats and
// reduction length.
int mma_choose(const Fmt& fa, const Fmt& fb, int64_t K);
// Layout conditions of the path: 16-byte chunks of codes on both operands.
bool mma_fits(const ConvGeom& ga, const uint8_t* A, int64_t K, int groups, const uint8_t* B,
              int64_t ldb, int b_layout);
// part: a workspace of at least mma_splitk(...) * M * N int32 for a dense GEMM
// whose reduction is split (NULL: no split).
hipError_t launch_mma(int op, int M, int N, int K, int groups, const ConvGeom& ga,
                      const uint8_t* A, const Fmt& fa, const float* alphaA, const uint8_t* B,
                      int64_t ldb, const Fmt& fb, const float* alphaB, int32_t* acc, float* y,
                      int64_t ldc, int32_t* part, hipStream_t s, const Post* post = nullptr);
// Ranges of the reduction split for a dense GEMM of this shape (1: none), and
// their length.
int mma_splitk(int64_t M, int64_t N, int64_t K, int* kchunk);

// The same contraction (op 1 formats) with both operands first decoded once to
// E4M3 into a workspace of mma_pre_workspace() bytes; A is a_rows rows of a_cols
// codes with pitch a_pitch (GEMM: M x K; convolution: the N*H*W pixels of C
// channels), B is b_rows rows of K codes with pitch ldb.
// mode 1: both formats lie inside OCP E2M1 (mma_f4ok) and the operands are
// decoded to packed E2M1 instead (half the bytes, fp4 MFMAs); a_cols and K are
// then multiples of 32.  mode 2: both inside OCP E2M3 (mma_f6ok), packed E2M3
// (3/4 of the bytes, fp6 MFMAs); K a multiple of 64 and, for a convolution,
// the channels per group too.  mode 0: E4M3.
size_t mma_pre_workspace(int64_t a_rows, int64_t a_cols, int64_t b_rows, int64_t K);
MmaDecode mma_decode_f4(const Fmt& f);
bool mma_f4ok(const Fmt& fa, const Fmt& fb, int64_t K);
MmaDecode mma_decode_f6(const Fmt& f);
bool mma_f6ok(const Fmt& fa, const Fmt& fb, int64_t K);
bool mma_f6_tiles(int64_t M, int64_t N, int groups);
hipError_t launch_mma_pre(int M, int N, int K, int groups, const ConvGeom& ga, const uint8_t* A,
                          int64_t a_rows, int64_t a_cols, int64_t a_pitch, const Fmt& fa,
                          const float* alphaA, const uint8_t* B, int64_t b_rows, int64_t ldb,
                          const Fmt& fb, const float* alphaB, int32_t* acc, float* y, int64_t ldc,
                          int mode, void* ws, const uint8_t* b_packed, bool split, hipStream_t s,
                          const Post* post = nullptr);
// b_packed: B given in packed E2M1 (mode 1 only), not decoded; split: a dense
// GEMM with too few tiles splits its reduction (mma_splitk), the int32 partial
// sums after the decoded operands in ws (see esb_gemm_packed_workspace_size).
hipError_t launch_pack_fp4(const uint8_t* codes, int64_t rows, int64_t K, int64_t ld, const Fmt& f,
                           uint8_t* packed, hipStream_t s);
// Skinny GEMM over packed E2M1 rows (A and B, K/2 bytes per row): one workgroup
// per 64 x 32 output tile, the reduction split over its four waves and summed
// in LDS.  fc_f4_fits: the shapes it takes (where 128 x 128 tiles would split the
// reduction over workgroups and 64 x 32 tiles give at least half the CUs one).
bool fc_f4_fits(int64_t M, int64_t N, int64_t K);
hipError_t launch_fc_f4(int M, int N, int K, const uint8_t* A_packed, int64_t lda_bytes,
                        const uint8_t* B_packed, int64_t ldb_bytes, int kA, int kB,
                        const float* alphaA, const float* alphaB, int32_t* acc, float* y,
                        int64_t ldc, hipStream_t s);

// Glue between layers: NHWC max pooling, the global average pool, max |x|.
struct PoolGeom {
    int N, H, W, C, R, S, sh, sw, ph, pw, P, Q;
};
hipError_t launch_maxpool(const float* x, const PoolGeom& g, float* out, hipStream_t s);
hipError_t launch_avgpool(const float* x, int N, int HW, int C, float* out, float* absmax,
                          hipStream_t s);
hipError_t launch_absmax(const float* x, int64_t len, float* absmax, hipStream_t s);

// Stem: convolution (stride 2, C <= 3, 64 output channels, int8 integers), the
// post-processing with a ReLU, and the 3x3 / stride-2 / pad-1 max pool, fused;
// y (or post.codes) receives the pooled outputs [N, PP, QQ, 64].
// Direct 3x3 / stride-1 / pad-1 convolution with input and output channels
// that are multiples of 64, on the fp8 MFMA (op 1 of mma_choose; dense NHWC
// input and KRSC filter, both 16-byte aligned): results identical to the
// implicit-GEMM path.
bool conv3x3_fits(const ConvGeom& g, int K, int groups, int op, const uint8_t* x,
                  const uint8_t* w);
hipError_t launch_conv3x3(const ConvGeom& g, int K, const uint8_t* x, const Fmt& fx,
                          const float* alphaX, const uint8_t* w, const Fmt& fw,
                          const float* alphaW, int32_t* acc, float* y, hipStream_t s,
                          const Post* post);

bool stem_fits(const ConvGeom& g, int K, int groups, const Fmt& fx, const Fmt& fw, int pool_r,
               int pool_stride, int pool_pad);
hipError_t launch_stem(const ConvGeom& g, const uint8_t* x, const Fmt& fx, const float* alphaX,
                       const uint8_t* w, const Fmt& fw, const float* alphaW, float* y, int PP,
                       int QQ, const Post& post, hipStream_t s);

// Depthwise convolution (groups == C == K): VALU kernel, HBM bound.
hipError_t launch_dwconv(const ConvGeom& g, const uint8_t* x, const Fmt& fx, const float* alphaX,
                         const uint8_t* w, const Fmt& fw, const float* alphaW, int32_t* acc,
                         float* y, hipStream_t s, const Post* post = nullptr);

}  // namespace esb
