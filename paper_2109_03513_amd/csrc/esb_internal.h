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

hipError_t launch_project(const float* x, int64_t len, const float* alpha, const Fmt& f,
                          uint8_t* codes, const float* dn, hipStream_t s);

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
                              int out_col_per_group, hipStream_t s);

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
                      int64_t ldc, int32_t* part, hipStream_t s);
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
                          int mode, void* ws, const uint8_t* b_packed, bool split, hipStream_t s);
// b_packed: B given in packed E2M1 (mode 1 only), not decoded; split: a dense
// GEMM with too few tiles splits its reduction (mma_splitk), the int32 partial
// sums after the decoded operands in ws (see esb_gemm_packed_workspace_size).
hipError_t launch_pack_fp4(const uint8_t* codes, int64_t rows, int64_t K, int64_t ld, const Fmt& f,
                           uint8_t* packed, hipStream_t s);

// Depthwise convolution (groups == C == K): VALU kernel, HBM bound.
hipError_t launch_dwconv(const ConvGeom& g, const uint8_t* x, const Fmt& fx, const float* alphaX,
                         const uint8_t* w, const Fmt& fw, const float* alphaW, int32_t* acc,
                         float* y, hipStream_t s);

}  // namespace esb
