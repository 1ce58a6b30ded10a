/*
 * libesb — the data-parallel hot path of elastic significant bit (ESB)
 * quantization (Gong et al., "Elastic Significant Bit Quantization and
 * Acceleration for Deep Neural Networks", IEEE TPDS 2021) on AMD MI355X
 * (gfx950).
 *
 * C ABI.  Every pointer argument documented "device" is a HIP device pointer
 * on the current device; "host" pointers are ordinary CPU memory.  `stream` is
 * a hipStream_t passed as void* (NULL = the null stream).  All device work is
 * enqueued asynchronously on `stream`; functions return once it is enqueued.
 * The caller owns every buffer; the library allocates no device memory (it
 * holds one static scratch array per GPU for esb_dda_align_noalloc).  Calls
 * keep no state between them and may be made from several host threads;
 * calls that share a workspace (or, for esb_dda_align_noalloc, a GPU) must not
 * overlap.
 *
 * Errors: every call returns an int status.  Arguments are validated on the
 * host before any launch; on error nothing is enqueued.  ESB_E_HIP means a HIP
 * runtime call failed; esb_last_hip_error() returns its hipError_t (per thread).
 *
 * Parameters of the format (Sec. 3.2, eq. (4)-(5)):
 *   n      total bits b, 2 <= n <= 8;
 *   k_sig  significant bits, 1 <= k_sig <= n-1.  The paper's k (fraction bits)
 *          is k = k_sig - 1: ESB(b, k) holds values with at most k+1
 *          significant bits.  Examples: (n=4, k_sig=2) is the paper's ESB(4,1);
 *          (n=3, k_sig=1) is ESB(3,0), powers of two; (n=3, k_sig=2) is
 *          ESB(3,1), a uniform grid.
 *
 * Code layout (ESB float format, eq. (14)): one code per byte, bits
 *   [n-1] sign | [n-2 .. k] exponent e | [k-1 .. 0] fraction f,
 * value 0.f when e is all ones (the subnormal binade), else 2^e * 1.f.  Zero
 * is always produced with sign 0; the code with sign 1 and value 0 is accepted
 * as input.  Bits above bit n-1 of an input code are ignored.
 */
#ifndef ESB_H
#define ESB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ESB_OK 0
#define ESB_E_INVALID (-1)     /* bad n/k_sig, sizes, NULL pointer, layout, descriptor */
#define ESB_E_OVERFLOW (-3)    /* reduction length * max|mA| * max|mB| > 2^31 - 1 */
#define ESB_E_UNSUPPORTED (-4) /* decoded integers exceed the split int8 range (|m| > 32639),
                                  or a format / length outside the packed 4-bit storage */
#define ESB_E_HIP (-5)         /* HIP launch / runtime failure, see esb_last_hip_error() */
#define ESB_E_WORKSPACE (-6)   /* workspace NULL or smaller than its *_workspace_size() */
#define ESB_E_SCRATCH (-7)     /* input larger than the static scratch of a *_noalloc call */

#define ESB_B_NK 0 /* B stored N x K, row-major (K contiguous) */
#define ESB_B_KN 1 /* B stored K x N, row-major (N contiguous) */

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int esb_version(void);

/* Human-readable name of a status code (static string). */
const char* esb_strerror(int status);

/* hipError_t of the last ESB_E_HIP returned on this thread (0 if none). */
int esb_last_hip_error(void);

/*
 * Value set, eq. (4)-(5) (Sec. 3.2).  Host only.
 * Writes the 2^n - 1 unscaled values of Q_e(1, n, k) in ascending order
 * (negatives, 0, positives) to vals_out[0 .. 2^n-2] (host, capacity `cap`
 * floats) and the count to *count_out (host).  The values are exact in fp32.
 * Returns ESB_E_INVALID for bad (n, k_sig), NULL pointers or cap < 2^n - 1.
 */
int esb_valueset(int n, int k_sig, float* vals_out, int cap, int* count_out);

/*
 * Projection operator Pi, eq. (6)-(8) (Sec. 3.3), emitting eq. (14) codes.
 *   x       device, len fp32 values, any layout;
 *   alpha   device, one fp32 scale (read on the device, so a preceding
 *           esb_dda_align on the same stream can produce it);
 *   codes   device, len bytes, same element order as x.
 * For each element: v = fl32(x / alpha) (IEEE binary32 division), clipped to
 * [-C, C] with C the largest set value, then rounded to the nearest set value
 * with ties going to the larger magnitude, sign restored (Pi(-x) = -Pi(x)).
 * NaN inputs give the +0 code; +-Inf give +-C.  If *alpha is not a positive
 * finite number every code is the +0 code.  len == 0 enqueues nothing.
 */
int esb_project(const float* x, int64_t len, const float* alpha, int n, int k_sig,
                uint8_t* codes, void* stream);

/*
 * Dequantization: out[i] = fl32(alpha * q(codes[i])), the values alpha * P(v)
 * of eq. (8).  codes, alpha, out are device pointers; len elements.
 */
int esb_dequantize(const uint8_t* codes, int64_t len, const float* alpha, int n, int k_sig,
                   float* out, void* stream);

/*
 * Bytes of device workspace esb_dda_align needs for these arguments (0 for
 * invalid arguments).  Deterministic in its arguments.
 */
size_t esb_dda_workspace_size(int64_t len, int n, int k_sig, int G);

/*
 * Distribution difference aligner: the search for the scale alpha of eq. (13)
 * over a candidate grid, with the objective of eq. (9) taken on the data
 * (the empirical distribution of x in place of p, both signs):
 *   D_j = sum_i (x_i - alpha_j * q_j(x_i))^2,   j = 0 .. G-1,
 * where q_j(x_i) is the projection of x_i under alpha_j (as esb_project).
 *   x          device, len fp32 values;
 *   grid       device, G fp32 candidate scales, 1 <= G and G * (2^(n-1)-1) <= 8192;
 *   alpha_out  device, one fp32: receives grid[j*];
 *   D_out      device, G doubles (may be NULL): the objective per candidate;
 *   workspace  device, at least esb_dda_workspace_size(len, n, k_sig, G) bytes.
 * j* is the smallest index with the least D_j.  A candidate that is not a
 * positive finite number gets D_j = NaN and ranks above every number; if any
 * x_i is NaN every D_j is NaN, else if any is +-Inf every D_j is +Inf (so
 * j* = 0).  D_j is accumulated in fp64 from exact per-interval partial sums;
 * it is deterministic for a given (len, grid) and agrees with the exact sum to
 * about 1e-12 relative.  Concurrent calls must use distinct workspaces.
 */
int esb_dda_align(const float* x, int64_t len, int n, int k_sig, const float* grid, int G,
                  float* alpha_out, double* D_out, void* workspace, size_t ws_bytes,
                  void* stream);

/*
 * Contraction over codes (Sec. 4.2, Forward(A_q, W_q); multiplication eq. (15)):
 *   acc[i][j] = sum_k mA[i][k] * mB[k][j]     (exact, int32)
 *   y[i][j]   = fl32(s * fl32(acc[i][j])),   s = 2^-(kA+kB) * fl32(alphaA * alphaB)
 * where m = q * 2^k is the exact integer of a code (q its unscaled value, k
 * the paper's fraction bits) and kA = kA_sig - 1, kB = kB_sig - 1.
 *   A        device, M x K codes, row-major with row pitch lda >= K bytes;
 *   B        device, N x K codes (b_layout ESB_B_NK, ldb >= K) or K x N codes
 *            (ESB_B_KN, ldb >= N);
 *   alphaA, alphaB  device, one fp32 each (only used for y);
 *   acc      device, M x N int32 with row pitch ldc elements, or NULL;
 *   y        device, M x N fp32 with row pitch ldc elements, or NULL;
 *            at least one of acc, y must be non-NULL.
 * ESB_E_UNSUPPORTED if an operand's largest decoded integer exceeds 32639
 * (operands above 127 use a split high/low int8 decomposition); ESB_E_OVERFLOW
 * if K * max|mA| * max|mB| > 2^31 - 1.  M, N or K == 0 is allowed (K == 0
 * writes zeros).
 */
int esb_gemm(int M, int N, int K, const uint8_t* A, int64_t lda, int nA, int kA_sig,
             const float* alphaA, const uint8_t* B, int64_t ldb, int nB, int kB_sig,
             const float* alphaB, int b_layout, int32_t* acc, float* y, int64_t ldc,
             void* stream);

/*
 * Bytes of device workspace that esb_gemm_ws may use (0 when it would use
 * none).  Two uses: decoding both operands once ahead of the contraction, for
 * pairs of formats whose values are exact in OCP E4M3 (or E2M3, E2M1) and
 * whose products and partial sums over K stay exact in the fp32 accumulation
 * of the fp8/fp6/fp4 matrix cores; and int32 partial sums when a GEMM with too
 * few output tiles to fill the GPU splits its reduction.  Deterministic in
 * its arguments.
 */
size_t esb_gemm_workspace_size(int M, int N, int K, int nA, int kA_sig, int nB, int kB_sig);

/*
 * esb_gemm with a caller workspace (device, at least esb_gemm_workspace_size()
 * bytes, or NULL).  Results are bit-identical to esb_gemm.  For shapes with
 * enough work per operand byte the codes of A and B are first decoded (to
 * packed E2M1, packed E2M3 or E4M3) into the workspace and the contraction
 * reads the decoded bytes; skinny shapes split the reduction and keep exact
 * int32 partial sums there; otherwise the workspace is unused.
 * ESB_E_WORKSPACE if workspace is non-NULL and ws_bytes is too small.  The
 * workspace carries nothing between calls; concurrent calls need distinct ones.
 */
int esb_gemm_ws(int M, int N, int K, const uint8_t* A, int64_t lda, int nA, int kA_sig,
                const float* alphaA, const uint8_t* B, int64_t ldb, int nB, int kB_sig,
                const float* alphaB, int b_layout, int32_t* acc, float* y, int64_t ldc,
                void* workspace, size_t ws_bytes, void* stream);

/*
 * Packed 4-bit code storage (the b-bit format of Sec. 4.1 at b <= 4, two codes
 * per byte).  For formats inside OCP FP4 E2M1 (at most 2 exponent bits and
 * k_sig <= 2: ESB(4,1) itself, every ESB(3,.) and ESB(2,.)), each code becomes
 * its E2M1 nibble with the same value q, 32 codes of a row per 16 bytes in a
 * fixed order (byte i of dword w holds codes 8w+i, low nibble, and 8w+4+i),
 * which is the operand layout of the fp4 matrix cores: a weight matrix packed
 * once is read in place by esb_gemm_packed, at half the bytes of one code per
 * byte and with no decoding in the contraction.
 *   esb_pack_size  bytes of `rows` packed rows of K codes: rows * K/2, or 0 when
 *                  the format is not inside E2M1 or K % 32 != 0;
 *   esb_pack       codes: device, rows x K codes with row pitch ld >= K (both
 *                  16-byte aligned); packed: device, esb_pack_size bytes, rows of
 *                  K/2 bytes.  ESB_E_UNSUPPORTED for formats outside E2M1 or
 *                  K % 32 != 0.
 */
size_t esb_pack_size(int rows, int K, int n, int k_sig);
int esb_pack(const uint8_t* codes, int rows, int K, int64_t ld, int n, int k_sig,
             uint8_t* packed, void* stream);

/*
 * GEMM with B given packed by esb_pack (N rows of K/2 bytes), A as codes (packed
 * per call into the workspace), results bit-identical to esb_gemm with
 * ESB_B_NK.  Both formats inside E2M1, K % 32 == 0, K * max|mA| * max|mB| < 2^24
 * (else ESB_E_UNSUPPORTED / ESB_E_OVERFLOW).  Skinny shapes (fully connected
 * layers at a small batch) split the reduction: over the four waves of one
 * workgroup per 64 x 32 output tile, summed exactly in LDS, where such tiles give
 * at least half the CUs a workgroup; otherwise over workgroups, with exact int32
 * partial sums in the workspace.
 *   workspace  device, at least esb_gemm_packed_workspace_size() bytes
 *              (ESB_E_WORKSPACE otherwise); A 16-byte aligned, lda % 16 == 0.
 */
size_t esb_gemm_packed_workspace_size(int M, int N, int K, int nA, int kA_sig, int nB,
                                      int kB_sig);
int esb_gemm_packed(int M, int N, int K, const uint8_t* A, int64_t lda, int nA, int kA_sig,
                    const float* alphaA, const uint8_t* B_packed, int nB, int kB_sig,
                    const float* alphaB, int32_t* acc, float* y, int64_t ldc, void* workspace,
                    size_t ws_bytes, void* stream);

/*
 * The aligner with its grid-only work done once: a plan.  Every call of
 * esb_dda_align first derives, from the candidates alone, each candidate's
 * exact cell thresholds, their merged sorted bounds and a bin table over them;
 * for a small tensor that set-up takes as long as the pass over the data.
 * esb_dda_plan builds it once, on the device, for candidates factors[j]
 * (device, G fp32); esb_dda_align_planned then searches the candidates
 *   alpha_j = 2^E * factors[j],   2^(E-1) <= |*scale| < 2^E   (E = 0 when *scale == 0),
 * a data-dependent power-of-two multiple of the factors (for example factors
 * spanning (0, 1/C] and *scale = max|x| from esb_absmax or an epilogue, so that
 * the grid spans (0, 2^E/C] with 2^E in (max|x|, 2 max|x|]).  Multiplying a
 * candidate by a power of two multiplies its exact thresholds by the same
 * power, so the plan's tables are shifted in the exponent instead of being
 * rebuilt; when the shifted tables would leave the normal fp32 range the call
 * rebuilds them.  Results are those of esb_dda_align with grid[j] =
 * ldexp(factors[j], E) (identical alpha, D within its stated accuracy and
 * deterministic); a *scale that is not finite makes every candidate NaN
 * (D_j = NaN, alpha_out = NaN).
 *   esb_dda_plan_size    bytes of a plan (0 for invalid arguments);
 *   esb_dda_plan         plan: device, 16-byte aligned, esb_dda_plan_size bytes
 *                        (ESB_E_WORKSPACE otherwise); written on `stream`;
 *   esb_dda_align_planned  n, k_sig, G as given to esb_dda_plan; scale: device
 *                        scalar; workspace: esb_dda_workspace_size(len, n, k_sig,
 *                        G) bytes.  A plan built for other arguments (or not a
 *                        plan) is not used: the call then rebuilds the tables
 *                        from the factors it finds there.
 */
size_t esb_dda_plan_size(int n, int k_sig, int G);
int esb_dda_plan(int n, int k_sig, const float* factors, int G, void* plan, size_t plan_bytes,
                 void* stream);
int esb_dda_align_planned(const float* x, int64_t len, int n, int k_sig, const void* plan, int G,
                          const float* scale, float* alpha_out, double* D_out, void* workspace,
                          size_t ws_bytes, void* stream);

/*
 * Quantization of one tensor with a plan (eq. (9), (13), then eq. (6)-(8)): the
 * planned aligner's alpha (and D_j), then the codes of x under that alpha, in
 * one call.  Results are those of esb_dda_align_planned followed by esb_project
 * with its alpha_out (identical alpha, D and codes).  For small tensors (at most
 * 2048 * (CUs) elements, 16-byte aligned x, 4-byte aligned codes, the aligner's
 * finishing step within one block of 256 threads) every block of the projection
 * derives alpha itself instead of waiting for a separate finishing kernel.
 *   arguments as esb_dda_align_planned; codes: device, len bytes (may be NULL
 *   when len == 0); D_out may be NULL.
 */
int esb_quantize_planned(const float* x, int64_t len, int n, int k_sig, const void* plan, int G,
                         const float* scale, float* alpha_out, double* D_out, uint8_t* codes,
                         void* workspace, size_t ws_bytes, void* stream);

/*
 * esb_dda_align for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, search and results as esb_dda_align (alpha and D
 * bit-identical), without a workspace: the call's scratch (the per-block
 * partial objectives) lives in a static device array of
 * ESB_DDA_NOALLOC_SCRATCH bytes that the library holds on every GPU it runs
 * on until the process ends; the call itself allocates nothing.
 *   Limit: esb_dda_workspace_size(len, n, k_sig, G) <= ESB_DDA_NOALLOC_SCRATCH
 *   (with G = 64 about 2^31 elements), else ESB_E_SCRATCH before any launch.
 *   Sharing: every call on one GPU uses that GPU's one array, so calls that
 *   overlap on a GPU (several streams or host threads) race; serialize them
 *   on one stream.  Nothing carries over from one call to the next.
 *   The first call on each device looks up that device's array address
 *   (hipGetSymbolAddress, with the device current); a failure returns
 *   ESB_E_HIP.
 */
#define ESB_DDA_NOALLOC_SCRATCH ((size_t)4 << 20)
int esb_dda_align_noalloc(const float* x, int64_t len, int n, int k_sig, const float* grid, int G,
                          float* alpha_out, double* D_out, void* stream);

/*
 * Batches of independent problems in one launch of each kernel: the DDA or the
 * projection of several tensors (for example a layer's weights and its input,
 * or every layer's weights), each with its own format, grid and outputs, with
 * results identical to one esb_dda_align / esb_project call per job.  Small
 * tensors leave most of the GPU idle and pay a fixed latency per launch; a
 * batch pays it once.  jobs: host array of count entries.  The DDA workspace
 * (device) holds every job's workspace, 256-byte aligned, in job order:
 * esb_dda_batch_workspace_size() bytes (0 for an invalid job).  Errors as the
 * single calls; a job that fails validation fails the whole batch before any
 * launch.
 */
typedef struct esb_dda_job {
    const float* x;     /* device, len fp32 */
    int64_t len;
    int n, k_sig;
    const float* grid;  /* device, G fp32 candidates */
    int G;
    float* alpha_out;   /* device, one fp32 */
    double* D_out;      /* device, G doubles, or NULL */
    const float* grid_scale;  /* device scalar, or NULL: candidate j is then
                                 fl32(grid_scale[0] * grid[j]) (one rounding), e.g. a grid of
                                 factors times a max|x| computed on the device */
} esb_dda_job;
size_t esb_dda_batch_workspace_size(int count, const esb_dda_job* jobs);
int esb_dda_align_batch(int count, const esb_dda_job* jobs, void* workspace, size_t ws_bytes,
                        void* stream);

typedef struct esb_project_job {
    const float* x;      /* device, len fp32 */
    int64_t len;
    const float* alpha;  /* device scalar */
    int n, k_sig;
    uint8_t* codes;      /* device, len codes */
} esb_project_job;
int esb_project_batch(int count, const esb_project_job* jobs, void* stream);

/*
 * Data normalization (Sec. 3.4, the DN equation) and the aligner in its analytic
 * form (eq. (9), (13) with p = N(0,1), "Resolving extremum"), the paper's own
 * flow of Alg. 1: W_q = ESB(DN(W)) with alpha* found offline for N(0,1).
 *
 * esb_dn_stats: stats_out (device, two fp32) = the mean and the population
 *   standard deviation sqrt((1/d) sum (x - mean)^2) of x, from one read of x:
 *   fp64 sums and squared deviations per chunk of 16384 elements, combined by
 *   the pairwise update in a fixed order (deterministic), rounded to binary32;
 *   NaN, NaN for len == 0.  workspace: device, 8-byte aligned, at least
 *   esb_dn_workspace_size(len) bytes (16 per chunk; ESB_E_WORKSPACE otherwise).
 * esb_project_dn: codes of the normalized values
 *   xh = fl32( fl32(x - mean) / fl32(std + 1e-7) ),   code = esb_project(xh, alpha),
 *   stats (device, two fp32 mean, std: e.g. from esb_dn_stats, or running
 *   averages kept by the caller); alpha device, as esb_project.
 * esb_dda_normal: for each candidate grid[j] (device, G >= 1 fp32), the
 *   one-sided analytic objective D_j = E[(t - Pi(t))^2; t >= 0], t ~ N(0,1),
 *   with nearest-neighbour cells [alpha mid_c, alpha mid_{c+1}) (the top cell
 *   open), in fp64 (erfc, exp); Table 1 of the paper prints 2 * D.  D_out
 *   (device, G doubles, required); dD_out (device, G doubles, may be NULL)
 *   = dD/dalpha at each candidate, -2 sum_c q_c (M1_c - alpha q_c M0_c) with
 *   M0, M1 the cell's probability and first moment (the zeros the paper's
 *   "Resolving extremum" looks for); alpha_out (device, one fp32) = grid[j*],
 *   j* the smallest index with the least D; non-positive or non-finite
 *   candidates get NaN and rank last.
 */
size_t esb_dn_workspace_size(int64_t len);
int esb_dn_stats(const float* x, int64_t len, float* stats_out, void* workspace, size_t ws_bytes,
                 void* stream);
int esb_project_dn(const float* x, int64_t len, const float* stats, const float* alpha, int n,
                   int k_sig, uint8_t* codes, void* stream);
int esb_dda_normal(int n, int k_sig, const float* grid, int G, float* alpha_out, double* D_out,
                   double* dD_out, void* stream);

/*
 * Glue between quantized layers (Sec. 4.2: the post-processing after a
 * convolution, "MP&ReLU", and the pooled features before the classifier), so
 * that a forward pass between two contractions runs only library kernels.
 * fp32, NHWC; every pointer device; asynchronous on `stream`.
 * esb_maxpool2d: out[n][p][q][c] = max over the R x S window at
 *   (p*stride - pad, q*stride - pad) of the input elements inside the image
 *   (padding is never selected; requires pad < R and pad < S so that every
 *   window holds one); a NaN in a window gives NaN.  out is [N, P, Q, C] with
 *   P = (H + 2 pad - R)/stride + 1, Q likewise.
 * esb_avgpool_global: out[n][c] = fl32( (sum over the HW positions, in
 *   position order, of (double)x[n][i][c]) / HW ), x [N, HW, C], out [N, C];
 *   absmax_out (or NULL) is raised to max |out| as below.
 * esb_absmax: *absmax_out = max(*absmax_out, max_i |x_i|), compared as fp32 bit
 *   patterns with the sign cleared (a NaN wins over every number); the caller
 *   sets the initial value (0 to start).  A DDA grid scaled by this maximum
 *   (esb_dda_job.grid_scale) needs no host round trip.
 */
int esb_maxpool2d(const float* x, int N, int H, int W, int C, int R, int S, int stride, int pad,
                  float* out, void* stream);
int esb_avgpool_global(const float* x, int N, int HW, int C, float* out, float* absmax_out,
                       void* stream);
int esb_absmax(const float* x, int64_t len, float* absmax_out, void* stream);

/* Convolution geometry.  Output P = (H + 2*pad_h - R)/stride_h + 1, Q likewise. */
typedef struct esb_conv_desc {
    int N, H, W, C;          /* input batch, height, width, channels (NHWC) */
    int K, R, S;             /* output channels, filter height, filter width */
    int stride_h, stride_w;  /* >= 1 */
    int pad_h, pad_w;        /* >= 0, zero padding by value 0 */
    int groups;              /* divides C and K; groups == C == K is depthwise */
} esb_conv_desc;

/*
 * Convolution stage of Sec. 4.2 (Fig. "computing_logic"): cross-correlation of
 * ESB-coded activations with ESB-coded filters, as an implicit GEMM with
 * M = N*P*Q, N = K, reduction R*S*C/groups, scaled like esb_gemm.
 *   x      device, NHWC codes [N, H, W, C];
 *   w      device, KRSC codes [K, R, S, C/groups];
 *   acc    device, NHWC int32 [N, P, Q, K], or NULL;
 *   y      device, NHWC fp32 [N, P, Q, K], or NULL (at least one non-NULL).
 * Errors as esb_gemm, with the reduction length R*S*C/groups.
 */
int esb_conv2d(const esb_conv_desc* d, const uint8_t* x, int nX, int kX_sig,
               const float* alphaX, const uint8_t* w, int nW, int kW_sig,
               const float* alphaW, int32_t* acc, float* y, void* stream);

/*
 * Workspace bytes for esb_conv2d_ws (0 when unused: depthwise convolutions and
 * formats outside the E4M3 path).  The decoded activations keep the NHWC
 * layout and the decoded filters the KRSC layout.
 */
size_t esb_conv2d_workspace_size(const esb_conv_desc* d, int nX, int kX_sig, int nW, int kW_sig);

/* esb_conv2d with a caller workspace; same contract as esb_gemm_ws. */
int esb_conv2d_ws(const esb_conv_desc* d, const uint8_t* x, int nX, int kX_sig,
                  const float* alphaX, const uint8_t* w, int nW, int kW_sig,
                  const float* alphaW, int32_t* acc, float* y, void* workspace,
                  size_t ws_bytes, void* stream);

/*
 * Fused post-processing of a contraction's outputs (Sec. 4.2: the "BN and DN"
 * step of eq. (16), folded offline into a per-channel a x + b, then the "ESB
 * quantization" step that hands the next layer its codes), in the epilogue of
 * the contraction kernels, so that the next layer's input is written as codes
 * (1 byte per output) instead of fp32.  For each output with scaled value
 * y0 = fl32(s fl32(acc)) (s as in esb_gemm) in channel j (the output column of
 * a GEMM, the output channel of a convolution):
 *   z = fma(a[j], y0, b[j])     one rounding; a[j] = 1 when a is NULL, b[j] = 0
 *                               when b is NULL (so -0 becomes +0);
 *   z = fl32(z + residual[o])   when residual is not NULL;
 *   z = z > 0 ? z : 0           when relu is nonzero (NaN gives 0);
 *   y[o] = z                    when y is not NULL (instead of y0);
 *   codes[o] = code of z under *alpha in ESB(n, k_sig), as esb_project, when
 *              codes is not NULL.
 *   *absmax_out = max(*absmax_out, |z|) over every output, when absmax_out is
 *              not NULL: the next layer's max|x| (e.g. for a DDA grid scaled by
 *              it) without another pass; the comparison is on the fp32 bit
 *              patterns, so a NaN z leaves a NaN; the caller sets the initial
 *              value (0 to start).
 * residual and codes have the layout of y (GEMM: M rows of pitch ldc; conv:
 * NHWC [N, P, Q, K]); residual may be the same buffer as y (read before the
 * write of the same element).  acc, when not NULL, still receives the integer
 * sums.  The scale of the outputs must be known before the layer (the
 * paper's offline / running-average scales): alpha is a device scalar.
 * Errors: ESB_E_INVALID if post is given without alphaA / alphaB, if codes is
 * given without alpha or with an invalid (n, k_sig), or if acc, y, codes and
 * absmax_out are all NULL; otherwise as esb_gemm_ws / esb_conv2d_ws (workspace may be NULL).
 */
typedef struct esb_post {
    const float* a;         /* device, one fp32 per output channel, or NULL */
    const float* b;         /* device, one fp32 per output channel, or NULL */
    const float* residual;  /* device fp32 in the layout of y, or NULL */
    int relu;               /* nonzero: clamp at 0 */
    const float* alpha;     /* device scalar: scale of the output codes */
    int n, k_sig;           /* format of the output codes */
    uint8_t* codes;         /* device, one code per output in the layout of y, or NULL */
    float* absmax_out;      /* device scalar, or NULL: raised to max |z| of this call */
} esb_post;

int esb_gemm_post(int M, int N, int K, const uint8_t* A, int64_t lda, int nA, int kA_sig,
                  const float* alphaA, const uint8_t* B, int64_t ldb, int nB, int kB_sig,
                  const float* alphaB, int b_layout, int32_t* acc, float* y, int64_t ldc,
                  const esb_post* post, void* workspace, size_t ws_bytes, void* stream);
int esb_conv2d_post(const esb_conv_desc* d, const uint8_t* x, int nX, int kX_sig,
                    const float* alphaX, const uint8_t* w, int nW, int kW_sig,
                    const float* alphaW, int32_t* acc, float* y, const esb_post* post,
                    void* workspace, size_t ws_bytes, void* stream);

/*
 * A convolution followed by the post-processing of esb_conv2d_post with a
 * ReLU and by max pooling (Sec. 4.2: the convolution stage, then "MP&ReLU"),
 * the stem of a convolutional network:
 *   z[n][p][q][k]  = relu(fma(a[k], fl32(s fl32(acc[n][p][q][k])), b[k]))  (as esb_conv2d_post)
 *   y[n][i][j][k]  = max of z over the pool_window x pool_window window at
 *                    (i pool_stride - pool_pad, j pool_stride - pool_pad), positions
 *                    outside z left out (pool_pad < pool_window: every window holds one);
 * y: device fp32 [N, PP, QQ, K] (PP = (P + 2 pool_pad - pool_window)/pool_stride + 1,
 * QQ likewise), or NULL; post: relu nonzero, residual NULL, a / b optional; its codes
 * (with alpha, n, k_sig) receive the codes of y and absmax_out is raised to max |y|.
 * Where the fused kernel applies (stride 2, C <= 3, S*C <= 32, R <= 8, K == 64, pool
 * 3 / 2 / 1, decoded integers within int8, x 4-byte aligned) nothing else is
 * written: the full-resolution z never reaches memory.  Elsewhere z is computed into
 * the workspace (device, esb_conv2d_relu_maxpool_workspace_size bytes, 0 where the
 * fused kernel applies) and pooled from there, with the same results.
 * Errors: ESB_E_INVALID for a missing post, relu == 0, a residual, a window made only
 * of padding, or no output; otherwise as esb_conv2d_post.
 */
size_t esb_conv2d_relu_maxpool_workspace_size(const esb_conv_desc* d, int nX, int kX_sig, int nW,
                                              int kW_sig, int pool_window, int pool_stride,
                                              int pool_pad);
int esb_conv2d_relu_maxpool(const esb_conv_desc* d, const uint8_t* x, int nX, int kX_sig,
                            const float* alphaX, const uint8_t* w, int nW, int kW_sig,
                            const float* alphaW, const esb_post* post, int pool_window,
                            int pool_stride, int pool_pad, float* y, void* workspace,
                            size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ESB_H */
