// C ABI of libesb: argument validation, format tables, dispatch.
#include <math.h>
#include <string.h>

#include "../../include/esb.h"
#include <atomic>
#include <mutex>
#include <vector>

#include "esb_internal.h"

namespace esb {

bool valid_fmt(int n, int k_sig) { return n >= 2 && n <= 8 && k_sig >= 1 && k_sig <= n - 1; }

// ESB(b, k) as a minifloat: 1 sign bit, b-k-1 exponent bits, k fraction bits,
// the all-ones exponent being the subnormal binade (eq. (14)).
Fmt make_fmt(int n, int k_sig) {
    Fmt f;
    f.n = n;
    f.k = k_sig - 1;
    f.ebits = n - f.k - 1;
    f.N = (1 << f.ebits) - 1;
    f.zero_code = (uint32_t)f.N << f.k;
    f.c_code = ((uint32_t)(f.N - 1) << f.k) | ((1u << f.k) - 1u);
    f.sign_bit = 1u << (n - 1);
    f.C = ldexpf((float)((1 << (f.k + 1)) - 1), f.N - f.k - 1);
    uint32_t cb;
    memcpy(&cb, &f.C, 4);
    f.c_bits = cb;
    const double mi = ldexp((double)((1 << (f.k + 1)) - 1), f.N - 1);
    f.max_int = mi > 2147483647.0 ? 2147483647 : (int)mi;
    return f;
}

double decode_value(const Fmt& f, uint32_t code) {
    code &= (1u << f.n) - 1u;
    const uint32_t e = (code >> f.k) & (uint32_t)f.N;
    const uint32_t fr = code & ((1u << f.k) - 1u);
    const double mag = (e == (uint32_t)f.N) ? ldexp((double)fr, -f.k)
                                             : ldexp((double)((1u << f.k) | fr), (int)e - f.k);
    return (code & f.sign_bit) ? -mag : mag;
}

int decode_int(const Fmt& f, uint32_t code) {
    const double v = ldexp(decode_value(f, code), f.k);
    return v > 2147483647.0 ? 2147483647 : (v < -2147483647.0 ? -2147483647 : (int)v);
}

int num_cus() {
    static std::atomic<int> cached[64];   // zero-initialized (static storage)
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cached[dev].load(std::memory_order_relaxed);
    if (!v) {   // racing threads store the same value
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
            v = 256;
        cached[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

}  // namespace esb

using namespace esb;

static thread_local int g_last_hip = 0;

static int hip_status(hipError_t e) {
    if (e == hipSuccess) return ESB_OK;
    g_last_hip = (int)e;
    return ESB_E_HIP;
}

// Scratch of the entry point that allocates nothing (esb_dda_align_noalloc):
// one array per GPU, held until the process ends.  In host code `scratch` only
// names the symbol; its device address comes from hipGetSymbolAddress, looked
// up once per device with that device current.
constexpr size_t kScratchBytes = ESB_DDA_NOALLOC_SCRATCH;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

static std::mutex g_scratch_mu;
static std::atomic<void*> g_scratch_ptr[64];

static hipError_t scratch_address(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
        if (!p) {
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (!p) return hipErrorInvalidSymbol;
            g_scratch_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return hipSuccess;
}

extern "C" {

int esb_version(void) { return 200; }   // 0.2.0: fused epilogue, packed codes, DN, batches

const char* esb_strerror(int status) {
    switch (status) {
        case ESB_OK: return "ok";
        case ESB_E_INVALID: return "invalid argument";
        case ESB_E_OVERFLOW: return "int32 accumulator bound exceeded";
        case ESB_E_UNSUPPORTED: return "decoded integers exceed the split int8 range";
        case ESB_E_HIP: return "HIP runtime error";
        case ESB_E_WORKSPACE: return "workspace missing or too small";
        case ESB_E_SCRATCH: return "input needs more scratch than the static device buffer holds";
        default: return "unknown status";
    }
}

int esb_last_hip_error(void) { return g_last_hip; }

int esb_valueset(int n, int k_sig, float* vals_out, int cap, int* count_out) {
    if (!valid_fmt(n, k_sig) || !vals_out || !count_out) return ESB_E_INVALID;
    const int count = (1 << n) - 1;
    if (cap < count) return ESB_E_INVALID;
    const Fmt f = make_fmt(n, k_sig);
    float v[256];
    int m = 0;
    for (uint32_t c = 0; c < (1u << n); c++) {
        if ((c & f.sign_bit) && ((c & ~f.sign_bit) == f.zero_code)) continue;   // -0
        v[m++] = (float)decode_value(f, c);
    }
    for (int i = 1; i < m; i++)
        for (int t = i; t > 0 && v[t] < v[t - 1]; t--) {
            const float tmp = v[t]; v[t] = v[t - 1]; v[t - 1] = tmp;
        }
    memcpy(vals_out, v, sizeof(float) * (size_t)m);
    *count_out = m;
    return ESB_OK;
}

int esb_project(const float* x, int64_t len, const float* alpha, int n, int k_sig, uint8_t* codes,
                void* stream) {
    if (!valid_fmt(n, k_sig) || len < 0 || !alpha) return ESB_E_INVALID;
    if (len > 0 && (!x || !codes)) return ESB_E_INVALID;
    return hip_status(launch_project(x, len, alpha, make_fmt(n, k_sig), codes, nullptr,
                                     (hipStream_t)stream));
}

int esb_dequantize(const uint8_t* codes, int64_t len, const float* alpha, int n, int k_sig,
                   float* out, void* stream) {
    if (!valid_fmt(n, k_sig) || len < 0 || !alpha) return ESB_E_INVALID;
    if (len > 0 && (!codes || !out)) return ESB_E_INVALID;
    return hip_status(launch_dequantize(codes, len, alpha, make_fmt(n, k_sig), out, (hipStream_t)stream));
}

size_t esb_dda_workspace_size(int64_t len, int n, int k_sig, int G) {
    if (!valid_fmt(n, k_sig)) return 0;
    DdaLayout L;
    if (!dda_layout(len, make_fmt(n, k_sig), G, &L)) return 0;
    return L.total;
}

int esb_dda_align(const float* x, int64_t len, int n, int k_sig, const float* grid, int G,
                  float* alpha_out, double* D_out, void* workspace, size_t ws_bytes, void* stream) {
    if (!valid_fmt(n, k_sig) || len < 0 || !grid || !alpha_out) return ESB_E_INVALID;
    if (len > 0 && !x) return ESB_E_INVALID;
    const Fmt f = make_fmt(n, k_sig);
    DdaLayout L;
    if (!dda_layout(len, f, G, &L)) return ESB_E_INVALID;
    if (!workspace || ws_bytes < L.total) return ESB_E_WORKSPACE;
    return hip_status(launch_dda(x, len, f, grid, G, alpha_out, D_out, workspace, L, (hipStream_t)stream));
}

int esb_dda_align_noalloc(const float* x, int64_t len, int n, int k_sig, const float* grid, int G,
                          float* alpha_out, double* D_out, void* stream) {
    if (!valid_fmt(n, k_sig) || len < 0 || !grid || !alpha_out) return ESB_E_INVALID;
    if (len > 0 && !x) return ESB_E_INVALID;
    const Fmt f = make_fmt(n, k_sig);
    DdaLayout L;
    if (!dda_layout(len, f, G, &L)) return ESB_E_INVALID;
    if (L.total > kScratchBytes) return ESB_E_SCRATCH;
    void* ws = nullptr;
    const hipError_t e = scratch_address(&ws);
    if (e != hipSuccess) return hip_status(e);
    return hip_status(launch_dda(x, len, f, grid, G, alpha_out, D_out, ws, L, (hipStream_t)stream));
}

size_t esb_dda_plan_size(int n, int k_sig, int G) {
    if (!valid_fmt(n, k_sig)) return 0;
    DdaLayout L;
    if (!dda_layout(0, make_fmt(n, k_sig), G, &L)) return 0;
    return dda_plan_bytes(make_fmt(n, k_sig), G);
}

int esb_dda_plan(int n, int k_sig, const float* factors, int G, void* plan, size_t plan_bytes,
                 void* stream) {
    if (!valid_fmt(n, k_sig) || !factors) return ESB_E_INVALID;
    const Fmt f = make_fmt(n, k_sig);
    DdaLayout L;
    if (!dda_layout(0, f, G, &L)) return ESB_E_INVALID;
    if (!plan || plan_bytes < dda_plan_bytes(f, G) || (uintptr_t)plan % 16) return ESB_E_WORKSPACE;
    return hip_status(launch_dda_plan(f, factors, G, plan, (hipStream_t)stream));
}

int esb_dda_align_planned(const float* x, int64_t len, int n, int k_sig, const void* plan, int G,
                          const float* scale, float* alpha_out, double* D_out, void* workspace,
                          size_t ws_bytes, void* stream) {
    if (!valid_fmt(n, k_sig) || len < 0 || !plan || !scale || !alpha_out) return ESB_E_INVALID;
    if (len > 0 && !x) return ESB_E_INVALID;
    if ((uintptr_t)plan % 16) return ESB_E_INVALID;
    DdaJobDesc d{};
    d.f = make_fmt(n, k_sig);
    if (!dda_layout(len, d.f, G, &d.L)) return ESB_E_INVALID;
    if (!workspace || ws_bytes < d.L.total) return ESB_E_WORKSPACE;
    d.x = x; d.len = len; d.grid = nullptr; d.G = G;
    d.alpha_out = alpha_out; d.D_out = D_out; d.ws = workspace;
    d.gscale = scale;
    d.plan = (const uint8_t*)plan;
    return hip_status(launch_dda_batch(&d, 1, (hipStream_t)stream));
}

int esb_quantize_planned(const float* x, int64_t len, int n, int k_sig, const void* plan, int G,
                         const float* scale, float* alpha_out, double* D_out, uint8_t* codes,
                         void* workspace, size_t ws_bytes, void* stream) {
    if (!valid_fmt(n, k_sig) || len < 0 || !plan || !scale || !alpha_out) return ESB_E_INVALID;
    if (len > 0 && (!x || !codes)) return ESB_E_INVALID;
    if ((uintptr_t)plan % 16) return ESB_E_INVALID;
    DdaJobDesc d{};
    d.f = make_fmt(n, k_sig);
    if (!dda_layout(len, d.f, G, &d.L)) return ESB_E_INVALID;
    if (!workspace || ws_bytes < d.L.total) return ESB_E_WORKSPACE;
    d.x = x; d.len = len; d.grid = nullptr; d.G = G;
    d.alpha_out = alpha_out; d.D_out = D_out; d.ws = workspace;
    d.gscale = scale;
    d.plan = (const uint8_t*)plan;
    return hip_status(launch_dda_quantize(d, codes, (hipStream_t)stream));
}

size_t esb_dda_batch_workspace_size(int count, const esb_dda_job* jobs) {
    if (count < 0 || (count > 0 && !jobs)) return 0;
    size_t total = 0;
    for (int i = 0; i < count; i++) {
        const esb_dda_job& j = jobs[i];
        if (!valid_fmt(j.n, j.k_sig)) return 0;
        DdaLayout L;
        if (!dda_layout(j.len, make_fmt(j.n, j.k_sig), j.G, &L)) return 0;
        total += (L.total + 255) & ~(size_t)255;
    }
    return total;
}

int esb_dda_align_batch(int count, const esb_dda_job* jobs, void* workspace, size_t ws_bytes,
                        void* stream) {
    if (count < 0 || (count > 0 && !jobs)) return ESB_E_INVALID;
    if (count == 0) return ESB_OK;
    std::vector<DdaJobDesc> d((size_t)count);
    size_t off = 0;
    for (int i = 0; i < count; i++) {
        const esb_dda_job& j = jobs[i];
        if (!valid_fmt(j.n, j.k_sig) || j.len < 0 || !j.grid || !j.alpha_out) return ESB_E_INVALID;
        if (j.len > 0 && !j.x) return ESB_E_INVALID;
        DdaJobDesc& e = d[(size_t)i];
        e.f = make_fmt(j.n, j.k_sig);
        if (!dda_layout(j.len, e.f, j.G, &e.L)) return ESB_E_INVALID;
        e.x = j.x; e.len = j.len; e.grid = j.grid; e.G = j.G;
        e.alpha_out = j.alpha_out; e.D_out = j.D_out;
        e.gscale = j.grid_scale;
        e.plan = nullptr;
        e.ws = (char*)workspace + off;
        off += (e.L.total + 255) & ~(size_t)255;
    }
    if (!workspace || ws_bytes < off) return ESB_E_WORKSPACE;
    return hip_status(launch_dda_batch(d.data(), count, (hipStream_t)stream));
}

int esb_maxpool2d(const float* x, int N, int H, int W, int C, int R, int S, int stride, int pad,
                  float* out, void* stream) {
    if (N < 0 || H < 1 || W < 1 || C < 1 || R < 1 || S < 1 || stride < 1 || pad < 0 ||
        pad >= R || pad >= S || H + 2 * pad < R || W + 2 * pad < S)
        return ESB_E_INVALID;
    PoolGeom g;
    g.N = N; g.H = H; g.W = W; g.C = C; g.R = R; g.S = S; g.sh = stride; g.sw = stride;
    g.ph = pad; g.pw = pad;
    g.P = (H + 2 * pad - R) / stride + 1;
    g.Q = (W + 2 * pad - S) / stride + 1;
    if ((int64_t)N * g.P * g.Q * C > 0 && (!x || !out)) return ESB_E_INVALID;
    return hip_status(launch_maxpool(x, g, out, (hipStream_t)stream));
}

int esb_avgpool_global(const float* x, int N, int HW, int C, float* out, float* absmax_out,
                       void* stream) {
    if (N < 0 || HW < 1 || C < 1) return ESB_E_INVALID;
    if (N > 0 && (!x || !out)) return ESB_E_INVALID;
    return hip_status(launch_avgpool(x, N, HW, C, out, absmax_out, (hipStream_t)stream));
}

int esb_absmax(const float* x, int64_t len, float* absmax_out, void* stream) {
    if (len < 0 || !absmax_out || (len > 0 && !x)) return ESB_E_INVALID;
    return hip_status(launch_absmax(x, len, absmax_out, (hipStream_t)stream));
}

int esb_project_batch(int count, const esb_project_job* jobs, void* stream) {
    if (count < 0 || (count > 0 && !jobs)) return ESB_E_INVALID;
    std::vector<ProjJobDesc> d((size_t)count);
    for (int i = 0; i < count; i++) {
        const esb_project_job& j = jobs[i];
        if (!valid_fmt(j.n, j.k_sig) || j.len < 0 || !j.alpha) return ESB_E_INVALID;
        if (j.len > 0 && (!j.x || !j.codes)) return ESB_E_INVALID;
        d[(size_t)i] = ProjJobDesc{j.x, j.len, j.alpha, make_fmt(j.n, j.k_sig), j.codes};
    }
    if (count == 0) return ESB_OK;
    return hip_status(launch_project_batch(d.data(), count, (hipStream_t)stream));
}

static int contraction_contract(int64_t kred, const Fmt& a, const Fmt& b) {
    if (a.max_int > 32639 || b.max_int > 32639) return ESB_E_UNSUPPORTED;
    if ((double)kred * (double)a.max_int * (double)b.max_int > 2147483647.0) return ESB_E_OVERFLOW;
    return ESB_OK;
}

// Decoding both operands once ahead of the contraction pays when the work per
// decoded byte is high: then the decode pass (1 byte read and written per code)
// is small next to a contraction that no longer decodes in its inner loop.
static bool pre_worth(int64_t M, int64_t N, int64_t K, int64_t a_elems, int64_t b_elems) {
    const double ops = 2.0 * (double)M * (double)N * (double)K;
    return ops >= 1500.0 * (double)(a_elems + b_elems);
}

// Fused post-processing: the output scale needs both alphas; codes need their
// format and scale.
static bool post_ok(const esb_post* p, const float* alphaA, const float* alphaB) {
    if (!p) return true;
    if (!alphaA || !alphaB) return false;
    if (p->codes && (!p->alpha || !valid_fmt(p->n, p->k_sig))) return false;
    return true;
}

static Post make_post(const esb_post* p) {
    Post q{};
    if (!p) return q;
    q.a = p->a;
    q.b = p->b;
    q.res = p->residual;
    q.alpha = p->alpha;
    q.codes = p->codes;
    q.absmax = (uint32_t*)p->absmax_out;
    q.relu = p->relu != 0;
    q.on = 1;
    if (p->codes) q.pp = proj_params(make_fmt(p->n, p->k_sig));
    return q;
}

static int gemm_impl(int M, int N, int K, const uint8_t* A, int64_t lda, int nA, int kA_sig,
                     const float* alphaA, const uint8_t* B, int64_t ldb, int nB, int kB_sig,
                     const float* alphaB, int b_layout, int32_t* acc, float* y, int64_t ldc,
                     void* ws, size_t ws_bytes, void* stream, const esb_post* post = nullptr) {
    if (!valid_fmt(nA, kA_sig) || !valid_fmt(nB, kB_sig)) return ESB_E_INVALID;
    if (M < 0 || N < 0 || K < 0 || (b_layout != ESB_B_NK && b_layout != ESB_B_KN)) return ESB_E_INVALID;
    if (!post_ok(post, alphaA, alphaB)) return ESB_E_INVALID;
    if (!acc && !y && !(post && (post->codes || post->absmax_out))) return ESB_E_INVALID;
    const Post P = make_post(post);
    const Post* pp = post ? &P : nullptr;
    if (ldc < N || lda < K || (b_layout == ESB_B_NK ? ldb < K : ldb < N)) return ESB_E_INVALID;
    if (y && (!alphaA || !alphaB)) return ESB_E_INVALID;
    if ((int64_t)M * N > 0 && K > 0 && (!A || !B)) return ESB_E_INVALID;
    const Fmt fa = make_fmt(nA, kA_sig), fb = make_fmt(nB, kB_sig);
    const int st = contraction_contract(K, fa, fb);
    if (st) return st;
    if (ws && ws_bytes < esb_gemm_workspace_size(M, N, K, nA, kA_sig, nB, kB_sig)) return ESB_E_WORKSPACE;
    if (M == 0 || N == 0) return ESB_OK;
    ConvGeom g;
    g.Nb = M; g.H = 1; g.W = 1; g.C = K; g.pitch = (int)(lda > 0x7fffffff ? 0x7fffffff : lda);
    g.Cg = K; g.R = 1; g.S = 1; g.sh = 1; g.sw = 1; g.ph = 0; g.pw = 0; g.P = 1; g.Q = 1;
    if (lda > 0x7fffffff) return ESB_E_INVALID;
    const int op = mma_choose(fa, fb, K);
    // decode-once formats: packed E2M1 where both formats fit it, else packed E2M3, else E4M3
    const bool f4 = mma_f4ok(fa, fb, K) && K % 32 == 0;
    const bool f6 = !f4 && mma_f6ok(fa, fb, K) && K % 64 == 0 && mma_f6_tiles(M, N, 1);
    const hipStream_t s = (hipStream_t)stream;
    const bool fits = mma_fits(g, A, K, 1, B, ldb, b_layout);
    if (ws && fits && (f4 || op == 1) && pre_worth(M, N, K, (int64_t)M * K, (int64_t)N * K))
        return hip_status(launch_mma_pre(M, N, K, 1, g, A, M, K, lda, fa, alphaA, B, N, ldb, fb, alphaB,
                                         acc, y, ldc, f4 ? 1 : (f6 ? 2 : 0), ws, nullptr, false, s,
                                         pp));
    if (op >= 0 && fits)   // with a workspace, skinny shapes split the reduction
        return hip_status(launch_mma(op, M, N, K, 1, g, A, fa, alphaA, B, ldb, fb, alphaB, acc, y,
                                     ldc, (int32_t*)ws, s, pp));
    return hip_status(launch_contraction(M, N, K, 1, g, A, decode_info(fa), alphaA, B, ldb, b_layout,
                                         decode_info(fb), alphaB, acc, y, ldc, N, s, pp));
}

size_t esb_gemm_workspace_size(int M, int N, int K, int nA, int kA_sig, int nB, int kB_sig) {
    if (!valid_fmt(nA, kA_sig) || !valid_fmt(nB, kB_sig) || M < 0 || N < 0 || K < 0) return 0;
    const Fmt fa = make_fmt(nA, kA_sig), fb = make_fmt(nB, kB_sig);
    const int op = mma_choose(fa, fb, K);
    size_t need = 0;
    if (op == 1 || (mma_f4ok(fa, fb, K) && K % 32 == 0))
        need = mma_pre_workspace(M, K, N, K);   // E4M3 size; packed E2M1 / E2M3 need less
    if (op >= 0 && K % 16 == 0) {               // split reduction: int32 partial sums
        int kc = K;
        const int ks = mma_splitk(M, N, K, &kc);
        if (ks > 1) {
            const size_t p = (size_t)ks * (size_t)M * (size_t)N * sizeof(int32_t);
            if (p > need) need = p;
        }
    }
    return need;
}

int esb_gemm(int M, int N, int K, const uint8_t* A, int64_t lda, int nA, int kA_sig,
             const float* alphaA, const uint8_t* B, int64_t ldb, int nB, int kB_sig,
             const float* alphaB, int b_layout, int32_t* acc, float* y, int64_t ldc, void* stream) {
    return gemm_impl(M, N, K, A, lda, nA, kA_sig, alphaA, B, ldb, nB, kB_sig, alphaB, b_layout, acc, y,
                     ldc, nullptr, 0, stream);
}

int esb_gemm_ws(int M, int N, int K, const uint8_t* A, int64_t lda, int nA, int kA_sig,
                const float* alphaA, const uint8_t* B, int64_t ldb, int nB, int kB_sig,
                const float* alphaB, int b_layout, int32_t* acc, float* y, int64_t ldc,
                void* workspace, size_t ws_bytes, void* stream) {
    return gemm_impl(M, N, K, A, lda, nA, kA_sig, alphaA, B, ldb, nB, kB_sig, alphaB, b_layout, acc, y,
                     ldc, workspace, ws_bytes, stream);
}

// Checked geometry of a convolution descriptor (ESB_OK or ESB_E_INVALID).
static int conv_geom(const esb_conv_desc* d, ConvGeom* g, int64_t* Mrows, int64_t* kred) {
    if (!d) return ESB_E_INVALID;
    if (d->N < 0 || d->H < 1 || d->W < 1 || d->C < 1 || d->K < 1 || d->R < 1 || d->S < 1 ||
        d->stride_h < 1 || d->stride_w < 1 || d->pad_h < 0 || d->pad_w < 0 || d->groups < 1 ||
        d->C % d->groups || d->K % d->groups)
        return ESB_E_INVALID;
    if ((int64_t)d->H + 2 * d->pad_h < d->R || (int64_t)d->W + 2 * d->pad_w < d->S) return ESB_E_INVALID;
    const int P = (d->H + 2 * d->pad_h - d->R) / d->stride_h + 1;
    const int Q = (d->W + 2 * d->pad_w - d->S) / d->stride_w + 1;
    *Mrows = (int64_t)d->N * P * Q;
    if (*Mrows > 0x7fffffff) return ESB_E_INVALID;
    const int Cg = d->C / d->groups;
    *kred = (int64_t)d->R * d->S * Cg;
    if (*kred > 0x7fffffff) return ESB_E_INVALID;
    g->Nb = d->N; g->H = d->H; g->W = d->W; g->C = d->C; g->pitch = d->C; g->Cg = Cg;
    g->R = d->R; g->S = d->S; g->sh = d->stride_h; g->sw = d->stride_w; g->ph = d->pad_h; g->pw = d->pad_w;
    g->P = P; g->Q = Q;
    return ESB_OK;
}

static bool conv_is_depthwise(const esb_conv_desc* d) {
    return d->C / d->groups == 1 && d->K / d->groups == 1 && (int64_t)d->C * d->R * d->S <= 16384;
}

static int conv_impl(const esb_conv_desc* d, const uint8_t* x, int nX, int kX_sig, const float* alphaX,
                     const uint8_t* w, int nW, int kW_sig, const float* alphaW, int32_t* acc, float* y,
                     void* ws, size_t ws_bytes, void* stream, const esb_post* post = nullptr) {
    if (!d || !valid_fmt(nX, kX_sig) || !valid_fmt(nW, kW_sig)) return ESB_E_INVALID;
    if (!post_ok(post, alphaX, alphaW)) return ESB_E_INVALID;
    if (!acc && !y && !(post && (post->codes || post->absmax_out))) return ESB_E_INVALID;
    const Post P = make_post(post);
    const Post* pp = post ? &P : nullptr;
    if (y && (!alphaX || !alphaW)) return ESB_E_INVALID;
    ConvGeom g;
    int64_t Mrows = 0, kred = 0;
    if (conv_geom(d, &g, &Mrows, &kred) != ESB_OK) return ESB_E_INVALID;
    const int Kg = d->K / d->groups;
    if (Mrows > 0 && (!x || !w)) return ESB_E_INVALID;
    const Fmt fx = make_fmt(nX, kX_sig), fw = make_fmt(nW, kW_sig);
    const int st = contraction_contract(kred, fx, fw);
    if (st) return st;
    if (ws && ws_bytes < esb_conv2d_workspace_size(d, nX, kX_sig, nW, kW_sig)) return ESB_E_WORKSPACE;
    if (Mrows == 0) return ESB_OK;
    const hipStream_t s = (hipStream_t)stream;
    if (conv_is_depthwise(d))
        return hip_status(launch_dwconv(g, x, fx, alphaX, w, fw, alphaW, acc, y, s, pp));
    const int op = mma_choose(fx, fw, kred);
    if (conv3x3_fits(g, d->K, d->groups, op, x, w))
        return hip_status(launch_conv3x3(g, d->K, x, fx, alphaX, w, fw, alphaW, acc, y, s, pp));
    const bool f4 = mma_f4ok(fx, fw, kred) && g.Cg % 32 == 0;
    const bool f6 = !f4 && mma_f6ok(fx, fw, kred) && g.Cg % 64 == 0 && mma_f6_tiles(Mrows, Kg, d->groups);
    const bool fits = mma_fits(g, x, kred, d->groups, w, kred, ESB_B_NK);
    const int64_t xel = (int64_t)d->N * d->H * d->W * d->C, wel = (int64_t)d->K * kred;
    if (ws && fits && (f4 || op == 1) && pre_worth(Mrows, d->K, kred, xel, wel))
        return hip_status(launch_mma_pre((int)Mrows, Kg, (int)kred, d->groups, g, x,
                                         (int64_t)d->N * d->H * d->W, d->C, d->C, fx, alphaX, w, d->K,
                                         kred, fw, alphaW, acc, y, d->K, f4 ? 1 : (f6 ? 2 : 0), ws, nullptr,
                                         false, s, pp));
    if (op >= 0 && fits)
        return hip_status(launch_mma(op, (int)Mrows, Kg, (int)kred, d->groups, g, x, fx, alphaX, w,
                                     kred, fw, alphaW, acc, y, d->K, nullptr, s, pp));
    return hip_status(launch_contraction((int)Mrows, Kg, (int)kred, d->groups, g, x, decode_info(fx),
                                         alphaX, w, kred, ESB_B_NK, decode_info(fw), alphaW, acc, y,
                                         d->K, Kg, s, pp));
}

size_t esb_conv2d_workspace_size(const esb_conv_desc* d, int nX, int kX_sig, int nW, int kW_sig) {
    if (!valid_fmt(nX, kX_sig) || !valid_fmt(nW, kW_sig)) return 0;
    ConvGeom g;
    int64_t Mrows = 0, kred = 0;
    if (conv_geom(d, &g, &Mrows, &kred) != ESB_OK || conv_is_depthwise(d)) return 0;
    const Fmt fx = make_fmt(nX, kX_sig), fw = make_fmt(nW, kW_sig);
    if (mma_choose(fx, fw, kred) != 1 && !(mma_f4ok(fx, fw, kred) && g.Cg % 32 == 0)) return 0;
    return mma_pre_workspace((int64_t)d->N * d->H * d->W, d->C, d->K, kred);
}

int esb_conv2d(const esb_conv_desc* d, const uint8_t* x, int nX, int kX_sig, const float* alphaX,
               const uint8_t* w, int nW, int kW_sig, const float* alphaW, int32_t* acc, float* y,
               void* stream) {
    return conv_impl(d, x, nX, kX_sig, alphaX, w, nW, kW_sig, alphaW, acc, y, nullptr, 0, stream);
}

int esb_conv2d_ws(const esb_conv_desc* d, const uint8_t* x, int nX, int kX_sig, const float* alphaX,
                  const uint8_t* w, int nW, int kW_sig, const float* alphaW, int32_t* acc, float* y,
                  void* workspace, size_t ws_bytes, void* stream) {
    return conv_impl(d, x, nX, kX_sig, alphaX, w, nW, kW_sig, alphaW, acc, y, workspace, ws_bytes,
                     stream);
}

int esb_gemm_post(int M, int N, int K, const uint8_t* A, int64_t lda, int nA, int kA_sig,
                  const float* alphaA, const uint8_t* B, int64_t ldb, int nB, int kB_sig,
                  const float* alphaB, int b_layout, int32_t* acc, float* y, int64_t ldc,
                  const esb_post* post, void* workspace, size_t ws_bytes, void* stream) {
    return gemm_impl(M, N, K, A, lda, nA, kA_sig, alphaA, B, ldb, nB, kB_sig, alphaB, b_layout, acc, y,
                     ldc, workspace, ws_bytes, stream, post);
}

int esb_conv2d_post(const esb_conv_desc* d, const uint8_t* x, int nX, int kX_sig,
                    const float* alphaX, const uint8_t* w, int nW, int kW_sig,
                    const float* alphaW, int32_t* acc, float* y, const esb_post* post,
                    void* workspace, size_t ws_bytes, void* stream) {
    return conv_impl(d, x, nX, kX_sig, alphaX, w, nW, kW_sig, alphaW, acc, y, workspace, ws_bytes,
                     stream, post);
}


// Pooled output size of the fused convolution + ReLU + max pool (0 on error).
static int pool_dims(const ConvGeom& g, int pool_r, int pool_stride, int pool_pad, int* PP, int* QQ) {
    if (pool_r < 1 || pool_stride < 1 || pool_pad < 0 || pool_pad >= pool_r) return 0;
    if (g.P + 2 * pool_pad < pool_r || g.Q + 2 * pool_pad < pool_r) return 0;
    *PP = (g.P + 2 * pool_pad - pool_r) / pool_stride + 1;
    *QQ = (g.Q + 2 * pool_pad - pool_r) / pool_stride + 1;
    return 1;
}

size_t esb_conv2d_relu_maxpool_workspace_size(const esb_conv_desc* d, int nX, int kX_sig, int nW,
                                              int kW_sig, int pool_window, int pool_stride,
                                              int pool_pad) {
    if (!valid_fmt(nX, kX_sig) || !valid_fmt(nW, kW_sig)) return 0;
    ConvGeom g;
    int64_t Mrows = 0, kred = 0;
    if (conv_geom(d, &g, &Mrows, &kred) != ESB_OK) return 0;
    int PP = 0, QQ = 0;
    if (!pool_dims(g, pool_window, pool_stride, pool_pad, &PP, &QQ)) return 0;
    const Fmt fx = make_fmt(nX, kX_sig), fw = make_fmt(nW, kW_sig);
    // the fused kernel needs none
    if (stem_fits(g, d->K, d->groups, fx, fw, pool_window, pool_stride, pool_pad)) return 0;
    const auto al = [](size_t v) { return (v + 255) & ~(size_t)255; };
    return al((size_t)Mrows * (size_t)d->K * sizeof(float)) +
           al((size_t)d->N * PP * QQ * (size_t)d->K * sizeof(float));
}

int esb_conv2d_relu_maxpool(const esb_conv_desc* d, const uint8_t* x, int nX, int kX_sig,
                            const float* alphaX, const uint8_t* w, int nW, int kW_sig,
                            const float* alphaW, const esb_post* post, int pool_window,
                            int pool_stride, int pool_pad, float* y, void* workspace,
                            size_t ws_bytes, void* stream) {
    if (!d || !valid_fmt(nX, kX_sig) || !valid_fmt(nW, kW_sig) || !alphaX || !alphaW) return ESB_E_INVALID;
    if (!post || !post->relu || post->residual) return ESB_E_INVALID;
    if (!post_ok(post, alphaX, alphaW)) return ESB_E_INVALID;
    if (!y && !post->codes && !post->absmax_out) return ESB_E_INVALID;
    ConvGeom g;
    int64_t Mrows = 0, kred = 0;
    if (conv_geom(d, &g, &Mrows, &kred) != ESB_OK) return ESB_E_INVALID;
    int PP = 0, QQ = 0;
    if (!pool_dims(g, pool_window, pool_stride, pool_pad, &PP, &QQ)) return ESB_E_INVALID;
    if (Mrows > 0 && (!x || !w)) return ESB_E_INVALID;
    const Fmt fx = make_fmt(nX, kX_sig), fw = make_fmt(nW, kW_sig);
    const int st = contraction_contract(kred, fx, fw);
    if (st) return st;
    const hipStream_t s = (hipStream_t)stream;
    const Post P = make_post(post);
    if (stem_fits(g, d->K, d->groups, fx, fw, pool_window, pool_stride, pool_pad)) {
        if (Mrows == 0) return ESB_OK;
        return hip_status(launch_stem(g, x, fx, alphaX, w, fw, alphaW, y, PP, QQ, P, s));
    }
    // elsewhere: the convolution with its post-processing into the workspace, the pool, then
    // the codes and the maximum of the pooled values
    const size_t need = esb_conv2d_relu_maxpool_workspace_size(d, nX, kX_sig, nW, kW_sig,
                                                                pool_window, pool_stride, pool_pad);
    if (!workspace || ws_bytes < need) return ESB_E_WORKSPACE;
    if (Mrows == 0) return ESB_OK;
    const auto al = [](size_t v) { return (v + 255) & ~(size_t)255; };
    float* conv_out = (float*)workspace;
    float* pooled = y ? y : (float*)((char*)workspace + al((size_t)Mrows * (size_t)d->K * sizeof(float)));
    esb_post inner = *post;
    inner.codes = nullptr;
    inner.alpha = nullptr;
    inner.absmax_out = nullptr;
    int rc = conv_impl(d, x, nX, kX_sig, alphaX, w, nW, kW_sig, alphaW, nullptr, conv_out, nullptr, 0,
                       stream, &inner);
    if (rc) return rc;
    PoolGeom pg;
    pg.N = d->N; pg.H = g.P; pg.W = g.Q; pg.C = d->K; pg.R = pool_window; pg.S = pool_window;
    pg.sh = pool_stride; pg.sw = pool_stride; pg.ph = pool_pad; pg.pw = pool_pad; pg.P = PP; pg.Q = QQ;
    hipError_t e = launch_maxpool(conv_out, pg, pooled, s);
    const int64_t npool = (int64_t)d->N * PP * QQ * d->K;
    if (e == hipSuccess && post->codes)
        e = launch_project(pooled, npool, post->alpha, make_fmt(post->n, post->k_sig), post->codes,
                           nullptr, s);
    if (e == hipSuccess && post->absmax_out) e = launch_absmax(pooled, npool, post->absmax_out, s);
    return hip_status(e);
}

// ------------------------------------------------------------ packed codes
static bool packable(const Fmt& f) { return f.ebits <= 2 && f.k <= 1; }   // inside OCP E2M1

size_t esb_pack_size(int rows, int K, int n, int k_sig) {
    if (!valid_fmt(n, k_sig) || rows < 0 || K <= 0 || K % 32 != 0) return 0;
    if (!packable(make_fmt(n, k_sig))) return 0;
    return (size_t)rows * (size_t)(K / 2);
}

int esb_pack(const uint8_t* codes, int rows, int K, int64_t ld, int n, int k_sig, uint8_t* packed,
             void* stream) {
    if (!valid_fmt(n, k_sig) || rows < 0 || K <= 0 || ld < K) return ESB_E_INVALID;
    const Fmt f = make_fmt(n, k_sig);
    if (!packable(f) || K % 32 != 0) return ESB_E_UNSUPPORTED;
    if (rows == 0) return ESB_OK;
    if (!codes || !packed || (uintptr_t)codes % 16 != 0 || ld % 16 != 0 || (uintptr_t)packed % 16 != 0)
        return ESB_E_INVALID;
    return hip_status(launch_pack_fp4(codes, rows, K, ld, f, packed, (hipStream_t)stream));
}

size_t esb_gemm_packed_workspace_size(int M, int N, int K, int nA, int kA_sig, int nB, int kB_sig) {
    if (!valid_fmt(nA, kA_sig) || !valid_fmt(nB, kB_sig) || M < 0 || N < 0 || K <= 0) return 0;
    const Fmt fa = make_fmt(nA, kA_sig), fb = make_fmt(nB, kB_sig);
    if (!mma_f4ok(fa, fb, K) || K % 32 != 0) return 0;
    const auto al = [](size_t v) { return (v + 255) & ~(size_t)255; };
    size_t need = al((size_t)M * (size_t)(K / 2));            // A, packed per call
    int kc = K;
    const int ks = mma_splitk(M, N, K, &kc);
    // skinny shapes: the reduction split over the waves of one workgroup (no
    // partial sums in memory) when that fills the chip, else over workgroups
    if (ks > 1 && !fc_f4_fits(M, N, K)) need += (size_t)ks * (size_t)M * (size_t)N * sizeof(int32_t);
    return need > 0 ? need : 1;
}

int esb_gemm_packed(int M, int N, int K, const uint8_t* A, int64_t lda, int nA, int kA_sig,
                    const float* alphaA, const uint8_t* B_packed, int nB, int kB_sig,
                    const float* alphaB, int32_t* acc, float* y, int64_t ldc, void* workspace,
                    size_t ws_bytes, void* stream) {
    if (!valid_fmt(nA, kA_sig) || !valid_fmt(nB, kB_sig)) return ESB_E_INVALID;
    if (M < 0 || N < 0 || K <= 0 || lda < K || ldc < N) return ESB_E_INVALID;
    if (!acc && !y) return ESB_E_INVALID;
    if (y && (!alphaA || !alphaB)) return ESB_E_INVALID;
    const Fmt fa = make_fmt(nA, kA_sig), fb = make_fmt(nB, kB_sig);
    if (!packable(fa) || !packable(fb) || K % 32 != 0) return ESB_E_UNSUPPORTED;
    const int st = contraction_contract(K, fa, fb);
    if (st) return st;
    if (!mma_f4ok(fa, fb, K)) return ESB_E_OVERFLOW;   // fp32 sums exact only below 2^24
    const size_t need = esb_gemm_packed_workspace_size(M, N, K, nA, kA_sig, nB, kB_sig);
    if (!workspace || ws_bytes < need) return ESB_E_WORKSPACE;
    if (M == 0 || N == 0) return ESB_OK;
    if (!A || !B_packed || (uintptr_t)A % 16 != 0 || lda % 16 != 0 || (uintptr_t)B_packed % 16 != 0)
        return ESB_E_INVALID;
    if (lda > 0x7fffffff) return ESB_E_INVALID;
    ConvGeom g;
    g.Nb = M; g.H = 1; g.W = 1; g.C = K; g.pitch = (int)lda;
    g.Cg = K; g.R = 1; g.S = 1; g.sh = 1; g.sw = 1; g.ph = 0; g.pw = 0; g.P = 1; g.Q = 1;
    if (fc_f4_fits(M, N, K)) {
        uint8_t* dA = (uint8_t*)workspace;   // A packed like B, rows of K/2 bytes
        hipError_t e = launch_pack_fp4(A, M, K, lda, fa, dA, (hipStream_t)stream);
        if (e == hipSuccess)
            e = launch_fc_f4(M, N, K, dA, K / 2, B_packed, K / 2, fa.k, fb.k, alphaA, alphaB, acc, y,
                             ldc, (hipStream_t)stream);
        return hip_status(e);
    }
    return hip_status(launch_mma_pre(M, N, K, 1, g, A, M, K, lda, fa, alphaA, nullptr, N, K / 2, fb,
                                     alphaB, acc, y, ldc, 1, workspace, B_packed, true,
                                     (hipStream_t)stream));
}

// ------------------------------------------- normalization and analytic DDA
size_t esb_dn_workspace_size(int64_t len) { return len < 0 ? 0 : dn_workspace(len); }

int esb_dn_stats(const float* x, int64_t len, float* stats_out, void* workspace, size_t ws_bytes,
                 void* stream) {
    if (len < 0 || !stats_out || (len > 0 && !x)) return ESB_E_INVALID;
    if (!workspace || ws_bytes < dn_workspace(len)) return ESB_E_WORKSPACE;
    return hip_status(launch_dn_stats(x, len, stats_out, workspace, (hipStream_t)stream));
}

int esb_project_dn(const float* x, int64_t len, const float* stats, const float* alpha, int n,
                   int k_sig, uint8_t* codes, void* stream) {
    if (!valid_fmt(n, k_sig) || len < 0 || !alpha || !stats) return ESB_E_INVALID;
    if (len > 0 && (!x || !codes)) return ESB_E_INVALID;
    return hip_status(launch_project(x, len, alpha, make_fmt(n, k_sig), codes, stats,
                                     (hipStream_t)stream));
}

int esb_dda_normal(int n, int k_sig, const float* grid, int G, float* alpha_out, double* D_out,
                   double* dD_out, void* stream) {
    if (!valid_fmt(n, k_sig) || G < 1 || !grid || !alpha_out || !D_out) return ESB_E_INVALID;
    return hip_status(launch_dda_normal(make_fmt(n, k_sig), grid, G, alpha_out, D_out,
                                        dD_out, (hipStream_t)stream));
}

}  // extern "C"
