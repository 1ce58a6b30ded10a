/*
 * ESB oracle: a plain, slow, obviously-correct CPU implementation of the
 * elastic-significant-bit (ESB) hot path of Gong et al., "Elastic Significant
 * Bit Quantization and Acceleration for Deep Neural Networks" (IEEE TPDS 2021).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  The GPU product path
 * (libesb) shares no code, header, table or constant with it.
 *
 * Conventions (readings of the paper, fixed here and in libesb alike):
 *   - b = total bits, k_sig = number of significant bits; the paper's k
 *     (fraction bits) is k = k_sig - 1 (Sec. 3.2, eq. (4)-(5): Omega_i holds
 *     numbers with at most k+1 significant bits).
 *   - Projection of fp32 x with fp32 scale alpha: v = fl32(x / alpha) (IEEE
 *     binary32 division, round-to-nearest-even), clipped to [-C, C], then
 *     rounded to the nearest set value with ties going to the larger magnitude
 *     (eq. (6) uses half-open intervals [lo, hi)), symmetric for negatives.
 *     Below 1 the step is xi_0 = 2^-k (eq. (5)), i.e. the binade exponent used
 *     by the shift-round form (eq. (7)) is clamped at 0.
 *   - NaN input, or an alpha that is not a positive finite number, projects
 *     to +0.  Zero is always encoded with sign bit 0.
 *   - Code layout (eq. (14)): sign | exponent (b-k-1 bits) | fraction (k bits),
 *     most significant first; the all-ones exponent is the subnormal binade
 *     (value 0.f), any other exponent e gives 2^e * 1.f.
 *   - Code bits above bit b-1 are ignored.
 *
 * Every function below cites the passage it follows.  Parity pins for this
 * file live in the CPU test-suite (paper values, closed forms, brute force).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ESO_OK 0
#define ESO_E_INVALID (-1)
#define ESO_E_OVERFLOW (-3)
#define ESO_E_UNSUPPORTED (-4)

static int valid_bk(int b, int k_sig) {
    return b >= 2 && b <= 8 && k_sig >= 1 && k_sig <= b - 1;
}

int eso_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* N = 2^(b-k-1) - 1, eq. (4). */
int eso_N(int b, int k_sig) {
    if (!valid_bk(b, k_sig)) return -1;
    int k = k_sig - 1;
    return (1 << (b - k - 1)) - 1;
}

/* C = max(xi_N * Omega_N), eq. (6): the largest unscaled set value. */
double eso_C(int b, int k_sig) {
    int k = k_sig - 1, N = eso_N(b, k_sig);
    if (N == 0) return 0.0;
    return ldexp((double)((1 << (k + 1)) - 1), N - k - 1);
}

static int cmp_double(const void* a, const void* b) {
    double x = *(const double*)a, y = *(const double*)b;
    return (x > y) - (x < y);
}

/*
 * Non-negative part Q*_e of the value set, eq. (4)-(5): the union over
 * i = 0..N of xi_i * Omega_i with Omega_0 = {0..2^k-1}, Omega_i = {2^k..2^(k+1)-1}
 * for i > 0, xi_0 = 2^-k and xi_i = 2^(i-k-1).  Written ascending, duplicates
 * removed; returns the count (2^(b-1)) or -1.
 */
int eso_valueset(int b, int k_sig, double* out, int cap) {
    if (!valid_bk(b, k_sig)) return -1;
    int k = k_sig - 1, N = eso_N(b, k_sig);
    int total = 0;
    double* tmp = (double*)malloc(sizeof(double) * (size_t)(1 << b));
    for (int i = 0; i <= N; i++) {
        double xi = (i == 0) ? ldexp(1.0, -k) : ldexp(1.0, i - k - 1);
        int lo = (i == 0) ? 0 : (1 << k);
        int hi = (i == 0) ? (1 << k) - 1 : (1 << (k + 1)) - 1;
        for (int w = lo; w <= hi; w++) tmp[total++] = (double)w * xi;
    }
    qsort(tmp, (size_t)total, sizeof(double), cmp_double);
    int n = 0;
    for (int i = 0; i < total; i++)
        if (n == 0 || tmp[i] != tmp[n - 1]) tmp[n++] = tmp[i];
    if (n > cap) { free(tmp); return -1; }
    memcpy(out, tmp, sizeof(double) * (size_t)n);
    free(tmp);
    return n;
}

/*
 * ESB float format, eq. (14): decode a b-bit code to its unscaled value.
 * sb = sign, e = exponent field, f = fraction field; e = 2^(b-k-1)-1 marks
 * the subnormal binade (value 0.f), otherwise the value is 2^e * 1.f.
 */
double eso_decode(int code, int b, int k_sig) {
    int k = k_sig - 1;
    int ebits = b - k - 1;
    int emax = (1 << ebits) - 1;
    code &= (1 << b) - 1;
    int sb = (code >> (b - 1)) & 1;
    int e = (code >> k) & emax;
    int f = code & ((1 << k) - 1);
    double mag;
    if (e == emax) mag = ldexp((double)f, -k);                 /* 0.f   */
    else mag = ldexp((double)((1 << k) + f), e - k);            /* 2^e*1.f */
    return sb ? -mag : mag;
}

/*
 * Inverse of eq. (14) on set members.  Returns the code, or -1 if q is not a
 * member of the (signed) set.  Zero always gets sign bit 0.
 */
int eso_encode(double q, int b, int k_sig) {
    if (!valid_bk(b, k_sig)) return -1;
    int k = k_sig - 1, N = eso_N(b, k_sig);
    int sb = q < 0.0;
    double a = fabs(q);
    int e;
    double f;
    if (a < 1.0) {
        e = N;
        f = ldexp(a, k);
    } else {
        int ex;
        frexp(a, &ex);
        e = ex - 1;                       /* floor(log2 a) */
        if (e > N - 1) return -1;
        f = ldexp(ldexp(a, -e) - 1.0, k);
    }
    if (f != floor(f) || f < 0 || f >= (double)(1 << k)) return -1;
    if (a == 0.0) sb = 0;
    return (sb << (b - 1)) | (e << k) | (int)f;
}

/* fl32(x / alpha) and the validity rule shared by projection and DDA. */
static int alpha_ok(float alpha) { return alpha > 0.0f && !isinf(alpha); }

/*
 * Projection of one element, eq. (7)-(8) with the readings above:
 * v = fl32(x/alpha); clip |v| to C; keep k+1 significant bits of |v| with
 * the binade exponent E = max(floor(log2|v|), 0), rounding half up in
 * magnitude; restore the sign.  Returns the signed unscaled value q.
 */
double eso_project_value(float x, float alpha, int b, int k_sig) {
    if (isnan(x) || !alpha_ok(alpha)) return 0.0;
    int k = k_sig - 1;
    float v = x / alpha;
    double a = fabs((double)v);
    double C = eso_C(b, k_sig);
    double q;
    if (a >= C) {
        q = C;
    } else {
        int E = 0;
        if (a >= 1.0) { int ex; frexp(a, &ex); E = ex - 1; }
        double h = ldexp(1.0, E - k);     /* step of the binade, xi_i */
        double t = a / h;                 /* exact: h is a power of two */
        double m = floor(t);
        if (t - m >= 0.5) m += 1.0;
        q = m * h;
    }
    if (q == 0.0) return 0.0;
    return (v < 0.0f) ? -q : q;
}

/*
 * Brute-force nearest neighbour, eq. (6): the member of Q*_e closest to
 * |fl32(x/alpha)|, ties to the larger member, sign restored.  Independent of
 * eso_project_value; used only to pin it.
 */
double eso_project_bruteforce(float x, float alpha, int b, int k_sig) {
    if (isnan(x) || !alpha_ok(alpha)) return 0.0;
    double vals[128];
    int n = eso_valueset(b, k_sig, vals, 128);
    float v = x / alpha;
    double a = fabs((double)v);
    double best = vals[0], bestd = INFINITY;
    for (int i = 0; i < n; i++) {
        double d = fabs(a - vals[i]);
        if (d <= bestd) { bestd = d; best = vals[i]; }   /* ascending: ties go up */
    }
    if (best == 0.0) return 0.0;
    return (v < 0.0f) ? -best : best;
}

/* Projection operator Pi, eq. (8), emitting eq. (14) codes. */
int eso_project(const float* x, int64_t n, float alpha, int b, int k_sig, uint8_t* codes) {
    if (!valid_bk(b, k_sig) || n < 0) return ESO_E_INVALID;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++)
        codes[i] = (uint8_t)eso_encode(eso_project_value(x[i], alpha, b, k_sig), b, k_sig);
    return ESO_OK;
}

/* Brute-force projection of a whole array (pin for eso_project). */
int eso_project_bf(const float* x, int64_t n, float alpha, int b, int k_sig, uint8_t* codes) {
    if (!valid_bk(b, k_sig) || n < 0) return ESO_E_INVALID;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++)
        codes[i] = (uint8_t)eso_encode(eso_project_bruteforce(x[i], alpha, b, k_sig), b, k_sig);
    return ESO_OK;
}

/* Dequantization: fl32(alpha * q) for each code (eq. (8): alpha * P(v)). */
int eso_dequantize(const uint8_t* codes, int64_t n, float alpha, int b, int k_sig, float* out) {
    if (!valid_bk(b, k_sig) || n < 0) return ESO_E_INVALID;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++)
        out[i] = (float)((double)alpha * eso_decode(codes[i], b, k_sig));
    return ESO_OK;
}

/*
 * Distribution difference aligner on data, eq. (9) and (13) with the
 * empirical distribution of x in place of p: for every candidate alpha_j,
 *   D_j = sum_i (x_i - alpha_j * q_j(x_i))^2,
 * q_j the projection under alpha_j.  Summed in long double.  Candidates that
 * are not positive finite numbers get D_j = NaN.  Returns j* = the smallest
 * index with the least D (NaN ranks above +Inf).
 */
int eso_dda(const float* x, int64_t n, int b, int k_sig, const float* grid, int G, double* D) {
    if (!valid_bk(b, k_sig) || n < 0 || G < 1) return ESO_E_INVALID;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int j = 0; j < G; j++) {
        float al = grid[j];
        if (!alpha_ok(al)) { D[j] = NAN; continue; }
        long double s = 0.0L;
        for (int64_t i = 0; i < n; i++) {
            double q = eso_project_value(x[i], al, b, k_sig);
            long double r = (long double)x[i] - (long double)al * (long double)q;
            s += r * r;
        }
        D[j] = (double)s;
    }
    int best = 0;
    for (int j = 1; j < G; j++)
        if (D[j] < D[best] || (isnan(D[best]) && !isnan(D[j]))) best = j;
    return best;
}

/*
 * Analytic eq. (9) for p = N(0,1) (Sec. 3.4, "Resolving extremum"): the
 * one-sided expected squared projection error over t >= 0 with
 * nearest-neighbour cells and the top cell open to +inf.
 *   int_lo^hi (t-q)^2 phi = M2 - 2 q M1 + q^2 M0,
 *   M0 = Phi(hi)-Phi(lo), M1 = phi(lo)-phi(hi), M2 = M0 + lo phi(lo) - hi phi(hi).
 */
static double nphi(double t) { return isinf(t) ? 0.0 : exp(-0.5 * t * t) / sqrt(2.0 * M_PI); }
static double nPhi_upper(double t) { return isinf(t) ? 0.0 : 0.5 * erfc(t / sqrt(2.0)); }

double eso_dda_normal(double alpha, int b, int k_sig) {
    double vals[128];
    int n = eso_valueset(b, k_sig, vals, 128);
    if (n < 0 || !(alpha > 0)) return NAN;
    double D = 0.0;
    for (int c = 0; c < n; c++) {
        double q = alpha * vals[c];
        double lo = (c == 0) ? 0.0 : 0.5 * alpha * (vals[c - 1] + vals[c]);
        double hi = (c == n - 1) ? INFINITY : 0.5 * alpha * (vals[c] + vals[c + 1]);
        double M0 = nPhi_upper(lo) - nPhi_upper(hi);
        double M1 = nphi(lo) - nphi(hi);
        double M2 = M0 + lo * nphi(lo) - (isinf(hi) ? 0.0 : hi * nphi(hi));
        D += M2 - 2.0 * q * M1 + q * q * M0;
    }
    return D;
}

/*
 * Derivative dD/dalpha of the analytic objective above (the quantity whose
 * zeros Sec. 3.4, "Resolving extremum", looks for).  Each cell's integrand
 * (t - alpha q_c)^2 phi(t) depends on alpha through alpha q_c and through the
 * cell ends alpha m_c; at an end shared by two nearest-neighbour cells the two
 * integrands are equal (the end is the midpoint), so the moving ends cancel and
 *   dD/dalpha = -2 sum_c q_c (M1_c - alpha q_c M0_c).
 */
double eso_dda_normal_deriv(double alpha, int b, int k_sig) {
    double vals[128];
    int n = eso_valueset(b, k_sig, vals, 128);
    if (n < 0 || !(alpha > 0)) return NAN;
    double d = 0.0;
    for (int c = 0; c < n; c++) {
        double lo = (c == 0) ? 0.0 : 0.5 * alpha * (vals[c - 1] + vals[c]);
        double hi = (c == n - 1) ? INFINITY : 0.5 * alpha * (vals[c] + vals[c + 1]);
        double M0 = nPhi_upper(lo) - nPhi_upper(hi);
        double M1 = nphi(lo) - nphi(hi);
        d += -2.0 * vals[c] * (M1 - alpha * vals[c] * M0);
    }
    return d;
}

/*
 * Data normalization, Sec. 3.4 ("Normalization", the DN equation): the mean
 * and the population standard deviation sqrt((1/d) sum (x - mu)^2), two passes
 * in long double.  n == 0 gives NaN for both.
 */
int eso_dn_stats(const float* x, int64_t n, double* mean, double* std) {
    if (n < 0) return ESO_E_INVALID;
    if (n == 0) { *mean = NAN; *std = NAN; return ESO_OK; }
    long double s = 0.0L;
    for (int64_t i = 0; i < n; i++) s += (long double)x[i];
    const long double mu = s / (long double)n;
    long double v = 0.0L;
    for (int64_t i = 0; i < n; i++) {
        const long double d = (long double)x[i] - mu;
        v += d * d;
    }
    *mean = (double)mu;
    *std = (double)sqrtl(v / (long double)n);
    return ESO_OK;
}

/*
 * Projection of normalized data (Alg. 1: ESB(DN(W))), in binary32 with the
 * given statistics (binary32 too) and epsilon = 1e-7 of the DN equation:
 *   xh = fl32( fl32(x - mean) / fl32(std + fl32(1e-7)) ),   code = Pi(xh)
 * with the projection of eso_project under alpha.
 */
int eso_project_dn(const float* x, int64_t n, float mean, float std, float alpha, int b, int k_sig,
                   uint8_t* codes) {
    if (!valid_bk(b, k_sig) || n < 0) return ESO_E_INVALID;
    volatile float eps = 1e-7f;
    const float den = std + eps;
    for (int64_t i = 0; i < n; i++) {
        volatile float d = x[i] - mean;
        const float xh = d / den;
        codes[i] = (uint8_t)eso_encode(eso_project_value(xh, alpha, b, k_sig), b, k_sig);
    }
    return ESO_OK;
}

/*
 * Post-processing of a contraction output (Sec. 4.2, the "BN and DN" step of
 * eq. (16) folded into a per-channel a x + b, then the "ESB quantization"
 * step): for the scaled output y of row i, channel j (row-major, pitch ld),
 *   z = fma(a_j, y, b_j)            one rounding; a_j = 1, b_j = 0 when absent,
 *   z = fl32(z + res_ij)            when a residual is given,
 *   z = z > 0 ? z : 0               when relu (NaN gives 0),
 *   code = projection of z with alpha (eq. (6)-(8)),
 * writing z to z_out and the code to codes_out (either may be NULL).
 */
int eso_post(const float* y, int64_t rows, int64_t cols, int64_t ld, const float* a,
             const float* bias, const float* res, int relu, float alpha, int b, int k_sig,
             float* z_out, uint8_t* codes_out) {
    if (!valid_bk(b, k_sig) || rows < 0 || cols < 0 || ld < cols) return ESO_E_INVALID;
    for (int64_t i = 0; i < rows; i++)
        for (int64_t j = 0; j < cols; j++) {
            const int64_t o = i * ld + j;
            float z = fmaf(a ? a[j] : 1.0f, y[o], bias ? bias[j] : 0.0f);
            if (res) z = z + res[o];
            if (relu) z = z > 0.0f ? z : 0.0f;
            if (z_out) z_out[o] = z;
            if (codes_out)
                codes_out[o] = (uint8_t)eso_encode(eso_project_value(z, alpha, b, k_sig), b, k_sig);
        }
    return ESO_OK;
}

/* Exact integer of a code: m = q * 2^k (eq. (14)-(15): fraction bits made integral). */
static int64_t code_int(int code, int b, int k_sig) {
    return (int64_t)ldexp(eso_decode(code, b, k_sig), k_sig - 1);
}

static double max_abs_int(int b, int k_sig) {
    return ldexp(eso_C(b, k_sig), k_sig - 1);
}

/* Contract of the contraction: the magnitude bound and the int32 bound. */
static int contraction_ok(int64_t Kred, int bA, int ksA, int bB, int ksB) {
    double MA = max_abs_int(bA, ksA), MB = max_abs_int(bB, ksB);
    if (MA > 32767.0 || MB > 32767.0) return ESO_E_UNSUPPORTED;
    if ((double)Kred * MA * MB > 2147483647.0) return ESO_E_OVERFLOW;
    return ESO_OK;
}

/* Output scale s = 2^-(kA+kB) * fl32(alphaA*alphaB), in binary32. */
static float out_scale(float alphaA, float alphaB, int ksA, int ksB) {
    float p = alphaA * alphaB;
    return ldexpf(p, -((ksA - 1) + (ksB - 1)));
}

/*
 * Dense contraction over codes (Sec. 4.2, Forward(A_q, W_q) with the
 * multiplication of eq. (15)): acc[i][j] = sum_k mA[i][k] * mB[k][j] in int64,
 * stored as int32, and y = fl32(s * fl32(acc)).
 * A: M x K row-major (lda).  B: layout 0 = N x K row-major (K contiguous),
 * layout 1 = K x N row-major.  acc / y may be NULL.
 */
int eso_gemm(int M, int N, int K,
             const uint8_t* A, int64_t lda, int bA, int ksA, float alphaA,
             const uint8_t* B, int64_t ldb, int bB, int ksB, float alphaB, int b_layout,
             int32_t* acc, float* y, int64_t ldc) {
    if (!valid_bk(bA, ksA) || !valid_bk(bB, ksB) || M < 0 || N < 0 || K < 0) return ESO_E_INVALID;
    int st = contraction_ok(K, bA, ksA, bB, ksB);
    if (st) return st;
    int64_t tA[256], tB[256];
    for (int c = 0; c < 256; c++) { tA[c] = code_int(c, bA, ksA); tB[c] = code_int(c, bB, ksB); }
    float s = out_scale(alphaA, alphaB, ksA, ksB);
    #pragma omp parallel for schedule(static)
    for (int i = 0; i < M; i++) {
        for (int j = 0; j < N; j++) {
            int64_t sum = 0;
            for (int kk = 0; kk < K; kk++) {
                uint8_t cb = b_layout == 0 ? B[(int64_t)j * ldb + kk] : B[(int64_t)kk * ldb + j];
                sum += tA[A[(int64_t)i * lda + kk]] * tB[cb];
            }
            if (acc) acc[(int64_t)i * ldc + j] = (int32_t)sum;
            if (y) y[(int64_t)i * ldc + j] = s * (float)(int32_t)sum;
        }
    }
    return ESO_OK;
}

/*
 * Convolution stage of Sec. 4.2 (op count h*w*K*K*c_in*c_out): direct
 * cross-correlation, NHWC codes x KRSC codes (C/groups channels per filter),
 * zero padding by value 0, strides sh/sw, pads ph/pw, groups.  Output NHWC
 * [N, P, Q, Kout] as int32 accumulators and/or scaled fp32.
 */
int eso_conv2d(int Nb, int H, int W, int C, int Kout, int R, int S,
               int sh, int sw, int ph, int pw, int groups,
               const uint8_t* x, int bX, int ksX, float alphaX,
               const uint8_t* w, int bW, int ksW, float alphaW,
               int32_t* acc, float* y) {
    if (!valid_bk(bX, ksX) || !valid_bk(bW, ksW)) return ESO_E_INVALID;
    if (Nb < 0 || H < 1 || W < 1 || C < 1 || Kout < 1 || R < 1 || S < 1 || sh < 1 || sw < 1 ||
        ph < 0 || pw < 0 || groups < 1 || C % groups || Kout % groups)
        return ESO_E_INVALID;
    int P = (H + 2 * ph - R) / sh + 1, Q = (W + 2 * pw - S) / sw + 1;
    if (H + 2 * ph < R || W + 2 * pw < S) return ESO_E_INVALID;
    int Cg = C / groups, Kg = Kout / groups;
    int st = contraction_ok((int64_t)R * S * Cg, bX, ksX, bW, ksW);
    if (st) return st;
    int64_t tX[256], tW[256];
    for (int c = 0; c < 256; c++) { tX[c] = code_int(c, bX, ksX); tW[c] = code_int(c, bW, ksW); }
    float s = out_scale(alphaX, alphaW, ksX, ksW);
    int64_t npix = (int64_t)Nb * P * Q;
    #pragma omp parallel for schedule(static)
    for (int64_t pix = 0; pix < npix; pix++) {
        int n = (int)(pix / ((int64_t)P * Q));
        int p = (int)((pix / Q) % P);
        int q = (int)(pix % Q);
        for (int ko = 0; ko < Kout; ko++) {
            int g = ko / Kg;
            int64_t sum = 0;
            for (int r = 0; r < R; r++) {
                int ih = p * sh - ph + r;
                if (ih < 0 || ih >= H) continue;
                for (int t = 0; t < S; t++) {
                    int iw = q * sw - pw + t;
                    if (iw < 0 || iw >= W) continue;
                    const uint8_t* xp = x + (((int64_t)n * H + ih) * W + iw) * C + (int64_t)g * Cg;
                    const uint8_t* wp = w + (((int64_t)ko * R + r) * S + t) * Cg;
                    for (int c = 0; c < Cg; c++) sum += tX[xp[c]] * tW[wp[c]];
                }
            }
            if (acc) acc[pix * Kout + ko] = (int32_t)sum;
            if (y) y[pix * Kout + ko] = s * (float)(int32_t)sum;
        }
    }
    return ESO_OK;
}
