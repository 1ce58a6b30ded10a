// Distribution difference aligner (eq. (9), (13)) on the data, gfx950.
//
// Objective per candidate scale alpha_j:  D_j = sum_i (|x_i| - alpha_j q_j(x_i))^2
//   = S2 - 2 alpha_j sum_i |x_i| q_j(x_i) + alpha_j^2 sum_i q_j(x_i)^2,
// with S2 = sum_i x_i^2.  q_j(x) depends on x only through which cell of
// candidate j holds |x|, and the cell boundaries are exact fp32 thresholds:
// T_{j,c} = the smallest fp32 X with fl32(X / alpha_j) >= mu_c, mu_c the
// midpoint between set values c-1 and c (ties go up, as in the projection).
// Sorting all G*M thresholds splits [0, inf) into "atoms"; every candidate's
// cell is a union of consecutive atoms.  So one pass over x suffices:
//   1. setup (1 block): thresholds by bisection over bit patterns, bitonic
//      sort, atom ranks, and a bin table over the threshold bit range;
//   2. histogram (<= 256 blocks): per element find its atom (bin lookup +
//      short scan), add (count, |x| in fixed point) to an LDS histogram with
//      integer atomics, accumulate x^2 in fp64; the unbounded top atom sums
//      |x| in fp64; per-block partials go to the workspace;
//   3. reduce: per atom, sum the partials over blocks (integers, exact);
//   4. finalize (1 block): per candidate, walk the atoms with the cell index,
//      A_j = sum Q_c S1, B_j = sum Q_c^2 S0, D_j = S2 + a (a B_j - 2 A_j),
//      then the argmin with ties to the lowest index.
// Fixed point: an atom [U_a, U_{a+1}) is bounded with U_{a+1} <= 3 U_a + ulps
// (neighbouring midpoints differ by at most a factor 3), so |x| / ulp(U_a) is
// an integer below 2^26 and a uint64 per atom holds >= 2^38 elements exactly.
// Everything is integer or fixed-order fp64: the result is deterministic.
#include "esb_internal.h"

namespace esb {

struct DdaArgs {
    float mids[128];   // mu_c, c = 1..M (index c-1)
    float q[128];      // Q_c, c = 0..M (unscaled values, ascending)
    int G, M, A, nblk;
};

struct DdaWs {   // pointers into the caller's workspace
    uint32_t* ubits;   // [A+2]: 0, sorted threshold bits (1..A), 0xffffffff
    int32_t* rank;     // [G*M]: atom index where cell c of candidate j starts
    uint32_t* bins;    // [kDdaBins]: first atom of each bin
    uint32_t* meta;    // lo, shift, nbins, A_fin, hi
    uint32_t* pcnt;    // [nblk][A+1]
    uint64_t* psum;    // [nblk][A+1]
    double* pscal;     // [nblk][4]: sum x^2, top-atom sum |x|, top count, flags
    double* s0;        // [A+1]
    double* s1;        // [A+1]
};

static DdaWs ws_ptrs(void* ws, const DdaLayout& L) {
    char* b = (char*)ws;
    DdaWs w;
    w.ubits = (uint32_t*)(b + L.off_ubits);
    w.rank = (int32_t*)(b + L.off_rank);
    w.bins = (uint32_t*)(b + L.off_bins);
    w.meta = (uint32_t*)(b + L.off_meta);
    w.pcnt = (uint32_t*)(b + L.off_pcnt);
    w.psum = (uint64_t*)(b + L.off_psum);
    w.pscal = (double*)(b + L.off_pscal);
    w.s0 = (double*)(b + L.off_s0);
    w.s1 = (double*)(b + L.off_s1);
    return w;
}

static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

bool dda_layout(int64_t len, const Fmt& f, int G, DdaLayout* L) {
    const int M = (1 << (f.n - 1)) - 1;
    if (G < 1 || G > kDdaMaxG || (int64_t)G * M > kDdaMaxThresholds || len < 0) return false;
    L->G = G;
    L->M = M;
    L->A = G * M;
    int64_t nb = (len + 16383) / 16384;
    L->nblk = (int)(nb < 1 ? 1 : (nb > kDdaMaxBlocks ? kDdaMaxBlocks : nb));
    const size_t A1 = (size_t)L->A + 1;
    size_t o = 0;
    L->off_ubits = o; o = align256(o + sizeof(uint32_t) * (A1 + 1));
    L->off_rank = o;  o = align256(o + sizeof(int32_t) * (size_t)L->A);
    L->off_bins = o;  o = align256(o + sizeof(uint32_t) * kDdaBins);
    L->off_meta = o;  o = align256(o + sizeof(uint32_t) * 8);
    L->off_pcnt = o;  o = align256(o + sizeof(uint32_t) * A1 * L->nblk);
    L->off_psum = o;  o = align256(o + sizeof(uint64_t) * A1 * L->nblk);
    L->off_pscal = o; o = align256(o + sizeof(double) * 4 * L->nblk);
    L->off_s0 = o;    o = align256(o + sizeof(double) * A1);
    L->off_s1 = o;    o = align256(o + sizeof(double) * A1);
    L->total = o;
    return true;
}

__device__ __forceinline__ bool alpha_ok(float a) { return a > 0.0f && a < __builtin_inff(); }

// Smallest fp32 X >= 0 (as bits) with fl32(X / alpha) >= mu: bisection over the
// monotone predicate on [0, +inf]; pred(0) is false (mu > 0), pred(inf) true.
__device__ uint32_t threshold_bits(float alpha, float mu) {
    uint32_t lo = 0u, hi = 0x7f800000u;
    while (hi - lo > 1u) {
        const uint32_t mid = lo + ((hi - lo) >> 1);
        if (__uint_as_float(mid) / alpha >= mu) hi = mid; else lo = mid;
    }
    return hi;
}

// ------------------------------------------------------------------- setup
__global__ __launch_bounds__(1024) void k_dda_setup(const float* __restrict__ grid, DdaArgs a,
                                                    DdaWs w) {
    __shared__ uint64_t keys[kDdaMaxThresholds];
    const int A = a.A, tid = threadIdx.x;
    int P = 1;
    while (P < A) P <<= 1;
    for (int i = tid; i < P; i += blockDim.x) {
        uint64_t key = ~0ull;
        if (i < A) {
            const int j = i / a.M, c = i % a.M;
            const float al = grid[j];
            const uint32_t t = alpha_ok(al) ? threshold_bits(al, a.mids[c]) : 0x7f800000u;
            key = ((uint64_t)t << 32) | (uint32_t)i;
        }
        keys[i] = key;
    }
    __syncthreads();
    // bitonic sort, ascending; keys are unique (index in the low word)
    for (int size = 2; size <= P; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = tid; i < P / 2; i += blockDim.x) {
                const int lo = 2 * i - (i & (stride - 1));
                const int hi = lo + stride;
                const bool up = ((lo & size) == 0);
                const uint64_t x = keys[lo], y = keys[hi];
                if ((x > y) == up) { keys[lo] = y; keys[hi] = x; }
            }
            __syncthreads();
        }
    }
    for (int p = tid; p < A; p += blockDim.x) {
        const uint64_t key = keys[p];
        w.ubits[p + 1] = (uint32_t)(key >> 32);
        w.rank[(uint32_t)key] = p + 1;
    }
    if (tid == 0) { w.ubits[0] = 0u; w.ubits[A + 1] = 0xffffffffu; }
    // number of finite thresholds
    __shared__ int s_afin;
    if (tid == 0) s_afin = 0;
    __syncthreads();
    for (int p = tid; p < A; p += blockDim.x) {
        const bool fin = (uint32_t)(keys[p] >> 32) < 0x7f800000u;
        const bool next_fin = (p + 1 < A) && ((uint32_t)(keys[p + 1] >> 32) < 0x7f800000u);
        if (fin && !next_fin) s_afin = p + 1;
    }
    __syncthreads();
    const int afin = s_afin;
    uint32_t lo = 0x7f800000u, hi = 0x7f800000u, shift = 0, nb = 1;
    if (afin > 0) {
        lo = (uint32_t)(keys[0] >> 32);
        hi = (uint32_t)(keys[afin - 1] >> 32);
        const uint32_t range = hi - lo;
        while ((range >> shift) >= (uint32_t)(kDdaBins - 1)) shift++;
        nb = (range >> shift) + 1;
    }
    // bins[b] = #{p in 1..A : U_p <= lo + (b << shift)} (>= 1 when afin > 0)
    for (uint32_t b = tid; b < nb; b += blockDim.x) {
        const uint32_t v = lo + (b << shift);
        int l = 0, r = afin;   // count of sorted finite keys with value <= v
        while (l < r) {
            const int mid = (l + r) >> 1;
            if ((uint32_t)(keys[mid] >> 32) <= v) l = mid + 1; else r = mid;
        }
        w.bins[b] = (uint32_t)l;
    }
    if (tid == 0) {
        w.meta[0] = lo; w.meta[1] = shift; w.meta[2] = nb; w.meta[3] = (uint32_t)afin;
        w.meta[4] = hi;
    }
}

// --------------------------------------------------------------- histogram
template <int BS>
__device__ __forceinline__ double block_sum(double v, double* red) {
    const int tid = threadIdx.x;
    red[tid] = v;
    __syncthreads();
    for (int s = BS / 2; s > 0; s >>= 1) {
        if (tid < s) red[tid] += red[tid + s];
        __syncthreads();
    }
    const double r = red[0];
    __syncthreads();
    return r;
}

constexpr int kHistThreads = 1024;

__global__ __launch_bounds__(kHistThreads) void k_dda_hist(const float* __restrict__ x, int64_t len,
                                                           DdaArgs a, DdaWs w) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int A = a.A, A1 = A + 1;
    uint64_t* hsum = (uint64_t*)smem;                       // [A+1]
    uint32_t* ub = (uint32_t*)(hsum + A1);                  // [A+2]
    uint32_t* hcnt = ub + (A + 2);                          // [A+1]
    uint32_t* bins = hcnt + A1;                             // [nb]
    __shared__ double red[kHistThreads];
    const uint32_t lo = w.meta[0], shift = w.meta[1], nb = w.meta[2], afin = w.meta[3];
    const uint32_t hi = w.meta[4];
    for (int i = threadIdx.x; i < A1; i += blockDim.x) { hsum[i] = 0; hcnt[i] = 0; }
    for (int i = threadIdx.x; i < A + 2; i += blockDim.x) ub[i] = w.ubits[i];
    for (uint32_t i = threadIdx.x; i < nb; i += blockDim.x) bins[i] = w.bins[i];
    __syncthreads();

    double sumsq = 0.0, top_s1 = 0.0;
    uint32_t top_cnt = 0, flags = 0;
    auto visit = [&](float xf) {
        const uint32_t ab = __float_as_uint(xf) & 0x7fffffffu;
        if (ab >= 0x7f800000u) { flags |= (ab > 0x7f800000u) ? 2u : 1u; return; }
        const double xd = (double)__uint_as_float(ab);
        sumsq = fma(xd, xd, sumsq);
        if (ab < lo) return;                              // atom 0: q = 0 for all candidates
        if (ab >= hi) { top_s1 += xd; top_cnt++; return; }  // top atom, unbounded
        uint32_t at = bins[(ab - lo) >> shift];
        while (ub[at + 1] <= ab) at++;
        const uint32_t eb = max(ub[at] >> 23, 1u);
        const uint32_t ex = max(ab >> 23, 1u);
        const uint32_t sig = (ab & 0x7fffffu) | ((ab >> 23) ? 0x800000u : 0u);
        atomicAdd(&hsum[at], (uint64_t)sig << (ex - eb));
        atomicAdd(&hcnt[at], 1u);
    };
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t tid0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (((uintptr_t)x & 15) == 0) {
        const int64_t n4 = len >> 2;
        const f32x4* x4 = (const f32x4*)x;
        for (int64_t i = tid0; i < n4; i += stride) {
            const f32x4 v = __builtin_nontemporal_load(&x4[i]);
            visit(v.x); visit(v.y); visit(v.z); visit(v.w);
        }
        for (int64_t i = (n4 << 2) + tid0; i < len; i += stride) visit(x[i]);
    } else {
        for (int64_t i = tid0; i < len; i += stride) visit(x[i]);
    }
    if (afin > 0 && top_cnt) atomicAdd(&hcnt[afin], top_cnt);
    const double s_sumsq = block_sum<kHistThreads>(sumsq, red);
    const double s_top = block_sum<kHistThreads>(top_s1, red);
    __shared__ uint32_t s_flags;
    if (threadIdx.x == 0) s_flags = 0;
    __syncthreads();
    if (flags) atomicOr(&s_flags, flags);
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * A1;
    for (int i = threadIdx.x; i < A1; i += blockDim.x) {
        w.pcnt[base + i] = hcnt[i];
        w.psum[base + i] = hsum[i];
    }
    if (threadIdx.x == 0) {
        double* ps = w.pscal + 4 * blockIdx.x;
        ps[0] = s_sumsq; ps[1] = s_top; ps[2] = 0.0; ps[3] = (double)s_flags;
    }
}

// ------------------------------------------------------------------ reduce
__global__ __launch_bounds__(256) void k_dda_reduce(DdaArgs a, DdaWs w) {
    const int A1 = a.A + 1;
    const int at = blockIdx.x * blockDim.x + threadIdx.x;
    if (at >= A1) return;
    const uint32_t afin = w.meta[3];
    uint64_t c = 0, s = 0;
    for (int b = 0; b < a.nblk; b++) {
        c += w.pcnt[(int64_t)b * A1 + at];
        s += w.psum[(int64_t)b * A1 + at];
    }
    double s1 = 0.0;
    if (at >= 1 && (uint32_t)at < afin) {
        const int eb = (int)max(w.ubits[at] >> 23, 1u);
        s1 = ldexp((double)s, eb - 150);
    } else if ((uint32_t)at == afin && afin > 0) {
        for (int b = 0; b < a.nblk; b++) s1 += w.pscal[4 * b + 1];
    }
    w.s0[at] = (double)c;
    w.s1[at] = (at == 0) ? 0.0 : s1;
}

// ---------------------------------------------------------------- finalize
constexpr int kFinThreads = 1024;

__global__ __launch_bounds__(kFinThreads) void k_dda_finalize(const float* __restrict__ grid,
                                                              DdaArgs a, DdaWs w,
                                                              float* __restrict__ alpha_out,
                                                              double* __restrict__ D_out) {
    __shared__ double red[kFinThreads];
    __shared__ double sA[kFinThreads], sB[kFinThreads];
    __shared__ double Dv[kDdaMaxG];
    const int tid = threadIdx.x;
    double ss = 0.0;
    uint32_t fl = 0;
    for (int b = tid; b < a.nblk; b += blockDim.x) {
        ss += w.pscal[4 * b];
        fl |= (uint32_t)w.pscal[4 * b + 3];
    }
    const double sumsq = block_sum<kFinThreads>(ss, red);
    __shared__ uint32_t s_fl;
    if (tid == 0) s_fl = 0;
    __syncthreads();
    if (fl) atomicOr(&s_fl, fl);
    const int G = a.G, M = a.M;
    const int T = kFinThreads / G;            // threads per candidate (>= 1)
    const int afin = (int)w.meta[3];
    const int natoms = afin;                  // atoms 1..afin carry q > 0 possibly
    const int j = tid / T, part = tid % T;
    double Aj = 0.0, Bj = 0.0;
    if (j < G && natoms > 0) {
        const int per = (natoms + T - 1) / T;
        const int a0 = 1 + part * per;
        const int a1 = min(natoms + 1, a0 + per);
        if (a0 < a1) {
            const int32_t* rk = w.rank + (int64_t)j * M;   // rk[c-1]: start atom of cell c
            int l = 0, r = M;                              // cell = #{c : rank_c <= a0}
            while (l < r) {
                const int mid = (l + r) >> 1;
                if (rk[mid] <= a0) l = mid + 1; else r = mid;
            }
            int c = l;
            for (int at = a0; at < a1; at++) {
                while (c < M && rk[c] <= at) c++;
                const double q = (double)a.q[c];
                Aj = fma(q, w.s1[at], Aj);
                Bj = fma(q * q, w.s0[at], Bj);
            }
        }
    }
    sA[tid] = Aj;
    sB[tid] = Bj;
    __syncthreads();
    if (part == 0 && j < G) {
        double ta = 0.0, tb = 0.0;
        for (int p = 0; p < T; p++) { ta += sA[tid + p]; tb += sB[tid + p]; }
        const float al = grid[j];
        const double ad = (double)al;
        double D = fma(ad, fma(ad, tb, -2.0 * ta), sumsq);
        if (!alpha_ok(al) || (s_fl & 2u)) D = __builtin_nan("");
        else if (s_fl & 1u) D = __builtin_inf();
        Dv[j] = D;
    }
    __syncthreads();
    if (tid == 0) {
        int best = 0;
        for (int jj = 1; jj < G; jj++) {
            const double d = Dv[jj], db = Dv[best];
            if (d < db || (db != db && d == d)) best = jj;
        }
        *alpha_out = grid[best];
    }
    if (D_out)
        for (int jj = tid; jj < G; jj += blockDim.x) D_out[jj] = Dv[jj];
}

hipError_t launch_dda(const float* x, int64_t len, const Fmt& f, const float* grid, int G,
                      float* alpha_out, double* D_out, void* ws, const DdaLayout& L,
                      hipStream_t s) {
    DdaArgs a;
    const int M = L.M;
    double vals[128];
    int nv = 0;
    for (uint32_t c = 0; c < (1u << f.n); c++) {   // non-negative values, ascending
        if (c & f.sign_bit) continue;
        vals[nv++] = decode_value(f, c);
    }
    for (int i = 1; i < nv; i++)
        for (int t = i; t > 0 && vals[t] < vals[t - 1]; t--) {
            const double tmp = vals[t]; vals[t] = vals[t - 1]; vals[t - 1] = tmp;
        }
    // drop the duplicate zero only if present (it is not: the -0 code is skipped)
    for (int c = 0; c <= M; c++) a.q[c] = (float)vals[c];
    for (int c = 1; c <= M; c++) a.mids[c - 1] = (float)(0.5 * (vals[c - 1] + vals[c]));
    a.G = G; a.M = M; a.A = L.A; a.nblk = L.nblk;
    const DdaWs w = ws_ptrs(ws, L);
    k_dda_setup<<<1, 1024, 0, s>>>(grid, a, w);
    const size_t smem = sizeof(uint64_t) * (L.A + 1) + sizeof(uint32_t) * ((L.A + 2) + (L.A + 1) + kDdaBins);
    static bool lds_attr_set[64] = {false};
    int dev = 0;
    if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < 64 && !lds_attr_set[dev]) {
        const hipError_t e = hipFuncSetAttribute((const void*)k_dda_hist,
                                                 hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 150 * 1024);
        if (e != hipSuccess) return e;
        lds_attr_set[dev] = true;
    }
    k_dda_hist<<<L.nblk, kHistThreads, smem, s>>>(x, len, a, w);
    k_dda_reduce<<<(L.A + 1 + 255) / 256, 256, 0, s>>>(a, w);
    k_dda_finalize<<<1, kFinThreads, 0, s>>>(grid, a, w, alpha_out, D_out);
    return hipGetLastError();
}

}  // namespace esb
