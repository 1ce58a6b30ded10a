// Data normalization (Sec. 3.4, the DN equation) and the distribution
// difference aligner in its analytic form for normalized data (eq. (9), (13)
// with p = N(0,1), "Resolving extremum"), gfx950.
//
// Statistics: the mean and the population standard deviation
// sqrt((1/d) sum (x - mean)^2), one read of x.  Block b holds a contiguous
// chunk of 16384 elements in registers (64 per thread), sums it in fp64, and
// sums the squared deviations from its own chunk mean (the two-pass form,
// inside the block); the chunks are combined exactly as in Chan, Golub and
// LeVeque's pairwise update: M2 = sum_b M2_b + sum_b n_b (mean_b - mean)^2,
// in fp64, in block order.  The result is deterministic; the statistics are
// returned rounded to binary32 (the form the projection uses).
//
// Analytic objective: for each candidate alpha_j, the one-sided expected
// squared projection error over t >= 0 of N(0,1) with nearest-neighbour cells
// [alpha mid_c, alpha mid_{c+1}) around alpha q_c, the top cell open:
//   int_lo^hi (t - v)^2 phi(t) dt = (1 + v^2) M0 - 2 v M1 + (lo phi(lo) - hi phi(hi)),
//   M0 = Phi(hi) - Phi(lo), M1 = phi(lo) - phi(hi),
// in fp64 (erfc, exp), and its slope in alpha (the moving cell ends cancel:
// they are midpoints, where neighbouring integrands agree)
//   dD/dalpha = -2 sum_c q_c (M1_c - alpha q_c M0_c).
// The argmin takes the smallest index among equal
// values; a candidate that is not a positive finite number gets NaN.
#include "esb_internal.h"

namespace esb {

constexpr int kDnThreads = 256;
constexpr int kDnPer = 64;                               // elements per thread
constexpr int64_t kDnChunk = (int64_t)kDnThreads * kDnPer;   // elements per block
constexpr int kDnRedThreads = 1024;

static int64_t dn_blocks(int64_t len) { return len <= 0 ? 1 : (len + kDnChunk - 1) / kDnChunk; }

size_t dn_workspace(int64_t len) { return sizeof(double) * 2 * (size_t)dn_blocks(len); }

// Fixed-order sum over the workgroup (xor butterfly in each wave, then the
// waves in order); every thread gets the total.
template <int NT>
__device__ __forceinline__ double group_sum(double v, double* sh) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    const int w = threadIdx.x >> 6;
    __syncthreads();   // sh may still be read from a previous call
    if ((threadIdx.x & 63) == 0) sh[w] = v;
    __syncthreads();
    double t = sh[0];
#pragma unroll
    for (int i = 1; i < NT / 64; i++) t += sh[i];
    return t;
}

// part[2b] = sum of chunk b, part[2b+1] = sum of squared deviations from the
// chunk's mean.  VEC: 16-byte loads (x 16-byte aligned); the last, partial
// chunk of the vector launch takes the scalar loads.
template <bool VEC>
__global__ __launch_bounds__(kDnThreads) void k_dn_chunk(const float* __restrict__ x, int64_t len,
                                                        double* __restrict__ part) {
    __shared__ double sh[kDnThreads / 64];
    const int64_t b0 = (int64_t)blockIdx.x * kDnChunk;
    const int nb = (int)(len - b0 < kDnChunk ? len - b0 : kDnChunk);
    const int t = threadIdx.x;
    float v[kDnPer];
    if (VEC && nb == kDnChunk) {
        const f32x4* x4 = (const f32x4*)(x + b0);
#pragma unroll
        for (int u = 0; u < kDnPer / 4; u++) {
            const f32x4 q = __builtin_nontemporal_load(&x4[u * kDnThreads + t]);
            v[4 * u] = q.x;
            v[4 * u + 1] = q.y;
            v[4 * u + 2] = q.z;
            v[4 * u + 3] = q.w;
        }
    } else {
        // element of v[4u + c] is 4 (u * 256 + t) + c, as in the vector layout
#pragma unroll
        for (int u = 0; u < kDnPer / 4; u++)
#pragma unroll
            for (int c = 0; c < 4; c++) {
                const int i = 4 * (u * kDnThreads + t) + c;
                v[4 * u + c] = i < nb ? x[b0 + i] : 0.0f;
            }
    }
    double s = 0.0;
#pragma unroll
    for (int e = 0; e < kDnPer; e++) s += (double)v[e];   // padding adds zeros
    const double S = group_sum<kDnThreads>(s, sh);
    const double m = S / (double)nb;
    double q = 0.0;
    if (VEC && nb == kDnChunk) {
#pragma unroll
        for (int e = 0; e < kDnPer; e++) {
            const double d = (double)v[e] - m;
            q = fma(d, d, q);
        }
    } else {
#pragma unroll
        for (int u = 0; u < kDnPer / 4; u++)
#pragma unroll
            for (int c = 0; c < 4; c++) {
                const double d = (double)v[4 * u + c] - m;
                if (4 * (u * kDnThreads + t) + c < nb) q = fma(d, d, q);
            }
    }
    const double M2 = group_sum<kDnThreads>(q, sh);
    if (t == 0) {
        part[2 * blockIdx.x] = S;
        part[2 * blockIdx.x + 1] = M2;
    }
}

// The chunks combined in block order: the binary32 mean and standard deviation.
__global__ __launch_bounds__(kDnRedThreads) void k_dn_combine(int64_t nblk, int64_t len,
                                                              const double* __restrict__ part,
                                                              float* __restrict__ stats) {
    __shared__ double sh[kDnRedThreads / 64];
    double s = 0.0;
    for (int64_t b = threadIdx.x; b < nblk; b += kDnRedThreads) s += part[2 * b];
    const double mean = group_sum<kDnRedThreads>(s, sh) / (double)len;
    double q = 0.0;
    for (int64_t b = threadIdx.x; b < nblk; b += kDnRedThreads) {
        const int64_t n = (b + 1 < nblk) ? kDnChunk : len - b * kDnChunk;
        const double d = part[2 * b] / (double)n - mean;
        q += part[2 * b + 1] + (double)n * d * d;
    }
    const double M2 = group_sum<kDnRedThreads>(q, sh);
    if (threadIdx.x == 0) {
        stats[0] = (float)mean;
        stats[1] = (float)sqrt(M2 / (double)len);
    }
}

__global__ void k_dn_empty(float* stats) {
    stats[0] = __builtin_nanf("");
    stats[1] = __builtin_nanf("");
}

hipError_t launch_dn_stats(const float* x, int64_t len, float* stats, void* ws, hipStream_t s) {
    if (len <= 0) {
        k_dn_empty<<<1, 1, 0, s>>>(stats);
        return hipGetLastError();
    }
    const int64_t nb = dn_blocks(len);
    if (nb > 0x7fffffff) return hipErrorInvalidValue;
    double* part = (double*)ws;
    if ((uintptr_t)x % 16 == 0) k_dn_chunk<true><<<(unsigned)nb, kDnThreads, 0, s>>>(x, len, part);
    else k_dn_chunk<false><<<(unsigned)nb, kDnThreads, 0, s>>>(x, len, part);
    k_dn_combine<<<1, kDnRedThreads, 0, s>>>(nb, len, part, stats);
    return hipGetLastError();
}

// ------------------------------------------------------------ analytic DDA
__device__ __forceinline__ double nphi(double t) {   // standard normal density
    return exp(-0.5 * t * t) * 0.3989422804014327;
}
__device__ __forceinline__ double nupper(double t) {   // 1 - Phi(t)
    return 0.5 * erfc(t * 0.7071067811865476);
}

// One thread per (candidate, cell): 256 / CELLS candidates per workgroup, the
// cells of a candidate on consecutive lanes.  Each thread evaluates phi and
// 1 - Phi at its cell's lower end once; the upper end is the next lane's lower
// end (the top cell's is +inf).  The cell terms of a candidate are summed by a
// butterfly inside its aligned lane group (and across the two waves of a
// candidate when CELLS = 128), a fixed order.
template <int CELLS>
__global__ __launch_bounds__(256) void k_dda_normal_eval(const float* __restrict__ grid, int G, int k,
                                                         double* __restrict__ D_out,
                                                         double* __restrict__ dD_out) {
    constexpr int kCpb = 256 / CELLS;
    __shared__ double s_phi[256], s_up[256], s_red[2][4];
    const int t = threadIdx.x, c = t % CELLS;
    const int j = blockIdx.x * kCpb + t / CELLS;
    const float al = j < G ? grid[j] : 1.0f;
    const bool valid = j < G && al > 0.0f && al < __builtin_inff();
    const double a = valid ? (double)al : 1.0;
    const double lo = c == 0 ? 0.0 : a * (double)set_mid(c, k);
    const double plo = nphi(lo), ulo = nupper(lo);
    s_phi[t] = plo;
    s_up[t] = ulo;
    __syncthreads();
    const bool top = c + 1 == CELLS;
    const double phi_hi = top ? 0.0 : s_phi[t + 1];
    const double up_hi = top ? 0.0 : s_up[t + 1];
    const double hphi_hi = top ? 0.0 : a * (double)set_mid(c + 1, k) * phi_hi;
    const double q = (double)set_value(c, k), v = a * q;
    const double M0 = ulo - up_hi, M1 = plo - phi_hi;
    const double M2 = M0 + lo * plo - hphi_hi;
    double D = M2 - 2.0 * v * M1 + v * v * M0;
    double dD = -2.0 * q * (M1 - v * M0);
#pragma unroll
    for (int off = (CELLS < 64 ? CELLS : 64) / 2; off > 0; off >>= 1) {
        D += __shfl_xor(D, off);
        dD += __shfl_xor(dD, off);
    }
    if (CELLS == 128) {
        if ((t & 63) == 0) {
            s_red[0][t >> 6] = D;
            s_red[1][t >> 6] = dD;
        }
        __syncthreads();
        D = s_red[0][(t >> 7) * 2] + s_red[0][(t >> 7) * 2 + 1];
        dD = s_red[1][(t >> 7) * 2] + s_red[1][(t >> 7) * 2 + 1];
    }
    if (c == 0 && j < G) {
        D_out[j] = valid ? D : __builtin_nan("");
        if (dD_out) dD_out[j] = valid ? dD : __builtin_nan("");
    }
}

// The smallest index with the least D, NaN ranking last.
__global__ __launch_bounds__(1024) void k_dda_normal_pick(const float* __restrict__ grid, int G,
                                                          const double* __restrict__ D,
                                                          float* __restrict__ alpha_out) {
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    double bd = 0.0;
    int bj = 0x7fffffff;   // none yet
    for (int j = tid; j < G; j += blockDim.x) {
        const double d = D[j];
        if (bj == 0x7fffffff || d < bd || (bd != bd && d == d)) { bd = d; bj = j; }
    }
    auto pick = [](double& bd, int& bj, double od, int oj) {
        const bool onan = od != od, mnan = bd != bd;
        const bool better = (oj != 0x7fffffff) &&
                            ((bj == 0x7fffffff) || (!onan && mnan) ||
                             (onan == mnan && (od < bd || ((od == bd || onan) && oj < bj))));
        if (better) { bd = od; bj = oj; }
    };
    for (int off = 32; off > 0; off >>= 1) {
        const double od = __shfl_xor(bd, off);
        const int oj = __shfl_xor(bj, off);
        pick(bd, bj, od, oj);
    }
    __shared__ double s_bd[16];
    __shared__ int s_bj[16];
    if (lane == 0) { s_bd[wid] = bd; s_bj[wid] = bj; }
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < (int)(blockDim.x / 64); w++) pick(bd, bj, s_bd[w], s_bj[w]);
        *alpha_out = grid[bj];
    }
}

template <int CELLS>
static void eval_t(const float* grid, int G, int k, double* D, double* dD, hipStream_t s) {
    const int cpb = 256 / CELLS;
    k_dda_normal_eval<CELLS><<<(G + cpb - 1) / cpb, 256, 0, s>>>(grid, G, k, D, dD);
}

hipError_t launch_dda_normal(const Fmt& f, const float* grid, int G, float* alpha_out,
                             double* D_out, double* dD_out, hipStream_t s) {
    switch (f.n) {
        case 2: eval_t<2>(grid, G, f.k, D_out, dD_out, s); break;
        case 3: eval_t<4>(grid, G, f.k, D_out, dD_out, s); break;
        case 4: eval_t<8>(grid, G, f.k, D_out, dD_out, s); break;
        case 5: eval_t<16>(grid, G, f.k, D_out, dD_out, s); break;
        case 6: eval_t<32>(grid, G, f.k, D_out, dD_out, s); break;
        case 7: eval_t<64>(grid, G, f.k, D_out, dD_out, s); break;
        case 8: eval_t<128>(grid, G, f.k, D_out, dD_out, s); break;
        default: return hipErrorInvalidValue;
    }
    const int nt = G >= 1024 ? 1024 : (G + 63) / 64 * 64;
    k_dda_normal_pick<<<1, nt, 0, s>>>(grid, G, D_out, alpha_out);
    return hipGetLastError();
}

}  // namespace esb
