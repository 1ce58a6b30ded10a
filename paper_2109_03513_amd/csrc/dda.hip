// Distribution difference aligner (eq. (9), (13)) on the data, gfx950.
//
// Objective per candidate scale alpha_j:  D_j = sum_i (|x_i| - alpha_j q_j(x_i))^2
//   = S2 - 2 alpha_j sum_i |x_i| q_j(x_i) + alpha_j^2 sum_i q_j(x_i)^2,
// with S2 = sum_i x_i^2.  q_j(x) depends on x only through which cell of
// candidate j holds |x|, and the cell boundaries are exact fp32 thresholds:
// T_{j,c} = the smallest fp32 X with fl32(X / alpha_j) >= mu_c, mu_c the
// midpoint between set values c-1 and c (ties go up, as in the projection).
// All G*M thresholds, sorted and further split at every power of two, cut
// [0, inf) into "atoms": every candidate's cell is a union of consecutive atoms
// and every bounded atom lies inside one binade.  One pass over x suffices:
//
// k_dda_hist (<= 256 blocks of 1024 threads), per block:
//   set-up in LDS: thresholds by a local search around fl32(alpha mu); their
//   ranks in the sorted order from branch-free binary searches in the other
//   candidates' (already ascending) lists; power-of-two split points; a bin
//   table over the threshold bit range whose entries name the atom directly
//   unless a boundary falls inside the bin;
//   pass: per element its atom, and one LDS atomic adding (significand << 20) + 1
//   to a packed 64-bit (sum, count) cell; x^2 in fp64; the unbounded top atom in
//   fp64.  Every 2^19 elements the packed cells are flushed to per-block totals.
// k_dda_reduce (only for many blocks): sums the per-block totals in slices.
// k_dda_finalize (1 block): per-atom sums, prefix sums over atoms, then per
//   candidate A_j = sum_c Q_c (P1[end_c] - P1[start_c]), B_j likewise with P0 and
//   Q_c^2, D_j = S2 + a (a B_j - 2 A_j); argmin with ties to the lowest index.
// Integer sums are exact; fp64 sums run in a fixed order: the result is
// deterministic.
#include <type_traits>

#include "esb_internal.h"

namespace esb {

constexpr int kHistThreads = 1024;
constexpr int kMaxSplits = 256;          // power-of-two split points (at most 254)
constexpr int kChunk4 = 4096;            // float4 per chunk: 16384 elements
constexpr int kFlushChunks = 32;         // 2^19 elements between flushes
constexpr int kReduceSlices = 16;

struct DdaArgs {
    float mids[128];   // mu_c, c = 1..M (index c-1)
    float q[128];      // Q_c, c = 0..M (unscaled values, ascending)
    int G, M, A, Aa, nblk, nslice;
    int rk_lds;        // the finalize keeps the cell starts in LDS (when they fit)
};

struct DdaWs {   // pointers into the caller's workspace
    uint32_t* ubits;   // [Aa+2]: augmented sorted bounds of the atoms
    int32_t* rank;     // [A]: atom where cell c of candidate j starts (j*M + c-1)
    uint32_t* meta;    // afin (top atom), Aprime (number of bounds)
    uint64_t* pcnt;    // [nblk][Aa+1] per-block element counts
    uint64_t* psum;    // [nblk][Aa+1] per-block significand sums
    double* pscal;     // [nblk][4]: sum x^2, top-atom sum |x|, top count, flags
    uint64_t* rcnt;    // [nslice][Aa+1] sliced sums (k_dda_reduce)
    uint64_t* rsum;    // [nslice][Aa+1]
};

__host__ __device__ static inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

static int dda_nblk(int64_t len) {
    const int64_t chunks = (len + 4 * kChunk4 - 1) / (4 * kChunk4);
    return (int)(chunks < 1 ? 1 : (chunks > kDdaMaxBlocks ? kDdaMaxBlocks : chunks));
}

bool dda_layout(int64_t len, const Fmt& f, int G, DdaLayout* L) {
    const int M = (1 << (f.n - 1)) - 1;
    if (G < 1 || G > kDdaMaxG || (int64_t)G * M > kDdaMaxThresholds || len < 0) return false;
    L->G = G;
    L->M = M;
    L->A = G * M;
    L->nblk = dda_nblk(len);
    const size_t Aa1 = (size_t)L->A + kMaxSplits + 1;
    const size_t ns = kReduceSlices;
    size_t o = 0;
    L->off_ubits = o; o = align256(o + sizeof(uint32_t) * (Aa1 + 1));
    L->off_rank = o;  o = align256(o + sizeof(int32_t) * (size_t)L->A);
    L->off_meta = o;  o = align256(o + sizeof(uint32_t) * 8);
    L->off_pcnt = o;  o = align256(o + sizeof(uint64_t) * Aa1 * L->nblk);
    L->off_psum = o;  o = align256(o + sizeof(uint64_t) * Aa1 * L->nblk);
    L->off_pscal = o; o = align256(o + sizeof(double) * 4 * L->nblk);
    L->off_s0 = o;    o = align256(o + sizeof(uint64_t) * Aa1 * ns);
    L->off_s1 = o;    o = align256(o + sizeof(uint64_t) * Aa1 * ns);
    L->off_bins = 0;
    L->total = o;
    return true;
}

static DdaWs ws_ptrs(void* ws, const DdaLayout& L) {
    char* b = (char*)ws;
    DdaWs w;
    w.ubits = (uint32_t*)(b + L.off_ubits);
    w.rank = (int32_t*)(b + L.off_rank);
    w.meta = (uint32_t*)(b + L.off_meta);
    w.pcnt = (uint64_t*)(b + L.off_pcnt);
    w.psum = (uint64_t*)(b + L.off_psum);
    w.pscal = (double*)(b + L.off_pscal);
    w.rcnt = (uint64_t*)(b + L.off_s0);
    w.rsum = (uint64_t*)(b + L.off_s1);
    return w;
}

__device__ __forceinline__ bool alpha_ok(float a) { return a > 0.0f && a < __builtin_inff(); }

__device__ __forceinline__ bool reaches(uint32_t xbits, float alpha, float mu) {
    return __uint_as_float(xbits) / alpha >= mu;   // fl32(X / alpha) >= mu, IEEE division
}

// Smallest fp32 X >= 0 (as bits) with fl32(X / alpha) >= mu.  The predicate is
// monotone in X, false at 0 (mu > 0) and true at +inf.  Local search from
// fl32(alpha * mu), which is within a few ulps of the answer; bisection if the
// walk does not settle.
__device__ uint32_t threshold_bits(float alpha, float mu) {
    uint32_t b = __float_as_uint(alpha * mu);
    if (b > 0x7f800000u) b = 0x7f800000u;
    int it = 0;
    if (reaches(b, alpha, mu)) {
        while (b > 0u && it < 32 && reaches(b - 1u, alpha, mu)) { b--; it++; }
    } else {
        while (it < 32 && !reaches(b, alpha, mu)) { b++; it++; }
    }
    if (it < 32) return b;
    uint32_t lo = 0u, hi = 0x7f800000u;
    while (hi - lo > 1u) {
        const uint32_t mid = lo + ((hi - lo) >> 1);
        if (reaches(mid, alpha, mu)) hi = mid; else lo = mid;
    }
    return hi;
}

// Number of powers of two strictly between bit patterns lo < hi (both finite).
__device__ __forceinline__ uint32_t splits_between(uint32_t lo, uint32_t hi) {
    const uint32_t e1 = lo >> 23, e2 = hi >> 23;
    const uint32_t last = (hi & 0x7fffffu) ? e2 : e2 - 1u;   // exponent of the last start < hi
    const uint32_t first = e1 + 1u;                           // first binade start > lo
    return (e2 > e1 && last >= first) ? last - first + 1u : 0u;
}

// Block-wide exclusive scan (1024 threads), fixed summation order.
template <typename T>
__device__ __forceinline__ T block_exclusive_scan(T v, T* sh, T* total) {
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, nw = blockDim.x >> 6;
    T x = v;
    for (int off = 1; off < 64; off <<= 1) {
        const T y = __shfl_up(x, off);
        if (lane >= off) x += y;
    }
    if (lane == 63) sh[wid] = x;
    __syncthreads();
    if (wid == 0) {
        T s = lane < nw ? sh[lane] : (T)0;
        for (int off = 1; off < 64; off <<= 1) {
            const T y = __shfl_up(s, off);
            if (lane >= off) s += y;
        }
        if (lane < nw) sh[lane] = s;
    }
    __syncthreads();
    const T before = (wid > 0 ? sh[wid - 1] : (T)0) + x - v;
    if (total) *total = sh[nw - 1];
    __syncthreads();
    return before;
}

// Block-wide exclusive scan of N fp64 components at once (one set of barriers).
template <int N>
__device__ __forceinline__ void block_exclusive_scan_n(const double (&v)[N], double (*sh)[16],
                                                       double (&before)[N], double (&total)[N]) {
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, nw = blockDim.x >> 6;
    double x[N];
#pragma unroll
    for (int c = 0; c < N; c++) x[c] = v[c];
    for (int off = 1; off < 64; off <<= 1) {
#pragma unroll
        for (int c = 0; c < N; c++) {
            const double y = __shfl_up(x[c], off);
            if (lane >= off) x[c] += y;
        }
    }
    if (lane == 63) {
#pragma unroll
        for (int c = 0; c < N; c++) sh[c][wid] = x[c];
    }
    __syncthreads();
    if (wid == 0) {
#pragma unroll
        for (int c = 0; c < N; c++) {
            double t = lane < nw ? sh[c][lane] : 0.0;
            for (int off = 1; off < 64; off <<= 1) {
                const double y = __shfl_up(t, off);
                if (lane >= off) t += y;
            }
            if (lane < nw) sh[c][lane] = t;
        }
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < N; c++) {
        before[c] = (wid > 0 ? sh[c][wid - 1] : 0.0) + x[c] - v[c];
        total[c] = sh[c][nw - 1];
    }
    __syncthreads();
}

// Block-wide sums of N fp64 components in a fixed order (deterministic): a
// butterfly inside each wave, then the wave totals added in wave order.  All
// threads receive the totals.  One barrier pair.
template <int N>
__device__ __forceinline__ void block_sum_n(double (&v)[N], double (*sh)[16]) {
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, nw = blockDim.x >> 6;
#pragma unroll
    for (int c = 0; c < N; c++)
        for (int off = 32; off > 0; off >>= 1) v[c] += __shfl_xor(v[c], off);
    if (lane == 0) {
#pragma unroll
        for (int c = 0; c < N; c++) sh[c][wid] = v[c];
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < N; c++) {
        double t = 0.0;
        for (int w = 0; w < nw; w++) t += sh[c][w];
        v[c] = t;
    }
    __syncthreads();
}

// Wave-level min / max / sum of 32-bit values (all 64 lanes take part).
__device__ __forceinline__ uint32_t wave_min(uint32_t v) {
    for (int off = 32; off > 0; off >>= 1) v = min(v, (uint32_t)__shfl_xor((int)v, off));
    return v;
}
__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
    for (int off = 32; off > 0; off >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, off));
    return v;
}
__device__ __forceinline__ uint32_t wave_add(uint32_t v) {
    for (int off = 32; off > 0; off >>= 1) v += (uint32_t)__shfl_xor((int)v, off);
    return v;
}

template <typename T>
__device__ __forceinline__ T block_sum(T v, T* sh) {
    T t;
    block_exclusive_scan<T>(v, sh, &t);
    return t;
}

// Dynamic LDS of k_dda_hist:
//   U     u32[Aa + 2]   sorted atom bounds: U[0] = 0, U[1..Ap] boundaries, U[Ap+1] = ~0
//   binfo u32[nbins]    per bin: first atom (low 16 bits) | boundaries inside (high 16);
//                       for the pass it becomes u32[2 * nbins]: the pair
//                       {first atom | bounds inside << 16, the first bound after it}
//   TH    u32[A]        thresholds, later their atom positions (the cell starts)
//   KH    u64[Aa + 65]  (value << 32 | id) bucket keys, later the packed histogram;
//                       the last 64 cells take the zero adds of lanes outside
//                       [lo, hi), one per lane, so that they never collide
__host__ __device__ static inline int hist_nbins(int A) {
    return A <= 2048 ? 8192 : (A <= 4096 ? 4096 : 2048);
}
static size_t hist_lds_bytes(int A) {
    const size_t Aa = (size_t)A + kMaxSplits;
    return align256(sizeof(uint32_t) * (Aa + 2)) + sizeof(uint32_t) * 2 * hist_nbins(A) +
           align256(sizeof(uint32_t) * A) + sizeof(uint64_t) * (Aa + 1 + 64);
}

__global__ __launch_bounds__(kHistThreads) void k_dda_hist(const float* __restrict__ x, int64_t len,
                                                           const float* __restrict__ grid,
                                                           DdaArgs a, DdaWs w) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int A = a.A, M = a.M, tid = threadIdx.x;
    const int nbins = hist_nbins(A);
    const size_t Aa = (size_t)A + kMaxSplits;
    uint32_t* U = (uint32_t*)smem;
    uint32_t* binfo = (uint32_t*)(smem + align256(sizeof(uint32_t) * (Aa + 2)));
    uint32_t* TH = binfo + 2 * nbins;
    uint64_t* KH = (uint64_t*)((unsigned char*)TH + align256(sizeof(uint32_t) * A));
    uint64_t* hist = KH;
    __shared__ float s_mids[128];
    __shared__ uint32_t s_lo, s_hi, s_nfin, s_flags;
    __shared__ uint32_t s_scan[16];
    __shared__ double s_red3[3][16];

    // ---- 0. this block's chunks of x; the first one is requested now, so its
    //         loads overlap the set-up.  Loads are unconditional (clamped
    //         address, value zeroed outside the range), so the compiler can
    //         leave a chunk in flight across the binning of the previous one.
    const bool vec = ((uintptr_t)x & 15) == 0;
    const int64_t n4 = vec ? (len >> 2) : (len + 3) >> 2;   // scalar path: chunks of 4 elements
    const int64_t nchunks = (n4 + kChunk4 - 1) / kChunk4;
    const int64_t cpb = (nchunks + gridDim.x - 1) / gridDim.x;
    const int64_t c0 = (int64_t)blockIdx.x * cpb;
    const int64_t c1 = min(nchunks, c0 + cpb);
    auto load_chunk_t = [&](auto VEC, int64_t ch, uint32_t (&g)[16]) {
        if constexpr (decltype(VEC)::value) {
            const f32x4* x4 = (const f32x4*)x;
#pragma unroll
            for (int u = 0; u < 4; u++) {
                const int64_t i4 = ch * kChunk4 + tid + u * kHistThreads;
                const bool in = ch < c1 && i4 < n4;
                const f32x4 v = __builtin_nontemporal_load(&x4[in ? i4 : 0]);
                g[4 * u + 0] = in ? __float_as_uint(v.x) : 0u;
                g[4 * u + 1] = in ? __float_as_uint(v.y) : 0u;
                g[4 * u + 2] = in ? __float_as_uint(v.z) : 0u;
                g[4 * u + 3] = in ? __float_as_uint(v.w) : 0u;
            }
        } else {
#pragma unroll
            for (int u = 0; u < 16; u++) {
                const int64_t i = ch * (4 * kChunk4) + tid + (int64_t)u * kHistThreads;
                const bool in = ch < c1 && i < len;
                const uint32_t v = __float_as_uint(x[in ? i : 0]);
                g[u] = in ? v : 0u;   // zeros: atom 0, add nothing
            }
        }
    };
    uint32_t gn[16];
    if (c0 < c1) {   // (a block with no chunk touches no element: x may be empty)
        if (vec) load_chunk_t(std::integral_constant<bool, true>{}, c0, gn);
        else load_chunk_t(std::integral_constant<bool, false>{}, c0, gn);
    }

    // ---- 1. thresholds, their finite range and count
    if (tid < M) s_mids[tid] = a.mids[tid];
    if (tid == 0) { s_lo = 0x7f800000u; s_hi = 0u; s_nfin = 0u; s_flags = 0u; }
    __syncthreads();
    {
        uint32_t wlo = 0x7f800000u, whi = 0u, wn = 0u;
        for (int i0 = 0; i0 < A; i0 += kHistThreads) {      // uniform trip count
            const int i = i0 + tid;
            if (i < A) {
                const int j = i / M, c = i - j * M;
                const float al = grid[j];
                const uint32_t t = alpha_ok(al) ? threshold_bits(al, s_mids[c]) : 0x7f800000u;
                TH[i] = t;
                if (t < 0x7f800000u) { wlo = min(wlo, t); whi = max(whi, t); wn++; }
            }
        }
        wlo = wave_min(wlo);
        whi = wave_max(whi);
        wn = wave_add(wn);
        if ((tid & 63) == 0 && wn) {
            atomicMin(&s_lo, wlo);
            atomicMax(&s_hi, whi);
            atomicAdd(&s_nfin, wn);
        }
    }
    __syncthreads();
    const uint32_t nfin = s_nfin;
    uint32_t lo = 0x7f800000u, hi = 0x7f800000u, shift = 0, base = 0, nb = 0, nsplit = 0;
    if (nfin > 0) {
        lo = s_lo;
        hi = s_hi;
        while (((hi >> shift) - (lo >> shift)) >= (uint32_t)(nbins - 1)) shift++;   // <= 19
        base = lo >> shift;
        nb = (hi >> shift) - base + 1;
        if (hi > lo) {
            const uint32_t e_lo = lo >> 23, e_hi = (hi - 1u) >> 23;   // binade starts in (lo, hi)
            nsplit = e_hi - e_lo;
        }
    }
    // ---- 2. boundaries per bin: finite thresholds and the powers of two in (lo, hi)
    for (uint32_t b = tid; b < nb; b += kHistThreads) binfo[b] = 0u;
    __syncthreads();
    for (int i = tid; i < A; i += kHistThreads) {
        const uint32_t t = TH[i];
        if (t < 0x7f800000u) atomicAdd(&binfo[(t >> shift) - base], 1u);
    }
    for (uint32_t e = tid; e < nsplit; e += kHistThreads) {
        const uint32_t v = ((lo >> 23) + 1u + e) << 23;
        atomicAdd(&binfo[(v >> shift) - base], 1u);
    }
    __syncthreads();
    // ---- 3. first atom of every bin: exclusive scan of the counts
    const uint32_t Ap = nfin + nsplit;
    {
        const int per = (int)((nb + kHistThreads - 1) / kHistThreads);
        uint32_t mysum = 0;
        for (int e = 0; e < per; e++) {
            const uint32_t b = (uint32_t)(tid * per + e);
            if (b < nb) mysum += binfo[b];
        }
        uint32_t run = block_exclusive_scan<uint32_t>(mysum, s_scan, nullptr);
        for (int e = 0; e < per; e++) {
            const uint32_t b = (uint32_t)(tid * per + e);
            if (b < nb) {
                const uint32_t c = binfo[b];
                binfo[b] = run;                 // fill counter (high half) starts at 0
                run += c;
            }
        }
    }
    __syncthreads();
    // ---- 4. scatter the keys into their buckets; non-finite thresholds start past the top
    for (int i = tid; i < A; i += kHistThreads) {
        const uint32_t t = TH[i];
        if (t < 0x7f800000u) {
            const uint32_t old = atomicAdd(&binfo[(t >> shift) - base], 0x10000u);
            KH[(old & 0xffffu) + (old >> 16)] = ((uint64_t)t << 32) | (uint32_t)i;
        } else {
            TH[i] = Ap + 1u;
        }
    }
    for (uint32_t e = tid; e < nsplit; e += kHistThreads) {
        const uint32_t v = ((lo >> 23) + 1u + e) << 23;
        const uint32_t old = atomicAdd(&binfo[(v >> shift) - base], 0x10000u);
        KH[(old & 0xffffu) + (old >> 16)] = ((uint64_t)v << 32) | (uint32_t)(A + e);
    }
    __syncthreads();
    // ---- 5. order inside each bucket by counting: position = first + #smaller keys
    for (uint32_t k = tid; k < Ap; k += kHistThreads) {
        const uint64_t key = KH[k];
        const uint32_t v = (uint32_t)(key >> 32), id = (uint32_t)key;
        const uint32_t bi = binfo[(v >> shift) - base];
        const uint32_t o = bi & 0xffffu, n = bi >> 16;
        uint32_t pos = o;
        for (uint32_t t = o; t < o + n; t++) pos += (KH[t] < key) ? 1u : 0u;
        U[pos + 1] = v;
        if (id < (uint32_t)A) TH[id] = pos + 1;      // atom where this cell starts
    }
    if (tid == 0) { U[0] = 0u; U[Ap + 1] = 0xffffffffu; }
    const uint32_t afin = Ap;                        // the top atom [hi, inf)
    __syncthreads();   // the keys are dead: KH becomes the histogram
    // ---- 5b. bin pairs {first atom | bounds inside << 16, next bound}: with at
    //          most one bound inside, the atom of a value is first + (v >= next)
    {
        constexpr int kPer = 8192 / kHistThreads;
        uint32_t bv[kPer];
#pragma unroll
        for (int k = 0; k < kPer; k++) {
            const uint32_t b = (uint32_t)(tid + k * kHistThreads);
            bv[k] = b < nb ? binfo[b] : 0u;
        }
        for (uint32_t i = tid; i <= Ap; i += kHistThreads) hist[i] = 0;
        __syncthreads();
#pragma unroll
        for (int k = 0; k < kPer; k++) {
            const uint32_t b = (uint32_t)(tid + k * kHistThreads);
            if (b < nb || (b == 0 && nb == 0)) {
                binfo[2 * b] = bv[k];
                binfo[2 * b + 1] = U[(bv[k] & 0xffffu) + 1];
            }
        }
    }
    __syncthreads();

    // ---- 6. the pass
    double sumsq = 0.0, top_s1 = 0.0;
    uint32_t top_cnt = 0, flags = 0;
    constexpr int E = 8;
    // Per element: x^2 into the fp64 sum; |x| in [lo, hi) to its atom (bin
    // table, then one comparison against the next bound; a loop only where a
    // bin holds two or more bounds) and one LDS atomic adding
    // (mantissa << 20) + 1.  Every atom lies inside one binade, so the sum of
    // the 23-bit mantissas and the count give the exact sum of |x| over the
    // atom.  |x| >= hi (the top atom) and non-finite x are rare: a branch.
    const uint32_t span = hi - lo;
    const uint32_t bmax = base + (nb > 0 ? nb - 1u : 0u);
    const uint2* bins = (const uint2*)binfo;
    const uint32_t spare = (uint32_t)Aa + 1u + (uint32_t)(tid & 63);
    auto visit = [&](const uint32_t (&xb)[E]) {
        uint32_t ab[E], t[E];
        uint2 bi[E];
        bool mid[E];
        uint32_t mx = 0;
#pragma unroll
        for (int e = 0; e < E; e++) {
            ab[e] = xb[e] & 0x7fffffffu;
            const double xd = (double)__uint_as_float(ab[e]);
            sumsq = fma(xd, xd, sumsq);
            mx = max(mx, ab[e]);
            mid[e] = ab[e] - lo < span;                // atom 0 (q = 0 for all) adds nothing
            const uint32_t b = min(max(ab[e] >> shift, base), bmax) - base;
            bi[e] = bins[b];
        }
        bool walk = false;
#pragma unroll
        for (int e = 0; e < E; e++) {
            t[e] = (bi[e].x & 0xffffu) + ((ab[e] >= bi[e].y) ? 1u : 0u);
            walk |= mid[e] && bi[e].x >= 0x20000u;
        }
        if (walk) {                                    // a bin with two or more bounds
#pragma unroll
            for (int e = 0; e < E; e++)
                if (mid[e] && bi[e].x >= 0x20000u)
                    while (U[t[e] + 1] <= ab[e]) t[e]++;
        }
        if (mx >= hi) {                                // the top atom, non-finite x
#pragma unroll
            for (int e = 0; e < E; e++) {
                if (ab[e] >= hi) {
                    if (ab[e] < 0x7f800000u) {
                        top_s1 += (double)__uint_as_float(ab[e]);
                        top_cnt += 1u;
                    } else {
                        flags |= (ab[e] > 0x7f800000u) ? 2u : 1u;
                    }
                }
            }
        }
#pragma unroll
        for (int e = 0; e < E; e++) {   // outside [lo, hi): zero into the lane's own spare cell
            const uint32_t mant = ab[e] & 0x7fffffu;
            const uint64_t v = mid[e] ? (((uint64_t)mant << 20) | 1u) : 0u;
            atomicAdd(&hist[mid[e] ? t[e] : spare], v);
        }
    };
    const int64_t cnt_base = (int64_t)blockIdx.x * (int64_t)(Aa + 1);
    bool first_flush = true;
    auto flush = [&]() {
        __syncthreads();
        for (uint32_t i = tid; i <= Ap; i += kHistThreads) {
            const uint64_t v = hist[i];
            hist[i] = 0;
            const uint64_t c = v & 0xfffffu, s = v >> 20;
            if (first_flush) { w.pcnt[cnt_base + i] = c; w.psum[cnt_base + i] = s; }
            else if (v) { w.pcnt[cnt_base + i] += c; w.psum[cnt_base + i] += s; }
        }
        first_flush = false;
        __syncthreads();
    };
    // The pass, one chunk of loads ahead of the chunk being binned (the first
    // chunk was requested before the set-up).
    auto pass = [&](auto VEC) {
        auto load_chunk = [&](int64_t ch, uint32_t (&g)[16]) { load_chunk_t(VEC, ch, g); };
        int since = 0;
        for (int64_t ch = c0; ch < c1; ch++) {
            uint32_t g[16];
#pragma unroll
            for (int u = 0; u < 16; u++) g[u] = gn[u];
            load_chunk(ch + 1, gn);
#pragma unroll
            for (int h = 0; h < 2; h++) {
                uint32_t gg[E];
#pragma unroll
                for (int e = 0; e < E; e++) gg[e] = g[E * h + e];
                visit(gg);
            }
            if (++since == kFlushChunks) { flush(); since = 0; }
        }
    };
    if (c0 < c1) {
        if (vec) pass(std::integral_constant<bool, true>{});
        else pass(std::integral_constant<bool, false>{});
    }
    if (vec && blockIdx.x == gridDim.x - 1 && tid < (int)(len & 3)) {   // tail of the vector path
        uint32_t gg[E];
        gg[0] = __float_as_uint(x[(len & ~(int64_t)3) + tid]);
#pragma unroll
        for (int e = 1; e < E; e++) gg[e] = 0u;
        visit(gg);
    }
    flush();

    // ---- 7. block scalars; block 0 also publishes the tables
    if (flags) atomicOr(&s_flags, flags);
    {
        double v3[3] = {sumsq, top_s1, (double)top_cnt};   // counts exact in fp64
        block_sum_n<3>(v3, s_red3);
        if (tid == 0) {
            double* ps = w.pscal + 4 * blockIdx.x;
            ps[0] = v3[0]; ps[1] = v3[1]; ps[2] = v3[2]; ps[3] = (double)s_flags;
        }
    }
    if (blockIdx.x == 0) {
        for (uint32_t i = tid; i <= Ap + 1; i += kHistThreads) w.ubits[i] = U[i];
        for (int i = tid; i < A; i += kHistThreads) w.rank[i] = (int32_t)TH[i];
        if (tid == 0) { w.meta[0] = afin; w.meta[1] = Ap; }
    }
}

// -------------------------------------------------------------------- reduce
// Slice s of the blocks, per atom: sums of the per-block totals (integers).
__global__ __launch_bounds__(256) void k_dda_reduce(DdaArgs a, DdaWs w) {
    const int at = blockIdx.x * 256 + threadIdx.x;
    const int Aa1 = a.Aa + 1;
    if (at >= Aa1) return;
    const uint32_t Ap = w.meta[1];
    if ((uint32_t)at > Ap) return;
    const int s = blockIdx.y, per = (a.nblk + a.nslice - 1) / a.nslice;
    const int b0 = s * per, b1 = min(a.nblk, b0 + per);
    uint64_t c = 0, t = 0;
    for (int b = b0; b < b1; b++) {
        c += w.pcnt[(int64_t)b * Aa1 + at];
        t += w.psum[(int64_t)b * Aa1 + at];
    }
    w.rcnt[(int64_t)s * Aa1 + at] = c;
    w.rsum[(int64_t)s * Aa1 + at] = t;
}

// ------------------------------------------------------------------ finalize
constexpr int kFinThreads = 1024;

// The reduction over blocks and the per-candidate objective, for a block of
// kFinThreads threads.  P0, P1: LDS of (afin + 2) doubles each; Dv: LDS of G
// doubles.  ubits: the
// sorted atom bounds; rks: the atom where each cell starts (LDS or global).
// nsrc rows of per-atom partial sums in srcc / srcs, nblk rows of block scalars.
__device__ void finalize_core(const float* __restrict__ grid, const DdaArgs& a, const DdaWs& w,
                              float* __restrict__ alpha_out, double* __restrict__ D_out,
                              double* P0, double* P1, const uint32_t* ubits, const int32_t* rks,
                              uint32_t afin, int nsrc, const uint64_t* srcc, const uint64_t* srcs,
                              int nblk, double* Dv) {
    const int tid = threadIdx.x, G = a.G, M = a.M;
    const int Aa1 = a.Aa + 1;
    __shared__ double s_red3[3][16];
    __shared__ double sq[128];
    __shared__ uint32_t s_fl;
    if (tid <= M) sq[tid] = (double)a.q[tid];
    if (tid == 0) s_fl = 0;
    // block scalars
    double v3[3] = {0.0, 0.0, 0.0};
    uint32_t fl = 0;
    for (int b = tid; b < nblk; b += kFinThreads) {
        const double* ps = w.pscal + 4 * b;
        v3[0] += ps[0]; v3[1] += ps[1]; v3[2] += ps[2]; fl |= (uint32_t)ps[3];
    }
    block_sum_n<3>(v3, s_red3);
    const double sumsq = v3[0], top_s1 = v3[1], top_c = v3[2];
    if (fl) atomicOr(&s_fl, fl);
    // per-atom sums S0, S1 for atoms 0..afin (atom 0 carries q = 0 for everyone),
    // loaded coalesced into LDS, then an in-place exclusive prefix scan over atoms
    for (int at = tid; at <= (int)afin + 1; at += kFinThreads) {
        double s0 = 0.0, s1 = 0.0;
        if (at >= 1 && (uint32_t)at < afin) {
            uint64_t c = 0, t = 0;
#pragma unroll 8
            for (int b = 0; b < nsrc; b++) {
                c += srcc[(int64_t)b * Aa1 + at];
                t += srcs[(int64_t)b * Aa1 + at];
            }
            // mantissa sums: add the implicit bit of a normal binade per element
            const uint32_t ex = ubits[at] >> 23;
            if (ex) t += c << 23;
            s0 = (double)c;
            s1 = ldexp((double)t, (int)max(ex, 1u) - 150);
        } else if (afin > 0 && (uint32_t)at == afin) {
            s0 = top_c;
            s1 = top_s1;
        }
        P0[at] = s0;
        P1[at] = s1;
    }
    __syncthreads();
    {
        const int per = ((int)afin + 2 + kFinThreads - 1) / kFinThreads;
        double m0 = 0.0, m1 = 0.0;
        for (int e = 0; e < per; e++) {
            const int at = tid * per + e;
            if (at <= (int)afin + 1) { m0 += P0[at]; m1 += P1[at]; }
        }
        const double m2[2] = {m0, m1};
        double bef[2], tot[2];
        block_exclusive_scan_n<2>(m2, s_red3, bef, tot);
        double r0 = bef[0], r1 = bef[1];
        for (int e = 0; e < per; e++) {
            const int at = tid * per + e;
            if (at <= (int)afin + 1) {
                const double v0 = P0[at], v1 = P1[at];
                P0[at] = r0;
                P1[at] = r1;
                r0 += v0;
                r1 += v1;
            }
        }
    }
    __syncthreads();
    // per candidate: cells as atom ranges [start_c, start_{c+1}), the last one to afin+1
    for (int j = tid; j < G; j += kFinThreads) {
        const int32_t* rkj = rks + (int64_t)j * M;
        const int end = (int)afin + 1;
        double Aj = 0.0, Bj = 0.0;
        int start = min(rkj[0], end);
        for (int c = 1; c <= M; c++) {
            const int next = (c < M) ? min(rkj[c], end) : end;
            const double q = sq[c];
            Aj = fma(q, P1[next] - P1[start], Aj);
            Bj = fma(q * q, P0[next] - P0[start], Bj);
            start = next;
        }
        const float al = grid[j];
        const double ad = (double)al;
        double D = fma(ad, fma(ad, Bj, -2.0 * Aj), sumsq);
        if (!alpha_ok(al) || (s_fl & 2u)) D = __builtin_nan("");
        else if (s_fl & 1u) D = __builtin_inf();
        Dv[j] = D;
    }
    __syncthreads();
    if (tid < 64) {
        // argmin over (isnan(D), D, j) in lexicographic order: the smallest index
        // with the least D, NaN ranking above every number
        double bd = __builtin_nan("");
        int bj = 0x7fffffff;
        for (int jj = tid; jj < G; jj += 64) {
            const double d = Dv[jj];
            const bool better = (d < bd) || (bd != bd && d == d) || (bj == 0x7fffffff);
            if (better) { bd = d; bj = jj; }
        }
        for (int off = 32; off > 0; off >>= 1) {
            const double od = __shfl_xor(bd, off);
            const int oj = __shfl_xor(bj, off);
            const bool onan = od != od, mnan = bd != bd;
            const bool better = (!onan && mnan) || (onan == mnan && (od < bd || (od == bd && oj < bj))) ||
                                (onan && mnan && oj < bj);
            if (better) { bd = od; bj = oj; }
        }
        if (tid == 0) *alpha_out = grid[bj];
    }
    if (D_out)
        for (int jj = tid; jj < G; jj += kFinThreads) D_out[jj] = Dv[jj];
}

__global__ __launch_bounds__(kFinThreads) void k_dda_finalize(const float* __restrict__ grid,
                                                              DdaArgs a, DdaWs w,
                                                              float* __restrict__ alpha_out,
                                                              double* __restrict__ D_out) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x;
    const int Aa1 = a.Aa + 1;
    double* P0 = (double*)smem;                  // [Aa+2] prefix sums of counts
    double* P1 = P0 + (Aa1 + 1);                 // [Aa+2] prefix sums of |x|
    double* Dv = P1 + (Aa1 + 1);                 // [G] objective per candidate
    int32_t* rk = (int32_t*)(Dv + a.G);         // [A] first atom of every cell
    if (a.rk_lds)
        for (int i = tid; i < a.A; i += kFinThreads) rk[i] = w.rank[i];
    const bool sliced = a.nslice > 0;
    finalize_core(grid, a, w, alpha_out, D_out, P0, P1, w.ubits, a.rk_lds ? rk : w.rank, w.meta[0],
                  sliced ? a.nslice : a.nblk, sliced ? w.rcnt : w.pcnt, sliced ? w.rsum : w.psum,
                  a.nblk, Dv);
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
    for (int c = 0; c <= M; c++) a.q[c] = (float)vals[c];
    for (int c = 1; c <= M; c++) a.mids[c - 1] = (float)(0.5 * (vals[c - 1] + vals[c]));
    a.G = G; a.M = M; a.A = L.A; a.Aa = L.A + kMaxSplits; a.nblk = L.nblk;
    a.nslice = L.nblk > 2 * kReduceSlices ? kReduceSlices : 0;
    a.rk_lds = 0;
    const DdaWs w = ws_ptrs(ws, L);
    static bool lds_attr_set[64] = {false};
    int dev = 0;
    if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < 64 && !lds_attr_set[dev]) {
        hipError_t e = hipFuncSetAttribute((const void*)k_dda_hist,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 150 * 1024);
        if (e != hipSuccess) return e;
        e = hipFuncSetAttribute((const void*)k_dda_finalize,
                                hipFuncAttributeMaxDynamicSharedMemorySize, 150 * 1024);
        if (e != hipSuccess) return e;
        lds_attr_set[dev] = true;
    }
    k_dda_hist<<<L.nblk, kHistThreads, hist_lds_bytes(L.A), s>>>(x, len, grid, a, w);
    if (a.nslice > 0) {
        dim3 rg((a.Aa + 1 + 255) / 256, a.nslice);
        k_dda_reduce<<<rg, 256, 0, s>>>(a, w);
    }
    size_t fin_lds = sizeof(double) * (2 * (size_t)(a.Aa + 2) + (size_t)G);
    a.rk_lds = fin_lds + sizeof(int32_t) * (size_t)a.A <= 140 * 1024;
    if (a.rk_lds) fin_lds += sizeof(int32_t) * (size_t)a.A;
    k_dda_finalize<<<1, kFinThreads, fin_lds, s>>>(grid, a, w, alpha_out, D_out);
    return hipGetLastError();
}

}  // namespace esb
