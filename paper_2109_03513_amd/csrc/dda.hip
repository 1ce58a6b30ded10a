// Distribution difference aligner (eq. (9), (13)) on the data, gfx950.
//
// Objective per candidate scale alpha_j:  D_j = sum_i (|x_i| - alpha_j q_j(x_i))^2
//   = S2 - 2 alpha_j sum_i |x_i| q_j(x_i) + alpha_j^2 sum_i q_j(x_i)^2,
// with S2 = sum_i x_i^2.  q_j(x) depends on x only through which cell of
// candidate j holds |x|, and the cell boundaries are exact fp32 thresholds:
// T_{j,c} = the smallest fp32 X with fl32(X / alpha_j) >= mu_c, mu_c the
// midpoint between set values c-1 and c (ties go up, as in the projection).
// The distinct values among all G*M thresholds and the powers of two between
// them cut [0, inf) into "atoms": every candidate's cell is a union of
// consecutive atoms and every bounded atom lies inside one binade.  (Grids of
// scales such as fl32(s (j+1)/64) make many thresholds coincide: merging them
// leaves few bins holding two bounds.)  One pass over x suffices.
//
// k_dda_hist (blocks of 1024 threads, each over at most 2^19 elements):
//   set-up in LDS: thresholds by a local search around fl32(alpha mu); bucket
//   placement by bin of the bit pattern (counts, scan, scatter, order inside a
//   bucket by counting), a scan that merges equal bounds, which gives the
//   distinct sorted bounds and each cell's first atom; then a table of 8-byte
//   bin entries {first atom | flags, the next
//   bound}, so that the atom of a value is first + (value >= that bound)
//   unless the bin holds two or more bounds (a flagged walk over the sorted
//   bounds; large inputs use 16384 bins, where such bins are rare).
//   The pass: per element one entry read and one LDS atomic adding
//   {significand, 1} to a packed 64-bit (count << 44 | sum) cell; x^2 in fp64.
//   Values below the smallest threshold fall in atom 0, where q = 0 for every
//   candidate: they add nothing (ReLU zeros never touch one LDS address).
//   Values at or above the largest threshold (the unbounded top atom) and
//   non-finite values land in the flagged last bin and are summed in fp64.
//   At the end the block turns its own cells into its share of the objective:
//   per-atom moments, prefix sums over atoms (counts in integers, sums of |x|
//   in fp64), then per candidate A_j = sum_c Q_c (P1[end_c] - P1[start_c]) and
//   B_j = sum_c Q_c^2 (P0[end_c] - P0[start_c]), written with the block's
//   sum x^2 as one short vector.
// k_dda_finalize (1 block): sums the block vectors in block order, D_j =
//   S2 + a (a B_j - 2 A_j), argmin with ties to the lowest index.
// Per-atom sums are exact integers; fp64 sums run in a fixed order: the result
// is deterministic.  Wave-level scans and reductions use DPP lane moves.
#include <atomic>

#include "esb_internal.h"

namespace esb {

constexpr int kHistThreads = 1024;
constexpr int kFinThreads = 1024;
constexpr int kMaxSplits = 256;            // powers of two between thresholds (at most 254)
constexpr int kRowElems = 4 * kHistThreads; // one float4 per thread
constexpr int kMaxRowsPerBlock = 128;      // 2^19 elements: a packed cell cannot overflow
constexpr uint32_t kFlagWalk = 1u << 31;   // bin holds two or more bounds
constexpr uint32_t kFlagTop = 1u << 30;    // last bin: values >= the largest threshold
constexpr uint32_t kAtomMask = (1u << 29) - 1u;
constexpr uint64_t kSumMask = (1ull << 44) - 1ull;

struct DdaArgs {
    int G, M, A, Aa;        // candidates, midpoints, thresholds G*M, A + kMaxSplits
    int n, k;               // format (k fraction bits)
    int lbins;              // log2 of the bin count of the pass
    int nblk, rows_pb;      // blocks of k_dda_hist, rows of kRowElems per block
};

// Per block of k_dda_hist, 2G + 2 doubles: A_0 .. A_{G-1}, B_0 .. B_{G-1}, the
// block's sum x^2, its flags (1: +-inf seen, 2: NaN seen).
__host__ __device__ inline int part_stride(int G) { return 2 * G + 2; }
// Above kGroupAbove blocks, k_dda_group first sums groups of kGroup
// consecutive block vectors (many CUs, one round of loads each); the finalize
// then reads the group vectors.
constexpr int kGroup = 16;
constexpr int kGroupAbove = 32;
__host__ __device__ inline int dda_groups(int nblk) {
    return nblk > kGroupAbove ? (nblk + kGroup - 1) / kGroup : 0;
}

__host__ __device__ static inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }
__host__ __device__ static inline size_t align16(size_t v) { return (v + 15) & ~(size_t)15; }

// Block geometry: rows of 4096 elements; two rows per block for small inputs
// (short passes on many CUs), at most 128 per block.
static void dda_blocks(int64_t len, int* nblk, int* rows_pb) {
    const int64_t rows = (len + kRowElems - 1) / kRowElems;
    int64_t rpb = 2;
    if (rows > 2 * 256) {
        rpb = (rows + 255) / 256;
        rpb = (rpb + 1) & ~(int64_t)1;
        if (rpb > kMaxRowsPerBlock) rpb = kMaxRowsPerBlock;
    }
    int64_t nb = (rows + rpb - 1) / rpb;
    *nblk = (int)(nb < 1 ? 1 : nb);
    *rows_pb = (int)rpb;
}

bool dda_layout(int64_t len, const Fmt& f, int G, DdaLayout* L) {
    const int M = (1 << (f.n - 1)) - 1;
    if (G < 1 || G > kDdaMaxG || (int64_t)G * M > kDdaMaxThresholds || len < 0) return false;
    if (len > ((int64_t)1 << 46)) return false;
    L->G = G;
    L->M = M;
    L->A = G * M;
    int rpb = 0;
    dda_blocks(len, &L->nblk, &rpb);
    const size_t ps = sizeof(double) * (size_t)part_stride(G);
    L->off_part = 0;
    L->off_group = align256(ps * (size_t)L->nblk);
    L->total = L->off_group + align256(ps * (size_t)dda_groups(L->nblk));
    return true;
}

// ------------------------------------------------------------ wave primitives
// DPP lane moves (gfx9): row_shr:n = 0x110 + n, row_bcast:15 = 0x142 (lane 15
// of each row to the next row), row_bcast:31 = 0x143 (lane 31 to rows 2, 3).
// A lane whose source is outside its row, or whose row is masked off, keeps
// `old` (the identity of the operation).
template <int CTRL, int ROWMASK>
__device__ __forceinline__ uint32_t dpp(uint32_t old, uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROWMASK, 0xf, false);
}
template <int CTRL, int ROWMASK>
__device__ __forceinline__ double dpp_f64(double v) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = dpp<CTRL, ROWMASK>(0u, (uint32_t)b);
    const uint32_t hi = dpp<CTRL, ROWMASK>(0u, (uint32_t)(b >> 32));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Inclusive scans over the 64 lanes of a wave (Hillis-Steele inside rows of 16,
// then the row totals carried across rows).  Fixed order: deterministic.
__device__ __forceinline__ uint32_t wave_scan_add(uint32_t v) {
    v += dpp<0x111, 0xf>(0u, v);
    v += dpp<0x112, 0xf>(0u, v);
    v += dpp<0x114, 0xf>(0u, v);
    v += dpp<0x118, 0xf>(0u, v);
    v += dpp<0x142, 0xa>(0u, v);
    v += dpp<0x143, 0xc>(0u, v);
    return v;
}
__device__ __forceinline__ double wave_scan_add(double v) {
    v += dpp_f64<0x111, 0xf>(v);
    v += dpp_f64<0x112, 0xf>(v);
    v += dpp_f64<0x114, 0xf>(v);
    v += dpp_f64<0x118, 0xf>(v);
    v += dpp_f64<0x142, 0xa>(v);
    v += dpp_f64<0x143, 0xc>(v);
    return v;
}
__device__ __forceinline__ uint32_t wave_scan_min(uint32_t v) {
    v = min(v, dpp<0x111, 0xf>(~0u, v));
    v = min(v, dpp<0x112, 0xf>(~0u, v));
    v = min(v, dpp<0x114, 0xf>(~0u, v));
    v = min(v, dpp<0x118, 0xf>(~0u, v));
    v = min(v, dpp<0x142, 0xa>(~0u, v));
    v = min(v, dpp<0x143, 0xc>(~0u, v));
    return v;
}
__device__ __forceinline__ uint32_t wave_scan_max(uint32_t v) {
    v = max(v, dpp<0x111, 0xf>(0u, v));
    v = max(v, dpp<0x112, 0xf>(0u, v));
    v = max(v, dpp<0x114, 0xf>(0u, v));
    v = max(v, dpp<0x118, 0xf>(0u, v));
    v = max(v, dpp<0x142, 0xa>(0u, v));
    v = max(v, dpp<0x143, 0xc>(0u, v));
    return v;
}
__device__ __forceinline__ uint32_t wave_scan_or(uint32_t v) {
    v |= dpp<0x111, 0xf>(0u, v);
    v |= dpp<0x112, 0xf>(0u, v);
    v |= dpp<0x114, 0xf>(0u, v);
    v |= dpp<0x118, 0xf>(0u, v);
    v |= dpp<0x142, 0xa>(0u, v);
    v |= dpp<0x143, 0xc>(0u, v);
    return v;
}
__device__ __forceinline__ uint32_t lane63(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}
__device__ __forceinline__ double lane63(double v) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), 63);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Workgroup barrier for LDS only.  __syncthreads() also waits for every global
// load in flight (here: the prefetched chunk of x, which the set-up is meant
// to overlap); all communication between threads in these kernels is through
// LDS.  The memory clobber keeps the compiler from moving LDS accesses across.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}


// Median of three (v_med3_u32): x clamped to [lo, hi] when lo <= hi.
__device__ __forceinline__ uint32_t med3_u32(uint32_t x, uint32_t lo, uint32_t hi) {
    uint32_t r;
    asm("v_med3_u32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "v"(lo), "v"(hi));
    return r;
}

__device__ __forceinline__ bool alpha_ok(float a) { return a > 0.0f && a < __builtin_inff(); }

// Smallest fp32 X >= 0 (as bits) with fl32(X / alpha) >= mu (IEEE division,
// round to nearest even), for alpha > 0 finite and mu a positive normal fp32
// whose significand is even (a set midpoint has at most k + 2 significant
// bits).  With p the fp32 just below mu, the quotient rounds to mu or above
// exactly when X / alpha >= m = (p + mu) / 2 (a tie goes to the even mu), that
// is X >= alpha * m.  That product has at most 24 + 25 significant bits, so it
// is exact in fp64, and X is its rounding up to fp32 (+inf past the largest).
__device__ __forceinline__ uint32_t threshold_bits(float alpha, float mu) {
    const double m = 0.5 * ((double)__uint_as_float(__float_as_uint(mu) - 1u) + (double)mu);
    const double t = (double)alpha * m;
    const float f = (float)t;
    uint32_t b = __float_as_uint(f);
    if ((double)f < t) b++;
    return b > 0x7f800000u ? 0x7f800000u : b;
}

// Bins of the pass: more bins make crowded bins (two or more bounds, a walk)
// rarer but cost set-up time, which dominates for small inputs.
static inline int hist_lbins(int A, bool large) {
    if (A <= 960) return large ? 13 : 12;
    if (A <= 4096) return large ? 13 : 12;
    return 11;
}
// Dynamic LDS of k_dda_hist:
//   ENT  uint2[nbins]  bin entries; during the set-up its start holds the bin
//                      counts u32[nbins] (first atom | count << 16)
//   U    u32[Aa + 4]   sorted atom bounds, padded with ~0
//   TH   u32[A]        thresholds, then the atom where each cell starts
//   KH   u64[C(Aa+1)+64] (bound << 32 | id) bucket keys, then the packed
//                      histogram: C interleaved copies (cell C*atom + lane % C,
//                      so that lanes on one dense atom add into different
//                      banks), then one spare cell per lane
struct HistLds {
    size_t u, th, kh, total;
};
__host__ __device__ static inline int hist_lcopies(int A) { return A <= 256 ? 4 : (A <= 960 ? 2 : 0); }
__host__ __device__ static inline HistLds hist_lds(int A, int lbins) {
    HistLds h;
    const size_t Aa = (size_t)A + kMaxSplits;
    h.u = (size_t)8 << lbins;
    h.th = h.u + align16(sizeof(uint32_t) * (Aa + 4));
    h.kh = h.th + align16(sizeof(uint32_t) * (size_t)A);
    h.total = h.kh + sizeof(uint64_t) * (((Aa + 1) << hist_lcopies(A)) + 64);
    return h;
}

// A plan: the grid-only part of the set-up for candidates factor_j (scale 1),
// dumped from LDS once, so that a call with candidates 2^E factor_j loads it
// instead of rebuilding it.  Multiplying a candidate by 2^E multiplies each of
// its exact thresholds by 2^E (the quotient fl32(X / alpha) is unchanged when
// X and alpha both scale and stay normal), and adding E << 23 to a normal fp32
// bit pattern is that multiplication, so the loaded bounds are the bounds of
// the scaled grid bit for bit while E lies in [emin, emax] (every threshold and
// every candidate stays normal).  Layout: this header, the G factors, the bin
// entries (nbins uint2), the distinct bounds U (A + 260 u32), the cell starts
// TH (A u32), each 16-byte aligned.
struct DdaPlanHead {
    uint32_t magic;
    int n, k, G, M, A, lbins;
    uint32_t shift, base, nb, hi, Dp;
    int emin, emax;
};
constexpr uint32_t kPlanMagic = 0x45534250u;   // "ESBP"
__host__ __device__ inline size_t plan_factors_off() { return align16(sizeof(DdaPlanHead)); }
__host__ __device__ inline size_t plan_ent_off(int G) {
    return plan_factors_off() + align16(sizeof(float) * (size_t)G);
}
__host__ __device__ inline size_t plan_u_off(int G, int lbins) {
    return plan_ent_off(G) + ((size_t)8 << lbins);
}
__host__ __device__ inline size_t plan_th_off(int G, int A, int lbins) {
    return plan_u_off(G, lbins) + align16(sizeof(uint32_t) * ((size_t)A + kMaxSplits + 4));
}
__host__ __device__ inline size_t plan_total(int G, int A, int lbins) {
    return plan_th_off(G, A, lbins) + align16(sizeof(uint32_t) * (size_t)A);
}
// Plans use the bins of large inputs (few crowded bins); loading them costs
// the same at every size.
inline int plan_lbins(int A) { return hist_lbins(A, true); }

// One block (local index bid of its job) of the histogram pass.  plan_in: the
// job's candidates are 2^E factor_j (factor_j = grid[j], E the binary exponent
// of |*gscale|) and the grid-only tables come from this plan when E is inside
// its range (else they are rebuilt as without a plan).  plan_out: build a plan
// (x empty): dump the tables after the set-up and return.
__device__ __forceinline__ void dda_hist_block(const float* __restrict__ x, int64_t len,
                                               const float* __restrict__ grid,
                                               const float* __restrict__ gscale, const DdaArgs a,
                                               double* __restrict__ part, const int bid,
                                               const uint8_t* __restrict__ plan_in,
                                               uint8_t* __restrict__ plan_out) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int A = a.A, M = a.M, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int nbins = 1 << a.lbins;
    const uint32_t lcop = (uint32_t)hist_lcopies(A);   // log2 of the histogram copies
    const HistLds hl = hist_lds(A, a.lbins);
    uint2* ENT = (uint2*)smem;
    uint32_t* binc = (uint32_t*)smem;
    uint32_t* U = (uint32_t*)(smem + hl.u);
    uint32_t* TH = (uint32_t*)(smem + hl.th);
    uint64_t* KH = (uint64_t*)(smem + hl.kh);
    uint64_t* hist = KH;
    __shared__ float s_mid[128];
    __shared__ uint32_t s_u[4][16];
    __shared__ double s_d[3][16];

    // ---- 0. requests first: this thread's candidate scales and the first chunk
    //         of x, so that both latencies overlap the clearing of the bins.
    constexpr int kMaxTpt = kDdaMaxThresholds / kHistThreads;   // thresholds per thread
    const float gsc = gscale ? *gscale : 1.0f;   // candidates fl32(gsc * grid[j])
    // planned: candidates 2^pe factor_j, 2^(pe-1) <= |gsc| < 2^pe (pe = 0 for 0); a
    // scale that is not finite makes every candidate NaN
    int pe = 0;
    bool use_plan = false;
    const bool sc_ok = __builtin_isfinite(gsc);
    if (plan_in) {
        frexpf(fabsf(gsc), &pe);
        const DdaPlanHead& ph = *(const DdaPlanHead*)plan_in;
        const bool head_ok = ph.magic == kPlanMagic && ph.n == a.n && ph.k == a.k && ph.G == a.G &&
                             ph.M == M && ph.A == A && ph.lbins == a.lbins &&
                             ph.nb <= (uint32_t)nbins && nbins <= (1 << 13) &&
                             ph.Dp <= (uint32_t)a.Aa && ph.shift < 23u;
        use_plan = head_ok && sc_ok && pe >= ph.emin && pe <= ph.emax;
    }
    float al[kMaxTpt];
#pragma unroll
    for (int r = 0; r < kMaxTpt; r++) {
        const int i = tid + r * kHistThreads;
        float v = 1.0f;
        if (i < A) {
            if (plan_in) v = sc_ok ? ldexpf(grid[i / M], pe) : __builtin_nanf("");
            else v = gscale ? gsc * grid[i / M] : grid[i / M];
        }
        al[r] = v;
    }
    const bool vec = ((uintptr_t)x & 15) == 0;
    const int64_t e0 = (int64_t)bid * a.rows_pb * kRowElems;
    const int64_t e1 = min(len, e0 + (int64_t)a.rows_pb * kRowElems);
    // element range of the vector path: whole float4 only; the last block takes
    // the len % 4 tail separately
    const int64_t v1 = vec ? (e1 & ~(int64_t)3) : e1;
    auto load_chunk = [&](int64_t c, uint32_t (&g)[16]) {   // c: first element of the chunk
        if (vec) {
            const f32x4* x4 = (const f32x4*)x;
#pragma unroll
            for (int u = 0; u < 4; u++) {
                const int64_t e = c + 4 * ((int64_t)u * kHistThreads + tid);
                const bool in = e < v1;
                const f32x4 v = __builtin_nontemporal_load(&x4[in ? (e >> 2) : 0]);
                g[4 * u + 0] = in ? __float_as_uint(v.x) : 0u;
                g[4 * u + 1] = in ? __float_as_uint(v.y) : 0u;
                g[4 * u + 2] = in ? __float_as_uint(v.z) : 0u;
                g[4 * u + 3] = in ? __float_as_uint(v.w) : 0u;
            }
        } else {
#pragma unroll
            for (int u = 0; u < 16; u++) {
                const int64_t e = c + 4 * ((int64_t)(u >> 2) * kHistThreads + tid) + (u & 3);
                const bool in = e < v1;
                g[u] = in ? __float_as_uint(x[in ? e : 0]) : 0u;
            }
        }
    };
    auto load_full = [&](int64_t c, uint32_t (&g)[16]) {    // a whole chunk inside [e0, v1)
        if (vec) {
            const f32x4* x4 = (const f32x4*)x + (c >> 2) + tid;
#pragma unroll
            for (int u = 0; u < 4; u++) {
                const f32x4 v = __builtin_nontemporal_load(&x4[u * kHistThreads]);
                g[4 * u + 0] = __float_as_uint(v.x);
                g[4 * u + 1] = __float_as_uint(v.y);
                g[4 * u + 2] = __float_as_uint(v.z);
                g[4 * u + 3] = __float_as_uint(v.w);
            }
        } else {
#pragma unroll
            for (int u = 0; u < 16; u++)
                g[u] = __float_as_uint(x[c + 4 * ((int64_t)(u >> 2) * kHistThreads + tid) + (u & 3)]);
        }
    };
    uint32_t gn[16];
    constexpr int64_t kChunkElems = 4 * 4 * kHistThreads;
    if (e0 + kChunkElems <= v1) load_full(e0, gn);
    else if (e0 < v1) load_chunk(e0, gn);   // (x may be NULL when len == 0)
    uint32_t shift = 0, base = 0, nb = 1, lo = 0x7f800000u, hi = 0x7f800000u, Dp = 0;
    uint32_t ec_lo = 255u, ec_hi = 0u, plan_bad = 0u;   // plan building only
    if (use_plan) {
        // the tables of the plan, every bound multiplied by 2^pe (pe << 23 added to
        // its bit pattern); padding (~0) and the zero lower bound of atom 0 stay
        const DdaPlanHead& ph = *(const DdaPlanHead*)plan_in;
        const uint32_t d = (uint32_t)pe << 23;
        shift = ph.shift;
        base = ph.base + (uint32_t)(pe * (1 << (23 - (int)ph.shift)));
        nb = ph.nb;
        hi = ph.hi + d;
        Dp = ph.Dp;
        const uint2* pe = (const uint2*)(plan_in + plan_ent_off(ph.G));
        const uint32_t* pu = (const uint32_t*)(plan_in + plan_u_off(ph.G, ph.lbins));
        const uint32_t* pt = (const uint32_t*)(plan_in + plan_th_off(ph.G, ph.A, ph.lbins));
        // every load in flight before the first store (at most 8192 bins, A + 260
        // bounds and A cell starts: 8, 9 and 8 per thread)
        constexpr int kB = (1 << 13) / kHistThreads;
        constexpr int kU = (kDdaMaxThresholds + kMaxSplits + 4 + kHistThreads - 1) / kHistThreads;
        constexpr int kT = kDdaMaxThresholds / kHistThreads;
        uint2 ev[kB];
        uint32_t uv[kU], tv[kT];
#pragma unroll
        for (int q = 0; q < kB; q++) {
            const uint32_t b = (uint32_t)(tid + q * kHistThreads);
            ev[q] = b < nb ? pe[b] : make_uint2(0u, 0u);
        }
#pragma unroll
        for (int q = 0; q < kU; q++) {
            const uint32_t i = (uint32_t)(tid + q * kHistThreads);
            uv[q] = i < Dp + 4u ? pu[i] : 0u;
        }
#pragma unroll
        for (int q = 0; q < kT; q++) {
            const int i = tid + q * kHistThreads;
            tv[q] = i < A ? pt[i] : 0u;
        }
#pragma unroll
        for (int q = 0; q < kB; q++) {
            const uint32_t b = (uint32_t)(tid + q * kHistThreads);
            if (b < nb) {
                uint2 e = ev[q];
                e.y = e.y == 0xffffffffu ? e.y : e.y + d;
                ENT[b] = e;
            }
        }
#pragma unroll
        for (int q = 0; q < kU; q++) {
            const uint32_t i = (uint32_t)(tid + q * kHistThreads);
            if (i < Dp + 4u) U[i] = (i == 0u || uv[q] == 0xffffffffu) ? uv[q] : uv[q] + d;
        }
#pragma unroll
        for (int q = 0; q < kT; q++) {
            const int i = tid + q * kHistThreads;
            if (i < A) TH[i] = tv[q];
        }
        for (uint32_t i = tid; i < ((Dp + 1u) << lcop); i += kHistThreads) hist[i] = 0ull;
        lds_barrier();
    } else {
        if (tid < M) s_mid[tid] = set_mid(tid + 1, a.k);
        for (int b = tid; b < nbins; b += kHistThreads) binc[b] = 0u;
        lds_barrier();

        // ---- 1. thresholds, their finite range and count
        {
            uint32_t wlo = 0x7f800000u, whi = 0u, wn = 0u;
    #pragma unroll
            for (int r = 0; r < kMaxTpt; r++) {
                const int i = tid + r * kHistThreads;
                if (r * kHistThreads < A && i < A) {
                    const int c = i - (i / M) * M;
                    const bool ok = alpha_ok(al[r]);
                    const uint32_t t = ok ? threshold_bits(al[r], s_mid[c]) : 0x7f800000u;
                    TH[i] = t;
                    if (t < 0x7f800000u) { wlo = min(wlo, t); whi = max(whi, t); wn++; }
                    if (ok) {   // for a plan: the exponents a scaled grid must keep normal
                        const uint32_t ec = __float_as_uint(al[r]) >> 23;
                        ec_lo = min(ec_lo, ec);
                        ec_hi = max(ec_hi, ec);
                        if (ec == 0u || t < 0x00800000u) plan_bad |= 1u;   // subnormal
                        if (t >= 0x7f800000u) plan_bad |= 2u;              // overflowed
                    }
                }
            }
            wlo = wave_scan_min(wlo);
            whi = wave_scan_max(whi);
            wn = wave_scan_add(wn);
            if (lane == 63) { s_u[0][wid] = wlo; s_u[1][wid] = whi; s_u[2][wid] = wn; }
        }
        lds_barrier();
        uint32_t nfin = 0u;
        lo = 0x7f800000u;
        hi = 0u;
    #pragma unroll
        for (int v = 0; v < kHistThreads / 64; v++) {
            lo = min(lo, s_u[0][v]);
            hi = max(hi, s_u[1][v]);
            nfin += s_u[2][v];
        }
        if (nfin == 0) { lo = 0x7f800000u; hi = 0x7f800000u; }
        shift = 0;
        while (((hi >> shift) - (lo >> shift)) >= (uint32_t)(nbins - 1)) shift++;   // <= 21
        base = lo >> shift;
        nb = (hi >> shift) - base + 1u;
        // binade starts strictly inside (lo, hi)
        const uint32_t nsplit = (hi > lo) ? ((hi - 1u) >> 23) - (lo >> 23) : 0u;
        const uint32_t Ap = nfin + nsplit;

        // ---- 2. bounds per bin: finite thresholds and the powers of two in (lo, hi)
        for (int i = tid; i < A; i += kHistThreads) {
            const uint32_t t = TH[i];
            if (t < 0x7f800000u) atomicAdd(&binc[(t >> shift) - base], 1u);
        }
        for (uint32_t e = tid; e < nsplit; e += kHistThreads)
            atomicAdd(&binc[((((lo >> 23) + 1u + e) << 23) >> shift) - base], 1u);
        lds_barrier();

        // ---- 3. first atom of every bin: exclusive scan of the counts, P bins per thread
        const int P = nbins / kHistThreads;   // 16, 8, 4 or 2 bins per thread
        {
            uint32_t cnt[16];
            uint4* b4 = (uint4*)binc;
    #pragma unroll
            for (int q = 0; q < 4; q++) {
                if (4 * q < P && P >= 4) {
                    const uint4 u = b4[tid * (P / 4) + q];
                    cnt[4 * q] = u.x; cnt[4 * q + 1] = u.y; cnt[4 * q + 2] = u.z; cnt[4 * q + 3] = u.w;
                } else {
                    cnt[4 * q] = cnt[4 * q + 1] = cnt[4 * q + 2] = cnt[4 * q + 3] = 0u;
                }
            }
            if (P == 2) {
                const uint2 u = ((const uint2*)binc)[tid];
                cnt[0] = u.x; cnt[1] = u.y;
            }
            uint32_t mine = 0;
    #pragma unroll
            for (int e = 0; e < 16; e++) mine += cnt[e];
            const uint32_t incl = wave_scan_add(mine);
            if (lane == 63) s_u[3][wid] = incl;
            lds_barrier();
            uint32_t run = incl - mine;
            for (int v = 0; v < wid; v++) run += s_u[3][v];
            uint32_t st[16];                        // fill counter (high half) starts at 0
    #pragma unroll
            for (int e = 0; e < 16; e++) { st[e] = run; run += cnt[e]; }
    #pragma unroll
            for (int q = 0; q < 4; q++)
                if (4 * q < P && P >= 4)
                    b4[tid * (P / 4) + q] = make_uint4(st[4 * q], st[4 * q + 1], st[4 * q + 2], st[4 * q + 3]);
            if (P == 2) ((uint2*)binc)[tid] = make_uint2(st[0], st[1]);
        }
        lds_barrier();

        // ---- 4. scatter the keys into their buckets; non-finite thresholds start past the top
        for (int i = tid; i < A; i += kHistThreads) {
            const uint32_t t = TH[i];
            if (t < 0x7f800000u) {
                const uint32_t old = atomicAdd(&binc[(t >> shift) - base], 0x10000u);
                KH[(old & 0xffffu) + (old >> 16)] = ((uint64_t)t << 32) | (uint32_t)i;
            } else {
                TH[i] = Ap + 1u;
            }
        }
        for (uint32_t e = tid; e < nsplit; e += kHistThreads) {
            const uint32_t v = ((lo >> 23) + 1u + e) << 23;
            const uint32_t old = atomicAdd(&binc[(v >> shift) - base], 0x10000u);
            KH[(old & 0xffffu) + (old >> 16)] = ((uint64_t)v << 32) | (uint32_t)(A + e);
        }
        lds_barrier();

        // ---- 5. order inside each bucket by counting: position = first + #smaller keys
        for (uint32_t k = tid; k < Ap; k += kHistThreads) {
            const uint64_t key = KH[k];
            const uint32_t v = (uint32_t)(key >> 32), id = (uint32_t)key;
            const uint32_t bi = binc[(v >> shift) - base];
            const uint32_t o = bi & 0xffffu, n = bi >> 16;
            uint32_t pos = o;
            for (uint32_t t = o; t < o + n; t++) pos += (KH[t] < key) ? 1u : 0u;
            U[pos + 1] = v;
            if (id < (uint32_t)A) TH[id] = pos + 1;      // atom where this cell starts
        }
        if (tid == 0) U[0] = 0u;
        lds_barrier();

        // ---- 5b. merge equal bounds: R[i] = number of distinct values among
        //          U[1..i] (the atom whose lower bound is U[i]); the distinct values
        //          move to U[1..Dp] in place.  R lives where the keys were.
        uint32_t* R = (uint32_t*)KH;                     // [Ap + 1]
        Dp = 0;
        {
            constexpr int kPerMax = (kDdaMaxThresholds + kMaxSplits + kHistThreads - 1) / kHistThreads;
            const int per = (int)((Ap + kHistThreads - 1) / kHistThreads);
            uint32_t uv[kPerMax], nf[kPerMax];
            uint32_t mine = 0;
    #pragma unroll
            for (int e = 0; e < kPerMax; e++) {
                const uint32_t i = 1u + (uint32_t)(tid * per + e);
                uv[e] = 0u;
                nf[e] = 0u;
                if (e < per && i <= Ap) {
                    uv[e] = U[i];
                    nf[e] = uv[e] != U[i - 1] ? 1u : 0u;
                    mine += nf[e];
                }
            }
            const uint32_t incl = wave_scan_add(mine);
            if (lane == 63) s_u[3][wid] = incl;
            lds_barrier();                               // every read of U above is done
            uint32_t run = incl - mine;
    #pragma unroll
            for (int v = 0; v < kHistThreads / 64; v++) {
                if (v < wid) run += s_u[3][v];
                Dp += s_u[3][v];
            }
    #pragma unroll
            for (int e = 0; e < kPerMax; e++) {
                const uint32_t i = 1u + (uint32_t)(tid * per + e);
                if (e < per && i <= Ap) {
                    run += nf[e];
                    R[i] = run;
                    if (nf[e]) U[run] = uv[e];
                }
            }
            if (tid == 0) R[0] = 0u;
            if (tid < 3) U[Dp + 1u + (uint32_t)tid] = 0xffffffffu;
        }
        lds_barrier();

        // ---- 6. cell starts in distinct atoms; bin entries {first | flags, next
        //         bound}; then KH becomes the histogram
        for (int i = tid; i < A; i += kHistThreads) {
            const uint32_t p = TH[i];
            TH[i] = p <= Ap ? R[p] : Dp + 1u;
        }
        {
            uint32_t ef[16], ey[16];
    #pragma unroll
            for (int e = 0; e < 16; e++) {
                ef[e] = 0u;
                ey[e] = 0u;
                const uint32_t b = (uint32_t)(tid + e * kHistThreads);
                if (e < P && b < nb) {
                    const uint32_t bv = binc[b];
                    const uint32_t o = bv & 0xffffu, n = bv >> 16;
                    const uint32_t f = R[o], nd = R[o + n] - f;   // distinct bounds inside
                    ef[e] = f | (nd >= 2u ? kFlagWalk : 0u) | (b == nb - 1u ? kFlagTop : 0u);
                    ey[e] = U[f + 1];
                }
            }
            lds_barrier();   // the counts alias the entries; R aliases the histogram
    #pragma unroll
            for (int e = 0; e < 16; e++) {
                const uint32_t b = (uint32_t)(tid + e * kHistThreads);
                if (e < P && b < nb) ENT[b] = make_uint2(ef[e], ey[e]);
            }
            for (uint32_t i = tid; i < ((Dp + 1u) << lcop); i += kHistThreads) hist[i] = 0ull;
        }
        lds_barrier();
    }
    if (plan_out) {   // dump the tables and the range of pe that keeps them exact
        uint32_t m0 = wave_scan_min(ec_lo), m1 = wave_scan_max(ec_hi), m2 = wave_scan_or(plan_bad);
        if (lane == 63) { s_u[0][wid] = m0; s_u[1][wid] = m1; s_u[2][wid] = m2; }
        lds_barrier();
        if (tid == 0) {
            uint32_t elo = 255u, ehi = 0u, bad = 0u;
            for (int v = 0; v < kHistThreads / 64; v++) {
                elo = min(elo, s_u[0][v]); ehi = max(ehi, s_u[1][v]); bad |= s_u[2][v];
            }
            int emin = -1000, emax = 1000;
            if (elo <= ehi) { emin = 1 - (int)elo; emax = 254 - (int)ehi; }
            if (lo < 0x7f800000u) {
                emin = max(emin, 1 - (int)(lo >> 23));
                emax = min(emax, 254 - (int)(hi >> 23));
            }
            if (bad & 2u) emin = max(emin, 0);
            if ((bad & 1u) || lo >= 0x7f800000u) { emin = 0; emax = 0; }   // nothing to shift
            if (emin > emax) { emin = 1; emax = 0; }   // empty: never used
            DdaPlanHead h;
            h.magic = kPlanMagic; h.n = a.n; h.k = a.k; h.G = a.G; h.M = M; h.A = A;
            h.lbins = a.lbins; h.shift = shift; h.base = base; h.nb = nb; h.hi = hi; h.Dp = Dp;
            h.emin = emin; h.emax = emax;
            *(DdaPlanHead*)plan_out = h;
        }
        float* pf = (float*)(plan_out + plan_factors_off());
        for (int j = tid; j < a.G; j += kHistThreads) pf[j] = grid[j];
        uint2* pe = (uint2*)(plan_out + plan_ent_off(a.G));
        for (uint32_t b = tid; b < nb; b += kHistThreads) pe[b] = ENT[b];
        uint32_t* pu = (uint32_t*)(plan_out + plan_u_off(a.G, a.lbins));
        for (uint32_t i = tid; i < Dp + 4u; i += kHistThreads) pu[i] = U[i];
        uint32_t* pt = (uint32_t*)(plan_out + plan_th_off(a.G, A, a.lbins));
        for (int i = tid; i < A; i += kHistThreads) pt[i] = TH[i];
        return;
    }

    // ---- 7. the pass
    double ss0 = 0.0, ss1 = 0.0, top_s1 = 0.0;
    uint32_t top_cnt = 0, flags = 0;
    constexpr int E = 8;
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    typedef const __attribute__((address_space(3))) u32x2 lds_u32x2;
    // LDS byte address of the entry of bin (v >> shift) is (v >> shift) * 8 + ent_b
    // (unsigned wrap-around), with the bin clamped to [base, base + nb - 1]
    const uint32_t ent_b = (uint32_t)(uintptr_t)(lds_u32x2*)(u32x2*)ENT - (base << 3);
    const uint32_t bhi = base + nb - 1u;
    // lanes whose value lies in atom 0 (q = 0 for every candidate) add into a
    // cell of their own, so that ReLU zeros never pile up on one LDS address
    const uint32_t spare = (((uint32_t)a.Aa + 1u) << lcop) + (uint32_t)lane;
    const uint32_t copy = (uint32_t)lane & ((1u << lcop) - 1u);
    auto visit = [&](const uint32_t* xb) {
        uint32_t ab[E], t[E], fx[E];
        u32x2 en[E];
#pragma unroll
        for (int e = 0; e < E; e++) ab[e] = xb[e] & 0x7fffffffu;
        // every entry read in flight before the first is used
#pragma unroll
        for (int e = 0; e < E; e++) {
            const uint32_t bi = med3_u32(ab[e] >> shift, base, bhi);
            en[e] = *(lds_u32x2*)(uintptr_t)((bi << 3) + ent_b);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int e = 0; e < E; e++) {
            const double xd = (double)__uint_as_float(ab[e]);
            if (e & 1) ss1 = fma(xd, xd, ss1); else ss0 = fma(xd, xd, ss0);
        }
        uint32_t any = 0;
#pragma unroll
        for (int e = 0; e < E; e++) {
            t[e] = en[e].x + (ab[e] >= en[e].y ? 1u : 0u);
            fx[e] = en[e].x;
            any |= en[e].x;
        }
        if (any & (kFlagWalk | kFlagTop)) {            // rare: crowded bins, the top bin
#pragma unroll
            for (int e = 0; e < E; e++) {
                t[e] &= kAtomMask;
                if (fx[e] & kFlagWalk)
                    while (U[t[e] + 1] <= ab[e]) t[e]++;
                if ((fx[e] & kFlagTop) && ab[e] >= hi) {
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
        for (int e = 0; e < E; e++) {
            const uint32_t at = t[e] != 0u ? (t[e] << lcop) + copy : spare;
            atomicAdd(&hist[at], (1ull << 44) | (uint64_t)(ab[e] & 0x7fffffu));
        }
    };
    const int64_t cstep = 4 * kHistThreads * 4;   // elements per chunk
    for (int64_t c = e0; c < v1; c += cstep) {
        uint32_t g[16];
#pragma unroll
        for (int u = 0; u < 16; u++) g[u] = gn[u];
        const int64_t cn = c + cstep;
        if (cn + cstep <= v1) load_full(cn, gn);
        else if (cn < v1) load_chunk(cn, gn);
        visit(g);
        if (c + 2 * 4 * kHistThreads < v1) visit(g + 8);   // rows 2, 3 of the chunk
    }
    if (vec && bid == a.nblk - 1 && tid < (int)(len & 3)) {   // tail of the vector path
        uint32_t g[E];
        g[0] = __float_as_uint(x[(len & ~(int64_t)3) + tid]);
#pragma unroll
        for (int e = 1; e < E; e++) g[e] = 0u;
        visit(g);
    }
    lds_barrier();

    // ---- 8. the block's share of the objective.  Per atom: S0 = count, S1 =
    //         sum |x| (the significand sums carry the binade of the atom's lower
    //         bound U[at]).  Atom 0 has q = 0 for every candidate (its values went
    //         to the spare cells); the top atom Dp is taken from the fp64 sums.
    //         Exclusive prefix sums over atoms 0 .. Dp: P0 (u32) over U, P1
    //         (fp64) over the histogram, once both are read.
    constexpr int kPerMax = (kDdaMaxThresholds + kMaxSplits + 2 + kHistThreads - 1) / kHistThreads;
    const int per = (int)((Dp + 2u + kHistThreads - 1) / kHistThreads);   // atoms 0 .. Dp+1
    uint32_t c0[kPerMax];
    double c1[kPerMax];
    uint32_t m0 = 0;
    double m1 = 0.0;
#pragma unroll
    for (int e = 0; e < kPerMax; e++) {
        const uint32_t at = (uint32_t)(tid * per + e);
        c0[e] = 0u;
        c1[e] = 0.0;
        if (e < per && at >= 1u && at < Dp) {
            uint64_t v = 0;
            for (uint32_t c = 0; c < (1u << lcop); c++) v += hist[(at << lcop) + c];   // fields stay apart
            const uint32_t cnt = (uint32_t)(v >> 44);
            uint64_t t = v & kSumMask;
            const uint32_t ex = U[at] >> 23;
            if (ex) t += (uint64_t)cnt << 23;            // the implicit bit of a normal binade
            c0[e] = cnt;
            c1[e] = ldexp((double)t, (int)max(ex, 1u) - 150);
        }
        m0 += c0[e];
        m1 += c1[e];
    }
    {
        const uint32_t i0 = wave_scan_add(m0);
        const double i1 = wave_scan_add(m1);
        const double ss = wave_scan_add(ss0 + ss1), t1 = wave_scan_add(top_s1);
        const uint32_t tc = wave_scan_add(top_cnt), fl = wave_scan_or(flags);
        if (lane == 63) {
            s_u[0][wid] = i0; s_d[0][wid] = i1;
            s_u[1][wid] = tc; s_u[2][wid] = fl; s_d[1][wid] = ss; s_d[2][wid] = t1;
        }
        lds_barrier();   // wave totals published; every read of the histogram and U is done
        uint32_t r0 = i0 - m0;
        double r1 = i1 - m1;
        for (int v = 0; v < wid; v++) { r0 += s_u[0][v]; r1 += s_d[0][v]; }
        uint32_t* P0 = U;
        double* P1 = (double*)KH;
#pragma unroll
        for (int e = 0; e < kPerMax; e++) {
            const uint32_t at = (uint32_t)(tid * per + e);
            if (e < per && at <= Dp + 1u) {
                P0[at] = r0;
                P1[at] = r1;
                r0 += c0[e];
                r1 += c1[e];
            }
        }
    }
    lds_barrier();

    // ---- 9. per cell (j, c), c >= 1: atoms [start_c, start_{c+1}), the last
    //         one up to Dp; the top atom joins the cell that holds Dp.  One
    //         thread per cell writes Q_c S1 and Q_c^2 S0 of the cell; thread j
    //         then sums the cells of candidate j in order.  Cells are taken
    //         1024 at a time; the terms live where the bin entries were.
    {
        const uint32_t* P0 = U;
        const double* P1 = (const double*)KH;
        double2* T = (double2*)smem;                 // [kHistThreads], 16 KB <= the entries
        double ssb = 0.0, t1b = 0.0;
        uint32_t tcb = 0, flb = 0;
#pragma unroll
        for (int v = 0; v < kHistThreads / 64; v++) {
            ssb += s_d[1][v]; t1b += s_d[2][v]; tcb += s_u[1][v]; flb |= s_u[2][v];
        }
        const uint32_t end = Dp + 1u;
        double Aj = 0.0, Bj = 0.0;
        for (int i0 = 0; i0 < A; i0 += kHistThreads) {
            const int i = i0 + tid;
            if (i < A) {
                const int j = i / M, c = i - j * M + 1;
                const uint32_t st = min(TH[i], end);
                const uint32_t nx = (c < M) ? min(TH[i + 1], end) : end;
                const double q = (double)set_value(c, a.k);
                double d1 = P1[nx] - P1[st];
                uint32_t d0 = P0[nx] - P0[st];
                if (st <= Dp && Dp < nx) { d1 += t1b; d0 += tcb; }
                T[tid] = make_double2(q * d1, (q * q) * (double)d0);
            }
            lds_barrier();
            if (tid < a.G) {
                const int lo = max(tid * M, i0), hi = min(tid * M + M, i0 + kHistThreads);
                for (int c = lo; c < hi; c += 4) {     // four reads in flight, sums in order
                    double2 t[4];
#pragma unroll
                    for (int u = 0; u < 4; u++) t[u] = T[min(c + u, hi - 1) - i0];
#pragma unroll
                    for (int u = 0; u < 4; u++)
                        if (c + u < hi) { Aj += t[u].x; Bj += t[u].y; }
                }
            }
            lds_barrier();
        }
        double* out = part + (int64_t)bid * part_stride(a.G);
        if (tid < a.G) {
            out[tid] = Aj;
            out[a.G + tid] = Bj;
        }
        if (tid == 0) {
            out[2 * a.G] = ssb;
            out[2 * a.G + 1] = (double)flb;
        }
    }
}

// ---------------------------------------------------------------- batches
// Several independent problems in one launch of each kernel: the blocks of job
// i are blk0 .. blk0 + nblk - 1 of the histogram grid (groups: grp0 ..), and
// block i of the finalize grid.  Small tensors leave most CUs idle and the
// fixed latency of the set-up, epilogue and finalize dominates, so running
// them side by side costs about as much as one.
constexpr int kDdaMaxJobs = 8;
struct DdaJob {
    const float* x;
    int64_t len;
    const float* grid;
    const float* gscale;   // NULL, or a device scalar multiplying every candidate (planned:
                           // its binary exponent E gives the candidates 2^E grid[j])
    const uint8_t* plan;   // NULL, or the job's plan (grid points at its factors)
    float* alpha_out;
    double* D_out;
    double* part;       // block vectors
    double* grp;        // group vectors (jobs with groups)
    DdaArgs a;
    int blk0, grp0, ngrp;
};
struct DdaBatch {
    DdaJob job[kDdaMaxJobs];
    int count;
};

__device__ __forceinline__ int dda_job_of_block(const DdaBatch& B, int b) {
    int j = 0;
    for (int i = 1; i < B.count; i++)
        if (B.job[i].blk0 <= b) j = i;
    return j;
}

__global__ __launch_bounds__(kHistThreads) void k_dda_hist(DdaBatch B) {
    const int j = dda_job_of_block(B, (int)blockIdx.x);
    const DdaJob& J = B.job[j];
    dda_hist_block(J.x, J.len, J.grid, J.gscale, J.a, J.part, (int)blockIdx.x - J.blk0, J.plan,
                   nullptr);
}

// One block: the set-up for the candidates factors[j] (scale 1), dumped as a plan.
__global__ __launch_bounds__(kHistThreads) void k_dda_plan(DdaArgs a, const float* factors,
                                                           uint8_t* plan) {
    dda_hist_block(nullptr, 0, factors, nullptr, a, nullptr, 0, nullptr, plan);
}

// --------------------------------------------------------------------- group
// Group g: the sums of block vectors kGroup g .. kGroup g + kGroup - 1 in block
// order (flags or-ed), one thread per vector entry.
__global__ __launch_bounds__(256) void k_dda_group(DdaBatch B) {
    int jb = 0;
    for (int i = 1; i < B.count; i++)
        if (B.job[i].ngrp > 0 && B.job[i].grp0 <= (int)blockIdx.x) jb = i;
    const DdaJob& J = B.job[jb];
    const DdaArgs a = J.a;
    const double* __restrict__ part = J.part;
    double* __restrict__ grp = J.grp;
    const int ps = part_stride(a.G), g = (int)blockIdx.x - J.grp0;
    const int b0 = g * kGroup, nb = min(kGroup, a.nblk - b0);
    for (int e = threadIdx.x; e < ps; e += 256) {
        double v[kGroup];
#pragma unroll
        for (int u = 0; u < kGroup; u++) v[u] = part[(int64_t)(b0 + min(u, nb - 1)) * ps + e];
        double t = 0.0;
        uint32_t fl = 0;
#pragma unroll
        for (int u = 0; u < kGroup; u++)
            if (u < nb) { t += v[u]; fl |= (uint32_t)v[u]; }
        grp[(int64_t)g * ps + e] = (e == ps - 1) ? (double)fl : t;
    }
}

// ------------------------------------------------------------------ finalize
// Threads per candidate: enough that no thread sums more than 8 block vectors,
// at most 16 and at most kFinThreads / G.
__host__ __device__ inline int fin_split(int G, int nblk) {
    int S = 1;
    while (S < 16 && S * 8 < nblk && 2 * S * G <= kFinThreads) S *= 2;
    return S;
}

// One block of G * S threads (rounded up to whole waves).  Thread (j, p) sums
// the vectors of blocks p, p + S, p + 2S, ... in that order, then the S partial
// sums of a candidate combine in a fixed butterfly; D_j = S2 + a (a B_j - 2 A_j)
// and the argmin over (isnan(D), D, j), ties to the lowest index.
// Block i of the grid finalizes job i (block vectors, or group vectors when
// the job has groups).
// The finishing step of job J inside one block (blockDim.x a multiple of 64 and at
// least G * S): writes D_out[j] when D_out is given and *alpha_out from thread 0 when
// alpha_out is given, and returns the chosen candidate to every thread.
__device__ __forceinline__ float dda_finish(const DdaJob& J, float* __restrict__ alpha_out,
                                            double* __restrict__ D_out) {
    const float* __restrict__ grid = J.grid;
    const double* __restrict__ part = J.ngrp > 0 ? J.grp : J.part;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int G = J.a.G, nb = J.ngrp > 0 ? J.ngrp : J.a.nblk, ps = part_stride(G);
    const int S = fin_split(G, nb);
    const int p = tid & (S - 1), j = tid / S;
    const bool live = j < G;
    float al = 0.0f;
    if (live) {
        if (J.plan) {   // 2^E grid[j], E the binary exponent of |scale|
            const float sc = *J.gscale;
            int E = 0;
            frexpf(fabsf(sc), &E);
            al = __builtin_isfinite(sc) ? ldexpf(grid[j], E) : __builtin_nanf("");
        } else {
            al = J.gscale ? *J.gscale * grid[j] : grid[j];
        }
    }
    double A = 0.0, B = 0.0, S2 = 0.0;
    uint32_t fl = 0;
    if (live) {
        for (int b0 = p; b0 < nb; b0 += 8 * S) {    // eight vectors in flight
            double v[8][4];
#pragma unroll
            for (int u = 0; u < 8; u++) {
                const int b = min(b0 + u * S, nb - 1);
                const double* r = part + (int64_t)b * ps;
                v[u][0] = r[j]; v[u][1] = r[G + j]; v[u][2] = r[2 * G]; v[u][3] = r[2 * G + 1];
            }
#pragma unroll
            for (int u = 0; u < 8; u++)
                if (b0 + u * S < nb) {
                    A += v[u][0]; B += v[u][1]; S2 += v[u][2]; fl |= (uint32_t)v[u][3];
                }
        }
    }
    for (int o = 1; o < S; o <<= 1) {               // the S lanes of a candidate are adjacent
        A += __shfl_xor(A, o);
        B += __shfl_xor(B, o);
        S2 += __shfl_xor(S2, o);
        fl |= (uint32_t)__shfl_xor((int)fl, o);
    }
    double bd = __builtin_nan("");
    int bj = 0x7fffffff;                            // none
    float ba = 0.0f;
    if (live && p == 0) {
        const double ad = (double)al;
        double D = fma(ad, fma(ad, B, -2.0 * A), S2);
        if (!alpha_ok(al) || (fl & 2u)) D = __builtin_nan("");
        else if (fl & 1u) D = __builtin_inf();
        if (D_out) D_out[j] = D;
        bd = D; bj = j; ba = al;
    }
    // (isnan(D), D, j) is a total order: the result does not depend on the order of
    // the comparisons, and after the butterfly every lane of a wave holds its best
    auto pick = [](double& bd, int& bj, float& ba, double od, int oj, float oa) {
        const bool onan = od != od, mnan = bd != bd;
        const bool better = (oj != 0x7fffffff) &&
                            ((bj == 0x7fffffff) || (!onan && mnan) ||
                             (onan == mnan && (od < bd || (od == bd && oj < bj))));
        if (better) { bd = od; bj = oj; ba = oa; }
    };
    for (int off = 32; off > 0; off >>= 1) {
        const double od = __shfl_xor(bd, off);
        const int oj = __shfl_xor(bj, off);
        const float oa = __shfl_xor(ba, off);
        pick(bd, bj, ba, od, oj, oa);
    }
    if (blockDim.x == 64) {
        if (alpha_out && lane == 0) *alpha_out = ba;
        return ba;
    }
    __shared__ double s_bd[kFinThreads / 64];
    __shared__ int s_bj[kFinThreads / 64];
    __shared__ float s_ba[kFinThreads / 64];
    __shared__ float s_alpha;
    if (lane == 0) { s_bd[wid] = bd; s_bj[wid] = bj; s_ba[wid] = ba; }
    lds_barrier();
    if (tid == 0) {
        for (int v = 1; v < (int)(blockDim.x / 64); v++) pick(bd, bj, ba, s_bd[v], s_bj[v], s_ba[v]);
        if (alpha_out) *alpha_out = ba;
        s_alpha = ba;
    }
    lds_barrier();
    return s_alpha;
}

__global__ __launch_bounds__(kFinThreads) void k_dda_finalize(DdaBatch jobs) {
    const DdaJob& J = jobs.job[blockIdx.x];
    dda_finish(J, J.alpha_out, J.D_out);
}

// The finishing step fused with the projection onto the chosen scale (eq. (6)-(8)),
// for one job: every block derives alpha itself with the finalize's arithmetic (the
// same value everywhere), block 0 also writes alpha_out and D_out, and each block
// then projects its tile of kQTile4 float4 of x (its loads issued before the
// finishing sums); the last block also takes the len % 4 tail.  Results equal
// k_dda_finalize followed by the projection.
constexpr int kQTile4 = 4 * 256;
__global__ __launch_bounds__(256) void k_dda_project(DdaBatch jobs, const float* __restrict__ x,
                                                     int64_t len, ProjParams pp,
                                                     uint8_t* __restrict__ codes) {
    const DdaJob& J = jobs.job[0];
    const int tid = threadIdx.x;
    const int64_t n4 = len >> 2;
    const f32x4* x4 = (const f32x4*)x;
    uint32_t* out4 = (uint32_t*)codes;
    const int64_t i0 = (int64_t)blockIdx.x * kQTile4 + tid;
    const bool whole = i0 + 3 * 256 < n4;
    f32x4 v[4];
    if (whole) {
#pragma unroll
        for (int u = 0; u < 4; u++) v[u] = __builtin_nontemporal_load(&x4[i0 + u * 256]);
    }
    const bool first = blockIdx.x == 0;
    const float alpha = dda_finish(J, first ? J.alpha_out : nullptr, first ? J.D_out : nullptr);
    const bool ok = alpha_valid(alpha);
    const bool fast = fast_scale(alpha);
    const float r = 1.0f / alpha;
    const uint32_t z4 = pp.zero_code * 0x01010101u;
    if (whole) {
#pragma unroll
        for (int u = 0; u < 4; u++)
            __builtin_nontemporal_store(ok ? code4(v[u], alpha, r, fast, pp) : z4, &out4[i0 + u * 256]);
    } else {
#pragma unroll
        for (int u = 0; u < 4; u++) {
            const int64_t i = i0 + u * 256;
            if (i < n4) out4[i] = ok ? code4(x4[i], alpha, r, fast, pp) : z4;
        }
    }
    if (blockIdx.x == gridDim.x - 1 && tid < (int)(len - 4 * n4)) {
        const int64_t i = 4 * n4 + tid;
        codes[i] = (uint8_t)(ok ? esb_code(x[i], alpha, pp) : pp.zero_code);
    }
}

// The set-up kernels use up to 156 KB of dynamic LDS; set once per device
// (racing threads set the same attributes).
static hipError_t set_lds_attributes() {
    static std::atomic<bool> lds_attr_set[64];
    int dev = 0;
    if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < 64 &&
        !lds_attr_set[dev].load(std::memory_order_acquire)) {
        hipError_t e = hipFuncSetAttribute((const void*)k_dda_hist,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 156 * 1024);
        if (e != hipSuccess) return e;
        e = hipFuncSetAttribute((const void*)k_dda_plan, hipFuncAttributeMaxDynamicSharedMemorySize,
                                156 * 1024);
        if (e != hipSuccess) return e;
        lds_attr_set[dev].store(true, std::memory_order_release);
    }
    return hipSuccess;
}

static hipError_t launch_batch(DdaBatch& B, int max_lds, int max_fin_threads, int nhist, int ngroups,
                              hipStream_t s) {
    const hipError_t e = set_lds_attributes();
    if (e != hipSuccess) return e;
    k_dda_hist<<<nhist, kHistThreads, max_lds, s>>>(B);
    if (ngroups > 0) k_dda_group<<<ngroups, 256, 0, s>>>(B);
    k_dda_finalize<<<B.count, max_fin_threads, 0, s>>>(B);
    return hipGetLastError();
}

// The launch set-up of up to kDdaMaxJobs jobs: their blocks, groups and LDS.
static void build_batch(const DdaJobDesc* jobs, int count, DdaBatch& B, int& nhist, int& ngroups,
                        int& max_lds, int& max_fin) {
    B.count = count;
    nhist = 0; ngroups = 0; max_lds = 0; max_fin = 64;
    for (int i = 0; i < B.count; i++) {
        const DdaJobDesc& d = jobs[i];
        DdaJob& J = B.job[i];
        DdaArgs& a = J.a;
        a.G = d.G; a.M = d.L.M; a.A = d.L.A; a.Aa = d.L.A + kMaxSplits;
        a.n = d.f.n; a.k = d.f.k;
        dda_blocks(d.len, &a.nblk, &a.rows_pb);
        a.lbins = d.plan ? plan_lbins(d.L.A) : hist_lbins(d.L.A, a.rows_pb >= 8);
        J.x = d.x; J.len = d.len; J.grid = d.grid; J.gscale = d.gscale;
        J.plan = d.plan;
        if (d.plan) J.grid = (const float*)(d.plan + plan_factors_off());
        J.alpha_out = d.alpha_out; J.D_out = d.D_out;
        J.part = (double*)((char*)d.ws + d.L.off_part);
        J.grp = (double*)((char*)d.ws + d.L.off_group);
        J.blk0 = nhist;
        nhist += a.nblk;
        J.ngrp = dda_groups(a.nblk);
        J.grp0 = ngroups;
        ngroups += J.ngrp;
        const int lds = (int)hist_lds(d.L.A, a.lbins).total;
        if (lds > max_lds) max_lds = lds;
        const int nt = (d.G * fin_split(d.G, J.ngrp > 0 ? J.ngrp : a.nblk) + 63) / 64 * 64;
        if (nt > max_fin) max_fin = nt;   // <= kFinThreads
    }
}

hipError_t launch_dda_batch(const DdaJobDesc* jobs, int count, hipStream_t s) {
    for (int c0 = 0; c0 < count; c0 += kDdaMaxJobs) {
        DdaBatch B;
        int nhist = 0, ngroups = 0, max_lds = 0, max_fin = 64;
        build_batch(jobs + c0, count - c0 < kDdaMaxJobs ? count - c0 : kDdaMaxJobs, B, nhist, ngroups,
                    max_lds, max_fin);
        const hipError_t e = launch_batch(B, max_lds, max_fin, nhist, ngroups, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_dda_quantize(const DdaJobDesc& d, uint8_t* codes, hipStream_t s) {
    DdaBatch B;
    int nhist = 0, ngroups = 0, max_lds = 0, max_fin = 64;
    build_batch(&d, 1, B, nhist, ngroups, max_lds, max_fin);
    const DdaJob& J = B.job[0];
    const int nb = J.ngrp > 0 ? J.ngrp : J.a.nblk;
    // Fused when the finishing step's threads fit one block of 256, the vector path
    // applies and the projection has at most two tiles per CU: every block reads all
    // the group vectors, which for more blocks costs more than the finalize launch
    // saves (ESB(5,2), 64 factors, against the two calls: 32768 elements 16.4 against
    // 17.4 us, 1.6 M 22.9 against 24.1, 3.2 M equal, 12.8 M 52.0 against 43.2).
    const int64_t tiles = ((d.len >> 2) + kQTile4 - 1) / kQTile4;
    const bool fused = d.G * fin_split(d.G, nb) <= 256 && (uintptr_t)d.x % 16 == 0 &&
                       (uintptr_t)codes % 4 == 0 && tiles <= 2 * (int64_t)num_cus();
    if (!fused) {
        const hipError_t e = launch_batch(B, max_lds, max_fin, nhist, ngroups, s);
        if (e != hipSuccess) return e;
        return launch_project(d.x, d.len, d.alpha_out, d.f, codes, nullptr, s);
    }
    hipError_t e = set_lds_attributes();
    if (e != hipSuccess) return e;
    k_dda_hist<<<nhist, kHistThreads, max_lds, s>>>(B);
    if (ngroups > 0) k_dda_group<<<ngroups, 256, 0, s>>>(B);
    k_dda_project<<<(unsigned)(tiles > 0 ? tiles : 1), 256, 0, s>>>(B, d.x, d.len, proj_params(d.f),
                                                                    codes);
    return hipGetLastError();
}

hipError_t launch_dda(const float* x, int64_t len, const Fmt& f, const float* grid, int G,
                      float* alpha_out, double* D_out, void* ws, const DdaLayout& L,
                      hipStream_t s) {
    const DdaJobDesc d{x, len, f, grid, G, alpha_out, D_out, ws, L, nullptr, nullptr};
    return launch_dda_batch(&d, 1, s);
}

size_t dda_plan_bytes(const Fmt& f, int G) {
    const int A = G * ((1 << (f.n - 1)) - 1);
    return plan_total(G, A, plan_lbins(A));
}

hipError_t launch_dda_plan(const Fmt& f, const float* factors, int G, void* plan, hipStream_t s) {
    DdaArgs a{};
    a.G = G;
    a.M = (1 << (f.n - 1)) - 1;
    a.A = G * a.M;
    a.Aa = a.A + kMaxSplits;
    a.n = f.n;
    a.k = f.k;
    a.lbins = plan_lbins(a.A);
    a.nblk = 1;
    a.rows_pb = 1;
    const hipError_t e = set_lds_attributes();
    if (e != hipSuccess) return e;
    k_dda_plan<<<1, kHistThreads, (int)hist_lds(a.A, a.lbins).total, s>>>(a, factors, (uint8_t*)plan);
    return hipGetLastError();
}

}  // namespace esb
