// Skinny contraction over packed E2M1 operands, gfx950: fully connected layers at
// a small batch (few output tiles, a long reduction), eq. (15) on the fp4
// matrix cores.
//
// Each workgroup owns one 64 x 32 output tile and the whole reduction.  Its
// four waves take the 128-byte lines of the reduction (256 values of every row)
// round robin; each wave accumulates its own 64 x 32 partial on the 32x32x64
// fp4 MFMA, and the four partials meet in LDS at the end.  Every partial and
// the total are integers below 2^24 in units of 2^-(kA+kB) (the admission bound
// of the E2M1 path, K max|mA| max|mB| < 2^24), so the fp32 sums are exact in
// any order, and no partial sum leaves the chip.
//
// Each wave streams its lines from L2 into a private ring of D steps in LDS by
// DMA (global_load_lds, 16 bytes per lane: one instruction moves 8 rows x 128
// bytes), waits on its own vmcnt only (no workgroup barrier in the loop), and
// reads the step back in the MFMA layout: lane l serves row l % 32 of a 32-row
// block and, at MFMA step t of the line, the 16-byte piece 4(l / 32) + t.  Piece
// c of an A row always meets piece c of the B row, so the products are those of
// the reduction, summed in another order.  In LDS, piece c of row r sits in
// slot c ^ (r % 8) of the row's 128 bytes (reads of one piece over 32 rows fall
// in distinct banks).
//
// Per workgroup (64 + 32) * K/2 bytes cross from L2; 64 x 32 minimizes that sum
// for the tile area one workgroup per CU needs at batch 128.  Measured on the
// AlexNet FC (128 x 4096 x 9216) the kernel moves about 45 GB/s per CU from L2
// with or without the MFMAs, whatever the address pattern (rows at their pitch
// or line-blocked) and whether B comes from HBM or from L2: the L2 -> CU rate
// over all CUs, not the matrix cores, bounds it.  The workgroups of one 32-column
// slice of B (the M tiles) are adjacent in the run of tiles of one XCD (every
// eighth workgroup id), so the slice is fetched from HBM about once.
#include <type_traits>

#include "esb_internal.h"

namespace esb {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kFcWaves = 4;
constexpr int kFcDepth = 3;              // ring steps per wave
constexpr int kFcBM = 64, kFcBN = 32;

struct FcParams {
    const uint8_t* A;       // M rows of Kb bytes (pitch lda)
    const uint8_t* B;       // N rows of Kb bytes (pitch ldb)
    int64_t lda, ldb;
    int M, N, Kb;
    int TM, T;              // M tiles, tiles
    const float* alphaA;
    const float* alphaB;
    int32_t* acc;
    float* y;
    int64_t ldc;
    int kA, kB;             // fraction bits: acc = sum * 2^(kA + kB)
};

__device__ __align__(128) const uint8_t kFcZero[128] = {0};   // +0 in E2M1, both nibbles

typedef const __attribute__((address_space(1))) uint8_t* gptr;
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) const void gbl_cvoid_t;

template <int B, int E, class F>
__device__ __forceinline__ void unroll(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        unroll<B + 1, E>(f);
    }
}

template <int N>
__device__ __forceinline__ void vm_wait() {   // s_waitcnt vmcnt(N)
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ v8i wide(v4i v) { return v8i{v[0], v[1], v[2], v[3], 0, 0, 0, 0}; }

template <int NW, int D>
__global__ __launch_bounds__(64 * NW) void k_fc_f4(FcParams p) {
    constexpr int BM = kFcBM, BN = kFcBN, TILE = BM * BN, TI = BM / 32;
    constexpr int SA = BM * 128, STEP = (BM + BN) * 128, NDMA = (BM + BN) / 8;
    static_assert(NW * TILE * 4 <= NW * D * STEP, "the partials fit the rings");
    __shared__ __align__(16) uint8_t ring[NW * D * STEP];

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lr = lane & 31, lg = lane >> 5;
    // workgroup b runs on XCD b % 8; XCD x takes the contiguous run of tiles
    // x * per + min(x, rem) + j, j = b / 8, M tiles fastest
    int tm, tn;
    {
        const int b = blockIdx.x, per = p.T >> 3, rem = p.T & 7, x = b & 7, j = b >> 3;
        const int t = x * per + min(x, rem) + j;
        tm = t % p.TM;
        tn = t / p.TM;
    }
    const int m0 = tm * BM, n0 = tn * BN;
    // DMA instruction u of a step moves rows 8u .. 8u+7 (B rows, then A rows);
    // lane l serves row 8u + l/8 and lands in slot l % 8 of it, so it fetches piece
    // (l % 8) ^ (row % 8) = (l % 8) ^ (l / 8).  Rows past M or N read row M-1 /
    // N-1: their sums land in outputs never stored.
    const int drow = lane >> 3, dpiece = (lane & 7) ^ drow;
    gptr src[NDMA];
#pragma unroll
    for (int u = 0; u < BN / 8; u++)
        src[u] = (gptr)p.B + (int64_t)min(n0 + 8 * u + drow, p.N - 1) * p.ldb + 16 * dpiece;
#pragma unroll
    for (int u = 0; u < BM / 8; u++)
        src[BN / 8 + u] = (gptr)p.A + (int64_t)min(m0 + 8 * u + drow, p.M - 1) * p.lda + 16 * dpiece;
    const gptr zero = (gptr)kFcZero + 16 * dpiece;

    // Every wave runs the same number of steps, a multiple of D, with no branch
    // in the loop body; step st is line w + st * NW.  A piece past the end of the
    // rows (the partial last line, lines past the last) comes from a block of +0
    // codes shared by every lane: its products are 0.
    const int lines = (p.Kb + 127) >> 7;
    const int SS = ((lines + NW - 1) / NW + D - 1) / D * D;
    uint8_t* myring = ring + w * D * STEP;
    auto fetch = [&](auto Q, int st) {
        constexpr int q = decltype(Q)::value;
        const int64_t off = (int64_t)(w + st * NW) << 7;
        const bool in = off + 16 * dpiece < p.Kb;
        uint8_t* slot = myring + q * STEP;
        // B first: its lines are the ones likely to come from HBM
#pragma unroll
        for (int u = 0; u < NDMA; u++) {
            uint8_t* dst = u < BN / 8 ? slot + SA + 1024 * u : slot + 1024 * (u - BN / 8);
            __builtin_amdgcn_global_load_lds((gbl_cvoid_t*)(in ? src[u] + off : zero), (lds_void_t*)dst,
                                             16, 0, 0);
        }
    };
    v16f acc[TI];
#pragma unroll
    for (int i = 0; i < TI; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) acc[i][r] = 0.0f;
    auto compute = [&](auto Q) {
        constexpr int q = decltype(Q)::value;
        const uint8_t* slot = myring + q * STEP;
        v4i fa[TI][4], fb[4];
#pragma unroll
        for (int t = 0; t < 4; t++) {
            const int pc = 4 * lg + t;
#pragma unroll
            for (int i = 0; i < TI; i++) {
                const int row = 32 * i + lr;
                fa[i][t] = *(const v4i*)(slot + row * 128 + 16 * (pc ^ (row & 7)));
            }
            fb[t] = *(const v4i*)(slot + SA + lr * 128 + 16 * (pc ^ (lr & 7)));
        }
#pragma unroll
        for (int t = 0; t < 4; t++)
#pragma unroll
            for (int i = 0; i < TI; i++)
                acc[i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                    wide(fa[i][t]), wide(fb[t]), acc[i], 4, 4, 0, 127, 0, 127);
    };

    // The compiler does not see the DMA writes: the waits are explicit, and
    // scheduling barriers keep the LDS reads after them and the next DMA into a
    // slot after the reads of that slot have returned.
    unroll<0, D>([&](auto Q) { fetch(Q, decltype(Q)::value); });
    for (int st = 0; st < SS; st += D) {
        unroll<0, D>([&](auto Q) {
            vm_wait<(D - 1) * NDMA>();                     // this step's DMAs landed
            asm volatile("" ::: "memory");
            __builtin_amdgcn_sched_barrier(0);
            compute(Q);
            __builtin_amdgcn_s_waitcnt(0xc07f & ~0x0f00);  // lgkmcnt(0): the slot's reads are done
            asm volatile("" ::: "memory");
            __builtin_amdgcn_sched_barrier(0);
            fetch(Q, st + decltype(Q)::value + D);         // past the end: the zero block
            __builtin_amdgcn_sched_barrier(0);
        });
    }
    vm_wait<0>();
    __syncthreads();   // every ring is done: the partials take their place

    // the partials of the waves meet in LDS: register r of a 32x32 block is row
    // 8(r/4) + 4(lane/32) + r%4, column lane%32
    float* red = (float*)ring;
    float* mine = red + w * TILE;
#pragma unroll
    for (int i = 0; i < TI; i++)
#pragma unroll
        for (int r = 0; r < 16; r++)
            mine[(32 * i + 8 * (r >> 2) + 4 * lg + (r & 3)) * BN + lr] = acc[i][r];
    __syncthreads();

    const float s = p.y ? ldexpf(p.alphaA[0] * p.alphaB[0], -(p.kA + p.kB)) : 0.0f;
    const int shift = p.kA + p.kB;
    for (int e = 4 * tid; e < TILE; e += 4 * 64 * NW) {
        f32x4 v = *(const f32x4*)(red + e);
#pragma unroll
        for (int u = 1; u < NW; u++) {
            const f32x4 o = *(const f32x4*)(red + u * TILE + e);
            v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
        }
        const int row = m0 + e / BN, col = n0 + (e % BN);
        if (row >= p.M || col >= p.N) continue;
        const float f[4] = {ldexpf(v.x, shift), ldexpf(v.y, shift), ldexpf(v.z, shift), ldexpf(v.w, shift)};
        const int64_t o = (int64_t)row * p.ldc + col;
        const int nv = min(4, p.N - col);
        const bool vec = nv == 4 && (o & 3) == 0;
        if (p.acc) {
            if (vec && ((uintptr_t)p.acc & 15) == 0) {
                *(v4i*)(p.acc + o) = v4i{(int)f[0], (int)f[1], (int)f[2], (int)f[3]};
            } else {
                for (int u = 0; u < nv; u++) p.acc[o + u] = (int32_t)f[u];
            }
        }
        if (p.y) {
            if (vec && ((uintptr_t)p.y & 15) == 0) {
                *(f32x4*)(p.y + o) = f32x4{s * f[0], s * f[1], s * f[2], s * f[3]};
            } else {
                for (int u = 0; u < nv; u++) p.y[o + u] = s * f[u];
            }
        }
    }
}

}  // namespace

bool fc_f4_fits(int64_t M, int64_t N, int64_t K) {
    if (M <= 0 || N <= 0 || K <= 0 || K % 32 != 0 || K / 2 > 0x7fffffff) return false;
    const int64_t tiles = ((M + kFcBM - 1) / kFcBM) * ((N + kFcBN - 1) / kFcBN);
    if (tiles > 0x7fffffff) return false;
    // only where the 128 x 128 tiles would split the reduction over workgroups,
    // and with enough 64 x 32 tiles to give half the CUs a workgroup
    int kc = (int)K;
    return mma_splitk(M, N, K, &kc) > 1 && 2 * tiles >= num_cus();
}

hipError_t launch_fc_f4(int M, int N, int K, const uint8_t* A_packed, int64_t lda_bytes,
                        const uint8_t* B_packed, int64_t ldb_bytes, int kA, int kB,
                        const float* alphaA, const float* alphaB, int32_t* acc, float* y,
                        int64_t ldc, hipStream_t s) {
    if (M <= 0 || N <= 0) return hipSuccess;
    FcParams p;
    p.A = A_packed; p.B = B_packed; p.lda = lda_bytes; p.ldb = ldb_bytes;
    p.M = M; p.N = N; p.Kb = K / 2;
    p.TM = (M + kFcBM - 1) / kFcBM;
    p.T = p.TM * ((N + kFcBN - 1) / kFcBN);
    p.alphaA = alphaA; p.alphaB = alphaB; p.acc = acc; p.y = y; p.ldc = ldc;
    p.kA = kA; p.kB = kB;
    k_fc_f4<kFcWaves, kFcDepth><<<(unsigned)p.T, 64 * kFcWaves, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace esb
