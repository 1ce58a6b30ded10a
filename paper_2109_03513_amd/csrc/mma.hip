// Large-tile contraction over ESB codes on the 32x32 MFMA shapes of gfx950.
//
// The product of two ESB values is a short fraction product shifted by the
// two exponents (eq. (15)), so a contraction over codes is an exact integer
// dot product over m = q * 2^k.  This kernel decodes each code once per
// workgroup while its tile moves from HBM to LDS, into one of two exact
// machine formats:
//
//  * F8: OCP E4M3.  ESB(b, k) is a minifloat with ebits = b-k-1 exponent bits
//    whose all-ones exponent is the subnormal binade; adding 1 to the exponent
//    field modulo 2^ebits turns it into the E4M3 layout, with value
//    q * 2^-6 exactly (the all-ones binade lands on the E4M3 subnormals).
//    Five VALU operations per four codes.  The 32x32x64 f8f6f4 MFMA
//    accumulates in fp32.  Measured on gfx950: within one instruction,
//    products more than 2^13 below the largest product of that instruction are
//    dropped, and the accumulator input is added exactly.  The dispatcher only
//    takes this path when every product m_A * m_B is at most 2^12 and
//    K * max|m_A| * max|m_B| < 2^24, where every partial sum is an integer
//    multiple of 2^-(kA+kB+12) that fp32 holds exactly.
//  * I8: int8 m through one v_perm_b32 table lookup (codes of n <= 3 bits, 8
//    entries), then v_mfma_i32_32x32x32_i8 with int32 accumulation.
//
// Tiles: BM x BN per workgroup, WGM x WGN waves of (BM/WGM) x (BN/WGN), BK =
// 64 reduction bytes per stage.  Codes travel HBM -> LDS by DMA into a ring of
// R "raw" buffers, R - 1 stages ahead (no registers held); while the MFMAs of
// stage t run, each thread decodes the raw chunks of stage t+1 it fetched
// itself into the other half of a double-buffered, XOR-swizzled decoded tile.
// One LDS barrier per stage.  Workgroups are numbered so that each XCD (every
// eighth workgroup id) gets a contiguous run of tiles.
#include <type_traits>

#include "esb_internal.h"

namespace esb {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int BK = 64;
constexpr int CPR = BK / 16;   // 16-byte chunks per tile row

struct FastParams {
    int M, N, K;
    int tiles_m, tiles_n, ntiles;
    ConvGeom ga;
    const uint8_t* A;
    const uint8_t* B;
    int64_t ldb;
    int64_t blkA, blkB;     // packed E2M3: bytes of one 48-byte stage block of every row
    int ksplit, kchunk;     // k_mma on a dense GEMM: reduction split in ksplit ranges of kchunk
    int32_t* part;          // [ksplit][M][N] int32 partial sums (ksplit > 1)
    MmaDecode da, db;
    const float* alphaA;
    const float* alphaB;
    int32_t* acc;
    float* y;
    int64_t ldc;
    int out_shift;          // F8: acc_int = acc_f32 * 2^out_shift
    int kA, kB;
    int zrowA, zrowB;       // rows of kZeroRows holding each operand's +0 code
    Post post;              // fused post-processing of the outputs (post.on == 0: none)
};
constexpr int kZeroRowE4M3 = 7 * 8;

// The int32 sums of a wave's 32x32 blocks (register r of a block is row
// 8(r/4) + 4(lane/32) + r%4, column lane%32), `iv(i, j, r)` the value.
template <int TI, int TJ, class IV>
__device__ __forceinline__ void store_acc(const FastParams& g, int lane, int row0, int col0, int grp,
                                          IV iv) {
    const int lr = lane & 31, lg = lane >> 5;
#pragma unroll
    for (int i = 0; i < TI; i++)
#pragma unroll
        for (int j = 0; j < TJ; j++)
#pragma unroll
            for (int r = 0; r < 16; r++) {
                const int row = row0 + 32 * i + 8 * (r >> 2) + 4 * lg + (r & 3);
                const int col = col0 + 32 * j + lr;
                if (row < g.M && col < g.N) g.acc[(int64_t)row * g.ldc + (int64_t)grp * g.N + col] = iv(i, j, r);
            }
}

// Epilogue of the 32x32-block MFMA kernels with the fused post-processing.
// One row of blocks (index i) at a time, each wave writes its TJ blocks of
// scaled values y0(i, j, r) (register r of a block is row 8(r/4) + 4(lane/32)
// + r%4, column lane%32) to its own LDS slab of 32 x 32TJ floats, then reads
// them back as four consecutive outputs per lane: the post-processing code is
// emitted once per row of blocks, outside the unrolled register loops (whose
// full unrolling keeps the accumulators in registers), and its global
// accesses are contiguous.  Every thread of the workgroup calls this.
template <int TI, int TJ, class Y0>
__device__ __forceinline__ void post_epilogue(const FastParams& g, float* slab, int lane, int row0,
                                              int col0, int grp, Y0 y0) {
    constexpr int W = 32 * TJ;
    const int lr = lane & 31, lg = lane >> 5;
    const float qa = post_alpha(g.post);
    uint32_t amax = 0;
#pragma unroll
    for (int i = 0; i < TI; i++) {
        __syncthreads();   // the LDS is free: main loop or previous row done everywhere
#pragma unroll
        for (int j = 0; j < TJ; j++)
#pragma unroll
            for (int r = 0; r < 16; r++)
                slab[(8 * (r >> 2) + 4 * lg + (r & 3)) * W + 32 * j + lr] = y0(i, j, r);
        __syncthreads();
#pragma unroll 1
        for (int e = 4 * lane; e < 32 * W; e += 256) {
            const int rl = e / W, cl = e - rl * W;
            const int row = row0 + 32 * i + rl, col = col0 + cl;
            if (row < g.M && col < g.N) {
                const int64_t ch = (int64_t)grp * g.N + col;
                amax = max(amax, post_store4(g.post, g.y, (int64_t)row * g.ldc + ch, ch,
                                             *(const f32x4*)(slab + e), min(4, g.N - col), qa));
            }
        }
    }
    post_absmax_flush(g.post, amax);
}

__device__ __forceinline__ uint32_t dec_f8(uint32_t c, const MmaDecode& d) {
    const uint32_t t = (((c & d.lm) << d.shf) + d.inc) & d.lmf;   // exponent + 1 (mod 2^ebits)
    return ((c << d.shs) & 0x80808080u) | t;                       // sign to bit 7
}

// Four codes to four OCP E2M1 nibbles (low half of each byte), value q
// exactly: the same exponent-field increment as dec_f8 on a 1-bit fraction.
__device__ __forceinline__ uint32_t dec_f4(uint32_t c, const MmaDecode& d) {
    const uint32_t t = (((c & d.lm) << d.shf) + d.inc) & d.lmf;
    return ((c << d.shs) & 0x08080808u) | t;
}

// Four codes to four OCP E2M3 values (low six bits of each byte), value q
// exactly: the exponent-field increment on a 3-bit fraction, sign to bit 5.
__device__ __forceinline__ uint32_t dec_f6(uint32_t c, const MmaDecode& d) {
    const uint32_t t = (((c & d.lm) << d.shf) + d.inc) & d.lmf;
    return ((c << d.shs) & 0x20202020u) | t;
}
// Four 6-bit values (one per byte) into the low 24 bits, value 0 lowest.
__device__ __forceinline__ uint32_t pack6(uint32_t v) {
    return (v & 0x3fu) | ((v >> 2) & 0xfc0u) | ((v >> 4) & 0x3f000u) | ((v >> 6) & 0xfc0000u);
}

__device__ __forceinline__ uint32_t dec_i8(uint32_t c, const MmaDecode& d) {
    return __builtin_amdgcn_perm(d.t1, d.t0, c & d.sel);
}

__device__ __forceinline__ uint4 as_u4(v4i v) {
    return make_uint4((uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]);
}

template <int OP>
__device__ __forceinline__ uint4 dec16(uint4 v, const MmaDecode& d) {
    if (OP == 1) return make_uint4(dec_f8(v.x, d), dec_f8(v.y, d), dec_f8(v.z, d), dec_f8(v.w, d));
    return make_uint4(dec_i8(v.x, d), dec_i8(v.y, d), dec_i8(v.z, d), dec_i8(v.w, d));
}

// 16 bytes of the +0 code of every ESB(n, k) (index (n - 2) * 8 + k): the
// source of every chunk that lies outside the operand (padding, ragged edges,
// the reduction tail), so that loads need no branches.
struct ZeroRows {
    uint8_t b[7 * 8 + 1][16];   // the last row: 0x00 bytes, +0 of OCP E4M3
};
constexpr ZeroRows make_zero_rows() {
    ZeroRows z{};
    for (int n = 2; n <= 8; n++)
        for (int k = 0; k < 8; k++)
            for (int i = 0; i < 16; i++)
                z.b[(n - 2) * 8 + k][i] =
                    (k <= n - 2) ? (uint8_t)(((1u << (n - k - 1)) - 1u) << k) : (uint8_t)0;
    return z;
}
__device__ ZeroRows kZeroRows = make_zero_rows();   // read only; global, not constant, memory

// LDS offset of 16-byte chunk `chunk` of tile row `row`.  LDS has 64 banks of
// 4 bytes: 256 bytes, four 64-byte rows.  Rows 4q..4q+3 take their chunks in
// the order chunk ^ (q & 3), so 16 consecutive rows read at one logical chunk
// (one quarter-wave of a fragment load) hit 16 distinct bank groups.
__device__ __forceinline__ int lds_off(int row, int chunk) {
    return row * BK + ((chunk ^ ((row >> 2) & 3)) << 4);
}

// Tile id -> (tm, tn): contiguous runs per XCD, then groups of 8 tile rows.
__device__ __forceinline__ void tile_of(const FastParams& g, int& tm, int& tn) {
    const int b = blockIdx.x, T = g.ntiles;
    const int per = T >> 3, rem = T & 7, x = b & 7, j = b >> 3;
    const int t = x * per + min(x, rem) + j;
    constexpr int GM = 8;
    const int span = GM * g.tiles_n;
    const int grp = t / span, first = grp * GM;
    const int gm = min(g.tiles_m - first, GM);
    const int r = t - grp * span;
    tm = first + r % gm;
    tn = r / gm;
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) const void gbl_cvoid_t;

// One 16-byte chunk from global memory into LDS by DMA: lane l of the wave
// writes lds_wave_base + 16 * l (the base must be the same for the whole wave).
// Workgroup barrier for LDS only.  __syncthreads() also drains every
// outstanding global access, which would wait for the fetch of the stage after
// next; the raw chunks a thread reads back were fetched by its own lane, so
// its own wait on them is enough.  The memory clobber keeps the compiler from
// moving LDS accesses across.
__device__ __forceinline__ void lds_barrier() {
    // the same wait as a builtin first: the compiler's wait tracking then knows
    // that every LDS read issued so far is complete
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0), vmcnt and expcnt at their maxima
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Read 16 bytes of LDS outside the compiler's wait tracking.  Used for the
// raw chunks: the compiler cannot tell which fetch wrote which raw buffer and
// would wait for every fetch in flight.  The caller orders the read after its
// fetch with vm_wait<>() and the use after the read with lgkm_wait_on().
__device__ __forceinline__ v4i lds_read16_untracked(const uint8_t* p) {
    v4i v;
    const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)p;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a) : "memory");
    return v;
}

// s_waitcnt vmcnt(N) (gfx9 encoding; expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void vm_wait() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ void dma16(const uint8_t* g, uint8_t* lds_wave_base) {
    __builtin_amdgcn_global_load_lds((gbl_cvoid_t*)g, (lds_void_t*)lds_wave_base, 16, 0, 0);
}

template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}
template <int I>
using ic = std::integral_constant<int, I>;

// R: depth of the ring of raw buffers; the fetch of a stage is issued R - 1
// stages before its codes are decoded.
template <int BM, int BN, int WGM, int WGN, int OP, int CONV, int R>
__global__ __launch_bounds__(64 * WGM * WGN) void k_mma(FastParams g) {
    constexpr int NT = 64 * WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int TI = WM / 32, TJ = WN / 32;
    constexpr int CHA = BM * CPR / NT, CHB = BN * CPR / NT, CT = CHA + CHB;
    static_assert(CHA * NT == BM * CPR && CHB * NT == BN * CPR, "whole chunks per thread");
    constexpr int RSTEP = NT / CPR;       // tile rows between a thread's chunks
    constexpr int TILE = (BM + BN) * BK;  // bytes of one stage: A rows, then B rows
    static_assert(R >= 2 && R <= 6, "raw ring depth");
    // dec: decoded, swizzled tiles read by the MFMAs.  raw: codes as fetched;
    // chunk j of thread t sits at (j * NT + t) * 16, written and read by t only.
    // Separate arrays, addressed with compile-time slots, let the compiler
    // wait for exactly the fetch a read depends on.
    __shared__ __align__(16) uint8_t dec0[TILE];
    __shared__ __align__(16) uint8_t dec1[TILE];
    __shared__ __align__(16) uint8_t raw0[TILE];
    __shared__ __align__(16) uint8_t raw1[TILE];
    __shared__ __align__(16) uint8_t raw2[R > 2 ? TILE : 16];
    __shared__ __align__(16) uint8_t raw3[R > 3 ? TILE : 16];
    __shared__ __align__(16) uint8_t raw4[R > 4 ? TILE : 16];
    __shared__ __align__(16) uint8_t raw5[R > 5 ? TILE : 16];
    auto RAW = [&](auto I) -> uint8_t* {
        constexpr int i = decltype(I)::value;
        if constexpr (i == 0) return raw0;
        else if constexpr (i == 1) return raw1;
        else if constexpr (i == 2) return raw2;
        else if constexpr (i == 3) return raw3;
        else if constexpr (i == 4) return raw4;
        else return raw5;
    };
    auto DEC = [&](auto I) -> uint8_t* {
        if constexpr (decltype(I)::value == 0) return dec0;
        else return dec1;
    };

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int tm, tn;
    tile_of(g, tm, tn);
    // convolution: blockIdx.z is the group; dense GEMM: the reduction range
    const int grp = CONV ? (int)blockIdx.z : 0;
    const int kz = CONV ? 0 : (int)blockIdx.z;
    const int kbeg = kz * g.kchunk;
    const int Kl = CONV ? g.K : min(g.K - kbeg, g.kchunk);   // reduction length of this workgroup
    const int m0 = tm * BM, n0 = tn * BN;
    const int wr = (wave / WGN) * WM, wc = (wave % WGN) * WN;
    const ConvGeom& cg = g.ga;
    const int goffA = grp * cg.Cg;
    const int64_t brow0 = (int64_t)grp * g.N;
    const int ch = tid % CPR;      // chunk column of every chunk of this thread
    const int row0 = tid / CPR;

    // A rows of this thread.  Convolution: output pixels, whose (r, s, c)
    // reduction position is the same for every chunk of the thread; a row
    // outside M gets an input row far out of range.
    int64_t a_off[CHA];
    int a_ih[CHA], a_iw[CHA];
    int kr = 0, ks = 0, kc = 16 * ch;
    if (CONV) {
#pragma unroll
        for (int i = 0; i < CHA; i++) {
            const int m = m0 + row0 + i * RSTEP;
            const bool ok = m < g.M;
            const int mm = ok ? m : 0;
            const int pq = cg.P * cg.Q;
            const int img = mm / pq, rem = mm - img * pq;
            const int p = rem / cg.Q, q = rem - p * cg.Q;
            a_ih[i] = ok ? p * cg.sh - cg.ph : -0x40000000;
            a_iw[i] = q * cg.sw - cg.pw;
            a_off[i] = (((int64_t)img * cg.H + a_ih[i]) * cg.W + a_iw[i]) * cg.pitch + goffA;
        }
        const int rs = kc / cg.Cg;
        kc -= rs * cg.Cg;
        kr = rs / cg.S;
        ks = rs - kr * cg.S;
    }
    const uint8_t* aptr = g.A + (int64_t)(m0 + row0) * cg.pitch + 16 * ch + kbeg;
    const int64_t astep = (int64_t)RSTEP * cg.pitch;
    const int mrem = g.M - m0 - row0;   // dense: chunk i of A is inside M iff i * RSTEP < mrem
    const uint8_t* bptr = g.B + (brow0 + n0 + row0) * g.ldb + 16 * ch + kbeg;
    const int64_t bstep = (int64_t)RSTEP * g.ldb;
    const int nrem = g.N - n0 - row0;
    const uint8_t* zA = kZeroRows.b[g.zrowA];
    const uint8_t* zB = kZeroRows.b[g.zrowB];

    // fetch the codes of reduction offset k0 into a raw buffer
    auto fetch = [&](int k0, uint8_t* rawbuf) {
        const bool kin = k0 + 16 * ch < Kl;
        uint8_t* base = rawbuf + wave * 64 * 16;
        if (CONV) {
            const int64_t koff = ((int64_t)kr * cg.W + ks) * cg.pitch + kc;
#pragma unroll
            for (int i = 0; i < CHA; i++) {
                const int ih = a_ih[i] + kr, iw = a_iw[i] + ks;
                const bool ok = kin && (unsigned)ih < (unsigned)cg.H && (unsigned)iw < (unsigned)cg.W;
                dma16(ok ? g.A + a_off[i] + koff : zA, base + i * NT * 16);
            }
            kc += BK;
            while (kc >= cg.Cg) {
                kc -= cg.Cg;
                if (++ks == cg.S) { ks = 0; ++kr; }
            }
        } else {
#pragma unroll
            for (int i = 0; i < CHA; i++)
                dma16((kin && i * RSTEP < mrem) ? aptr + i * astep + k0 : zA, base + i * NT * 16);
        }
#pragma unroll
        for (int i = 0; i < CHB; i++)
            dma16((kin && i * RSTEP < nrem) ? bptr + i * bstep + k0 : zB, base + (CHA + i) * NT * 16);
    };
    v4i rv[CT];
    auto read_raw = [&](const uint8_t* rawbuf) {
#pragma unroll
        for (int j = 0; j < CT; j++) rv[j] = lds_read16_untracked(&rawbuf[(j * NT + tid) * 16]);
    };
    // s_waitcnt lgkmcnt(0), tied to the raw registers so no use moves above it
    auto raw_ready = [&]() {
#pragma unroll
        for (int j = 0; j < CT; j++) asm volatile("" : "+v"(rv[j]));
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int j = 0; j < CT; j++) asm volatile("" : "+v"(rv[j]));
    };
    auto decode_store = [&](uint8_t* d) {
#pragma unroll
        for (int j = 0; j < CHA; j++)
            *(uint4*)&d[lds_off(row0 + j * RSTEP, ch)] = dec16<OP>(as_u4(rv[j]), g.da);
#pragma unroll
        for (int j = 0; j < CHB; j++)
            *(uint4*)&d[BM * BK + lds_off(row0 + j * RSTEP, ch)] = dec16<OP>(as_u4(rv[CHA + j]), g.db);
    };

    typedef typename std::conditional<OP == 1, v16f, v16i>::type acc_t;
    acc_t acc[TI][TJ];
#pragma unroll
    for (int i = 0; i < TI; i++)
#pragma unroll
        for (int j = 0; j < TJ; j++)
#pragma unroll
            for (int r = 0; r < 16; r++) acc[i][j][r] = 0;

    const int lr = lane & 31, lg = lane >> 5;
    auto compute = [&](const uint8_t* d) {
        const uint8_t* tA = d;
        const uint8_t* tB = d + BM * BK;
        if (OP == 1) {
            v8i fb[TJ];
            const int c0 = 2 * lg;
#pragma unroll
            for (int j = 0; j < TJ; j++) {
                const int row = wc + 32 * j + lr;
                const v4i lo = *(const v4i*)&tB[lds_off(row, c0)];
                const v4i hi = *(const v4i*)&tB[lds_off(row, c0 + 1)];
                fb[j] = v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            }
#pragma unroll
            for (int i = 0; i < TI; i++) {
                const int row = wr + 32 * i + lr;
                const v4i lo = *(const v4i*)&tA[lds_off(row, c0)];
                const v4i hi = *(const v4i*)&tA[lds_off(row, c0 + 1)];
                const v8i fa = v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
                for (int j = 0; j < TJ; j++)
                    acc[i][j] = (acc_t)__builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                        fa, fb[j], (v16f)acc[i][j], 0, 0, 0, 127, 0, 127);
            }
        } else {
#pragma unroll
            for (int kb = 0; kb < BK / 32; kb++) {
                v4i fa[TI], fb[TJ];
                const int c0 = 2 * kb + lg;
#pragma unroll
                for (int i = 0; i < TI; i++) fa[i] = *(const v4i*)&tA[lds_off(wr + 32 * i + lr, c0)];
#pragma unroll
                for (int j = 0; j < TJ; j++) fb[j] = *(const v4i*)&tB[lds_off(wc + 32 * j + lr, c0)];
#pragma unroll
                for (int i = 0; i < TI; i++)
#pragma unroll
                    for (int j = 0; j < TJ; j++)
                        acc[i][j] = (acc_t)__builtin_amdgcn_mfma_i32_32x32x32_i8(
                            fa[i], fb[j], (v16i)acc[i][j], 0, 0, 0);
            }
        }
    };

    const int KT = (Kl + BK - 1) / BK;
    static_for<0, R>([&](auto Q) { fetch(decltype(Q)::value * BK, RAW(Q)); });
    vm_wait<(R - 1) * CT>();   // stage 0 landed
    read_raw(RAW(ic<0>{}));
    raw_ready();
    decode_store(DEC(ic<0>{}));
    lds_barrier();
    // Stage s: its codes sit in raw slot s % R, its decoded tile in dec slot s % 2.
    constexpr int U = (R % 2 == 0) ? R : 2 * R;
    for (int kt = 0; kt < KT; kt += U) {
        static_for<0, U>([&](auto Q) {
            constexpr int q = decltype(Q)::value;
            if (kt + q < KT) {
                // fetches in flight: stages s+1 .. s+R-1, CT instructions each
                vm_wait<(R - 2) * CT>();                    // stage s+1 landed
                read_raw(RAW(ic<(q + 1) % R>{}));
                fetch((kt + q + R) * BK, RAW(ic<q % R>{})); // stage s+R into the slot of stage s
                raw_ready();
                compute(DEC(ic<q % 2>{}));
                decode_store(DEC(ic<(q + 1) % 2>{}));
                lds_barrier();
            }
        });
    }

    // epilogue: register r of a 32x32 block holds row 8*(r/4) + 4*(lane/32) + r%4,
    // column lane % 32.
    float s = 0.0f;
    if (g.y || g.post.on) s = ldexpf(g.alphaA[0] * g.alphaB[0], -(g.kA + g.kB));
    if (g.post.on && (CONV || g.ksplit == 1)) {
        // two LDS buffers of TILE bytes each hold the slabs of half the waves
        constexpr int NW = WGM * WGN;
        static_assert((NW / 2) * 32 * 32 * TJ * 4 <= TILE, "post slabs fit the decode buffers");
        if (g.acc)
            store_acc<TI, TJ>(g, lane, m0 + wr, n0 + wc, grp, [&](int i, int j, int r) {
                return OP == 1 ? (int32_t)ldexpf((float)acc[i][j][r], g.out_shift) : (int32_t)acc[i][j][r];
            });
        float* slab = (float*)(wave < NW / 2 ? dec0 : dec1) + (wave % (NW / 2)) * (32 * 32 * TJ);
        post_epilogue<TI, TJ>(g, slab, lane, m0 + wr, n0 + wc, grp, [&](int i, int j, int r) {
            return OP == 1 ? s * ldexpf((float)acc[i][j][r], g.out_shift) : s * (float)(int32_t)acc[i][j][r];
        });
        return;
    }
#pragma unroll
    for (int i = 0; i < TI; i++)
#pragma unroll
        for (int j = 0; j < TJ; j++)
#pragma unroll
            for (int r = 0; r < 16; r++) {
                const int row = m0 + wr + 32 * i + 8 * (r >> 2) + 4 * lg + (r & 3);
                const int col = n0 + wc + 32 * j + lr;
                if (row < g.M && col < g.N) {
                    float fv;
                    int32_t iv;
                    if (OP == 1) {
                        fv = ldexpf((float)acc[i][j][r], g.out_shift);
                        iv = (int32_t)fv;
                    } else {
                        iv = (int32_t)acc[i][j][r];
                        fv = (float)iv;
                    }
                    if (!CONV && g.ksplit > 1) {          // partial sum of this range
                        g.part[((int64_t)kz * g.M + row) * g.N + col] = iv;
                        continue;
                    }
                    const int64_t o = (int64_t)row * g.ldc + (int64_t)grp * g.N + col;
                    if (g.acc) g.acc[o] = iv;
                    if (g.y) g.y[o] = s * fv;
                }
            }
}

// Sum of the ksplit partial sums of every output, in range order (int32 and
// exact: every partial and the total obey the accumulator bound; two's
// complement wrap-around), then the epilogue of the contraction.  Four
// consecutive outputs per thread when N % 4 == 0 (16-byte loads, the loads of
// eight ranges in flight together), else one.
__global__ __launch_bounds__(256) void k_splitk_sum(FastParams g) {
    const int64_t MN = (int64_t)g.M * g.N;
    float s = 0.0f;
    if (g.y || g.post.on) s = ldexpf(g.alphaA[0] * g.alphaB[0], -(g.kA + g.kB));
    const float qa = g.post.on ? post_alpha(g.post) : 0.0f;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t amax = 0;
    if (g.N % 4 == 0) {
        const int4* p = (const int4*)g.part;
        const int64_t MN4 = MN / 4;
        for (int64_t e = t0; e < MN4; e += stride) {
            uint32_t u0 = 0, u1 = 0, u2 = 0, u3 = 0;
            for (int z0 = 0; z0 < g.ksplit; z0 += 8) {
                int4 v[8];
#pragma unroll
                for (int z = 0; z < 8; z++) v[z] = p[(int64_t)min(z0 + z, g.ksplit - 1) * MN4 + e];
#pragma unroll
                for (int z = 0; z < 8; z++)
                    if (z0 + z < g.ksplit) {
                        u0 += (uint32_t)v[z].x; u1 += (uint32_t)v[z].y;
                        u2 += (uint32_t)v[z].z; u3 += (uint32_t)v[z].w;
                    }
            }
            const int64_t row = (4 * e) / g.N, col = 4 * e - row * g.N;
            const int64_t o = row * g.ldc + col;
            const int32_t t[4] = {(int32_t)u0, (int32_t)u1, (int32_t)u2, (int32_t)u3};
#pragma unroll
            for (int c = 0; c < 4; c++) {
                if (g.acc) g.acc[o + c] = t[c];
                amax = max(amax, out_store(g.post, g.y, o + c, col + c, s * (float)t[c], qa));
            }
        }
        post_absmax_flush(g.post, amax);
        return;
    }
    for (int64_t e = t0; e < MN; e += stride) {
        uint32_t u = 0;
        for (int z = 0; z < g.ksplit; z++) u += (uint32_t)g.part[z * MN + e];
        const int32_t t = (int32_t)u;
        const int64_t row = e / g.N, col = e - row * g.N;
        const int64_t o = row * g.ldc + col;
        if (g.acc) g.acc[o] = t;
        amax = max(amax, out_store(g.post, g.y, o, col, s * (float)t, qa));
    }
    post_absmax_flush(g.post, amax);
}

// ------------------------------------------------------ pre-decoded operands
// For contractions with enough work per operand byte, both operands are
// first decoded once to OCP E4M3 (the elementwise map of dec_f8) into the
// caller's workspace; k_mma_pre then moves E4M3 bytes by DMA straight into the
// swizzled tile that the MFMAs read, with no decode and no second pass
// through LDS in the loop.
struct DecodeJob {
    const uint8_t* src;
    int64_t rows, cols16, pitch;   // rows of cols16 16-byte chunks, row pitch in bytes
    MmaDecode d;
    uint8_t* dst;                  // dense rows of 16 * cols16 bytes
};
// Both operands in one launch: the first n0 chunks belong to job 0.
__global__ __launch_bounds__(256) void k_decode_e4m3(DecodeJob j0, DecodeJob j1) {
    const int64_t n0 = j0.rows * j0.cols16, n = n0 + j1.rows * j1.cols16;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += stride) {
        const bool second = t >= n0;
        const DecodeJob& j = second ? j1 : j0;
        const int64_t u = second ? t - n0 : t;
        const int64_t r = u / j.cols16, c = u - r * j.cols16;
        const uint4 v = *(const uint4*)(j.src + r * j.pitch + 16 * c);
        *(uint4*)(j.dst + 16 * u) = make_uint4(dec_f8(v.x, j.d), dec_f8(v.y, j.d), dec_f8(v.z, j.d),
                                               dec_f8(v.w, j.d));
    }
}

// Rows of 32-code groups to packed E2M1: 16 bytes per group, byte i of dword j
// holding codes 8j+i (low nibble) and 8j+4+i (high nibble) -- a permutation of
// the reduction order applied to both operands alike.  Here cols16 counts
// groups of 32 codes.
__global__ __launch_bounds__(256) void k_decode_fp4(DecodeJob j0, DecodeJob j1) {
    const int64_t n0 = j0.rows * j0.cols16, n = n0 + j1.rows * j1.cols16;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += stride) {
        const bool second = t >= n0;
        const DecodeJob& j = second ? j1 : j0;
        const int64_t u = second ? t - n0 : t;
        const int64_t r = u / j.cols16, c = u - r * j.cols16;
        const uint8_t* p = j.src + r * j.pitch + 32 * c;
        const uint4 a = *(const uint4*)p, b = *(const uint4*)(p + 16);
        *(uint4*)(j.dst + 16 * u) =
            make_uint4(dec_f4(a.x, j.d) | (dec_f4(a.y, j.d) << 4), dec_f4(a.z, j.d) | (dec_f4(a.w, j.d) << 4),
                       dec_f4(b.x, j.d) | (dec_f4(b.y, j.d) << 4), dec_f4(b.z, j.d) | (dec_f4(b.w, j.d) << 4));
    }
}

// Rows of codes to packed E2M3 in stage blocks: the 64 codes 64b .. 64b+63 of
// row r become 48 bytes at dst + (b * rows + r) * 48, so that the rows of one
// contraction stage are one contiguous run of memory.  Within each 24-byte
// half, value i sits at bits 6i .. 6i+5 (little endian).  One item per (block,
// row), rows fastest, so that a wave writes 3 KB of contiguous memory; here
// cols16 counts blocks of 64 codes per row.
__device__ __forceinline__ void pack24(const uint4& a, const uint4& b, const MmaDecode& d, uint32_t* o) {
    const uint32_t w0 = pack6(dec_f6(a.x, d)), w1 = pack6(dec_f6(a.y, d));
    const uint32_t w2 = pack6(dec_f6(a.z, d)), w3 = pack6(dec_f6(a.w, d));
    const uint32_t w4 = pack6(dec_f6(b.x, d)), w5 = pack6(dec_f6(b.y, d));
    const uint32_t w6 = pack6(dec_f6(b.z, d)), w7 = pack6(dec_f6(b.w, d));
    o[0] = w0 | (w1 << 24);
    o[1] = (w1 >> 8) | (w2 << 16);
    o[2] = (w2 >> 16) | (w3 << 8);
    o[3] = w4 | (w5 << 24);
    o[4] = (w5 >> 8) | (w6 << 16);
    o[5] = (w6 >> 16) | (w7 << 8);
}
__global__ __launch_bounds__(256) void k_decode_fp6(DecodeJob j0, DecodeJob j1) {
    const int64_t n0 = j0.rows * j0.cols16, n = n0 + j1.rows * j1.cols16;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += stride) {
        const bool second = t >= n0;
        const DecodeJob& j = second ? j1 : j0;
        const int64_t u = second ? t - n0 : t;
        const int64_t b = u / j.rows, r = u - b * j.rows;
        const uint4* p = (const uint4*)(j.src + r * j.pitch + 64 * b);
        const uint4 c0 = p[0], c1 = p[1], c2 = p[2], c3 = p[3];
        uint32_t o[12];
        pack24(c0, c1, j.d, o);
        pack24(c2, c3, j.d, o + 6);
        uint4* q = (uint4*)(j.dst + u * 48);
        q[0] = make_uint4(o[0], o[1], o[2], o[3]);
        q[1] = make_uint4(o[4], o[5], o[6], o[7]);
        q[2] = make_uint4(o[8], o[9], o[10], o[11]);
    }
}

// DMA layout: one global_load_lds of a wave writes 1 KB = 16 tile rows of 64
// bytes; lane l lands at row 16 q + l / 4, physical chunk l % 4, which under
// the swizzle of lds_off holds logical chunk (l % 4) ^ ((l / 16) % 4) — the same
// for every DMA of the lane, so each lane fetches one fixed 16-byte column of
// the reduction in every row it serves.
// F4: the operands hold packed E2M1 (a 64-byte row is 128 reduction values,
// two 32x32x64 fp4 MFMAs per stage); otherwise E4M3 (64 values, one MFMA).
// Reduction lengths, pitches and offsets are in bytes of the decoded rows.
template <int BM, int BN, int WGM, int WGN, int CONV, int R, int F4>
__global__ __launch_bounds__(64 * WGM * WGN) void k_mma_pre(FastParams g) {
    constexpr int NW = WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int TI = WM / 32, TJ = WN / 32;
    constexpr int CHA = BM / (16 * NW), CHB = BN / (16 * NW), CT = CHA + CHB;
    static_assert(CHA * 16 * NW == BM && CHB * 16 * NW == BN, "whole DMA rows per wave");
    constexpr int TILE = (BM + BN) * BK;
    static_assert(R >= 2 && R <= 4, "ring depth");
    __shared__ __align__(16) uint8_t ring[R * TILE];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int tm, tn;
    tile_of(g, tm, tn);
    // convolution: blockIdx.z is the group; dense GEMM: the reduction range
    const int grp = CONV ? (int)blockIdx.z : 0;
    const int kz = CONV ? 0 : (int)blockIdx.z;
    const int kbeg = kz * g.kchunk;                                   // bytes
    const int Kl = CONV ? g.K : min(g.K - kbeg, g.kchunk);
    const int m0 = tm * BM, n0 = tn * BN;
    const int wr = (wave / WGN) * WM, wc = (wave % WGN) * WN;
    const ConvGeom& cg = g.ga;
    const int goffA = grp * cg.Cg;
    const int64_t brow0 = (int64_t)grp * g.N;
    const int rsub = lane >> 2;
    const int lc = (lane & 3) ^ ((lane >> 4) & 3);   // logical 16-byte chunk of this lane

    int64_t a_off[CHA];
    int a_ih[CHA], a_iw[CHA];
    int arow_ok[CHA];
    int kr = 0, ks = 0, kc = 16 * lc;
#pragma unroll
    for (int i = 0; i < CHA; i++) {
        const int m = m0 + 16 * (wave + i * NW) + rsub;
        const bool ok = m < g.M;
        arow_ok[i] = ok;
        if (CONV) {
            const int mm = ok ? m : 0;
            const int pq = cg.P * cg.Q;
            const int img = mm / pq, rem = mm - img * pq;
            const int p = rem / cg.Q, q = rem - p * cg.Q;
            a_ih[i] = ok ? p * cg.sh - cg.ph : -0x40000000;
            a_iw[i] = q * cg.sw - cg.pw;
            a_off[i] = (((int64_t)img * cg.H + a_ih[i]) * cg.W + a_iw[i]) * cg.pitch + goffA;
        } else {
            a_off[i] = (int64_t)(ok ? m : 0) * cg.pitch + 16 * lc + kbeg;
        }
    }
    if (CONV) {
        const int rs = kc / cg.Cg;
        kc -= rs * cg.Cg;
        kr = rs / cg.S;
        ks = rs - kr * cg.S;
    }
    int64_t b_off[CHB];
    int brow_ok[CHB];
#pragma unroll
    for (int i = 0; i < CHB; i++) {
        const int nn = n0 + 16 * (wave + i * NW) + rsub;
        brow_ok[i] = nn < g.N;
        b_off[i] = (brow0 + (brow_ok[i] ? nn : 0)) * g.ldb + 16 * lc + (CONV ? 0 : kbeg);
    }
    const uint8_t* z = kZeroRows.b[kZeroRowE4M3];

    // the E4M3 bytes of reduction offset k0 into a ring slot (stages in order)
    auto fetch = [&](int k0, uint8_t* slot) {
        const bool kin = k0 + 16 * lc < Kl;
        if (CONV) {
            const int64_t koff = ((int64_t)kr * cg.W + ks) * cg.pitch + kc;
#pragma unroll
            for (int i = 0; i < CHA; i++) {
                const int ih = a_ih[i] + kr, iw = a_iw[i] + ks;
                const bool ok = kin && (unsigned)ih < (unsigned)cg.H && (unsigned)iw < (unsigned)cg.W;
                dma16(ok ? g.A + a_off[i] + koff : z, slot + 1024 * (wave + i * NW));
            }
            kc += BK;
            while (kc >= cg.Cg) {
                kc -= cg.Cg;
                if (++ks == cg.S) { ks = 0; ++kr; }
            }
        } else {
#pragma unroll
            for (int i = 0; i < CHA; i++)
                dma16((kin && arow_ok[i]) ? g.A + a_off[i] + k0 : z, slot + 1024 * (wave + i * NW));
        }
#pragma unroll
        for (int i = 0; i < CHB; i++)
            dma16((kin && brow_ok[i]) ? g.B + b_off[i] + k0 : z,
                  slot + BM * BK + 1024 * (wave + i * NW));
    };

    v16f acc[TI][TJ];
#pragma unroll
    for (int i = 0; i < TI; i++)
#pragma unroll
        for (int j = 0; j < TJ; j++)
#pragma unroll
            for (int r = 0; r < 16; r++) acc[i][j][r] = 0.0f;

    // Each stage's MFMAs come in two parts.  E4M3: the A rows i < TI0, then the
    // rest, over the same B fragments (kept for two stages, by stage parity);
    // F4: the first and the second 64 values of the stage's 128.  Part 0 of stage s is issued before the
    // barrier that ends the stage, part 1 after it, so the MFMAs keep running
    // while the waves meet; the fragments of part 0 of stage s+1 are read right
    // after that barrier, under the MFMAs of part 1.
    constexpr int TI0 = (TI + 1) / 2;
    const int lr = lane & 31, lg = lane >> 5;
    v8i fa[TI], fb[2][TJ];        // E4M3 fragments: 32 bytes per lane
    v4i ga[2][TI], gb[2][TJ];     // E2M1 fragments: 16 bytes = 32 values per lane, per part
    auto frag8 = [&](const uint8_t* t, int row, int c0) {
        const v4i lo = *(const v4i*)&t[lds_off(row, c0)];
        const v4i hi = *(const v4i*)&t[lds_off(row, c0 + 1)];
        return v8i{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    };
    auto frag4 = [&](const uint8_t* t, int row, int c0) { return *(const v4i*)&t[lds_off(row, c0)]; };
    auto wide = [](v4i v) { return v8i{v[0], v[1], v[2], v[3], 0, 0, 0, 0}; };
    // fragments of part 0 of the stage in slot d (B into buffer PAR)
    auto read0 = [&](const uint8_t* d, auto PAR) {
        constexpr int par = decltype(PAR)::value;
        const uint8_t* tA = d;
        const uint8_t* tB = d + BM * BK;
        if constexpr (F4) {
#pragma unroll
            for (int j = 0; j < TJ; j++) gb[0][j] = frag4(tB, wc + 32 * j + lr, lg);
#pragma unroll
            for (int i = 0; i < TI; i++) ga[0][i] = frag4(tA, wr + 32 * i + lr, lg);
        } else {
#pragma unroll
            for (int j = 0; j < TJ; j++) fb[par][j] = frag8(tB, wc + 32 * j + lr, 2 * lg);
#pragma unroll
            for (int i = 0; i < TI0; i++) fa[i] = frag8(tA, wr + 32 * i + lr, 2 * lg);
        }
    };
    auto read1 = [&](const uint8_t* d) {
        const uint8_t* tA = d;
        const uint8_t* tB = d + BM * BK;
        if constexpr (F4) {
#pragma unroll
            for (int j = 0; j < TJ; j++) gb[1][j] = frag4(tB, wc + 32 * j + lr, 2 + lg);
#pragma unroll
            for (int i = 0; i < TI; i++) ga[1][i] = frag4(tA, wr + 32 * i + lr, 2 + lg);
        } else {
#pragma unroll
            for (int i = TI0; i < TI; i++) fa[i] = frag8(tA, wr + 32 * i + lr, 2 * lg);
        }
    };
    auto mfma = [&](auto PART, auto PAR) {
        constexpr int part = decltype(PART)::value, par = decltype(PAR)::value;
        if constexpr (F4) {
#pragma unroll
            for (int i = 0; i < TI; i++)
#pragma unroll
                for (int j = 0; j < TJ; j++)
                    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                        wide(ga[part][i]), wide(gb[part][j]), acc[i][j], 4, 4, 0, 127, 0, 127);
        } else {
#pragma unroll
            for (int i = part ? TI0 : 0; i < (part ? TI : TI0); i++)
#pragma unroll
                for (int j = 0; j < TJ; j++)
                    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                        fa[i], fb[par][j], acc[i][j], 0, 0, 0, 127, 0, 127);
        }
    };

    // stage s lives in slot s % R; its fetch is issued R stages ahead, so at
    // the barrier of stage s the fetches of stages s+2 .. s+R-1 may still be
    // in flight (CT instructions each) while stage s+1 has landed
    static_assert(R == 2 || R == 4, "ring depth");
    const int KT = (Kl + BK - 1) / BK;
    static_for<0, R>([&](auto Q) {
        constexpr int q = decltype(Q)::value;
        fetch(q * BK, ring + q * TILE);
    });
    vm_wait<(R - 1) * CT>();   // stage 0 landed
    lds_barrier();
    read0(ring, ic<0>{});
    // One stage; no branches inside, so that the compiler's waits track every
    // fragment exactly.  Past the last stage read0 reads a slot it never uses.
    auto stage = [&](int st, auto PAR) {
        constexpr int par = decltype(PAR)::value;
        uint8_t* slot = ring + (st & (R - 1)) * TILE;
        mfma(ic<0>{}, PAR);
        read1(slot);
        __builtin_amdgcn_sched_barrier(0);
        vm_wait<(R - 2) * CT>();       // this thread's part of stage st+1 landed
        lds_barrier();                 // all of it; every read of this slot is done
        fetch((st + R) * BK, slot);
        read0(ring + ((st + 1) & (R - 1)) * TILE, ic<par ^ 1>{});
        __builtin_amdgcn_sched_barrier(0);
        mfma(ic<1>{}, PAR);
    };
    int st = 0;
    for (; st + 1 < KT; st += 2) {
        stage(st, ic<0>{});
        stage(st + 1, ic<1>{});
    }
    if (st < KT) stage(st, ic<0>{});
    vm_wait<0>();   // the fetches past the end (+0 rows) land before the workgroup ends

    float s = 0.0f;
    if (g.y || g.post.on) s = ldexpf(g.alphaA[0] * g.alphaB[0], -(g.kA + g.kB));
    if (g.post.on && (CONV || g.ksplit == 1)) {
        static_assert(NW * 32 * 32 * TJ * 4 <= R * TILE, "post slabs fit the ring");
        if (g.acc)
            store_acc<TI, TJ>(g, lane, m0 + wr, n0 + wc, grp, [&](int i, int j, int r) {
                return (int32_t)ldexpf(acc[i][j][r], g.out_shift);
            });
        post_epilogue<TI, TJ>(g, (float*)ring + wave * (32 * 32 * TJ), lane, m0 + wr, n0 + wc, grp,
                              [&](int i, int j, int r) { return s * ldexpf(acc[i][j][r], g.out_shift); });
        return;
    }
#pragma unroll
    for (int i = 0; i < TI; i++)
#pragma unroll
        for (int j = 0; j < TJ; j++)
#pragma unroll
            for (int r = 0; r < 16; r++) {
                const int row = m0 + wr + 32 * i + 8 * (r >> 2) + 4 * lg + (r & 3);
                const int col = n0 + wc + 32 * j + lr;
                if (row < g.M && col < g.N) {
                    const float fv = ldexpf(acc[i][j][r], g.out_shift);
                    if (!CONV && g.ksplit > 1) {          // partial sum of this range
                        g.part[((int64_t)kz * g.M + row) * g.N + col] = (int32_t)fv;
                        continue;
                    }
                    const int64_t o = (int64_t)row * g.ldc + (int64_t)grp * g.N + col;
                    if (g.acc) g.acc[o] = (int32_t)fv;
                    if (g.y) g.y[o] = s * fv;
                }
            }
}

// Packed E2M3 operands (fp6): a stage is 64 reduction values = 48 bytes of
// every tile row, kept unswizzled in LDS (rows of 48 bytes, 12 banks apart:
// at most two lanes of a half-wave share a bank).  The DMA of a stage is
// (BM + BN) * 48 / 1024 wave instructions, CT per wave; each lane serves one
// 16-byte piece of one row per instruction.  An instruction never straddles
// the A/B boundary (BM * 48 is a multiple of 1024).  In the stage-blocked
// layout of k_decode_fp6 consecutive rows of a stage are contiguous, so an
// instruction reads whole 64-byte segments.  Convolution needs Cg % 64 == 0,
// so that a stage lies inside one filter tap (r, s): every lane of a stage
// then shares (r, s, channel block).  MFMA: 32x32x64 with
// cbsz = blgp = 2 (E2M3), six operand VGPRs; the MFMAs of a stage come in two
// parts around the barrier as in k_mma_pre.
template <int BM, int BN, int WGM, int WGN, int CONV, int R>
__global__ __launch_bounds__(64 * WGM * WGN) void k_mma_f6(FastParams g) {
    constexpr int NW = WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int TI = WM / 32, TJ = WN / 32;
    constexpr int RB = 48;                                // bytes per row per stage
    constexpr int NI = (BM + BN) * RB / 1024, CT = NI / NW;
    static_assert(CT * NW == NI && (BM * RB) % 1024 == 0, "whole DMA instructions per wave");
    constexpr int TILE = (BM + BN) * RB;
    static_assert(R >= 2 && R <= 6, "ring depth");
    __shared__ __align__(16) uint8_t ring[R * TILE];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int tm, tn;
    tile_of(g, tm, tn);
    const int grp = blockIdx.z;
    const int m0 = tm * BM, n0 = tn * BN;
    const int wr = (wave / WGN) * WM, wc = (wave % WGN) * WN;
    const ConvGeom& cg = g.ga;
    const int64_t brow0 = (int64_t)grp * g.N;

    // per DMA instruction i of this wave: operand, row, 16-byte piece of the lane
    int64_t off[CT];       // A: pixel-row or row byte offset; B: row byte offset (+ piece)
    int ih0[CT], iw0[CT];  // convolution: input position of the output pixel
    bool isa[CT], rok[CT];
    int piece[CT];
#pragma unroll
    for (int i = 0; i < CT; i++) {
        const int o = 1024 * (wave + i * NW) + 16 * lane;
        isa[i] = o < BM * RB;
        const int ob = isa[i] ? o : o - BM * RB;
        const int row = ob / RB;
        piece[i] = ob - row * RB;
        ih0[i] = iw0[i] = 0;
        if (isa[i]) {
            const int m = m0 + row;
            rok[i] = m < g.M;
            if (CONV) {
                const int mm = rok[i] ? m : 0;
                const int pq = cg.P * cg.Q;
                const int img = mm / pq, rem = mm - img * pq;
                const int p = rem / cg.Q, q = rem - p * cg.Q;
                ih0[i] = rok[i] ? p * cg.sh - cg.ph : -0x40000000;
                iw0[i] = q * cg.sw - cg.pw;
                off[i] = (((int64_t)img * cg.H + ih0[i]) * cg.W + iw0[i]) * RB + piece[i];
            } else {
                off[i] = (int64_t)(rok[i] ? m : 0) * RB + piece[i];
            }
        } else {
            const int nn = n0 + row;
            rok[i] = nn < g.N;
            off[i] = (brow0 + (rok[i] ? nn : 0)) * RB + piece[i];
        }
    }
    const uint8_t* z = kZeroRows.b[kZeroRowE4M3];   // 0x00: E2M3 +0
    const int KT = g.K / RB;                          // whole stages (K % 64 == 0 values)
    const int nbc = cg.Cg / RB;                       // convolution: stage blocks per tap
    int kr = 0, ks = 0, kb = 0;                       // convolution: tap and block of the next fetch

    auto fetch = [&](int st, uint8_t* slot) {
        const bool kin = st < KT;
        const int64_t kA = (int64_t)st * g.blkA, kB = (int64_t)st * g.blkB;
        int64_t koff = 0;
        if (CONV) koff = ((int64_t)kr * cg.W + ks) * RB + (int64_t)(grp * nbc + kb) * g.blkA;
#pragma unroll
        for (int i = 0; i < CT; i++) {
            bool ok = kin && rok[i];
            const uint8_t* src;
            if (isa[i]) {
                if (CONV) {
                    const int ih = ih0[i] + kr, iw = iw0[i] + ks;
                    ok = ok && (unsigned)ih < (unsigned)cg.H && (unsigned)iw < (unsigned)cg.W;
                    src = g.A + off[i] + koff;
                } else {
                    src = g.A + off[i] + kA;
                }
            } else {
                src = g.B + off[i] + kB;
            }
            dma16(ok ? src : z, slot + 1024 * (wave + i * NW));
        }
        if (CONV) {
            if (++kb == nbc) {
                kb = 0;
                if (++ks == cg.S) { ks = 0; ++kr; }
            }
        }
    };

    v16f acc[TI][TJ];
#pragma unroll
    for (int i = 0; i < TI; i++)
#pragma unroll
        for (int j = 0; j < TJ; j++)
#pragma unroll
            for (int r = 0; r < 16; r++) acc[i][j][r] = 0.0f;

    constexpr int TI0 = (TI + 1) / 2;
    const int lr = lane & 31, lg = lane >> 5;
    v8i fa[TI], fb[2][TJ];
    // (native vector loads through pointers into the ring: with HIP's struct
    // uint2 the compiler loses track of the address and waits for every DMA in
    // flight before the read)
    typedef int v2i __attribute__((ext_vector_type(2)));
    auto frag6 = [&](const uint8_t* t, int row) {   // 24 bytes: 32 values of this half of the stage
        const v2i* p = (const v2i*)(t + row * RB + 24 * lg);
        const v2i x0 = p[0], x1 = p[1], x2 = p[2];
        return v8i{x0[0], x0[1], x1[0], x1[1], x2[0], x2[1], 0, 0};
    };
    auto read0 = [&](const uint8_t* d, auto PAR) {
        constexpr int par = decltype(PAR)::value;
#pragma unroll
        for (int j = 0; j < TJ; j++) fb[par][j] = frag6(d + BM * RB, wc + 32 * j + lr);
#pragma unroll
        for (int i = 0; i < TI0; i++) fa[i] = frag6(d, wr + 32 * i + lr);
    };
    auto read1 = [&](const uint8_t* d) {
#pragma unroll
        for (int i = TI0; i < TI; i++) fa[i] = frag6(d, wr + 32 * i + lr);
    };
    auto mfma = [&](auto PART, auto PAR) {
        constexpr int part = decltype(PART)::value, par = decltype(PAR)::value;
#pragma unroll
        for (int i = part ? TI0 : 0; i < (part ? TI : TI0); i++)
#pragma unroll
            for (int j = 0; j < TJ; j++)
                acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa[i], fb[par][j], acc[i][j],
                                                                             2, 2, 0, 127, 0, 127);
    };

    static_for<0, R>([&](auto Q) {
        constexpr int q = decltype(Q)::value;
        fetch(q, ring + q * TILE);
    });
    vm_wait<(R - 1) * CT>();   // stage 0 landed
    lds_barrier();
    read0(ring, ic<0>{});
    auto stage = [&](int st, auto PAR) {
        constexpr int par = decltype(PAR)::value;
        uint8_t* slot = ring + (st % R) * TILE;
        mfma(ic<0>{}, PAR);
        read1(slot);
        __builtin_amdgcn_sched_barrier(0);
        vm_wait<(R - 2) * CT>();       // this thread's part of stage st+1 landed
        lds_barrier();                 // all of it; every read of this slot is done
        fetch(st + R, slot);
        read0(ring + ((st + 1) % R) * TILE, ic<par ^ 1>{});
        __builtin_amdgcn_sched_barrier(0);
        mfma(ic<1>{}, PAR);
    };
    int st = 0;
    for (; st + 1 < KT; st += 2) {
        stage(st, ic<0>{});
        stage(st + 1, ic<1>{});
    }
    if (st < KT) stage(st, ic<0>{});
    vm_wait<0>();   // the fetches past the end (+0 rows) land before the workgroup ends

    float s = 0.0f;
    if (g.y || g.post.on) s = ldexpf(g.alphaA[0] * g.alphaB[0], -(g.kA + g.kB));
    if (g.post.on && (CONV || g.ksplit == 1)) {
        static_assert(NW * 32 * 32 * TJ * 4 <= R * TILE, "post slabs fit the ring");
        if (g.acc)
            store_acc<TI, TJ>(g, lane, m0 + wr, n0 + wc, grp, [&](int i, int j, int r) {
                return (int32_t)ldexpf(acc[i][j][r], g.out_shift);
            });
        post_epilogue<TI, TJ>(g, (float*)ring + wave * (32 * 32 * TJ), lane, m0 + wr, n0 + wc, grp,
                              [&](int i, int j, int r) { return s * ldexpf(acc[i][j][r], g.out_shift); });
        return;
    }
#pragma unroll
    for (int i = 0; i < TI; i++)
#pragma unroll
        for (int j = 0; j < TJ; j++)
#pragma unroll
            for (int r = 0; r < 16; r++) {
                const int row = m0 + wr + 32 * i + 8 * (r >> 2) + 4 * lg + (r & 3);
                const int col = n0 + wc + 32 * j + lr;
                if (row < g.M && col < g.N) {
                    const float fv = ldexpf(acc[i][j][r], g.out_shift);
                    const int64_t o = (int64_t)row * g.ldc + (int64_t)grp * g.N + col;
                    if (g.acc) g.acc[o] = (int32_t)fv;
                    if (g.y) g.y[o] = s * fv;
                }
            }
}

template <int BM, int BN, int WGM, int WGN, int R>
hipError_t launch_f6_t(FastParams g, int groups, bool conv, hipStream_t s) {
    g.tiles_m = (g.M + BM - 1) / BM;
    g.tiles_n = (g.N + BN - 1) / BN;
    g.ntiles = g.tiles_m * g.tiles_n;
    dim3 grid(g.ntiles, 1, groups);
    const int nt = 64 * WGM * WGN;
    if (conv) k_mma_f6<BM, BN, WGM, WGN, 1, R><<<grid, nt, 0, s>>>(g);
    else k_mma_f6<BM, BN, WGM, WGN, 0, R><<<grid, nt, 0, s>>>(g);
    return hipGetLastError();
}

template <int BM, int BN, int WGM, int WGN, int R>
hipError_t launch_pre_t(FastParams g, int groups, bool conv, bool f4, hipStream_t s) {
    g.tiles_m = (g.M + BM - 1) / BM;
    g.tiles_n = (g.N + BN - 1) / BN;
    g.ntiles = g.tiles_m * g.tiles_n;
    dim3 grid(g.ntiles, 1, conv ? groups : g.ksplit);
    const int nt = 64 * WGM * WGN;
    if (f4) {
        if (conv) k_mma_pre<BM, BN, WGM, WGN, 1, R, 1><<<grid, nt, 0, s>>>(g);
        else k_mma_pre<BM, BN, WGM, WGN, 0, R, 1><<<grid, nt, 0, s>>>(g);
    } else {
        if (conv) k_mma_pre<BM, BN, WGM, WGN, 1, R, 0><<<grid, nt, 0, s>>>(g);
        else k_mma_pre<BM, BN, WGM, WGN, 0, R, 0><<<grid, nt, 0, s>>>(g);
    }
    if (!conv && g.ksplit > 1) {
        const int64_t MN = (int64_t)g.M * g.N;
        int64_t nb = (MN + 255) / 256;
        if (nb > 4 * num_cus()) nb = 4 * num_cus();
        k_splitk_sum<<<(unsigned)nb, 256, 0, s>>>(g);
    }
    return hipGetLastError();
}

template <int BM, int BN, int WGM, int WGN, int OP, int R>
hipError_t launch_t(FastParams g, int groups, hipStream_t s) {
    const bool conv = !(g.ga.H == 1 && g.ga.W == 1 && g.ga.R == 1 && g.ga.S == 1 && g.ga.ph == 0 &&
                        g.ga.pw == 0 && g.ga.Cg == g.K && groups == 1);
    g.tiles_m = (g.M + BM - 1) / BM;
    g.tiles_n = (g.N + BN - 1) / BN;
    g.ntiles = g.tiles_m * g.tiles_n;
    dim3 grid(g.ntiles, 1, conv ? groups : g.ksplit);
    if (conv) k_mma<BM, BN, WGM, WGN, OP, 1, R><<<grid, 64 * WGM * WGN, 0, s>>>(g);
    else k_mma<BM, BN, WGM, WGN, OP, 0, R><<<grid, 64 * WGM * WGN, 0, s>>>(g);
    if (!conv && g.ksplit > 1) {
        const int64_t MN = (int64_t)g.M * g.N;
        int64_t nb = (MN + 255) / 256;
        if (nb > 4 * num_cus()) nb = 4 * num_cus();
        k_splitk_sum<<<(unsigned)nb, 256, 0, s>>>(g);
    }
    return hipGetLastError();
}

template <int OP>
hipError_t launch_op(const FastParams& g, int groups, hipStream_t s) {
    if (g.ksplit > 1)   // the tiles mma_splitk planned with
        return g.M > 64 ? launch_t<128, 128, 2, 4, OP, 4>(g, groups, s) : launch_t<64, 64, 2, 2, OP, 4>(g, groups, s);
    const int64_t cus = num_cus();
    auto tiles = [&](int bm, int bn) {
        return (int64_t)((g.M + bm - 1) / bm) * ((g.N + bn - 1) / bn) * groups;
    };
    // Measured on MI355X (ESB(5,3) operands): 256 x 256 on eight waves is the
    // fastest tile wherever it fills the chip; below that, decoding per MAC
    // grows as (BM + BN) / (BM * BN), so the largest tile that keeps at least
    // half the CUs busy wins over a smaller one that fills them all.
    if (g.N > 128 && tiles(256, 256) >= cus) return launch_t<256, 256, 2, 4, OP, 2>(g, groups, s);
    if (g.N > 64 && tiles(128, 128) >= cus / 2) return launch_t<128, 128, 2, 4, OP, 2>(g, groups, s);
    if (tiles(128, 64) >= cus) return launch_t<128, 64, 2, 2, OP, 4>(g, groups, s);
    return launch_t<64, 64, 2, 2, OP, 4>(g, groups, s);
}

}  // namespace

MmaDecode mma_decode(const Fmt& f, int op) {
    MmaDecode d;
    const uint32_t rep = 0x01010101u;
    d.lm = ((1u << (f.n - 1)) - 1u) * rep;
    d.inc = ((1u << f.k) << (3 - f.k)) * rep;   // + 1 in the exponent field, after the shift
    d.shf = 3 - f.k;
    d.lmf = (((1u << (f.n - 1)) - 1u) << d.shf) * rep;
    d.shs = 8 - f.n;
    d.sel = (op == 1) ? 0u : ((1u << f.n) - 1u) * rep;
    uint32_t t[2] = {0, 0};
    if (op == 0) {
        for (uint32_t c = 0; c < 8; c++) {
            const uint32_t m = (uint32_t)decode_int(f, c & ((1u << f.n) - 1u)) & 0xffu;
            t[c >> 2] |= m << (8 * (c & 3));
        }
    }
    d.t0 = t[0];
    d.t1 = t[1];
    return d;
}

int mma_choose(const Fmt& fa, const Fmt& fb, int64_t K) {
    if (fa.n <= 3 && fb.n <= 3) return 0;
    auto f8ok = [](const Fmt& f) {
        return f.ebits <= 4 && f.k <= 3 && !(f.ebits == 4 && f.k == 3);
    };
    if (!f8ok(fa) || !f8ok(fb)) return -1;
    const double p = (double)fa.max_int * (double)fb.max_int;
    if (p > 4096.0 || (double)K * p >= 16777216.0) return -1;
    return 1;
}

MmaDecode mma_decode_f4(const Fmt& f) {
    MmaDecode d{};
    const uint32_t rep = 0x01010101u;
    d.shf = 1 - f.k;                                     // fraction to E2M1's one bit
    d.lm = ((1u << (f.n - 1)) - 1u) * rep;
    d.inc = 0x02u * rep;                                 // + 1 in the exponent field
    d.lmf = (((1u << (f.n - 1)) - 1u) << d.shf) * rep;
    d.shs = 4 - f.n;                                     // sign to bit 3
    return d;
}

bool mma_f4ok(const Fmt& fa, const Fmt& fb, int64_t K) {
    auto in_e2m1 = [](const Fmt& f) { return f.ebits <= 2 && f.k <= 1; };
    if (!in_e2m1(fa) || !in_e2m1(fb)) return false;
    return (double)K * (double)fa.max_int * (double)fb.max_int < 16777216.0;
}

// The fp6 path only for shapes that fill the chip with 256 x 256 tiles: there
// it matches the E4M3 path (kernel ~7 % faster, decode as fast); the smaller
// tiles that would fit its 48-byte rows run on four or two waves and lose.
bool mma_f6_tiles(int64_t M, int64_t N, int groups) {
    return N > 128 && ((M + 255) / 256) * ((N + 255) / 256) * groups >= num_cus();
}

MmaDecode mma_decode_f6(const Fmt& f) {
    MmaDecode d{};
    const uint32_t rep = 0x01010101u;
    d.shf = 3 - f.k;                                     // fraction to E2M3's three bits
    d.lm = ((1u << (f.n - 1)) - 1u) * rep;
    d.inc = 0x08u * rep;                                 // + 1 in the exponent field
    d.lmf = (((1u << (f.n - 1)) - 1u) << d.shf) * rep;
    d.shs = 6 - f.n;                                     // sign to bit 5
    return d;
}

bool mma_f6ok(const Fmt& fa, const Fmt& fb, int64_t K) {
    auto in_e2m3 = [](const Fmt& f) { return f.ebits <= 2 && f.k <= 3; };
    if (!in_e2m3(fa) || !in_e2m3(fb)) return false;
    return (double)K * (double)fa.max_int * (double)fb.max_int < 16777216.0;
}

bool mma_fits(const ConvGeom& ga, const uint8_t* A, int64_t K, int groups, const uint8_t* B,
              int64_t ldb, int b_layout) {
    return b_layout == 0 && K > 0 && ga.Cg >= 16 && ga.Cg % 16 == 0 && ga.pitch % 16 == 0 &&
           (uintptr_t)A % 16 == 0 && (int64_t)groups * ga.Cg <= ga.pitch && K % 16 == 0 &&
           ldb % 16 == 0 && (uintptr_t)B % 16 == 0 &&
           (int64_t)ga.Nb * ga.H * ga.W <= 0x7fffffff;
}

size_t mma_pre_workspace(int64_t a_rows, int64_t a_cols, int64_t b_rows, int64_t K) {
    const auto al = [](size_t v) { return (v + 255) & ~(size_t)255; };
    return al((size_t)a_rows * (size_t)a_cols) + al((size_t)b_rows * (size_t)K);
}

// Packed E2M1 rows (esb_pack): 32 codes to 16 bytes, the layout k_mma_pre reads.
hipError_t launch_pack_fp4(const uint8_t* codes, int64_t rows, int64_t K, int64_t ld, const Fmt& f,
                           uint8_t* packed, hipStream_t s) {
    if (rows <= 0 || K <= 0) return hipSuccess;
    DecodeJob j0{codes, rows, K / 32, ld, mma_decode_f4(f), packed};
    DecodeJob j1{codes, 0, 0, ld, mma_decode_f4(f), packed};
    int64_t blocks = (j0.rows * j0.cols16 + 255) / 256;
    const int64_t cap = (int64_t)num_cus() * 16;
    if (blocks > cap) blocks = cap;
    k_decode_fp4<<<(unsigned)(blocks < 1 ? 1 : blocks), 256, 0, s>>>(j0, j1);
    return hipGetLastError();
}

hipError_t launch_mma_pre(int M, int N, int K, int groups, const ConvGeom& ga, const uint8_t* A,
                          int64_t a_rows, int64_t a_cols, int64_t a_pitch, const Fmt& fa,
                          const float* alphaA, const uint8_t* B, int64_t b_rows, int64_t ldb,
                          const Fmt& fb, const float* alphaB, int32_t* acc, float* y, int64_t ldc,
                          int mode, void* ws, const uint8_t* b_packed, bool split, hipStream_t s,
                          const Post* post) {
    if (M <= 0 || N <= 0) return hipSuccess;
    const bool conv = !(ga.H == 1 && ga.W == 1 && ga.R == 1 && ga.S == 1 && ga.ph == 0 && ga.pw == 0 &&
                        ga.Cg == K && groups == 1);
    const bool f4 = mode == 1, f6 = mode == 2;
    // decoded bytes per code: 1 (E4M3), 1/2 (E2M1) or 3/4 (E2M3); lengths below are in bytes
    auto bytes = [&](int64_t codes) { return f4 ? codes / 2 : (f6 ? codes / 4 * 3 : codes); };
    const int64_t a_bytes = bytes(a_cols), kbytes = bytes(K);
    const auto al = [](size_t v) { return (v + 255) & ~(size_t)255; };
    uint8_t* dA = (uint8_t*)ws;
    uint8_t* dBw = dA + al((size_t)a_rows * (size_t)a_bytes);
    // B packed by esb_pack (E2M1 rows of K/2 bytes): used in place, not decoded
    uint8_t* dB = b_packed ? (uint8_t*)b_packed : dBw;
    int32_t* part = (int32_t*)(b_packed ? dBw : dBw + al((size_t)b_rows * (size_t)kbytes));
    const int grp = f6 ? 64 : (f4 ? 32 : 16);    // codes per decode item
    const MmaDecode da = f4 ? mma_decode_f4(fa) : (f6 ? mma_decode_f6(fa) : mma_decode(fa, 1));
    const MmaDecode db = f4 ? mma_decode_f4(fb) : (f6 ? mma_decode_f6(fb) : mma_decode(fb, 1));
    DecodeJob j0{A, a_rows, a_cols / grp, a_pitch, da, dA};
    DecodeJob j1{B, b_packed ? 0 : b_rows, (int64_t)K / grp, ldb, db, dB};
    const int64_t items = j0.rows * j0.cols16 + j1.rows * j1.cols16;
    int64_t blocks = (items + 255) / 256;
    const int64_t cap = (int64_t)num_cus() * 16;
    if (blocks > cap) blocks = cap;
    const unsigned nb = (unsigned)(blocks < 1 ? 1 : blocks);
    if (f4) k_decode_fp4<<<nb, 256, 0, s>>>(j0, j1);
    else if (f6) k_decode_fp6<<<nb, 256, 0, s>>>(j0, j1);
    else k_decode_e4m3<<<nb, 256, 0, s>>>(j0, j1);
    FastParams g;
    g.M = M; g.N = N; g.K = (int)kbytes; g.ga = ga;
    g.ga.pitch = (int)a_bytes;
    g.ga.Cg = (int)bytes(ga.Cg);
    g.A = dA; g.B = dB; g.ldb = kbytes;
    g.ksplit = 1; g.kchunk = (int)kbytes; g.part = nullptr;
    if (split && !conv && !f6) {
        int kc = K;
        const int ks = mma_splitk(M, N, K, &kc);
        if (ks > 1) {   // the same number of ranges, in 64-byte stages of decoded bytes
            const int64_t kcb = ((kbytes + ks - 1) / ks + 63) / 64 * 64;
            g.kchunk = (int)kcb;
            g.ksplit = (int)((kbytes + kcb - 1) / kcb);
            g.part = part;
        }
    }
    g.blkA = a_rows * 48;
    g.blkB = b_rows * 48;
    g.da = j0.d;
    g.db = j1.d;
    g.alphaA = alphaA; g.alphaB = alphaB; g.acc = acc; g.y = y; g.ldc = ldc;
    g.post = post ? *post : Post{};
    g.kA = fa.k; g.kB = fb.k;
    // E4M3 holds q * 2^-6 per operand; E2M1 and E2M3 hold q itself
    g.out_shift = fa.k + fb.k + ((f4 || f6) ? 0 : 12);
    g.zrowA = g.zrowB = kZeroRowE4M3;
    g.tiles_m = g.tiles_n = g.ntiles = 0;
    const int64_t cus = num_cus();
    auto tiles = [&](int bm, int bn) {
        return (int64_t)((M + bm - 1) / bm) * ((N + bn - 1) / bn) * groups;
    };
    if (f6) return launch_f6_t<256, 256, 2, 4, 4>(g, groups, conv, s);   // see mma_f6_tiles
    if (g.ksplit > 1)   // the tiles mma_splitk planned with
        return M > 64 ? launch_pre_t<128, 128, 2, 4, 4>(g, groups, conv, f4, s)
                      : launch_pre_t<64, 64, 2, 2, 4>(g, groups, conv, f4, s);
    if (N > 128 && tiles(256, 256) >= cus) return launch_pre_t<256, 256, 2, 4, 4>(g, groups, conv, f4, s);
    if (N > 64 && tiles(256, 128) >= cus) return launch_pre_t<256, 128, 4, 2, 4>(g, groups, conv, f4, s);
    if (N > 64 && tiles(128, 128) >= cus / 2) return launch_pre_t<128, 128, 2, 4, 4>(g, groups, conv, f4, s);
    if (tiles(128, 64) >= cus) return launch_pre_t<128, 64, 2, 2, 4>(g, groups, conv, f4, s);
    return launch_pre_t<64, 64, 2, 2, 4>(g, groups, conv, f4, s);
}

// Split of the reduction for a dense GEMM with too few output tiles to fill
// the chip (skinny shapes such as a fully connected layer at a small batch):
// ranges of kchunk (a multiple of 64, at least 4 stages) so that tiles x
// ranges reaches about one workgroup per CU (measured on the AlexNet FC at
// batch 128 with 128 x 64 tiles: 4 ranges 24.5 us, 8 ranges 26.3, 16 ranges
// 36.5; more partial sums cost more than the extra workgroups gain; 128 x 128
// tiles on eight waves with 8 ranges: 24.0 us); 1 when no split pays.
int mma_splitk(int64_t M, int64_t N, int64_t K, int* kchunk) {
    *kchunk = (int)K;
    const int64_t cus = num_cus();
    const int64_t bm = M > 64 ? 128 : 64;
    const int64_t bn = M > 64 ? 128 : 64;
    const int64_t tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
    if (2.0 * (double)M * (double)N * (double)K < 2147483648.0 || tiles * 2 >= cus) return 1;
    int64_t ks = (cus + tiles - 1) / tiles;
    if (ks > K / 256) ks = K / 256;
    if (ks > 16) ks = 16;
    if (ks < 2) return 1;
    const int64_t kc = ((K + ks - 1) / ks + 63) / 64 * 64;
    *kchunk = (int)kc;
    return (int)((K + kc - 1) / kc);
}

hipError_t launch_mma(int op, int M, int N, int K, int groups, const ConvGeom& ga,
                      const uint8_t* A, const Fmt& fa, const float* alphaA, const uint8_t* B,
                      int64_t ldb, const Fmt& fb, const float* alphaB, int32_t* acc, float* y,
                      int64_t ldc, int32_t* part, hipStream_t s, const Post* post) {
    if (M <= 0 || N <= 0) return hipSuccess;
    FastParams g;
    g.M = M; g.N = N; g.K = K; g.ga = ga;
    g.A = A; g.B = B; g.ldb = ldb;
    g.ksplit = 1;
    g.kchunk = K;
    g.part = nullptr;
    if (part && groups == 1) {
        int kc = K;
        const int ks = mma_splitk(M, N, K, &kc);
        if (ks > 1) { g.ksplit = ks; g.kchunk = kc; g.part = part; }
    }
    g.da = mma_decode(fa, op);
    g.db = mma_decode(fb, op);
    g.alphaA = alphaA; g.alphaB = alphaB; g.acc = acc; g.y = y; g.ldc = ldc;
    g.post = post ? *post : Post{};
    g.kA = fa.k; g.kB = fb.k;
    g.out_shift = fa.k + fb.k + 12;
    g.zrowA = (fa.n - 2) * 8 + fa.k;
    g.zrowB = (fb.n - 2) * 8 + fb.k;
    g.tiles_m = g.tiles_n = g.ntiles = 0;
    return op == 1 ? launch_op<1>(g, groups, s) : launch_op<0>(g, groups, s);
}

}  // namespace esb
