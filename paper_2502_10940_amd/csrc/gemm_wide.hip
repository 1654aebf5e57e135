// gemm_wide.hip -- the persistent 256 x 256 bf16 MFMA GEMM:
// C[M][N] = sum_k P(m, k) Q(n, k), fp32 accumulation, the fused epilogues of
// epilogue.hpp.
//
// Design (CDNA4, wave64, one workgroup per CU):
//  * 512 threads = 8 waves in a 2 x 4 grid, each wave a 128 x 64 block of C
//    as 4 x 2 tiles of v_mfma_f32_32x32x16_bf16 (128 fp32 accumulators per
//    lane), two waves per SIMD so that one issues MFMAs while the other waits.
//    One 256 x 256 tile per CU needs 1 KB of operands per unit of k, two
//    thirds of what two 256 x 128 tiles need.
//  * K advances in tiles of 32 through four LDS stages of 32 KB: while one K
//    tile is consumed the next three are in flight, loaded straight into LDS
//    (global_load_lds_dwordx4: no staging registers, no LDS write
//    instructions).  K tails and unaligned operands take guarded register
//    loads written to the same layout.
//  * One barrier per K tile, placed between its two 16-deep sub-steps.  The
//    fragments of each sub-step are read from LDS under the MFMAs of the one
//    before, and the stage the barrier frees is refilled at once.
//  * The grid is persistent (one workgroup per CU).  The last four K tiles of
//    an output tile prefetch the first four K tiles of the next one, so the
//    next tile's loads are in flight during the epilogue, and the epilogue's
//    stores drain under the next tile's MFMAs.
//  * Each wave counts the vector-memory operations it issues and waits for a
//    K tile with vmcnt(operations issued after it): a wave's vector-memory
//    operations complete in issue order.
//  * LDS layouts.  k-contiguous operands: [256 rows][32 k], 64-byte rows,
//    16-byte chunks XOR-swizzled by (row >> 2) & 3, read with ds_read_b128.
//    m-contiguous operands (the weight-gradient operands, the weights of the
//    backward products): [32 k][256 m], 512-byte rows, chunks swizzled by
//    4 (k & 3), read with the transposing ds_read_b64_tr_b16.  With gfx950's
//    64 banks neither read conflicts.
//  * Ragged edges: k-contiguous rows past the edge re-read the last row,
//    m-contiguous chunks past the edge re-read the last chunk (the chunk
//    holding the last column may run into the row's pitch padding, which the
//    ABI allows).  Those values reach only outputs that are not stored.
#include "internal.hpp"
#include "device_math.hpp"
#include "epilogue.hpp"

namespace cola {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef const __attribute__((address_space(1))) void* gptr_t;
typedef __attribute__((address_space(3))) void* lptr_t;
typedef __attribute__((address_space(3))) s16x4* lptr4_t;

constexpr int BM = 256;
constexpr int BN = 256;
constexpr int BK = 32;
constexpr int WAVES_M = 2;                     // wave grid of the workgroup
constexpr int WAVES_N = 4;
constexpr int NW = WAVES_M * WAVES_N;
constexpr int NT = 64 * NW;
constexpr int NSTAGE = 4;
constexpr int TILE = 256 * BK * 2;            // bytes of one operand tile (either layout)
constexpr int STAGE = 2 * TILE;
constexpr int WR = BM / WAVES_M;              // rows of a wave's block
constexpr int WC = BN / WAVES_N;              // columns of a wave's block
constexpr int TM = WR / 32;                   // MFMA tiles per wave
constexpr int TN = WC / 32;
constexpr int DTL_OPS = TILE / 1024 / NW;     // direct-to-LDS instructions per wave per operand tile
constexpr int SMEM = NSTAGE * STAGE;
static_assert(SMEM <= 160 * 1024, "LDS budget");

__device__ __forceinline__ bool aligned16(const void* p, int64_t ld) {
    return ((reinterpret_cast<uintptr_t>(p) & 15u) == 0) && ((ld & 7) == 0);
}

__device__ __forceinline__ void dtl16(const void* g, char* lds) {
    __builtin_amdgcn_global_load_lds((gptr_t)g, (lptr_t)lds, 16, 0, 0);
}

__device__ __forceinline__ uint4 load8_guarded(const uint16_t* p, int valid) {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const uint32_t lo = (2 * e < valid) ? p[2 * e] : 0u;
        const uint32_t hi = (2 * e + 1 < valid) ? p[2 * e + 1] : 0u;
        w[e] = lo | (hi << 16);
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

template <int LAYOUT>
struct Tile;

// ---- k-contiguous operand: LDS [256 rows][32 k] ----
template <>
struct Tile<KMAJ> {
    __device__ static __forceinline__ int off(int row, int c) {
        return row * 64 + ((c ^ ((row >> 2) & 3)) << 4);
    }

    // Wave w, instruction j fills LDS bytes [1024 (4w + j), +1024): rows
    // 16 (4w + j) .. +16, lane l -> row + l/4, physical chunk l % 4.
    __device__ static __forceinline__ void dtl(char* lds, const uint16_t* base, int64_t ld, int64_t row0,
                                               int64_t rows, int64_t k0) {
        const int wave = threadIdx.x >> 6;
        const int lane = threadIdx.x & 63;
#pragma unroll
        for (int j = 0; j < DTL_OPS; ++j) {
            const int blk = DTL_OPS * wave + j;
            const int row = 16 * blk + (lane >> 2);
            const int lc = (lane & 3) ^ ((row >> 2) & 3);
            int64_t grow = row0 + row;
            if (grow >= rows) grow = rows - 1;
            dtl16(base + grow * ld + k0 + 8 * lc, lds + 1024 * blk);
        }
    }

    // Guarded register path: chunk id -> (row id / 4, chunk id % 4).
    __device__ static __forceinline__ void load_store(char* lds, const uint16_t* base, int64_t ld, int64_t row0,
                                                      int64_t rows, int64_t k0, int64_t kend, bool aligned) {
#pragma unroll
        for (int i = 0; i < 256 * 4 / NT; ++i) {
            const int id = threadIdx.x + NT * i;
            const int64_t row = row0 + (id >> 2);
            const int64_t k = k0 + 8 * (id & 3);
            uint4 v;
            if (row < rows && k + 8 <= kend && aligned) {
                v = *reinterpret_cast<const uint4*>(base + row * ld + k);
            } else {
                const int64_t valid = row < rows ? kend - k : 0;
                v = load8_guarded(base + (row < rows ? row : 0) * ld + k,
                                  (int)(valid < 0 ? 0 : (valid > 8 ? 8 : valid)));
            }
            *reinterpret_cast<uint4*>(lds + off(id >> 2, id & 3)) = v;
        }
    }

    // 32 rows (row0 ..) x 16 k (16 s ..) fragment, s = 0 or 1
    __device__ static __forceinline__ bf16x8 frag(const char* lds, int row0, int s, int lane) {
        return *reinterpret_cast<const bf16x8*>(lds + off(row0 + (lane & 31), 2 * s + (lane >> 5)));
    }
};

// ---- m-contiguous operand: LDS [32 k][256 m] ----
template <>
struct Tile<MNMAJ> {
    __device__ static __forceinline__ int off(int k, int c) {
        return k * 512 + ((c ^ ((k & 3) << 2)) << 4);
    }

    // Wave w, instruction j fills LDS bytes [1024 (4w + j), +1024): k rows
    // 2 (4w + j) and 2 (4w + j) + 1, lane l -> k row + l/32, physical chunk
    // l % 32.  Chunks that start past the last column re-read the last chunk.
    __device__ static __forceinline__ void dtl(char* lds, const uint16_t* base, int64_t ld, int64_t m0,
                                               int64_t rows, int64_t k0) {
        const int wave = threadIdx.x >> 6;
        const int lane = threadIdx.x & 63;
        const int64_t mlast = ((rows - 1) >> 3) << 3;
#pragma unroll
        for (int j = 0; j < DTL_OPS; ++j) {
            const int blk = DTL_OPS * wave + j;
            const int k = 2 * blk + (lane >> 5);
            const int lc = (lane & 31) ^ ((k & 3) << 2);
            int64_t m = m0 + 8 * lc;
            if (m > mlast) m = mlast;
            dtl16(base + (k0 + k) * ld + m, lds + 1024 * blk);
        }
    }

    __device__ static __forceinline__ void load_store(char* lds, const uint16_t* base, int64_t ld, int64_t m0,
                                                      int64_t rows, int64_t k0, int64_t kend, bool aligned) {
#pragma unroll
        for (int i = 0; i < 32 * 32 / NT; ++i) {
            const int id = threadIdx.x + NT * i;
            const int64_t k = k0 + (id >> 5);
            const int64_t m = m0 + 8 * (id & 31);
            uint4 v;
            if (k < kend && m + 8 <= rows && aligned) {
                v = *reinterpret_cast<const uint4*>(base + k * ld + m);
            } else {
                const int64_t valid = k < kend ? rows - m : 0;
                v = load8_guarded(base + (k < kend ? k : 0) * ld + (valid > 0 ? m : 0),
                                  (int)(valid < 0 ? 0 : (valid > 8 ? 8 : valid)));
            }
            *reinterpret_cast<uint4*>(lds + off(id >> 5, id & 31)) = v;
        }
    }

    // 32 m (m0 ..) x 16 k (16 s ..) fragment via two transposing reads: in
    // each 16-lane group, lanes 4q..4q+3 point at k row q of a 4 x 16 block
    // (four consecutive m each) and lane i receives column m0 + i.
    __device__ static __forceinline__ bf16x8 frag(const char* lds, int m0, int s, int lane) {
        const int g = lane >> 4;
        const int i = lane & 15;
        const int m = m0 + 16 * (g & 1) + 4 * (i & 3);
        const int k = 16 * s + 8 * (g >> 1) + (i >> 2);
        const int byte = (m & 7) * 2;
        const int c = m >> 3;
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lptr4_t)(lds + off(k, c) + byte));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lptr4_t)(lds + off(k + 4, c) + byte));
        const s16x8 s8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        return __builtin_bit_cast(bf16x8, s8);
    }
};

// LDS barrier: this wave's LDS operations are complete, then all waves meet.
// (No memory fence: global stores stay in flight.)
__device__ __forceinline__ void barrier_lds() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most n of this wave's vector-memory operations are
// outstanding, n rounded down to a multiple of 4 (a longer wait, never a
// shorter one).
__device__ __forceinline__ void wait_vm_at_most(int n) {
    n = __builtin_amdgcn_readfirstlane(n);
    switch (n < 0 ? 0 : (n >= 60 ? 15 : n >> 2)) {
        case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
        case 1: asm volatile("s_waitcnt vmcnt(4)" ::: "memory"); break;
        case 2: asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
        case 3: asm volatile("s_waitcnt vmcnt(12)" ::: "memory"); break;
        case 4: asm volatile("s_waitcnt vmcnt(16)" ::: "memory"); break;
        case 5: asm volatile("s_waitcnt vmcnt(20)" ::: "memory"); break;
        case 6: asm volatile("s_waitcnt vmcnt(24)" ::: "memory"); break;
        case 7: asm volatile("s_waitcnt vmcnt(28)" ::: "memory"); break;
        case 8: asm volatile("s_waitcnt vmcnt(32)" ::: "memory"); break;
        case 9: asm volatile("s_waitcnt vmcnt(36)" ::: "memory"); break;
        case 10: asm volatile("s_waitcnt vmcnt(40)" ::: "memory"); break;
        case 11: asm volatile("s_waitcnt vmcnt(44)" ::: "memory"); break;
        case 12: asm volatile("s_waitcnt vmcnt(48)" ::: "memory"); break;
        case 13: asm volatile("s_waitcnt vmcnt(52)" ::: "memory"); break;
        case 14: asm volatile("s_waitcnt vmcnt(56)" ::: "memory"); break;
        default: asm volatile("s_waitcnt vmcnt(60)" ::: "memory"); break;
    }
}

// Vector-memory operations one wave issues in the epilogue of an interior
// tile with aligned outputs (4 TM TN groups of 4 columns per lane).  The bf16
// stores without an input take the whole-line path there (one 16-byte store
// per two groups, TN even).  An over-count would shorten a wait, so where the
// path is not certain the smaller count is used.
template <int EPI>
__device__ __forceinline__ int epilogue_ops(bool aux) {
    constexpr int G = 4 * TM * TN;
    static_assert(TN % 2 == 0, "whole-line epilogue");
    return EPI == EPI_STORE || EPI == EPI_H ? G / 2
         : EPI == EPI_STORE_F32 ? G
         : EPI == EPI_Z_H ? (aux ? G : G / 2)
         : (aux ? 3 * G : 2 * G);               // EPI_DZ: Z loads, dZ (and H) stores
}

struct TileCoord {
    int64_t m0, n0, kbeg, kend;
    int split, nk;
};

// The persistent grid walks the output tiles.  With a grid and a tile count
// that are multiples of 8, XCD x (blockIdx % 8) owns the contiguous tile range
// [x T/8, (x+1) T/8), which its workgroups sweep together (n fastest), so
// tiles that share operand rows run at the same time on the same L2.
__device__ __forceinline__ bool tile_at(const GemmArgs& a, int64_t i, TileCoord* t) {
    const int64_t tiles_n = (a.N + BN - 1) / BN;
    const int64_t tiles_m = (a.M + BM - 1) / BM;
    const int64_t per_split = tiles_m * tiles_n;
    const int64_t total = per_split * a.splits;
    const int64_t G = gridDim.x;
    int64_t idx;
    if ((G & 7) == 0 && (total & 7) == 0) {
        const int64_t x = blockIdx.x & 7;
        const int64_t j = (int64_t)(blockIdx.x >> 3) + i * (G >> 3);
        if (j >= (total >> 3)) return false;
        idx = x * (total >> 3) + j;
    } else {
        idx = (int64_t)blockIdx.x + i * G;
        if (idx >= total) return false;
    }
    t->split = (int)(idx / per_split);
    const int64_t rem = idx - (int64_t)t->split * per_split;
    t->m0 = (rem / tiles_n) * BM;
    t->n0 = (rem % tiles_n) * BN;
    t->kbeg = (int64_t)t->split * a.k_chunk;
    t->kend = min(a.K, t->kbeg + a.k_chunk);
    t->nk = (int)((t->kend - t->kbeg + BK - 1) / BK);
    return true;
}

template <int PL, int QL, int EPI, int TAG>
__global__ __launch_bounds__(NT, 1) void gemm_wide_kernel(GemmArgs a) {
    __shared__ __attribute__((aligned(1024))) char smem[SMEM];

    const uint16_t* P = reinterpret_cast<const uint16_t*>(a.p);
    const uint16_t* Q = reinterpret_cast<const uint16_t*>(a.q);
    const bool p_al = aligned16(a.p, a.ldp);
    const bool q_al = aligned16(a.q, a.ldq);
    const int64_t out_vec = (EPI == EPI_STORE_F32) ? 3 : 7;   // pitch granule of a 16-byte store
    bool out_al = ((reinterpret_cast<uintptr_t>(a.c) & 15u) == 0) && ((a.ldc & out_vec) == 0);
    if (EPI == EPI_Z_H || EPI == EPI_DZ)
        out_al = out_al && (!a.aux || (((reinterpret_cast<uintptr_t>(a.aux) & 15u) == 0) && ((a.ldaux & 7) == 0)));
    if (EPI == EPI_DZ)
        out_al = out_al && ((reinterpret_cast<uintptr_t>(a.zin) & 15u) == 0) && ((a.ldzin & 7) == 0);
    const int epi_ops = epilogue_ops<EPI>(a.aux != nullptr);

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;

    // Vector-memory operations this wave has issued (counted exactly, or
    // under-counted, which only lengthens a wait), and, one byte per stage,
    // that count modulo 256 right after the stage's K tile was issued (at most
    // three K tiles and one epilogue, under 256 operations, follow a K tile
    // before it is awaited).  All wave-uniform scalars.
    int issued = 0;
    uint32_t done_at = 0;
    int loaded = 0;                            // bit st: stage st holds an issued K tile
    auto ops_after = [&](int st) -> int {
        return (int)(((uint32_t)issued - (done_at >> (8 * st))) & 0xffu);
    };

    // Issue K tile kt of output tile t into stage kt % 4.  dtl_only: issue
    // only if both operands go direct to LDS (register-path tiles are issued
    // at the start of their output tile instead).
    auto issue = [&](const TileCoord& t, int kt, bool dtl_only) {
        const int st = kt & (NSTAGE - 1);
        char* As = smem + st * STAGE;
        char* Bs = As + TILE;
        const int64_t k0 = t.kbeg + (int64_t)kt * BK;
        const bool kfull = k0 + BK <= t.kend;
        const bool pd = kfull && p_al;
        const bool qd = kfull && q_al;
        if (dtl_only && !(pd && qd)) return;
        if (pd) {
            Tile<PL>::dtl(As, P, a.ldp, t.m0, a.M, k0);
            issued += DTL_OPS;
        } else {
            Tile<PL>::load_store(As, P, a.ldp, t.m0, a.M, k0, t.kend, p_al);
        }
        if (qd) {
            Tile<QL>::dtl(Bs, Q, a.ldq, t.n0, a.N, k0);
            issued += DTL_OPS;
        } else {
            Tile<QL>::load_store(Bs, Q, a.ldq, t.n0, a.N, k0, t.kend, q_al);
        }
        issued = __builtin_amdgcn_readfirstlane(issued);
        done_at = (done_at & ~(0xffu << (8 * st))) | (((uint32_t)issued & 0xffu) << (8 * st));
        loaded |= 1 << st;
    };

    TileCoord cur;
    if (!tile_at(a, 0, &cur)) return;
    constexpr int RD = TM * (PL == KMAJ ? 1 : 2) + TN * (QL == KMAJ ? 1 : 2);   // LDS reads per sub-step

    for (int64_t it = 0;; ++it) {
        TileCoord nxt;
        const bool more = tile_at(a, it + 1, &nxt);

        // K tiles of this output tile not prefetched yet (the first output
        // tile, or register-path tiles)
        for (int kt = 0; kt < NSTAGE && kt < cur.nk; ++kt)
            if (!((loaded >> kt) & 1)) issue(cur, kt, false);

        f32x16 acc[TM][TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

        bf16x8 fa[2][TM], fb[2][TN];
        if (cur.nk > 0) {
            wait_vm_at_most(ops_after(0));
            barrier_lds();
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[0][i] = Tile<PL>::frag(smem, wm * WR + 32 * i, 0, lane);
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[0][j] = Tile<QL>::frag(smem + TILE, wn * WC + 32 * j, 0, lane);
        }
        for (int kt = 0; kt < cur.nk; ++kt) {
            const int st = kt & (NSTAGE - 1);
            const int sn = (kt + 1) & (NSTAGE - 1);
            const char* As = smem + st * STAGE;
            // second sub-step's fragments, read under the first sub-step's MFMAs
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[1][i] = Tile<PL>::frag(As, wm * WR + 32 * i, 1, lane);
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[1][j] = Tile<QL>::frag(As + TILE, wn * WC + 32 * j, 1, lane);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0][i], fb[0][j], acc[i][j], 0, 0, 0);
            // one MFMA, then the reads, then the other 15: the first MFMA waits
            // only for reads issued a sub-step earlier
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, TM * TN - 1, 0);

            // K tile kt+1 has landed (this wave's loads; the barrier makes it
            // every wave's), and every wave is done reading K tile kt.
            wait_vm_at_most(kt + 1 < cur.nk ? ops_after(sn) : 64);
            barrier_lds();
            loaded &= ~(1 << st);
            if (kt + NSTAGE < cur.nk) issue(cur, kt + NSTAGE, false);
            else if (more && st < nxt.nk) issue(nxt, st, true);   // stage st is free for good

            // next K tile's first sub-step, read under this second sub-step's
            // MFMAs (after the last K tile the values read are not used)
            const char* An = smem + sn * STAGE;
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[0][i] = Tile<PL>::frag(An, wm * WR + 32 * i, 0, lane);
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[0][j] = Tile<QL>::frag(An + TILE, wn * WC + 32 * j, 0, lane);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1][i], fb[1][j], acc[i][j], 0, 0, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, TM * TN - 1, 0);
        }
        // stages the next output tile needs that this one never used (nk < 4)
        if (more)
            for (int kt = cur.nk; kt < NSTAGE && kt < nxt.nk; ++kt)
                if (!((loaded >> kt) & 1)) issue(nxt, kt, true);

        const int64_t row0 = cur.m0 + wm * WR;
        const int64_t col0 = cur.n0 + wn * WC;
        const bool interior = out_al && row0 + WR <= a.M && col0 + WC <= a.N;
        epilogue_block<EPI>(a, acc, row0, col0, lane, cur.split);
        if (interior) issued = __builtin_amdgcn_readfirstlane(issued + epi_ops);
        if (!more) break;
        cur = nxt;
    }
}

// Persistent grid: one workgroup per CU (256 on MI355X), fewer if there are
// fewer tiles; a multiple of 8 when possible so each XCD gets equal work.
constexpr int64_t kWideGrid = 256;

template <int PL, int QL, int EPI, int TAG>
hipError_t launch_w(const GemmArgs& a, hipStream_t s) {
    if (a.p_layout != PL || a.q_layout != QL || a.epi != EPI) return hipErrorInvalidValue;
    const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * (int64_t)a.splits;
    if (tiles <= 0) return hipSuccess;
    int64_t grid = tiles < kWideGrid ? tiles : kWideGrid;
    if (grid > 8 && (tiles & 7) == 0) grid &= ~int64_t(7);
    hipLaunchKernelGGL((gemm_wide_kernel<PL, QL, EPI, TAG>), dim3((unsigned)grid), dim3(NT), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_wide(const GemmArgs& a, hipStream_t s) {
    switch (a.tag) {
        case TAG_FWD_Z: return launch_w<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_Z>(a, s);
        case TAG_INFER_H: return launch_w<KMAJ, KMAJ, EPI_H, TAG_INFER_H>(a, s);
        case TAG_FWD_Y: return launch_w<KMAJ, KMAJ, EPI_STORE, TAG_FWD_Y>(a, s);
        case TAG_FWD_YP: return launch_w<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_YP>(a, s);
        case TAG_BWD_DZ: return launch_w<KMAJ, MNMAJ, EPI_DZ, TAG_BWD_DZ>(a, s);
        case TAG_BWD_DX: return launch_w<KMAJ, MNMAJ, EPI_STORE, TAG_BWD_DX>(a, s);
        case TAG_BWD_DA: return launch_w<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_BWD_DA>(a, s);
        case TAG_BWD_DB: return launch_w<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_BWD_DB>(a, s);
        case TAG_DENSE_FWD: return launch_w<KMAJ, KMAJ, EPI_STORE, TAG_DENSE_FWD>(a, s);
        case TAG_DENSE_DX: return launch_w<KMAJ, MNMAJ, EPI_STORE, TAG_DENSE_DX>(a, s);
        case TAG_DENSE_DW: return launch_w<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_DENSE_DW>(a, s);
        default: return hipErrorNotSupported;
    }
}

}  // namespace cola
