// gemm_wide.hip -- the 256 x 256 bf16 MFMA GEMM used when both output
// dimensions exceed 128:  C[M][N] = sum_k P(m, k) Q(n, k), fp32 accumulation,
// the fused epilogues of epilogue.hpp.
//
// Design (CDNA4, wave64, one workgroup per CU):
//  * 256 threads = 4 waves in a 2 x 2 grid, each wave a 128 x 128 block of C
//    as 4 x 4 tiles of v_mfma_f32_32x32x16_bf16 (256 fp32 accumulators per
//    lane).  The large wave tile halves the LDS bytes read per MFMA compared
//    with 128 x 64 wave tiles.
//  * K advances in tiles of 64 through two LDS stages (2 x 64 KB).  Interior
//    tiles are copied global -> LDS by the direct-to-LDS loads
//    (global_load_lds_dwordx4): no registers, no LDS write instructions; the
//    next tile's loads are in flight while the current tile's MFMAs run.
//  * Operands with contiguous k (KMAJ) sit in LDS as [row][k] with 128-byte
//    rows, 16-byte chunks XOR-swizzled by (row ^ row >> 3) & 7; fragments are
//    read with ds_read_b128.  Operands with contiguous m (MNMAJ: the operands
//    of the token-reduction weight gradients and the weights in the backward
//    products) sit in LDS as they are in memory, [k][m] with 512-byte rows,
//    chunks XOR-swizzled by 2 (k & 3); fragments are read with the gfx950
//    transposing LDS load ds_read_b64_tr_b16 (two per fragment), which hands
//    each lane four consecutive k of one m.
//  * Tiles on a ragged edge (or at the K tail, or with unaligned pitches) are
//    loaded through registers with per-chunk guards and written to the same
//    LDS layout at once (no staging registers live across the MFMA loop);
//    for k-contiguous operands rows past the edge simply re-read the last
//    row (those outputs are never stored).
#include "internal.hpp"
#include "device_math.hpp"
#include "epilogue.hpp"

namespace cola {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

constexpr int BM = 256;
constexpr int BN = 256;
constexpr int BK = 64;
constexpr int NT = 256;
constexpr int TILE = 256 * 128;        // bytes of one operand tile (either layout)
constexpr int STAGE = 2 * TILE;

__device__ __forceinline__ bool aligned16(const void* p, int64_t ld) {
    return ((reinterpret_cast<uintptr_t>(p) & 15u) == 0) && ((ld & 7) == 0);
}

typedef const __attribute__((address_space(1))) void* gptr_t;
typedef __attribute__((address_space(3))) void* lptr_t;
typedef __attribute__((address_space(3))) s16x4* lptr4_t;

__device__ __forceinline__ void dtl16(const void* g, char* lds) {
    __builtin_amdgcn_global_load_lds((gptr_t)g, (lptr_t)lds, 16, 0, 0);
}

// Eight bf16 from global memory, elements at or past `valid` read as zero.
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

// ---- k-contiguous operand: LDS [256 rows][64 k] ----
template <>
struct Tile<KMAJ> {
    uint4 v[8];

    __device__ static __forceinline__ int off(int row, int c) {
        return row * 128 + ((c ^ ((row ^ (row >> 3)) & 7)) << 4);
    }

    // Wave w, instruction j fills LDS bytes [1024 (8w + j), +1024): rows
    // 8 (8w + j) .. +8, lane l -> row + l/8, physical chunk l % 8.
    __device__ static __forceinline__ void dtl(char* lds, const uint16_t* base, int64_t ld, int64_t row0,
                                               int64_t rows, int64_t k0) {
        const int wave = threadIdx.x >> 6;
        const int lane = threadIdx.x & 63;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int blk = 8 * wave + j;
            const int row = 8 * blk + (lane >> 3);
            const int lc = (lane & 7) ^ ((row ^ (row >> 3)) & 7);
            int64_t grow = row0 + row;
            if (grow >= rows) grow = rows - 1;
            dtl16(base + grow * ld + k0 + 8 * lc, lds + 1024 * blk);
        }
    }

    __device__ __forceinline__ void load(const uint16_t* base, int64_t ld, int64_t row0, int64_t rows,
                                         int64_t k0, int64_t kend, bool aligned) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int id = threadIdx.x + NT * i;
            const int64_t row = row0 + (id >> 3);
            const int64_t k = k0 + 8 * (id & 7);
            if (row < rows && k + 8 <= kend && aligned) {
                v[i] = *reinterpret_cast<const uint4*>(base + row * ld + k);
            } else {
                const int64_t valid = row < rows ? kend - k : 0;
                v[i] = load8_guarded(base + (row < rows ? row : 0) * ld + k,
                                     (int)(valid < 0 ? 0 : (valid > 8 ? 8 : valid)));
            }
        }
    }

    __device__ __forceinline__ void store(char* lds) const {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int id = threadIdx.x + NT * i;
            *reinterpret_cast<uint4*>(lds + off(id >> 3, id & 7)) = v[i];
        }
    }

    // 32 rows (row0 ..) x 16 k (kbase ..) MFMA operand fragment
    __device__ static __forceinline__ bf16x8 frag(const char* lds, int row0, int kbase, int lane) {
        return *reinterpret_cast<const bf16x8*>(lds + off(row0 + (lane & 31), (kbase >> 3) + (lane >> 5)));
    }
};

// ---- m-contiguous operand: LDS [64 k][256 m] ----
template <>
struct Tile<MNMAJ> {
    uint4 v[8];

    __device__ static __forceinline__ int off(int k, int c) {
        return k * 512 + ((c ^ ((k & 3) << 1)) << 4);
    }

    // Wave w, instruction j fills LDS bytes [1024 (8w + j), +1024): k rows
    // 2 (8w + j) and 2 (8w + j) + 1, lane l -> k row + l/32, physical chunk
    // l % 32.  Chunks that start past the last column re-read the last chunk
    // (their outputs are never stored); the chunk holding the last column may
    // run into the row's pitch padding, which the ABI lets the library read.
    __device__ static __forceinline__ void dtl(char* lds, const uint16_t* base, int64_t ld, int64_t m0,
                                               int64_t rows, int64_t k0) {
        const int wave = threadIdx.x >> 6;
        const int lane = threadIdx.x & 63;
        const int64_t mlast = ((rows - 1) >> 3) << 3;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int blk = 8 * wave + j;
            const int k = 2 * blk + (lane >> 5);
            const int lc = (lane & 31) ^ ((k & 3) << 1);
            int64_t m = m0 + 8 * lc;
            if (m > mlast) m = mlast;
            dtl16(base + (k0 + k) * ld + m, lds + 1024 * blk);
        }
    }

    __device__ __forceinline__ void load(const uint16_t* base, int64_t ld, int64_t m0, int64_t rows,
                                         int64_t k0, int64_t kend, bool aligned) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int id = threadIdx.x + NT * i;
            const int64_t k = k0 + (id >> 5);
            const int64_t m = m0 + 8 * (id & 31);
            if (k < kend && m + 8 <= rows && aligned) {
                v[i] = *reinterpret_cast<const uint4*>(base + k * ld + m);
            } else {
                const int64_t valid = k < kend ? rows - m : 0;
                v[i] = load8_guarded(base + (k < kend ? k : 0) * ld + (valid > 0 ? m : 0),
                                     (int)(valid < 0 ? 0 : (valid > 8 ? 8 : valid)));
            }
        }
    }

    __device__ __forceinline__ void store(char* lds) const {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int id = threadIdx.x + NT * i;
            *reinterpret_cast<uint4*>(lds + off(id >> 5, id & 31)) = v[i];
        }
    }

    // 32 m (m0 ..) x 16 k (kbase ..) MFMA operand fragment.  Each transposing
    // read serves 16 lanes: lanes 4q..4q+3 point at k row q of a 4 x 16 block
    // (four consecutive m each), and lane i of the group receives the four k
    // values of column m0 + i.  Two reads give the lane's eight k.
    __device__ static __forceinline__ bf16x8 frag(const char* lds, int m0, int kbase, int lane) {
        const int g = lane >> 4;
        const int i = lane & 15;
        const int m = m0 + 16 * (g & 1) + 4 * (i & 3);
        const int k = kbase + 8 * (g >> 1) + (i >> 2);
        const int byte = (m & 7) * 2;
        const int c = m >> 3;
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lptr4_t)(lds + off(k, c) + byte));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lptr4_t)(lds + off(k + 4, c) + byte));
        const s16x8 s8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        return __builtin_bit_cast(bf16x8, s8);
    }
};

// LDS barrier: this wave's LDS writes are complete, then all waves meet.
// (Plain s_barrier: no memory fence, so global stores stay in flight.)
__device__ __forceinline__ void barrier_lds() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
// Wait until at most N vector-memory operations of this wave are outstanding
// (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Vector-memory operations one thread issues in the epilogue of an interior
// tile: 8 half slabs x 4 passes x (stores, plus loads of Z for EPI_DZ).
template <int EPI>
constexpr int epilogue_vm_ops(bool aux) {
    return EPI == EPI_STORE ? 32 : EPI == EPI_STORE_F32 ? 64 : EPI == EPI_Z_H ? (aux ? 64 : 32) : 0;
}

struct TileCoord {
    int64_t m0, n0, kbeg, kend;
    int split, nk;
};

// The persistent grid walks the output tiles.  With a grid and a tile count
// that are multiples of 8, XCD x (blockIdx % 8) owns the contiguous tile range
// [x T/8, (x+1) T/8), which its workgroups sweep together, so tiles that
// share operand rows are computed at the same time on the same L2.
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
    // the epilogue stages through the second LDS stage only
    static_assert(4 * 16 * (BN / 2 + 4) * 4 <= STAGE, "epilogue staging does not fit");
    __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

    const uint16_t* P = reinterpret_cast<const uint16_t*>(a.p);
    const uint16_t* Q = reinterpret_cast<const uint16_t*>(a.q);
    const bool p_al = aligned16(a.p, a.ldp);
    const bool q_al = aligned16(a.q, a.ldq);
    const int64_t out_vec = (EPI == EPI_STORE_F32) ? 3 : 7;   // pitch granule of a 16-byte store
    const bool out_al = ((reinterpret_cast<uintptr_t>(a.c) & 15u) == 0) && ((a.ldc & out_vec) == 0) &&
                        (!a.aux || (((reinterpret_cast<uintptr_t>(a.aux) & 15u) == 0) && ((a.ldaux & 7) == 0)));
    constexpr int EPI_OPS = epilogue_vm_ops<EPI>(true);

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int wm = wave >> 1;
    const int wn = wave & 1;

    // Issue the loads of one K tile into an LDS stage.  Interior tiles go
    // straight to LDS and stay in flight; edge tiles (rare) are loaded into
    // registers and written to LDS right away, so no staging registers stay
    // live across the MFMA loop.
    // `part` selects what to issue: 1 = direct-to-LDS loads only, 2 = the
    // register-path loads only, 3 = both.
    auto issue = [&](const TileCoord& t, int stage, int64_t k0, int part) {
        char* As = smem + stage * STAGE;
        char* Bs = As + TILE;
        const bool kfull = k0 + BK <= t.kend;
        if (kfull && p_al) {
            if (part & 1) Tile<PL>::dtl(As, P, a.ldp, t.m0, a.M, k0);
        } else if (part & 2) {
            Tile<PL> r;
            r.load(P, a.ldp, t.m0, a.M, k0, t.kend, p_al);
            r.store(As);
        }
        if (kfull && q_al) {
            if (part & 1) Tile<QL>::dtl(Bs, Q, a.ldq, t.n0, a.N, k0);
        } else if (part & 2) {
            Tile<QL> r;
            r.load(Q, a.ldq, t.n0, a.N, k0, t.kend, q_al);
            r.store(Bs);
        }
    };

    TileCoord cur;
    if (!tile_at(a, 0, &cur)) return;
    if (cur.nk > 0) issue(cur, 0, cur.kbeg, 3);
    bool drained = true;        // were the previous epilogue's memory operations counted exactly?

    for (int64_t it = 0;; ++it) {
        f32x16 acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

        for (int kt = 0; kt < cur.nk; ++kt) {
            // this stage's direct-to-LDS loads are the oldest outstanding
            // operations; the previous tile's epilogue stores may stay in flight
            if (kt == 0 && !drained) wait_vm<(EPI_OPS > 63 ? 63 : EPI_OPS)>();
            else wait_vm<0>();
            barrier_lds();
            if (kt + 1 < cur.nk) issue(cur, (kt + 1) & 1, cur.kbeg + (int64_t)(kt + 1) * BK, 3);
            const char* As = smem + (kt & 1) * STAGE;
            const char* Bs = As + TILE;
            bf16x8 fa[2][4], fb[2][4];
#pragma unroll
            for (int i = 0; i < 4; ++i) fa[0][i] = Tile<PL>::frag(As, wm * 128 + 32 * i, 0, lane);
#pragma unroll
            for (int j = 0; j < 4; ++j) fb[0][j] = Tile<QL>::frag(Bs, wn * 128 + 32 * j, 0, lane);
#pragma unroll
            for (int s = 0; s < BK / 16; ++s) {
                const int c = s & 1;
                if (s + 1 < BK / 16) {        // next sub-step's fragments, read under this one's MFMAs
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        fa[c ^ 1][i] = Tile<PL>::frag(As, wm * 128 + 32 * i, 16 * (s + 1), lane);
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        fb[c ^ 1][j] = Tile<QL>::frag(Bs, wn * 128 + 32 * j, 16 * (s + 1), lane);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[c][i], fb[c][j], acc[i][j],
                                                                            0, 0, 0);
            }
            // Pin the order: first sub-step's reads, then for each sub-step the
            // next sub-step's reads ahead of its 16 MFMAs.
            constexpr int RD = 4 * (PL == KMAJ ? 1 : 2) + 4 * (QL == KMAJ ? 1 : 2);
            __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
#pragma unroll
            for (int s = 0; s < BK / 16 - 1; ++s) {
                __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);
        }

        // Every wave is done with both stages: start the next tile's first K
        // tile (stage 0) before this tile's epilogue, which stages through
        // stage 1 and whose stores then drain under the next tile's MFMAs.
        TileCoord nxt;
        const bool more = tile_at(a, it + 1, &nxt);
        wait_vm<0>();
        barrier_lds();
        if (more && nxt.nk > 0) issue(nxt, 0, nxt.kbeg, 1);

        const bool interior = out_al && cur.m0 + BM <= a.M && cur.n0 + BN <= a.N &&
                              (EPI != EPI_DZ) && (EPI != EPI_Z_H || a.aux);
        float* stg = reinterpret_cast<float*>(smem + STAGE) + wave * 16 * (BN / 2 + 4);
        epi_slab<0, BM, BN, EPI>(a, acc, stg, cur.m0, cur.n0, wm, wn, lane, cur.split);
        epi_slab<1, BM, BN, EPI>(a, acc, stg, cur.m0, cur.n0, wm, wn, lane, cur.split);
        epi_slab<2, BM, BN, EPI>(a, acc, stg, cur.m0, cur.n0, wm, wn, lane, cur.split);
        epi_slab<3, BM, BN, EPI>(a, acc, stg, cur.m0, cur.n0, wm, wn, lane, cur.split);
        if (!more) break;
        drained = !interior;
        cur = nxt;
        if (cur.nk > 0) issue(cur, 0, cur.kbeg, 2);   // edge-tile loads, after the epilogue
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
        case TAG_FWD_Y: return launch_w<KMAJ, KMAJ, EPI_STORE, TAG_FWD_Y>(a, s);
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
