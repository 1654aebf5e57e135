// gemm_big.hip -- the 256 x 256 bf16 MFMA GEMM with one wave per SIMD:
// C[M][N] = sum_k P(m, k) Q(n, k), fp32 accumulation, the fused epilogues of
// epilogue.hpp.
//
// Design (CDNA4, wave64, one workgroup per CU):
//  * 256 threads = 4 waves in a 2 x 2 grid, one per SIMD; each wave owns a
//    128 x 128 block of C as 4 x 4 tiles of v_mfma_f32_32x32x16_bf16 (256
//    fp32 accumulators per lane, in the accumulation registers).  A 256 x 256
//    tile needs 1 KB of operands per unit of k: 32 bytes per clock per CU at
//    the MFMA peak.
//  * K advances in tiles of BK (32) through NSTAGE LDS stages (32 KB each):
//    NSTAGE - 1 K tiles are in flight while one is consumed, loaded straight
//    into LDS (global_load_lds_dwordx4: no staging registers, no LDS write
//    instructions), with per-lane offsets computed once per output tile and a
//    scalar base per K tile.
//  * Software pipeline inside each wave: the fragments of the next 16-deep
//    k step are read from LDS under the MFMAs of the current one; the loads
//    of the K tile NSTAGE - 1 ahead are issued one per MFMA; one barrier per
//    K tile, placed after the first MFMAs of the tile's last k step so that
//    the matrix pipe has work while the waves meet.  The hot loop has no
//    branches: the prefetching, draining and last K tiles are separate
//    instances of the same body, and a partial last K tile (K not a multiple
//    of BK) goes through guarded register loads after the loop.
//  * LDS layouts (as the other families).  k-contiguous operands:
//    [256 rows][BK k], 16-byte chunks XOR-swizzled by row, read with
//    ds_read_b128; m-contiguous operands (weight-gradient operands, the
//    weights of the backward products): [BK k][256 m], chunks swizzled by
//    4 (k & 3), read with the transposing ds_read_b64_tr_b16.  With gfx950's
//    64 LDS banks neither read conflicts.
//  * Ragged M / N edges: k-contiguous rows past the edge re-read the last row,
//    m-contiguous chunks past the edge re-read the last chunk; those values
//    reach only outputs that are not stored.  Operands must have 16-byte
//    aligned rows (the launcher falls back to the streaming family otherwise).
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
constexpr int NT = 256;
constexpr int WR = 128;          // rows of a wave's block
constexpr int WC = 128;          // columns of a wave's block
constexpr int TM = WR / 32;
constexpr int TN = WC / 32;

__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Buffer descriptor of a wave-uniform base address (raw buffer, no range
// check: every offset the kernel uses is in bounds by construction).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_of(const char* ubase) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(ubase), (short)0, 0x7fffffff, 0x00020000);
}
// 16 bytes per lane from base + voff (scalar descriptor, 32-bit per-lane
// offset: buffer_load_dwordx4 ... lds) to LDS bytes [lds + 16 lane, +16).
__device__ __forceinline__ void dtl16(__amdgpu_buffer_rsrc_t r, uint32_t voff, char* lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lptr_t)lds, 16, voff, 0, 0, 0);
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

template <int LAYOUT, int BK>
struct BTile;

// ---- k-contiguous operand: LDS [256 rows][BK k] ----
template <int BK>
struct BTile<KMAJ, BK> {
    static constexpr int CR = BK / 8;                 // 16-byte chunks per row
    static constexpr int RPI = 64 / CR;               // rows per 1 KB instruction
    static constexpr int BYTES = 256 * BK * 2;
    static constexpr int DPW = BYTES / 1024 / 4;      // direct-to-LDS instructions per wave
    static constexpr int FRAG_READS = 1;              // LDS reads per fragment
    static_assert(CR == 4 || CR == 8, "BK of 32 or 64");

    // chunk c of row r sits at chunk c ^ swz(r): the 16 rows a quarter-wave
    // reads cover all 64 banks once
    __device__ static __forceinline__ int swz(int row) { return (row / (16 / CR)) & (CR - 1); }
    __device__ static __forceinline__ int off(int row, int c) { return row * (2 * BK) + ((c ^ swz(row)) << 4); }

    // Per-lane byte offset of instruction j, relative to the K tile's first
    // element (row0, k0).  Rows past the edge re-read the last row.
    __device__ static __forceinline__ uint32_t voff(int j, int64_t ld, int64_t row0, int64_t rows) {
        const int lane = threadIdx.x & 63;
        const int blk = DPW * wave_id() + j;
        const int row = RPI * blk + lane / CR;
        const int lc = (lane % CR) ^ swz(row);
        const int64_t lrow = row0 + row < rows ? row : rows - 1 - row0;
        return 2u * ((uint32_t)lrow * (uint32_t)ld + 8u * (uint32_t)lc);
    }
    __device__ static __forceinline__ const char* gbase(const uint16_t* base, int64_t ld, int64_t row0, int64_t k0) {
        return reinterpret_cast<const char*>(base + row0 * ld + k0);
    }

    // Guarded register path (partial K tile): zeros past kend.
    __device__ static __forceinline__ void load_store(char* lds, const uint16_t* base, int64_t ld, int64_t row0,
                                                      int64_t rows, int64_t k0, int64_t kend) {
#pragma unroll
        for (int i = 0; i < 256 * CR / NT; ++i) {
            const int id = threadIdx.x + NT * i;
            const int64_t row = row0 + id / CR;
            const int64_t k = k0 + 8 * (id % CR);
            const int64_t valid = row < rows ? kend - k : 0;
            const uint4 v = load8_guarded(base + (row < rows ? row : 0) * ld + (valid > 0 ? k : 0),
                                          (int)(valid < 0 ? 0 : (valid > 8 ? 8 : valid)));
            *reinterpret_cast<uint4*>(lds + off(id / CR, id % CR)) = v;
        }
    }

    // 32 rows (row0 ..) x 16 k (16 s ..) fragment
    __device__ static __forceinline__ bf16x8 frag(const char* lds, int row0, int s, int lane) {
        return *reinterpret_cast<const bf16x8*>(lds + off(row0 + (lane & 31), 2 * s + (lane >> 5)));
    }
};

// ---- m-contiguous operand: LDS [BK k][256 m] (512-byte rows) ----
template <int BK>
struct BTile<MNMAJ, BK> {
    static constexpr int BYTES = BK * 256 * 2;
    static constexpr int DPW = BYTES / 1024 / 4;
    static constexpr int FRAG_READS = 2;

    __device__ static __forceinline__ int off(int k, int c) { return k * 512 + ((c ^ ((k & 3) << 2)) << 4); }

    // Instruction j fills k rows 2 blk, 2 blk + 1; chunks that start past the
    // last column re-read the last chunk.
    __device__ static __forceinline__ uint32_t voff(int j, int64_t ld, int64_t m0, int64_t rows) {
        const int lane = threadIdx.x & 63;
        const int64_t mlast = ((rows - 1) >> 3) << 3;
        const int blk = DPW * wave_id() + j;
        const int k = 2 * blk + (lane >> 5);
        const int lc = (lane & 31) ^ ((k & 3) << 2);
        const int64_t lm = m0 + 8 * lc <= mlast ? 8 * lc : mlast - m0;
        return 2u * ((uint32_t)k * (uint32_t)ld + (uint32_t)lm);
    }
    __device__ static __forceinline__ const char* gbase(const uint16_t* base, int64_t ld, int64_t m0, int64_t k0) {
        return reinterpret_cast<const char*>(base + k0 * ld + m0);
    }

    __device__ static __forceinline__ void load_store(char* lds, const uint16_t* base, int64_t ld, int64_t m0,
                                                      int64_t rows, int64_t k0, int64_t kend) {
#pragma unroll
        for (int i = 0; i < BK * 32 / NT; ++i) {
            const int id = threadIdx.x + NT * i;
            const int64_t k = k0 + id / 32;
            const int64_t m = m0 + 8 * (id % 32);
            const int64_t valid = k < kend ? rows - m : 0;
            const uint4 v = load8_guarded(base + (k < kend ? k : 0) * ld + (valid > 0 ? m : 0),
                                          (int)(valid < 0 ? 0 : (valid > 8 ? 8 : valid)));
            *reinterpret_cast<uint4*>(lds + off(id / 32, id % 32)) = v;
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

// Scheduling hints: sched_group_barrier masks (MFMA, all VMEM, DS read).
constexpr int SG_MFMA = 0x008;
constexpr int SG_VMEM = 0x010;
constexpr int SG_DSR = 0x100;

// Scheduling pattern of M MFMAs with R LDS reads and V vector-memory
// loads spread over them: after MFMA n come the reads and loads whose even
// share falls there (floor((n+1) R / M) - floor(n R / M) of each), so that no
// gap between two MFMAs holds more than a few instructions -- with one wave
// per SIMD, a gap longer than an MFMA's 32 cycles idles the matrix pipe.
template <int M, int R, int V, int N = 0>
__device__ __forceinline__ void sched_spread() {
    if constexpr (N < M) {
        constexpr int r = (N + 1) * R / M - N * R / M;
        constexpr int v = (N + 1) * V / M - N * V / M;
        __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
        if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(SG_DSR, r, 0);
        if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(SG_VMEM, v, 0);
        sched_spread<M, R, V, N + 1>();
    }
}

__device__ __forceinline__ void barrier_lds() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
template <int N>
__device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
template <class T, T V>
using ic = std::integral_constant<T, V>;

// f(ic<int, 0>), ..., f(ic<int, N - 1>): a loop whose index is a constant.
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (I < N) {
        f(ic<int, I>{});
        static_for<N, I + 1>(f);
    }
}

// Coordinates of one output tile (and K range) of a persistent workgroup.
struct BigTile {
    int64_t m0, n0, kbeg, kend;
    int split, nkf;               // nkf: whole K tiles
    bool tail;                    // a partial K tile follows them
};

// Output tile i (0, 1, ...) of this workgroup; false past the last one.  With
// a grid and a tile count that are multiples of 8, XCD x (blockIdx % 8) owns
// the contiguous tile range [x T/8, (x+1) T/8) and sweeps it with its
// workgroups together (n fastest), so tiles that share operand rows run at
// the same time on the same L2.
template <int BK>
__device__ __forceinline__ bool big_tile_at(const GemmArgs& a, int64_t i, BigTile* t) {
    const int64_t tiles_n = (a.N + BN - 1) / BN;
    const int64_t tiles_m = (a.M + BM - 1) / BM;
    const int64_t per_split = tiles_m * tiles_n;
    const int64_t total = per_split * a.splits;
    const int64_t G = gridDim.x;
    int64_t idx;
    if ((G & 7) == 0 && (total & 7) == 0) {
        const int64_t j = (int64_t)(blockIdx.x >> 3) + i * (G >> 3);
        if (j >= (total >> 3)) return false;
        idx = (int64_t)(blockIdx.x & 7) * (total >> 3) + j;
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
    t->nkf = (int)((t->kend - t->kbeg) / BK);
    t->tail = t->kbeg + (int64_t)t->nkf * BK < t->kend;
    return true;
}

// LDS rings: the P operand (the activations in every product of the layer)
// runs NP = 3 slots, two K tiles ahead; the Q operand NQ = 2 slots, one K
// tile ahead.  Five 32 KB slots fill the 160 KB of LDS.
constexpr int NP = 3;
constexpr int NQ = 2;

template <int BK, int PL, int QL, int EPI, int TAG>
__global__ __launch_bounds__(NT, 1) void gemm_big_kernel(GemmArgs a) {
    using TP = BTile<PL, BK>;
    using TQ = BTile<QL, BK>;
    constexpr int NSUB = BK / 16;                          // 16-deep k steps per K tile
    constexpr int RD = TM * TP::FRAG_READS + TN * TQ::FRAG_READS;   // LDS reads per k step
    constexpr int NMFMA = TM * TN;                         // MFMAs per k step
    constexpr int POPS = TP::DPW;                          // direct-to-LDS loads per wave, P tile
    constexpr int QOPS = TQ::DPW;
    static_assert(NSUB % 2 == 0, "fragment double buffer alternates per k step");
    constexpr int LPS = (QOPS + POPS + NSUB - 2) / (NSUB - 1);       // loads per k step
    static_assert(LPS <= NMFMA, "at most one direct-to-LDS load per MFMA");
    __shared__ __attribute__((aligned(1024))) char smem[NP * TP::BYTES + NQ * TQ::BYTES];
    char* const pring = smem;
    char* const qring = smem + NP * TP::BYTES;

    const uint16_t* P = reinterpret_cast<const uint16_t*>(a.p);
    const uint16_t* Q = reinterpret_cast<const uint16_t*>(a.q);
    const int wave = wave_id();
    const int lane = threadIdx.x & 63;
    const int wm = wave >> 1;
    const int wn = wave & 1;

    // Per-lane offsets of this wave's loads for a tile (they depend on the
    // tile only at the M / N edges).
    struct Offs {
        uint32_t p[POPS], q[QOPS];
    };
    auto offs_for = [&](const BigTile& t, Offs& o) {
#pragma unroll
        for (int j = 0; j < POPS; ++j) o.p[j] = TP::voff(j, a.ldp, t.m0, a.M);
#pragma unroll
        for (int j = 0; j < QOPS; ++j) o.q[j] = TQ::voff(j, a.ldq, t.n0, a.N);
    };
    // K tile kt of a tile whose first K tile has global number g0 sits in P
    // slot (g0 + kt) % NP and Q slot (g0 + kt) % NQ.
    auto pslot = [&](int g) -> char* { return pring + (g % NP) * TP::BYTES; };
    auto qslot = [&](int g) -> char* { return qring + (g % NQ) * TQ::BYTES; };

    // Direct-to-LDS load r of the P (Q) part of whole K tile kt of tile t into
    // the slot of global K tile g.
    auto issue_p1 = [&](const BigTile& t, const Offs& o, int r, int kt, int g) {
        const int64_t k0 = t.kbeg + (int64_t)kt * BK;
        dtl16(rsrc_of(TP::gbase(P, a.ldp, t.m0, k0)), o.p[r], pslot(g) + 1024 * (POPS * wave + r));
    };
    auto issue_q1 = [&](const BigTile& t, const Offs& o, int r, int kt, int g) {
        const int64_t k0 = t.kbeg + (int64_t)kt * BK;
        dtl16(rsrc_of(TQ::gbase(Q, a.ldq, t.n0, k0)), o.q[r], qslot(g) + 1024 * (QOPS * wave + r));
    };

    auto issue_p = [&](const BigTile& t, const Offs& o, int kt, int g) {
#pragma unroll
        for (int r = 0; r < POPS; ++r) issue_p1(t, o, r, kt, g);
    };
    auto issue_q = [&](const BigTile& t, const Offs& o, int kt, int g) {
#pragma unroll
        for (int r = 0; r < QOPS; ++r) issue_q1(t, o, r, kt, g);
    };

    f32x16 acc[TM][TN];
    bf16x8 fa[2][TM], fb[2][TN];
    auto read_frags = [&](const char* ps, const char* qs, int s, bf16x8 (&ra)[TM], bf16x8 (&rb)[TN]) {
#pragma unroll
        for (int i = 0; i < TM; ++i) ra[i] = TP::frag(ps, wm * WR + 32 * i, s, lane);
#pragma unroll
        for (int j = 0; j < TN; ++j) rb[j] = TQ::frag(qs, wn * WC + 32 * j, s, lane);
    };
    auto mfmas = [&](const bf16x8 (&ra)[TM], const bf16x8 (&rb)[TN]) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ra[i], rb[j], acc[i][j], 0, 0, 0);
    };

    BigTile cur, nxt;
    if (!big_tile_at<BK>(a, 0, &cur)) return;
    Offs oc, on;
    offs_for(cur, oc);
    int g0 = 0;              // global number of cur's first K tile
    bool ready = false;      // cur's P(0), Q(0), P(1) were prefetched, in that order
    for (int64_t it = 0;; ++it) {
        const bool more = big_tile_at<BK>(a, it + 1, &nxt);
        if (more) offs_for(nxt, on);
        const int nkf = cur.nkf;
        // the last two K tiles of cur prefetch P(0), Q(0), P(1) of the next tile
        const bool pf_next = more && nkf >= 2 && nxt.nkf >= 2;

#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;
        if (nkf > 0) {
            if (!ready) {
                // nothing of cur in flight: wait for every earlier load, meet
                // (every wave is done with the slots), then issue P(0), Q(0), P(1)
                wait_vm<0>();
                barrier_lds();
                issue_p(cur, oc, 0, g0);
                issue_q(cur, oc, 0, g0);
                if (nkf > 1) issue_p(cur, oc, 1, g0 + 1);
            }
            // P(0) and Q(0) are in once at most P(1)'s loads are pending (loads
            // complete in order; the previous epilogue's stores only lengthen
            // this wait)
            if (nkf > 1) wait_vm<POPS>();
            else wait_vm<0>();
            barrier_lds();
            read_frags(pslot(g0), qslot(g0), 0, fa[0], fb[0]);
        }

        // One whole K tile kt of cur, whose first k step's fragments are in
        // fa[0], fb[0].  Under the MFMAs of its first k step it issues Q of
        // K tile kt + 1 and P of K tile kt + 2 (their slots held K tile kt - 1,
        // which every wave finished reading before the barrier of K tile kt),
        // or the next tile's first K tiles in their place.  MODE 0: both from
        // cur; 1: Q from cur, P = the next tile's P(0); 2: the last K tile: Q =
        // the next tile's Q(0), P = its P(1).  Q, P: issue them (uniform).
        // NEXT: after the first MFMAs of the last k step, wait for K tile
        // kt + 1, meet at the barrier, and read its first k step's fragments
        // under the remaining MFMAs.
        // load r (of QOPS + POPS) of body kt: Q of K tile kt + 1, then P of kt + 2
        auto issue_qp = [&](int r, int kt) {
            if (r < QOPS) issue_q1(cur, oc, r, kt + 1, g0 + kt + 1);
            else issue_p1(cur, oc, r - QOPS, kt + 2, g0 + kt + 2);
        };
        auto body = [&](auto mode, auto next, int kt, bool do_q, bool do_p) {
            constexpr int MODE = decltype(mode)::value;
            const char* ps = pslot(g0 + kt);
            const char* qs = qslot(g0 + kt);
            static_for<NSUB - 1>([&](auto sc) {
                constexpr int s = decltype(sc)::value;
                read_frags(ps, qs, s + 1, fa[(s + 1) & 1], fb[(s + 1) & 1]);
                // the loads of the steady K tiles go out over the first NSUB - 1
                // k steps (a burst would outrun the load path, about half a
                // cache line per clock, and stall this wave's MFMA issue)
                constexpr int l0 = s * LPS, l1 = (s + 1) * LPS < QOPS + POPS ? (s + 1) * LPS : QOPS + POPS;
                if constexpr (MODE == 0) {
#pragma unroll
                    for (int r = l0; r < l1; ++r) issue_qp(r, kt);
                }
                mfmas(fa[s & 1], fb[s & 1]);
                // reads (and loads) spread over the MFMAs
                sched_spread<NMFMA, RD, MODE == 0 ? l1 - l0 : 0>();
                __builtin_amdgcn_sched_barrier(0);
                if constexpr (s == 0 && MODE != 0) {
                    // drain and hand-over K tiles: loads at once, if any
                    if (do_q) {
                        if constexpr (MODE == 1) issue_q(cur, oc, kt + 1, g0 + kt + 1);
                        else issue_q(nxt, on, 0, g0 + nkf);
                    }
                    if (do_p) {
                        if constexpr (MODE == 1) issue_p(nxt, on, 0, g0 + nkf);
                        else issue_p(nxt, on, 1, g0 + nkf + 1);
                    }
                }
            });
            constexpr int sl = NSUB - 1;
            if constexpr (decltype(next)::value) {
                // two MFMAs keep the matrix pipe busy through the wait and barrier
#pragma unroll
                for (int q = 0; q < 2; ++q)
                    acc[q / TN][q % TN] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        fa[sl & 1][q / TN], fb[sl & 1][q % TN], acc[q / TN][q % TN], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
                // K tile kt + 1 is in once at most the P loads issued after its
                // Q loads are pending
                if (do_p) wait_vm<POPS>();
                else wait_vm<0>();
                barrier_lds();
                __builtin_amdgcn_sched_barrier(0);
                read_frags(pslot(g0 + kt + 1), qslot(g0 + kt + 1), 0, fa[0], fb[0]);
#pragma unroll
                for (int q = 2; q < NMFMA; ++q)
                    acc[q / TN][q % TN] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        fa[sl & 1][q / TN], fb[sl & 1][q % TN], acc[q / TN][q % TN], 0, 0, 0);
                sched_spread<NMFMA - 2, RD, 0>();
                __builtin_amdgcn_sched_barrier(0);
            } else {
                mfmas(fa[sl & 1], fb[sl & 1]);
            }
        };
        int kt = 0;
        for (; kt + 2 < nkf; ++kt) body(ic<int, 0>{}, ic<bool, true>{}, kt, true, true);
        if (kt + 1 < nkf) {
            body(ic<int, 1>{}, ic<bool, true>{}, kt, true, pf_next);
            ++kt;
        }
        if (kt < nkf) body(ic<int, 2>{}, ic<bool, false>{}, kt, pf_next, pf_next);

        // partial last K tile: guarded register loads (zeros past kend) into
        // the slots no prefetch uses, once every wave is done with them
        if (cur.tail) {
            char* ps = pslot(g0 + nkf + NP - 1);
            char* qs = qslot(g0 + nkf + NQ - 1);
            const int64_t k0 = cur.kbeg + (int64_t)nkf * BK;
            barrier_lds();
            TP::load_store(ps, P, a.ldp, cur.m0, a.M, k0, cur.kend);
            TQ::load_store(qs, Q, a.ldq, cur.n0, a.N, k0, cur.kend);
            barrier_lds();
#pragma unroll
            for (int s = 0; s < NSUB; ++s) {
                read_frags(ps, qs, s, fa[0], fb[0]);
                mfmas(fa[0], fb[0]);
            }
        }
        epilogue_block<EPI>(a, acc, cur.m0 + wm * WR, cur.n0 + wn * WC, lane, cur.split);
        if (!more) break;
        g0 += nkf;
        ready = pf_next;
        cur = nxt;
        oc = on;
    }
}

// K tile 64: every direct-to-LDS load of a k-contiguous operand reads whole
// 128-byte lines (the load path's throughput is set by the lines it touches:
// 64-byte rows halve it, measured).
constexpr int kBigBK = 64;
// Persistent grid: one workgroup per CU (256 on MI355X), fewer if there are
// fewer tiles; a multiple of 8 when possible so each XCD gets equal work.
constexpr int64_t kBigGrid = 256;

template <int PL, int QL, int EPI, int TAG>
hipError_t launch_b(const GemmArgs& a, hipStream_t s) {
    if (a.p_layout != PL || a.q_layout != QL || a.epi != EPI) return hipErrorInvalidValue;
    const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * (int64_t)a.splits;
    if (tiles <= 0) return hipSuccess;
    int64_t grid = tiles < kBigGrid ? tiles : kBigGrid;
    if (grid > 8 && (tiles & 7) == 0) grid &= ~int64_t(7);
    hipLaunchKernelGGL((gemm_big_kernel<kBigBK, PL, QL, EPI, TAG>), dim3((unsigned)grid), dim3(NT), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_big(const GemmArgs& a, hipStream_t s) {
    switch (a.tag) {
        case TAG_FWD_Z: return launch_b<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_Z>(a, s);
        case TAG_INFER_H: return launch_b<KMAJ, KMAJ, EPI_H, TAG_INFER_H>(a, s);
        case TAG_FWD_Y: return launch_b<KMAJ, KMAJ, EPI_STORE, TAG_FWD_Y>(a, s);
        case TAG_FWD_YP: return launch_b<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_YP>(a, s);
        case TAG_BWD_DZ: return launch_b<KMAJ, MNMAJ, EPI_DZ, TAG_BWD_DZ>(a, s);
        case TAG_BWD_DX: return launch_b<KMAJ, MNMAJ, EPI_STORE, TAG_BWD_DX>(a, s);
        case TAG_BWD_DA: return launch_b<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_BWD_DA>(a, s);
        case TAG_BWD_DB: return launch_b<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_BWD_DB>(a, s);
        case TAG_DENSE_FWD: return launch_b<KMAJ, KMAJ, EPI_STORE, TAG_DENSE_FWD>(a, s);
        case TAG_DENSE_DX: return launch_b<KMAJ, MNMAJ, EPI_STORE, TAG_DENSE_DX>(a, s);
        case TAG_DENSE_DW: return launch_b<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_DENSE_DW>(a, s);
        default: return hipErrorNotSupported;
    }
}

}  // namespace cola
