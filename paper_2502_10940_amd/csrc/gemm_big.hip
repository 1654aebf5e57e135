// gemm_big.hip -- the 256 x 256 bf16 MFMA GEMM with one wave per SIMD:
// C[M][N] = sum_k P(m, k) Q(n, k), fp32 accumulation, the fused epilogues of
// epilogue.hpp.  An alternative to the ping-pong family (gemm_pp.hip), kept
// for comparisons (COLA_GEMM_FAMILY=big).
//
// Design (CDNA4, wave64, one persistent workgroup per CU):
//  * 256 threads = 4 waves in a 2 x 2 grid, one per SIMD; each wave owns a
//    128 x 128 block of C as 4 x 4 tiles of v_mfma_f32_32x32x16_bf16 (256
//    fp32 accumulators per lane, in the accumulation registers).  A 256 x 256
//    tile needs 1 KB of operands per unit of k: 32 bytes per clock per CU at
//    the MFMA peak.
//  * K tiles are 64 deep, so every load row is a whole 128-byte line (the
//    load path's throughput is set by the lines it touches).  LDS holds three
//    P slots (two K tiles ahead) and two Q slots (one ahead), 160 KB; loads go
//    straight into LDS (buffer_load ... lds) with per-lane offsets formed once
//    per output tile.
//  * Software pipeline inside each wave: the fragments of the next 16-deep
//    k step are read from LDS under the MFMAs of the current one, the loads
//    of later K tiles are spread over the first three k steps, and one
//    barrier per K tile comes after the first MFMAs of its last k step.  The
//    last two K tiles of an output tile prefetch the next tile's first ones.
//    With a single wave per SIMD every issue gap and the epilogue show on the
//    matrix pipe: about 87 % of it without loads, measured, against about
//    95 % for the ping-pong family.
//  * LDS layouts and ragged edges: lds_tile.hpp.  A partial last K tile goes
//    through guarded register loads after the loop.  Operands must have
//    16-byte aligned rows (the launcher falls back to the streaming family
//    otherwise).
#include "internal.hpp"
#include "device_math.hpp"
#include "epilogue.hpp"
#include "lds_tile.hpp"

namespace cola {
namespace {

constexpr int BM = 256;
constexpr int BN = 256;
constexpr int NT = 256;
constexpr int WR = 128;          // rows of a wave's block
constexpr int WC = 128;          // columns of a wave's block
constexpr int TM = WR / 32;
constexpr int TN = WC / 32;

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
        for (int j = 0; j < POPS; ++j) o.p[j] = TP::voff(POPS * wave + j, a.ldp, t.m0, a.M);
#pragma unroll
        for (int j = 0; j < QOPS; ++j) o.q[j] = TQ::voff(QOPS * wave + j, a.ldq, t.n0, a.N);
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
            TP::template load_store<NT>(ps, P, a.ldp, cur.m0, a.M, k0, cur.kend);
            TQ::template load_store<NT>(qs, Q, a.ldq, cur.n0, a.N, k0, cur.kend);
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
