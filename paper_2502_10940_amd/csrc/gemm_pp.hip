// gemm_pp.hip -- the 256 x 256 bf16 MFMA GEMM with two wave groups in
// ping-pong: C[M][N] = sum_k P(m, k) Q(n, k), fp32 accumulation, the fused
// epilogues of epilogue.hpp.
//
// Design (CDNA4, wave64, one workgroup of 8 waves per CU, two per SIMD):
//  * Group 0 (waves 0-3) owns rows 0-127 of the 256 x 256 tile, group 1
//    (waves 4-7) rows 128-255; each wave a 128 x 64 block as 4 x 2 tiles of
//    v_mfma_f32_32x32x16_bf16 (128 fp32 accumulators per lane).  The two
//    waves on a SIMD belong to different groups.  The Q fragment is the
//    MFMA's first operand, so the accumulators hold C^T tiles: four
//    consecutive columns of one row per register group, stored by the
//    transposed epilogue of epilogue.hpp without any transposes.
//  * Each group alternates a memory phase (read the whole K tile's fragments
//    from LDS into registers, issue its share of the direct-to-LDS loads)
//    and a compute phase (the K tile's 32 MFMAs, at raised wave priority
//    when the Q operand fits in L2).
//    Group 1 runs one phase behind group 0, and all eight waves meet at a
//    barrier between phases, so on every SIMD one wave issues MFMAs while
//    the other reads and loads: the matrix pipe never waits for LDS reads,
//    address arithmetic or barriers of the wave that is computing.
//  * K tiles are 64 deep (whole 128-byte lines per load row, which the load
//    path needs to reach its bandwidth).  LDS holds three P slots and two Q
//    slots of 32 KB (160 KB): group 1 loads P two K tiles ahead, group 0
//    loads Q one K tile ahead; a slot is refilled once both groups have read
//    it (two barriers later).
//  * A partial last K tile (K not a multiple of 64) is loaded through
//    guarded registers after the ping-pong, by all waves, and computed by
//    both groups.
//  * Ragged M / N edges as in the other families; operands need 16-byte
//    aligned rows (the launcher falls back otherwise).
#include "internal.hpp"
#include "device_math.hpp"
#include "epilogue.hpp"
#include "lds_tile.hpp"

namespace cola {
namespace {

constexpr int BM = 256;
constexpr int BN = 256;
constexpr int NTHR = 512;        // 8 waves
constexpr int WR = 128;          // rows of a wave's block
constexpr int WC = 64;           // columns of a wave's block
constexpr int TM = WR / 32;
constexpr int TN = WC / 32;
constexpr int NP = 3;            // P slots (two K tiles ahead)
constexpr int NQ = 2;            // Q slots (one K tile ahead)
// K tile of the persistent kernel and the launcher: 64, whole 128-byte lines
// per load row.
constexpr int kPPBK = 64;

// Byte offset of the ring slot of K tile i (i >= 0) among N slots of BYTES.
// It passes through an empty asm statement and a mask, so the compiler
// neither turns it into a running difference across iterations nor loses
// that it is small and non-negative: the constant parts of the fragment
// addresses then fold into the LDS instructions' offset fields instead of
// one VALU add per read.
template <int N, int BYTES>
__device__ __forceinline__ uint32_t slot_off(int i) {
    uint32_t o = ((uint32_t)i % (uint32_t)N) * (uint32_t)BYTES;
    asm volatile("" : "+s"(o));
    return o & 0x3ffffu;
}

// n / d for n, d < 2^21: one multiply by the hardware reciprocal (1 ulp) and
// a correction of at most one either way.  The product is within 1/2 of
// n / d (relative error below 1.5 * 2^-23, n / d < 2^21), so its truncation
// is off by at most one.
__device__ __forceinline__ int64_t fdiv21(int64_t n, int64_t d) {
    const uint32_t un = (uint32_t)n, ud = (uint32_t)d;
    uint32_t q = (uint32_t)((float)un * __builtin_amdgcn_rcpf((float)ud));
    const int32_t r = (int32_t)(un - q * ud);
    if (r < 0) --q;
    else if ((uint32_t)r >= ud) ++q;
    // the operands are wave-uniform: keep the quotient (and the tile
    // coordinates made from it) in scalar registers
    return (int64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)q);
}

// LDS of one workgroup: NP P slots and NQ Q slots.
template <int PL, int QL, int BK>
constexpr int pp_smem_bytes() {
    return NP * BTile<PL, BK>::BYTES + NQ * BTile<QL, BK>::BYTES;
}

// Block number with an XCD-aware renumbering (the hardware hands block b to
// XCD b % 8): with a grid that is a multiple of 8, XCD x gets the contiguous
// range [x G/8, (x+1) G/8) of output tiles.
__device__ __forceinline__ int64_t xcd_block() {
    const int64_t nb = gridDim.x;
    int64_t b = blockIdx.x;
    if ((nb & 7) == 0) b = (b & 7) * (nb >> 3) + (b >> 3);
    return b;
}

// One output tile (tile and split number b of the product a) of one
// workgroup, with the rings in smem.
template <int BK, int PL, int QL, int EPI>
__device__ __forceinline__ void pp_one_tile(const GemmArgs& a, int64_t b, char* smem) {
    using TP = BTile<PL, BK>;
    using TQ = BTile<QL, BK>;
    constexpr int NSUB = BK / 16;                 // 16-deep k steps per K tile
    constexpr int POPS = TP::DPW;                 // loads per loader wave per P tile (4 loaders)
    constexpr int QOPS = TQ::DPW;
    char* const pring = smem;
    char* const qring = smem + NP * TP::BYTES;

    const int64_t tiles_n = (a.N + BN - 1) / BN;
    const int64_t tiles_m = (a.M + BM - 1) / BM;
    const int64_t per_split = tiles_m * tiles_n;
    // below 2^21 tiles the reciprocal division (a few instructions instead of
    // a 64-bit division before the first load)
    const bool fast = per_split * a.splits < (int64_t(1) << 21);
    const int split = (int)(fast ? fdiv21(b, per_split) : b / per_split);
    const int64_t rem = b - (int64_t)split * per_split;
    const int64_t tm = fast ? fdiv21(rem, tiles_n) : rem / tiles_n;
    const int64_t m0 = tm * BM;
    const int64_t n0 = (rem - tm * tiles_n) * BN;
    const int64_t kbeg = (int64_t)split * a.k_chunk;
    const int64_t kend = min(a.K, kbeg + a.k_chunk);
    const int nk = (int)((kend - kbeg) / BK);     // whole K tiles
    const bool tail = kbeg + (int64_t)nk * BK < kend;

    const uint16_t* P = reinterpret_cast<const uint16_t*>(a.p);
    const uint16_t* Q = reinterpret_cast<const uint16_t*>(a.q);
    const int wave = wave_id();
    const int lane = threadIdx.x & 63;
    const int grp = wave >> 2;                    // 0: rows 0-127, loads Q; 1: rows 128-255, loads P
    const int wl = wave & 3;                      // loader index and column block in the group

    // this wave's share of the loads: group 0 fills Q tiles, group 1 P tiles
    uint32_t vo[POPS > QOPS ? POPS : QOPS];
    if (grp == 0) {
#pragma unroll
        for (int j = 0; j < QOPS; ++j) vo[j] = TQ::voff(QOPS * wl + j, a.ldq, n0, a.N);
    } else {
#pragma unroll
        for (int j = 0; j < POPS; ++j) vo[j] = TP::voff(POPS * wl + j, a.ldp, m0, a.M);
    }
    auto issue_p = [&](int kt) {
        const __amdgpu_buffer_rsrc_t r = rsrc_of(TP::gbase(P, a.ldp, m0, kbeg + (int64_t)kt * BK));
        char* slot = pring + (kt % NP) * TP::BYTES;
#pragma unroll
        for (int j = 0; j < POPS; ++j) dtl16(r, vo[j], slot + 1024 * (POPS * wl + j));
    };
    auto issue_q = [&](int kt) {
        const __amdgpu_buffer_rsrc_t r = rsrc_of(TQ::gbase(Q, a.ldq, n0, kbeg + (int64_t)kt * BK));
        char* slot = qring + (kt % NQ) * TQ::BYTES;
#pragma unroll
        for (int j = 0; j < QOPS; ++j) dtl16(r, vo[j], slot + 1024 * (QOPS * wl + j));
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    // Per-lane parts of the fragment read addresses, computed once: per k
    // step for k-contiguous tiles, per 32-row block for m-contiguous ones;
    // the rest of each address is wave-uniform or an immediate.
    constexpr int NLP = PL == KMAJ ? NSUB : TM;
    constexpr int NLQ = QL == KMAJ ? NSUB : TN;
    uint32_t lp[NLP], lq[NLQ];
#pragma unroll
    for (int u = 0; u < NLP; ++u) lp[u] = TP::lane_off(PL == KMAJ ? u : (grp * WR) / 32 + u, lane);
#pragma unroll
    for (int u = 0; u < NLQ; ++u) lq[u] = TQ::lane_off(QL == KMAJ ? u : (wl * WC) / 32 + u, lane);
    auto frag_p = [&](const char* ps, int i, int s) -> bf16x8 {
        if constexpr (PL == KMAJ) return TP::frag_at(ps, grp * WR + 32 * i, lp[s]);
        else return TP::frag_at(ps, s, lp[i]);
    };
    auto frag_q = [&](const char* qs, int j, int s) -> bf16x8 {
        if constexpr (QL == KMAJ) return TQ::frag_at(qs, wl * WC + 32 * j, lq[s]);
        else return TQ::frag_at(qs, s, lq[j]);
    };

    // the whole K tile's fragments of this wave
    bf16x8 fa[NSUB][TM], fb[NSUB][TN];
    auto read_tile = [&](const char* ps, const char* qs) {
#pragma unroll
        for (int s = 0; s < NSUB; ++s) {
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[s][i] = frag_p(ps, i, s);
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[s][j] = frag_q(qs, j, s);
        }
    };
    // Raised wave priority for the compute phase when the Q operand fits
    // comfortably in an XCD's L2 (measured on MI355X: it helps there, and
    // slows products whose Q operand misses in L2, whose memory phases need
    // the issue slots), and for the fp32 weight gradients, whose memory
    // phases are short since their fragment addresses fold into the LDS
    // offsets (measured: dA + dB -1 %).
    const bool prio = EPI == EPI_STORE_F32 || (int64_t)a.N * a.K * 2 <= (int64_t)(3 << 20);
    auto compute_tile = [&]() {
        if (prio) __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[s][j], fa[s][i], acc[i][j], 0, 0, 0);
        if (prio) __builtin_amdgcn_s_setprio(0);
    };

    // prologue: P(0), P(1) by group 1, Q(0) by group 0; K tile 0 complete
    // before the first barrier
    if (nk > 0) {
        if (grp == 0) {
            issue_q(0);
            wait_vm<0>();
        } else {
            issue_p(0);
            if (nk > 1) {
                issue_p(1);
                wait_vm<POPS>();
            } else {
                wait_vm<0>();
            }
        }
    }
    barrier_lds();

    // Ping-pong over the whole K tiles.  Barrier b(2j) opens group 0's memory
    // phase of K tile j, b(2j+1) its compute phase and group 1's memory phase
    // of K tile j, b(2j+2) group 1's compute phase.  Group 0 issues Q(j + 1)
    // in its memory phase of j (the slot of Q(j - 1), free since b(2j)) and
    // has it in before b(2j+2); group 1 issues P(j + 2) in its memory phase
    // of j (the slot of P(j - 1), free since b(2j)) and has P(j + 1) in
    // before b(2j+2).
    if (grp == 1) barrier_lds();
    for (int j = 0; j < nk; ++j) {
        read_tile(pring + slot_off<NP, TP::BYTES>(j), qring + slot_off<NQ, TQ::BYTES>(j));
        if (grp == 0) {
            if (j + 1 < nk) issue_q(j + 1);
        } else {
            if (j + 2 < nk) {
                issue_p(j + 2);
                wait_vm<POPS>();
            } else {
                wait_vm<0>();
            }
        }
        barrier_lds();                                // end of the memory phase
        __builtin_amdgcn_sched_barrier(0);
        compute_tile();
        __builtin_amdgcn_sched_barrier(0);
        if (grp == 0) wait_vm<0>();                   // Q(j + 1) in
        barrier_lds();                                // end of the compute phase
    }
    if (grp == 0) barrier_lds();

    // partial last K tile: guarded register loads (zeros past kend) by all
    // waves into slot 0 of each ring (every wave is done with the rings)
    if (tail) {
        const int64_t k0 = kbeg + (int64_t)nk * BK;
        TP::template load_store<NTHR>(pring, P, a.ldp, m0, a.M, k0, kend);
        TQ::template load_store<NTHR>(qring, Q, a.ldq, n0, a.N, k0, kend);
        barrier_lds();
        read_tile(pring, qring);
        compute_tile();
    }
    epilogue_block_t<EPI>(a, acc, m0 + grp * WR, n0 + wl * WC, lane, split);
}

// One workgroup per output tile (and split).
template <int BK, int PL, int QL, int EPI, int TAG>
__global__ __launch_bounds__(NTHR, 1) void gemm_pp_kernel(GemmArgs a) {
    __shared__ __attribute__((aligned(1024))) char smem[pp_smem_bytes<PL, QL, BK>()];
    pp_one_tile<BK, PL, QL, EPI>(a, xcd_block(), smem);
}

// Two products of the same kind in one grid: blocks [0, nb0) are the tiles
// and splits of a0, the rest those of a1 (the two weight gradients of a
// layer, which share K = T: one launch, one set of partials per split for
// both, and their tiles together fill the CUs).
template <int BK, int PL, int QL, int EPI, int TAG>
__global__ __launch_bounds__(NTHR, 1) void gemm_pp_pair_kernel(GemmArgs a0, GemmArgs a1, int64_t nb0) {
    __shared__ __attribute__((aligned(1024))) char smem[pp_smem_bytes<PL, QL, BK>()];
    const int64_t b = xcd_block();
    if (b < nb0) pp_one_tile<BK, PL, QL, EPI>(a0, b, smem);
    else pp_one_tile<BK, PL, QL, EPI>(a1, b - nb0, smem);
}

// ---- persistent variant (every K range a whole number of K tiles, at
// least two) ----
//
// One workgroup per CU walks its output tiles; the K tiles of all its tiles
// form one stream with global numbers g (P slot g % 3, Q slot g % 2), so the
// loads run ahead across tile boundaries exactly as inside a tile and the two
// groups keep their phase offset.  After the last K tile of a tile each group
// spends one phase on its epilogue (group 0's overlaps group 1's last compute
// phase), clears its accumulators and goes on with the next tile's first K
// tile: no prologue, no drain.  (The first k step of each tile's first K
// tile starts from zero accumulators, so nothing is cleared in between.)

struct PPTile {
    int64_t m0, n0, kbeg;
    int split, nk;
};

constexpr int64_t kBand = 8;

// Output tile i (0, 1, ...) of this workgroup; false past the last one.  With
// a grid and a tile count that are multiples of 8, XCD x (blockIdx % 8) owns
// the contiguous tile range [x T/8, (x+1) T/8), swept by its workgroups
// together, so tiles that share operand rows share an L2.  When that range
// is whole rows of tiles (one split), it is swept in column bands of
// kBand tiles (n fastest within a band, then the next row): the Q rows of a
// band (kBand x 256 rows, 2 MB for K = 512) stay in the XCD's 4 MB L2 while
// the band's rows stream, instead of every row of tiles pulling all of Q.
// Every dividend and divisor here is at most the tile count; below 2^21
// tiles (any realistic launch) the divisions take the short path, so the
// walk costs a few dozen instructions per tile instead of several
// thousand cycles of 64-bit division.
__device__ __forceinline__ bool pp_tile_at(const GemmArgs& a, int64_t i, PPTile* t) {
    // the launch constants pass through an empty asm statement so that the
    // walk is recomputed at each call rather than hoisted out of the tile
    // loop (its loop-invariant part would stay live in registers and spill)
    int64_t M = a.M, N = a.N, K = a.K, kc = a.k_chunk;
    int splits = a.splits;
    asm volatile("" : "+s"(M), "+s"(N), "+s"(K), "+s"(kc), "+s"(splits));
    const int64_t tiles_n = (N + BN - 1) / BN;             // shifts (BN, BM powers of two)
    const int64_t tiles_m = (M + BM - 1) / BM;
    const int64_t per_split = tiles_m * tiles_n;
    const int64_t total = per_split * splits;
    const bool fast = total < (int64_t(1) << 21);
    auto dv = [fast](int64_t n, int64_t d) { return fast ? fdiv21(n, d) : n / d; };
    const int64_t G = gridDim.x;
    int64_t idx;
    if ((G & 7) == 0 && (total & 7) == 0) {
        const int64_t per_xcd = total >> 3;
        const int64_t j = (int64_t)(blockIdx.x >> 3) + i * (G >> 3);
        if (j >= per_xcd) return false;
        const int64_t x = blockIdx.x & 7;
        const int64_t rows = dv(per_xcd, tiles_n);            // rows of tiles this XCD owns
        if (splits == 1 && rows * tiles_n == per_xcd && tiles_n > kBand) {
            const int64_t nbands = (tiles_n + kBand - 1) / kBand;
            int64_t band = dv(j, rows * kBand);
            if (band > nbands - 1) band = nbands - 1;
            const int64_t off = j - band * rows * kBand;
            const int64_t w = min(kBand, tiles_n - band * kBand);  // width of this band
            const int64_t r = w == kBand ? off / kBand : dv(off, w);
            idx = (x * rows + r) * tiles_n + band * kBand + (off - r * w);
        } else {
            idx = x * per_xcd + j;
        }
    } else {
        idx = (int64_t)blockIdx.x + i * G;
        if (idx >= total) return false;
    }
    t->split = (int)dv(idx, per_split);
    const int64_t rem = idx - (int64_t)t->split * per_split;
    const int64_t tm = dv(rem, tiles_n);
    t->m0 = tm * BM;
    t->n0 = (rem - tm * tiles_n) * BN;
    t->kbeg = (int64_t)t->split * kc;
    t->nk = (int)((min(K, t->kbeg + kc) - t->kbeg) / kPPBK);
    return true;
}

template <int BK, int PL, int QL, int EPI, int TAG>
__global__ __launch_bounds__(NTHR, 1) void gemm_pp_persist_kernel(GemmArgs a) {
    using TP = BTile<PL, BK>;
    using TQ = BTile<QL, BK>;
    constexpr int NSUB = BK / 16;
    constexpr int POPS = TP::DPW;
    constexpr int QOPS = TQ::DPW;
    __shared__ __attribute__((aligned(1024))) char smem[NP * TP::BYTES + NQ * TQ::BYTES];
    char* const pring = smem;
    char* const qring = smem + NP * TP::BYTES;

    const uint16_t* P = reinterpret_cast<const uint16_t*>(a.p);
    const uint16_t* Q = reinterpret_cast<const uint16_t*>(a.q);
    const int wave = wave_id();
    const int lane = threadIdx.x & 63;
    const int grp = wave >> 2;
    const int wl = wave & 3;

    // P (Q) part of K tile kt of tile t into the slot of global K tile g;
    // the per-lane offsets are formed here (they depend on the tile only at
    // the M / N edges)
    // Interior tiles: each load's offset is a per-lane part that depends on
    // the load only through its parity (two registers per wave, computed
    // once) plus a wave-uniform part in the scalar offset operand, so a load
    // costs no vector arithmetic.  Edge tiles form the clamped per-lane
    // offsets at each issue (the lane goes through an empty asm statement so
    // that they are not hoisted and kept live across the compute phase).
    uint32_t lpart[2];
#pragma unroll
    for (int par = 0; par < 2; ++par)
        lpart[par] = grp == 0 ? TQ::lane_part(par, a.ldq, lane) : TP::lane_part(par, a.ldp, lane);
    auto issue_p = [&](const PPTile& t, int kt, int g) {
        const __amdgpu_buffer_rsrc_t r = rsrc_of(TP::gbase(P, a.ldp, t.m0, t.kbeg + (int64_t)kt * BK));
        char* slot = pring + (g % NP) * TP::BYTES;
        if (TP::interior(t.m0, a.M)) {
#pragma unroll
            for (int j = 0; j < POPS; ++j)
                dtl16s(r, lpart[j & 1], TP::uniform_part(POPS * wl + j, a.ldp), slot + 1024 * (POPS * wl + j));
        } else {
            int ln = lane;
            asm volatile("" : "+v"(ln));
#pragma unroll
            for (int j = 0; j < POPS; ++j)
                dtl16(r, TP::voff_l(POPS * wl + j, a.ldp, t.m0, a.M, ln), slot + 1024 * (POPS * wl + j));
        }
    };
    auto issue_q = [&](const PPTile& t, int kt, int g) {
        const __amdgpu_buffer_rsrc_t r = rsrc_of(TQ::gbase(Q, a.ldq, t.n0, t.kbeg + (int64_t)kt * BK));
        char* slot = qring + (g % NQ) * TQ::BYTES;
        if (TQ::interior(t.n0, a.N)) {
#pragma unroll
            for (int j = 0; j < QOPS; ++j)
                dtl16s(r, lpart[j & 1], TQ::uniform_part(QOPS * wl + j, a.ldq), slot + 1024 * (QOPS * wl + j));
        } else {
            int ln = lane;
            asm volatile("" : "+v"(ln));
#pragma unroll
            for (int j = 0; j < QOPS; ++j)
                dtl16(r, TQ::voff_l(QOPS * wl + j, a.ldq, t.n0, a.N, ln), slot + 1024 * (QOPS * wl + j));
        }
    };

    constexpr int NLP = PL == KMAJ ? NSUB : TM;
    constexpr int NLQ = QL == KMAJ ? NSUB : TN;
    uint32_t lp[NLP], lq[NLQ];
#pragma unroll
    for (int u = 0; u < NLP; ++u) lp[u] = TP::lane_off(PL == KMAJ ? u : (grp * WR) / 32 + u, lane);
#pragma unroll
    for (int u = 0; u < NLQ; ++u) lq[u] = TQ::lane_off(QL == KMAJ ? u : (wl * WC) / 32 + u, lane);
    auto frag_p = [&](const char* ps, int i, int s) -> bf16x8 {
        if constexpr (PL == KMAJ) return TP::frag_at(ps, grp * WR + 32 * i, lp[s]);
        else return TP::frag_at(ps, s, lp[i]);
    };
    auto frag_q = [&](const char* qs, int j, int s) -> bf16x8 {
        if constexpr (QL == KMAJ) return TQ::frag_at(qs, wl * WC + 32 * j, lq[s]);
        else return TQ::frag_at(qs, s, lq[j]);
    };

    f32x16 acc[TM][TN];
    bf16x8 fa[NSUB][TM], fb[NSUB][TN];
    auto read_tile = [&](int g) {
        const char* ps = pring + slot_off<NP, TP::BYTES>(g);
        const char* qs = qring + slot_off<NQ, TQ::BYTES>(g);
#pragma unroll
        for (int s = 0; s < NSUB; ++s) {
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[s][i] = frag_p(ps, i, s);
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[s][j] = frag_q(qs, j, s);
        }
    };
    // Raised wave priority for the compute phase when the Q operand fits
    // comfortably in an XCD's L2 (measured on MI355X: it helps there, and
    // slows products whose Q operand misses in L2, whose memory phases need
    // the issue slots).
    const bool prio = (int64_t)a.N * a.K * 2 <= (int64_t)(3 << 20);
    // FIRST: the first K tile of an output tile, whose first k step starts
    // from zero accumulators (no separate clearing after the epilogue)
    auto compute_tile = [&](auto first) {
        if (prio) __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    if constexpr (decltype(first)::value) {
                        if (s == 0) {
                            const f32x16 zero = {};
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[s][j], fa[s][i], zero, 0, 0, 0);
                            continue;
                        }
                    }
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[s][j], fa[s][i], acc[i][j], 0, 0, 0);
                }
        if (prio) __builtin_amdgcn_s_setprio(0);
    };

    PPTile cur, nxt;
    if (!pp_tile_at(a, 0, &cur)) return;
    bool more = pp_tile_at(a, 1, &nxt);

    // prologue: P(0), P(1) by group 1, Q(0) by group 0 (every tile has at
    // least two K tiles)
    if (grp == 0) {
        issue_q(cur, 0, 0);
        wait_vm<0>();
    } else {
        issue_p(cur, 0, 0);
        issue_p(cur, 1, 1);
        wait_vm<POPS>();
    }
    barrier_lds();

    // The phases of both groups, one barrier after each: for every tile, a
    // memory and a compute phase per K tile, then the epilogue phase; group 1
    // one phase behind group 0.  Group 0 issues Q(g + 1) in its memory phase
    // of global K tile g and has it in by the end of its compute phase;
    // group 1 issues P(g + 2) in its memory phase of g and has P(g + 1) in by
    // the end of it.  The slots they fill (of g - 1) were read by both groups
    // before: group 1 read them in its memory phase of g - 1, group 0 one
    // phase earlier still.
    if (grp == 1) barrier_lds();
    int g = 0;
    for (int64_t it = 0;; ++it) {
        const int nk = cur.nk;
        for (int kt = 0; kt < nk; ++kt, ++g) {
            read_tile(g);
            if (grp == 0) {
                if (kt + 1 < nk) issue_q(cur, kt + 1, g + 1);
                else if (more) issue_q(nxt, 0, g + 1);
            } else {
                bool issued = true;
                if (kt + 2 < nk) issue_p(cur, kt + 2, g + 2);
                else if (more) issue_p(nxt, kt + 2 - nk, g + 2);
                else issued = false;
                if (issued) wait_vm<POPS>();
                else wait_vm<0>();
            }
            barrier_lds();                               // end of the memory phase
            __builtin_amdgcn_sched_barrier(0);
            if (kt == 0) compute_tile(ic<bool, true>{});
            else compute_tile(ic<bool, false>{});
            __builtin_amdgcn_sched_barrier(0);
            if (grp == 0) wait_vm<0>();                  // Q(g + 1) in
            barrier_lds();                               // end of the compute phase
        }
        // the epilogue's coordinates pass through an empty asm statement so
        // that none of its address arithmetic is hoisted above the K loop
        // (it would stay live across the loop and spill)
        // (tile coordinates are wave-uniform and below 2^31: M, N < 2^31)
        int em0 = __builtin_amdgcn_readfirstlane((int)(cur.m0 + grp * WR));
        int en0 = __builtin_amdgcn_readfirstlane((int)(cur.n0 + wl * WC));
        int esplit = __builtin_amdgcn_readfirstlane(cur.split);
        asm volatile("" : "+s"(em0), "+s"(en0), "+s"(esplit));
        epilogue_block_t<EPI>(a, acc, (int64_t)em0, (int64_t)en0, lane, esplit);
        barrier_lds();                                   // end of the epilogue phase
        if (!more) break;
        cur = nxt;
        more = pp_tile_at(a, it + 2, &nxt);
    }
    if (grp == 0) barrier_lds();
}

// Persistent grid: one workgroup per CU (256 on MI355X), a multiple of 8 when
// possible so each XCD gets equal work.
constexpr int64_t kPPGrid = 256;

template <int PL, int QL, int EPI, int TAG>
hipError_t launch_p(const GemmArgs& a, hipStream_t s) {
    if (a.p_layout != PL || a.q_layout != QL || a.epi != EPI) return hipErrorInvalidValue;
    const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * (int64_t)a.splits;
    if (tiles <= 0) return hipSuccess;
    if (tiles > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    // persistent when there are more tiles than CUs and every split is a whole
    // number (at least two) of K tiles
    const int64_t last = a.K - (int64_t)(a.splits - 1) * a.k_chunk;
    const bool whole = a.K % kPPBK == 0 && a.k_chunk % kPPBK == 0 && a.k_chunk >= 2 * kPPBK && last >= 2 * kPPBK;
    if (whole && tiles > kPPGrid) {
        int64_t grid = kPPGrid;
        if ((tiles & 7) == 0) grid &= ~int64_t(7);
        hipLaunchKernelGGL((gemm_pp_persist_kernel<kPPBK, PL, QL, EPI, TAG>), dim3((unsigned)grid), dim3(NTHR), 0,
                           s, a);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((gemm_pp_kernel<kPPBK, PL, QL, EPI, TAG>), dim3((unsigned)tiles), dim3(NTHR), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_pp_pair(const GemmArgs& a0, const GemmArgs& a1, hipStream_t s) {
    for (const GemmArgs* a : {&a0, &a1})
        if (a->p_layout != MNMAJ || a->q_layout != MNMAJ || a->epi != EPI_STORE_F32) return hipErrorInvalidValue;
    auto blocks = [](const GemmArgs& a) {
        return ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * (int64_t)a.splits;
    };
    const int64_t nb0 = blocks(a0), nb1 = blocks(a1);
    if (nb0 + nb1 <= 0) return hipSuccess;
    if (nb0 + nb1 > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((gemm_pp_pair_kernel<kPPBK, MNMAJ, MNMAJ, EPI_STORE_F32, TAG_BWD_DA>),
                       dim3((unsigned)(nb0 + nb1)), dim3(NTHR), 0, s, a0, a1, nb0);
    return hipGetLastError();
}

hipError_t launch_gemm_pp(const GemmArgs& a, hipStream_t s) {
    switch (a.tag) {
        case TAG_FWD_Z: return launch_p<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_Z>(a, s);
        case TAG_INFER_H: return launch_p<KMAJ, KMAJ, EPI_H, TAG_INFER_H>(a, s);
        case TAG_FWD_Y: return launch_p<KMAJ, KMAJ, EPI_STORE, TAG_FWD_Y>(a, s);
        case TAG_FWD_YP: return launch_p<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_YP>(a, s);
        case TAG_FWD_YG: return launch_p<KMAJ, KMAJ, EPI_GATE, TAG_FWD_YG>(a, s);
        case TAG_BWD_DXG: return launch_p<KMAJ, MNMAJ, EPI_DGATE, TAG_BWD_DXG>(a, s);
        case TAG_BWD_DZ: return launch_p<KMAJ, MNMAJ, EPI_DZ, TAG_BWD_DZ>(a, s);
        case TAG_BWD_DX: return launch_p<KMAJ, MNMAJ, EPI_STORE, TAG_BWD_DX>(a, s);
        case TAG_BWD_DA: return launch_p<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_BWD_DA>(a, s);
        case TAG_BWD_DB: return launch_p<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_BWD_DB>(a, s);
        case TAG_DENSE_FWD: return launch_p<KMAJ, KMAJ, EPI_STORE, TAG_DENSE_FWD>(a, s);
        case TAG_DENSE_DX: return launch_p<KMAJ, MNMAJ, EPI_STORE, TAG_DENSE_DX>(a, s);
        case TAG_DENSE_DW: return launch_p<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_DENSE_DW>(a, s);
        default: return hipErrorNotSupported;
    }
}

}  // namespace cola
