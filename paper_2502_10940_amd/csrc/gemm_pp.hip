// gemm_pp.hip -- the 256 x 256 bf16 MFMA GEMM with two wave groups in
// ping-pong: C[M][N] = sum_k P(m, k) Q(n, k), fp32 accumulation, the fused
// epilogues of epilogue.hpp.
//
// Design (CDNA4, wave64, one workgroup of 8 waves per CU, two per SIMD):
//  * Group 0 (waves 0-3) owns rows 0-127 of the 256 x 256 tile, group 1
//    (waves 4-7) rows 128-255; each wave a 128 x 64 block as 4 x 2 tiles of
//    v_mfma_f32_32x32x16_bf16 (128 fp32 accumulators per lane).  The two
//    waves on a SIMD belong to different groups.
//  * Each group alternates a memory phase (read the whole K tile's fragments
//    from LDS into registers, issue its share of the direct-to-LDS loads)
//    and a compute phase (the K tile's 32 MFMAs, at raised wave priority).
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

template <int BK, int PL, int QL, int EPI, int TAG>
__global__ __launch_bounds__(NTHR, 1) void gemm_pp_kernel(GemmArgs a) {
    using TP = BTile<PL, BK>;
    using TQ = BTile<QL, BK>;
    constexpr int NSUB = BK / 16;                 // 16-deep k steps per K tile
    constexpr int POPS = TP::DPW;                 // loads per loader wave per P tile (4 loaders)
    constexpr int QOPS = TQ::DPW;
    __shared__ __attribute__((aligned(1024))) char smem[NP * TP::BYTES + NQ * TQ::BYTES];
    char* const pring = smem;
    char* const qring = smem + NP * TP::BYTES;

    // output tile: XCD-aware renumbering (hardware hands block b to XCD b % 8)
    const int64_t nb = gridDim.x;
    int64_t b = blockIdx.x;
    if ((nb & 7) == 0) b = (b & 7) * (nb >> 3) + (b >> 3);
    const int64_t tiles_n = (a.N + BN - 1) / BN;
    const int64_t tiles_m = (a.M + BM - 1) / BM;
    const int64_t per_split = tiles_m * tiles_n;
    const int split = (int)(b / per_split);
    const int64_t rem = b - (int64_t)split * per_split;
    const int64_t m0 = (rem / tiles_n) * BM;
    const int64_t n0 = (rem % tiles_n) * BN;
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
    auto compute_tile = [&]() {
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s][i], fb[s][j], acc[i][j], 0, 0, 0);
        __builtin_amdgcn_s_setprio(0);
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
        read_tile(pring + (j % NP) * TP::BYTES, qring + (j % NQ) * TQ::BYTES);
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
    epilogue_block<EPI>(a, acc, m0 + grp * WR, n0 + wl * WC, lane, split);
}

// K tile 64: whole 128-byte lines per load row.
constexpr int kPPBK = 64;

template <int PL, int QL, int EPI, int TAG>
hipError_t launch_p(const GemmArgs& a, hipStream_t s) {
    if (a.p_layout != PL || a.q_layout != QL || a.epi != EPI) return hipErrorInvalidValue;
    const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * (int64_t)a.splits;
    if (tiles <= 0) return hipSuccess;
    if (tiles > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((gemm_pp_kernel<kPPBK, PL, QL, EPI, TAG>), dim3((unsigned)tiles), dim3(NTHR), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_pp(const GemmArgs& a, hipStream_t s) {
    switch (a.tag) {
        case TAG_FWD_Z: return launch_p<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_Z>(a, s);
        case TAG_INFER_H: return launch_p<KMAJ, KMAJ, EPI_H, TAG_INFER_H>(a, s);
        case TAG_FWD_Y: return launch_p<KMAJ, KMAJ, EPI_STORE, TAG_FWD_Y>(a, s);
        case TAG_FWD_YP: return launch_p<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_YP>(a, s);
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
