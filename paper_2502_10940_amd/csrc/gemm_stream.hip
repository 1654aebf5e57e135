// gemm_stream.hip -- the streaming bf16 MFMA GEMM: C[M][N] = sum_k P(m, k) Q(n, k)
// with fp32 accumulation and the fused epilogues of epilogue.hpp.
//
// Design (CDNA4, wave64, two workgroups per CU):
//  * 256 threads = 4 waves in a 2 x 2 grid; tile BM x 128 (BM = 256, or 128
//    when M <= 128); each wave owns (BM/2) x 64 of C as 32x32x16 MFMA tiles
//    (128 fp32 accumulators per lane at BM = 256), so two workgroups fit a
//    CU and one's barriers, waits and epilogue overlap the other's MFMAs.
//  * K advances in tiles of 32 through three LDS stages (72 KB at BM = 256):
//    the loads run two K tiles ahead.  Interior tiles use the direct-to-LDS
//    loads (global_load_lds_dwordx4): no staging registers and no LDS write
//    instructions.  They are issued one per two MFMAs: a burst of them right
//    after the barrier stalls the issuing wave on the address unit's queue.
//  * k-contiguous operands sit in LDS as [row][32 k], 64-byte rows, 16-byte
//    chunks XOR-swizzled by (row >> 2) & 3, read with ds_read_b128;
//    m-contiguous operands (token-reduction weight gradients, weights in the
//    backward products) sit as in memory, [32 k][rows], chunks swizzled by
//    4 (k & 3), read with the transposing ds_read_b64_tr_b16.  gfx950's LDS
//    has 64 four-byte banks (256 bytes per clock): a 32-lane half-wave of
//    either read touches 16 distinct 16-byte bank groups, so neither pattern
//    conflicts (measured: b128 reads at 4 clocks, tr reads at 2.5).
//  * Ragged edges: k-contiguous rows past the edge re-read the last row;
//    m-contiguous chunks past the edge re-read the last chunk (the chunk
//    holding the last column may run into the row's pitch padding, which the
//    ABI allows).  Those values only reach outputs that are not stored.  The
//    K tail and unaligned operands go through guarded register loads.
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

constexpr int BN = 128;
constexpr int NT = 256;

// Operands the direct-to-LDS path takes: 16-byte aligned rows, and a pitch
// small enough for 32-bit per-lane offsets within a tile (256 rows or 32 k).
__device__ __forceinline__ bool aligned16(const void* p, int64_t ld) {
    return ((reinterpret_cast<uintptr_t>(p) & 15u) == 0) && ((ld & 7) == 0) && ld < (int64_t(1) << 22);
}

// 16 bytes per lane from ubase + voff (wave-uniform base, 32-bit per-lane
// offset: the scalar-base form of the instruction) to LDS.
__device__ __forceinline__ void dtl16(const char* ubase, uint32_t voff, char* lds) {
    __builtin_amdgcn_global_load_lds((gptr_t)(ubase + voff), (lptr_t)lds, 16, 0, 0);
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

__device__ __forceinline__ void barrier_lds() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
template <int N>
__device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int R, int LAYOUT, int BK>
struct STile;

// ---- k-contiguous operand: LDS [R rows][BK k] (2 BK-byte rows) ----
// CR = BK / 8 16-byte chunks per row; chunk c of row r sits at chunk
// c ^ ((r / (16 / CR)) % CR): for BK = 32 (64-byte rows) (r >> 2) & 3, for
// BK = 16 (32-byte rows) (r >> 3) & 1.  Either way the 32 rows a half-wave
// reads cover all 64 banks once.
template <int R, int BK>
struct STile<R, KMAJ, BK> {
    static constexpr int CR = BK / 8;
    static constexpr int RPI = 64 / CR;                      // rows per 1 KB instruction
    static constexpr int BYTES = R * BK * 2;
    static constexpr int DTL_PER_WAVE = BYTES / 1024 / 4;   // 1 KB per wave instruction
    static_assert(CR == 2 || CR == 4, "BK of 16 or 32");

    __device__ static __forceinline__ int off(int row, int c) {
        return row * (2 * BK) + ((c ^ ((row / (16 / CR)) & (CR - 1))) << 4);
    }

    // Wave w, instruction j fills LDS bytes [1024 (DPW w + j), +1024): rows
    // RPI blk .. +RPI, lane l -> row + l / CR, physical chunk l % CR.
    __device__ static __forceinline__ void dtl_one(int j, char* lds, const uint16_t* base, int64_t ld,
                                                   int64_t row0, int64_t rows, int64_t k0) {
        const int wave = threadIdx.x >> 6;
        const int lane = threadIdx.x & 63;
        const int blk = DTL_PER_WAVE * wave + j;
        const int row = RPI * blk + lane / CR;
        const int lc = (lane % CR) ^ ((row / (16 / CR)) & (CR - 1));
        const int lrow = row0 + row < rows ? row : (int)(rows - 1 - row0);
        const uint32_t voff = 2u * ((uint32_t)lrow * (uint32_t)ld + 8u * (uint32_t)lc);
        dtl16(reinterpret_cast<const char*>(base + row0 * ld + k0), voff, lds + 1024 * blk);
    }
    __device__ static __forceinline__ void dtl(char* lds, const uint16_t* base, int64_t ld, int64_t row0,
                                               int64_t rows, int64_t k0) {
#pragma unroll
        for (int j = 0; j < DTL_PER_WAVE; ++j) dtl_one(j, lds, base, ld, row0, rows, k0);
    }

    // guarded: chunk id -> (row id / CR, chunk id % CR); R * CR chunks
    __device__ static __forceinline__ void load_store(char* lds, const uint16_t* base, int64_t ld, int64_t row0,
                                                      int64_t rows, int64_t k0, int64_t kend, bool aligned) {
#pragma unroll
        for (int i = 0; i < R * CR / NT; ++i) {
            const int id = threadIdx.x + NT * i;
            const int64_t row = row0 + id / CR;
            const int64_t k = k0 + 8 * (id % CR);
            uint4 v;
            if (row < rows && k + 8 <= kend && aligned) {
                v = *reinterpret_cast<const uint4*>(base + row * ld + k);
            } else {
                const int64_t valid = row < rows ? kend - k : 0;
                v = load8_guarded(base + (row < rows ? row : 0) * ld + k,
                                  (int)(valid < 0 ? 0 : (valid > 8 ? 8 : valid)));
            }
            *reinterpret_cast<uint4*>(lds + off(id / CR, id % CR)) = v;
        }
    }

    // 32 rows (row0 ..) x 16 k (16 s ..) fragment
    __device__ static __forceinline__ bf16x8 frag(const char* lds, int row0, int s, int lane) {
        return *reinterpret_cast<const bf16x8*>(lds + off(row0 + (lane & 31), 2 * s + (lane >> 5)));
    }
};

// ---- m-contiguous operand: LDS [BK k][R m] (2R-byte rows) ----
template <int R, int BK>
struct STile<R, MNMAJ, BK> {
    static constexpr int BYTES = BK * R * 2;
    static constexpr int DTL_PER_WAVE = BYTES / 1024 / 4;
    static constexpr int CPR = R / 8;                         // 16-byte chunks per k row
    static_assert(CPR >= 16, "the 4 (k & 3) chunk swizzle needs 16 chunks per row");

    __device__ static __forceinline__ int off(int k, int c) {
        return k * (2 * R) + ((c ^ ((k & 3) << 2)) << 4);
    }

    // Wave w, instruction j fills LDS bytes [1024 (DPW w + j), +1024): k rows
    // (1024 / 2R) blk .., lane l -> k row + l / CPR, physical chunk l % CPR.
    // Chunks that start past the last column re-read the last chunk.
    __device__ static __forceinline__ void dtl_one(int j, char* lds, const uint16_t* base, int64_t ld,
                                                   int64_t m0, int64_t rows, int64_t k0) {
        const int wave = threadIdx.x >> 6;
        const int lane = threadIdx.x & 63;
        const int64_t mlast = ((rows - 1) >> 3) << 3;
        const int blk = DTL_PER_WAVE * wave + j;
        const int k = (1024 / (2 * R)) * blk + lane / CPR;
        const int lc = (lane % CPR) ^ ((k & 3) << 2);
        const int lm = m0 + 8 * lc <= mlast ? 8 * lc : (int)(mlast - m0);
        const uint32_t voff = 2u * ((uint32_t)k * (uint32_t)ld + (uint32_t)lm);
        dtl16(reinterpret_cast<const char*>(base + k0 * ld + m0), voff, lds + 1024 * blk);
    }
    __device__ static __forceinline__ void dtl(char* lds, const uint16_t* base, int64_t ld, int64_t m0,
                                               int64_t rows, int64_t k0) {
#pragma unroll
        for (int j = 0; j < DTL_PER_WAVE; ++j) dtl_one(j, lds, base, ld, m0, rows, k0);
    }

    __device__ static __forceinline__ void load_store(char* lds, const uint16_t* base, int64_t ld, int64_t m0,
                                                      int64_t rows, int64_t k0, int64_t kend, bool aligned) {
#pragma unroll
        for (int i = 0; i < BK * CPR / NT; ++i) {
            const int id = threadIdx.x + NT * i;
            const int64_t k = k0 + id / CPR;
            const int64_t m = m0 + 8 * (id % CPR);
            uint4 v;
            if (k < kend && m + 8 <= rows && aligned) {
                v = *reinterpret_cast<const uint4*>(base + k * ld + m);
            } else {
                const int64_t valid = k < kend ? rows - m : 0;
                v = load8_guarded(base + (k < kend ? k : 0) * ld + (valid > 0 ? m : 0),
                                  (int)(valid < 0 ? 0 : (valid > 8 ? 8 : valid)));
            }
            *reinterpret_cast<uint4*>(lds + off(id / CPR, id % CPR)) = v;
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

// Wait until at most DTL_OPS * c vector-memory operations are outstanding.
template <int DTL_OPS, int D>
__device__ __forceinline__ void wait_tiles(int c) {
    static_assert(D <= 5, "up to four K tiles after the awaited one");
    switch (c) {
        case 0: wait_vm<0>(); break;
        case 1: wait_vm<DTL_OPS>(); break;
        case 2: if constexpr (D > 2) wait_vm<2 * DTL_OPS>(); else wait_vm<DTL_OPS>(); break;
        case 3: if constexpr (D > 3) wait_vm<3 * DTL_OPS>(); else wait_vm<DTL_OPS>(); break;
        default: if constexpr (D > 4) wait_vm<4 * DTL_OPS>(); else wait_vm<DTL_OPS>(); break;
    }
}

template <int BM, int BK, int NSTAGE, int PL, int QL, int EPI, int TAG>
__global__ __launch_bounds__(NT, 2) void gemm_stream_kernel(GemmArgs a) {
    using TP = STile<BM, PL, BK>;
    using TQ = STile<BN, QL, BK>;
    constexpr int TM = BM / 64;
    constexpr int TN = BN / 64;
    constexpr int NSUB = BK / 16;                                    // MFMA k-steps per K tile
    constexpr int D = NSTAGE - 1;                                    // K tiles loaded ahead
    constexpr int STAGE = TP::BYTES + TQ::BYTES;
    constexpr int DTL_OPS = TP::DTL_PER_WAVE + TQ::DTL_PER_WAVE;    // per wave per K tile
    constexpr int NMFMA = NSUB * TM * TN;                            // per wave per K tile
    static_assert(2 * DTL_OPS <= NMFMA, "one direct-to-LDS load per two MFMAs");
    __shared__ __attribute__((aligned(1024))) char smem[NSTAGE * STAGE];

    // XCD-aware renumbering: hardware hands block b to XCD b % 8
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
    const int nk = (int)((kend - kbeg + BK - 1) / BK);

    const uint16_t* P = reinterpret_cast<const uint16_t*>(a.p);
    const uint16_t* Q = reinterpret_cast<const uint16_t*>(a.q);
    const bool p_al = aligned16(a.p, a.ldp);
    const bool q_al = aligned16(a.q, a.ldq);
    // K tiles 0 .. nk_dtl-1 go direct to LDS: whole tiles of aligned operands
    const int nk_dtl = (p_al && q_al) ? (int)((kend - kbeg) / BK) : 0;
    // Row blocks start their K sweep at different K tiles (rotated by 5 tiles
    // per row block, when every K tile is whole and aligned), so the row
    // blocks running together do not all fetch the same rows of the shared
    // operand at the same moment.  The order of the sum is fixed per tile:
    // results stay bitwise reproducible.
    const int rot = (nk_dtl == nk && nk > 1) ? (int)(((rem / tiles_n) * 5) % nk) : 0;
    auto kofs = [&](int kt) -> int64_t {
        int p = kt + rot;
        if (p >= nk) p -= nk;
        return kbeg + (int64_t)p * BK;
    };

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int wm = wave >> 1;
    const int wn = wave & 1;

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    // Direct-to-LDS instruction r (of DTL_OPS) of K tile kt.
    auto issue_one = [&](int r, int kt) {
        char* As = smem + (kt % NSTAGE) * STAGE;
        const int64_t k0 = kofs(kt);
        if (r < TP::DTL_PER_WAVE) TP::dtl_one(r, As, P, a.ldp, m0, a.M, k0);
        else TQ::dtl_one(r - TP::DTL_PER_WAVE, As + TP::BYTES, Q, a.ldq, n0, a.N, k0);
    };
    // Whole K tile: direct-to-LDS, or the guarded register path (K tail,
    // unaligned operands; LDS written at once).
    auto issue = [&](int kt) {
        char* As = smem + (kt % NSTAGE) * STAGE;
        const int64_t k0 = kofs(kt);
        if (kt < nk_dtl) {
            TP::dtl(As, P, a.ldp, m0, a.M, k0);
            TQ::dtl(As + TP::BYTES, Q, a.ldq, n0, a.N, k0);
        } else {
            TP::load_store(As, P, a.ldp, m0, a.M, k0, kend, p_al);
            TQ::load_store(As + TP::BYTES, Q, a.ldq, n0, a.N, k0, kend, q_al);
        }
    };

    for (int kt = 0; kt < D && kt < nk; ++kt) issue(kt);
    for (int kt = 0; kt < nk; ++kt) {
        // K tile kt is complete once at most the direct-to-LDS operations of
        // the K tiles issued after it are outstanding (vector-memory
        // operations complete in issue order; register-path tiles leave none).
        {
            int after = min(kt + D - 1, nk - 1);
            if (after > nk_dtl - 1) after = nk_dtl - 1;
            wait_tiles<DTL_OPS, D>(after > kt ? after - kt : 0);
        }
        barrier_lds();                               // also: every wave is done with K tile kt-1's stage
        // K tile kt+D goes into the stage K tile kt-1 used.  Direct-to-LDS
        // loads are issued one per two MFMAs below: a burst of them would stall
        // this wave on the address unit's queue while its MFMA unit idles.
        // Register-path tiles are loaded here, at once.
        const bool pf = kt + D < nk_dtl;
        if (kt + D < nk && !pf) issue(kt + D);
        const char* As = smem + (kt % NSTAGE) * STAGE;
        const char* Bs = As + TP::BYTES;
        bf16x8 fa[NSUB][TM], fb[NSUB][TN];
#pragma unroll
        for (int s = 0; s < NSUB; ++s) {
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[s][i] = TP::frag(As, wm * (BM / 2) + 32 * i, s, lane);
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[s][j] = TQ::frag(Bs, wn * (BN / 2) + 32 * j, s, lane);
        }
        // Raised issue priority while this wave runs its MFMAs: the other
        // workgroup's wave on the SIMD fills the gaps with its loads and reads.
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int s = 0; s < NSUB; ++s)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s][i], fb[s][j], acc[i][j], 0, 0, 0);
                    const int n = (s * TM + i) * TN + j;          // MFMA index in this K tile
                    if ((n & 1) == 1 && (n >> 1) < DTL_OPS && pf) issue_one(n >> 1, kt + D);
                }
        __builtin_amdgcn_s_setprio(0);
    }
    epilogue_block<EPI>(a, acc, m0 + wm * (BM / 2), n0 + wn * (BN / 2), lane, split);
}

// K tile and LDS stages: 32 x 3 (72 KB at BM = 256, two K tiles in flight).
// (16 x 6 keeps more bytes in flight but halves the MFMAs between barriers;
// measured slower on MI355X.)
constexpr int kStreamBK = 32;
constexpr int kStreamStages = 3;

template <int BM, int PL, int QL, int EPI, int TAG>
hipError_t launch_s(const GemmArgs& a, hipStream_t s) {
    const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * (int64_t)a.splits;
    if (tiles <= 0) return hipSuccess;
    if (tiles > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((gemm_stream_kernel<BM, kStreamBK, kStreamStages, PL, QL, EPI, TAG>), dim3((unsigned)tiles),
                       dim3(NT), 0, s, a);
    return hipGetLastError();
}

template <int PL, int QL, int EPI, int TAG>
hipError_t launch_sl(const GemmArgs& a, hipStream_t s) {
    if (a.p_layout != PL || a.q_layout != QL || a.epi != EPI) return hipErrorInvalidValue;
    if (a.M > 128) return launch_s<256, PL, QL, EPI, TAG>(a, s);
    return launch_s<128, PL, QL, EPI, TAG>(a, s);
}

}  // namespace

hipError_t launch_gemm_stream(const GemmArgs& a, hipStream_t s) {
    switch (a.tag) {
        case TAG_FWD_Z: return launch_sl<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_Z>(a, s);
        case TAG_INFER_H: return launch_sl<KMAJ, KMAJ, EPI_H, TAG_INFER_H>(a, s);
        case TAG_FWD_Y: return launch_sl<KMAJ, KMAJ, EPI_STORE, TAG_FWD_Y>(a, s);
        case TAG_FWD_YP: return launch_sl<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_YP>(a, s);
        case TAG_BWD_DZ: return launch_sl<KMAJ, MNMAJ, EPI_DZ, TAG_BWD_DZ>(a, s);
        case TAG_BWD_DX: return launch_sl<KMAJ, MNMAJ, EPI_STORE, TAG_BWD_DX>(a, s);
        case TAG_BWD_DA: return launch_sl<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_BWD_DA>(a, s);
        case TAG_BWD_DB: return launch_sl<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_BWD_DB>(a, s);
        case TAG_DENSE_FWD: return launch_sl<KMAJ, KMAJ, EPI_STORE, TAG_DENSE_FWD>(a, s);
        case TAG_DENSE_DX: return launch_sl<KMAJ, MNMAJ, EPI_STORE, TAG_DENSE_DX>(a, s);
        case TAG_DENSE_DW: return launch_sl<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_DENSE_DW>(a, s);
        default: return hipErrorNotSupported;
    }
}

}  // namespace cola
