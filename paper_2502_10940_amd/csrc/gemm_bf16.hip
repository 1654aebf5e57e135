// gemm_bf16.hip -- the bf16 MFMA GEMM behind every CoLA and dense step on
// gfx950:  C[M][N] = sum_k P(m, k) Q(n, k), fp32 accumulation, with a fused
// epilogue (plain store, Z/H with sigma, dZ with sigma', fp32 partials).
//
// Design (CDNA4, wave64):
//  * 256 threads = 4 waves in a 2 x 2 grid; each wave owns a (BM/2) x (BN/2)
//    block of C, computed with v_mfma_f32_32x32x16_bf16 tiles (acc in fp32).
//    Two workgroups share a CU (128 accumulator registers per wave, 48-64 KB
//    of LDS per workgroup), so one workgroup's barriers and memory waits are
//    covered by the other's MFMAs.
//  * K advances in tiles of 64.  Both operand tiles live in LDS as [row][k]
//    with 128-byte rows; the eight 16-byte chunks of a row are XOR-swizzled
//    by (row ^ row >> 3) & 7, so the MFMA fragment reads (16 B per lane) and
//    the tile writes are free of bank conflicts.
//  * Operands with contiguous k (KMAJ) are copied global -> registers -> LDS
//    unchanged.  Operands with k strided (MNMAJ: the weight-gradient GEMMs,
//    whose reduction runs over tokens, and products with the small weight
//    matrices) are loaded as 16-byte runs along m and transposed in registers
//    (8 x 8 blocks of bf16, pure permutes) on their way into LDS, so the MFMA
//    core only ever sees k-contiguous fragments.
//  * One LDS tile per operand: the next K tile's global loads are issued
//    before the current tile's MFMAs and land in registers; they are written
//    to LDS between two barriers once the MFMAs are done with it.
//  * Workgroups are renumbered so that each XCD (blockIdx % 8 on MI355X)
//    receives a contiguous run of output tiles: tiles sharing an operand row
//    block share that XCD's L2.
//  * The epilogue works straight from the accumulator registers (quad
//    transposes, epilogue.hpp); ragged edges and unaligned pitches fall back
//    to guarded per-element accesses.
#include <stdlib.h>
#include <string.h>

#include "internal.hpp"
#include "device_math.hpp"
#include "epilogue.hpp"

namespace cola {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int BK = BF16_BK;   // 64
constexpr int NT = 256;

__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }
__device__ __forceinline__ int lds_off(int row, int chunk) {
    return row * 128 + ((chunk ^ swz(row)) << 4);
}

__device__ __forceinline__ bool aligned16(const void* p, int64_t ld) {
    return ((reinterpret_cast<uintptr_t>(p) & 15u) == 0) && ((ld & 7) == 0);
}

// ---------------------------------------------------------------------------
// operand tile loaders: global -> registers -> LDS tile [R rows][64 k]
// ---------------------------------------------------------------------------
template <int R, int LAYOUT>
struct Loader;

// k contiguous: thread t moves chunks (row t/8 + 32 i, chunk t%8).
template <int R>
struct Loader<R, KMAJ> {
    static constexpr int NV = R / 32;
    uint4 v[NV];

    // fast: the whole tile is in range and 16-byte aligned.  Otherwise each
    // 16-byte chunk is checked: whole chunks in range load as vectors (when
    // aligned), a chunk straddling the K end loads element by element, and
    // chunks out of range read as zero.
    __device__ __forceinline__ void load(const uint16_t* base, int64_t ld, int64_t row0,
                                         int64_t rows, int64_t k0, int64_t kend, bool fast,
                                         bool aligned) {
        const int t = threadIdx.x;
        const int c = t & 7;
        const int r = t >> 3;
        if (fast) {
            const uint16_t* p = base + (row0 + r) * ld + k0 + c * 8;
#pragma unroll
            for (int i = 0; i < NV; ++i)
                v[i] = *reinterpret_cast<const uint4*>(p + (int64_t)(32 * i) * ld);
        } else {
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const int64_t row = row0 + r + 32 * i;
                const int64_t k = k0 + c * 8;
                if (row < rows && k + 8 <= kend && aligned) {
                    v[i] = *reinterpret_cast<const uint4*>(base + row * ld + k);
                } else {
                    uint32_t w[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        uint32_t lo = 0, hi = 0;
                        if (row < rows && k + 2 * e < kend) lo = base[row * ld + k + 2 * e];
                        if (row < rows && k + 2 * e + 1 < kend) hi = base[row * ld + k + 2 * e + 1];
                        w[e] = lo | (hi << 16);
                    }
                    v[i] = make_uint4(w[0], w[1], w[2], w[3]);
                }
            }
        }
    }

    __device__ __forceinline__ void store(char* lds) const {
        const int t = threadIdx.x;
        const int c = t & 7;
        const int r = t >> 3;
#pragma unroll
        for (int i = 0; i < NV; ++i)
            *reinterpret_cast<uint4*>(lds + lds_off(r + 32 * i, c)) = v[i];
    }
};

// k strided: thread covers KR consecutive k rows x 8 consecutive m (one
// 16-byte load per k row), transposes the block in registers, and writes
// KR k-values per m row into the [m][k] LDS tile.
template <int R>
struct Loader<R, MNMAJ> {
    static constexpr int MB = R / 8;        // m blocks per tile
    static constexpr int KB = NT / MB;      // k blocks per tile
    static constexpr int KR = BK / KB;      // k rows per thread: 8 (R=256) or 4 (R=128)
    static_assert(KR == 8 || KR == 4, "unsupported tile");
    uint4 v[KR];

    __device__ __forceinline__ void load(const uint16_t* base, int64_t ld, int64_t row0,
                                         int64_t rows, int64_t k0, int64_t kend, bool fast,
                                         bool aligned) {
        const int t = threadIdx.x;
        const int mb = t % MB;
        const int kb = t / MB;
        const int64_t m = row0 + mb * 8;
        const int64_t k = k0 + kb * KR;
        if (fast) {
            const uint16_t* p = base + k * ld + m;
#pragma unroll
            for (int kk = 0; kk < KR; ++kk)
                v[kk] = *reinterpret_cast<const uint4*>(p + (int64_t)kk * ld);
        } else {
#pragma unroll
            for (int kk = 0; kk < KR; ++kk) {
                if (k + kk < kend && m + 8 <= rows && aligned) {
                    v[kk] = *reinterpret_cast<const uint4*>(base + (k + kk) * ld + m);
                } else {
                    uint32_t w[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        uint32_t lo = 0, hi = 0;
                        if (k + kk < kend && m + 2 * e < rows) lo = base[(k + kk) * ld + m + 2 * e];
                        if (k + kk < kend && m + 2 * e + 1 < rows) hi = base[(k + kk) * ld + m + 2 * e + 1];
                        w[e] = lo | (hi << 16);
                    }
                    v[kk] = make_uint4(w[0], w[1], w[2], w[3]);
                }
            }
        }
    }

    __device__ __forceinline__ void store(char* lds) const {
        const int t = threadIdx.x;
        const int mb = t % MB;
        const int kb = t / MB;
        const int kofs = kb * KR;              // first k of this thread within the tile
        const int chunk = kofs >> 3;
        const int inchunk = (kofs & 7) * 2;    // byte offset inside the chunk (0 or 8)
        uint32_t src[KR][4];
#pragma unroll
        for (int kk = 0; kk < KR; ++kk) {
            src[kk][0] = v[kk].x; src[kk][1] = v[kk].y; src[kk][2] = v[kk].z; src[kk][3] = v[kk].w;
        }
#pragma unroll
        for (int mm = 0; mm < 8; ++mm) {
            const int row = mb * 8 + mm;
            uint32_t d[KR / 2];
#pragma unroll
            for (int pp = 0; pp < KR / 2; ++pp) {
                const uint32_t a = src[2 * pp][mm >> 1];
                const uint32_t b = src[2 * pp + 1][mm >> 1];
                d[pp] = (mm & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
            }
            char* dst = lds + lds_off(row, chunk) + inchunk;
            if constexpr (KR == 8) {
                *reinterpret_cast<uint4*>(dst) = make_uint4(d[0], d[1], d[2], d[3]);
            } else {
                *reinterpret_cast<uint2*>(dst) = make_uint2(d[0], d[1]);
            }
        }
    }
};

// ---------------------------------------------------------------------------
// the kernel
// ---------------------------------------------------------------------------
// TAG is the kernel class (one symbol per step of the layer, so profiles
// name them apart); it does not change the code.
template <int BM, int BN, int PL, int QL, int EPI, int TAG>
__global__ __launch_bounds__(NT, 2) void gemm_bf16_kernel(GemmArgs a) {
    constexpr int TM = BM / 64;   // 32x32 MFMA tiles per wave along m
    constexpr int TN = BN / 64;   // ... along n
    constexpr int TILE = (BM + BN) * 128;
    __shared__ __attribute__((aligned(16))) char smem[TILE];

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
    const bool p_rows_full = m0 + BM <= a.M;
    const bool q_rows_full = n0 + BN <= a.N;

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

    Loader<BM, PL> lp;
    Loader<BN, QL> lq;
    char* As = smem;
    char* Bs = smem + BM * 128;

    if (nk > 0) {
        {
            const bool kfull = kbeg + BK <= kend;
            lp.load(P, a.ldp, m0, a.M, kbeg, kend, p_al && p_rows_full && kfull, p_al);
            lq.load(Q, a.ldq, n0, a.N, kbeg, kend, q_al && q_rows_full && kfull, q_al);
        }
        for (int kt = 0; kt < nk; ++kt) {
            if (kt > 0) __syncthreads();          // everyone is done reading the tile
            lp.store(As);
            lq.store(Bs);
            __syncthreads();                      // the new tile is visible
            if (kt + 1 < nk) {                    // next tile's loads fly during the MFMAs
                const int64_t k0 = kbeg + (int64_t)(kt + 1) * BK;
                const bool kfull = k0 + BK <= kend;
                lp.load(P, a.ldp, m0, a.M, k0, kend, p_al && p_rows_full && kfull, p_al);
                lq.load(Q, a.ldq, n0, a.N, k0, kend, q_al && q_rows_full && kfull, q_al);
            }
#pragma unroll
            for (int s = 0; s < BK / 16; ++s) {
                bf16x8 fa[TM], fb[TN];
                const int chunk = 2 * s + (lane >> 5);
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    fa[i] = *reinterpret_cast<const bf16x8*>(
                        As + lds_off(wm * (BM / 2) + 32 * i + (lane & 31), chunk));
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    fb[j] = *reinterpret_cast<const bf16x8*>(
                        Bs + lds_off(wn * (BN / 2) + 32 * j + (lane & 31), chunk));
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
            }
        }
    }
    // ---- epilogue straight from the accumulators ----
    epilogue_block<EPI>(a, acc, m0 + wm * (BM / 2), n0 + wn * (BN / 2), lane, split);
}

template <int BM, int BN, int PL, int QL, int EPI, int TAG>
hipError_t launch_t(const GemmArgs& a, hipStream_t s) {
    const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * (int64_t)a.splits;
    if (tiles <= 0) return hipSuccess;
    if (tiles > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, PL, QL, EPI, TAG>), dim3((unsigned)tiles), dim3(NT), 0, s, a);
    return hipGetLastError();
}

template <int PL, int QL, int EPI, int TAG>
hipError_t launch_layout(const GemmArgs& a, hipStream_t s) {
    if (a.p_layout != PL || a.q_layout != QL || a.epi != EPI) return hipErrorInvalidValue;
    if (a.M > 128) return launch_t<256, 128, PL, QL, EPI, TAG>(a, s);
    return launch_t<128, 128, PL, QL, EPI, TAG>(a, s);
}

}  // namespace

// The BIG and PP families take only operands with 16-byte aligned rows whose tile
// offsets fit its 32-bit per-lane offsets.
bool big_operands_ok(const GemmArgs& a) {
    auto al = [](const void* p, int64_t ld) {
        return (reinterpret_cast<uintptr_t>(p) & 15u) == 0 && (ld & 7) == 0 && ld < (int64_t(1) << 22);
    };
    return al(a.p, a.ldp) && al(a.q, a.ldq);
}

int gemm_family(int64_t M, int64_t N, int tag) {
    static const int forced = [] {
        const char* e = getenv("COLA_GEMM_FAMILY");
        if (!e) return -1;
        if (!strcmp(e, "reg")) return (int)FAM_REG;
        if (!strcmp(e, "stream")) return (int)FAM_STREAM;
        if (!strcmp(e, "wide")) return (int)FAM_WIDE;
        if (!strcmp(e, "big")) return (int)FAM_BIG;
        if (!strcmp(e, "pp")) return (int)FAM_PP;
        return -1;
    }();
    if (forced == FAM_WIDE || forced == FAM_BIG || forced == FAM_PP) return bf16_wide_ok(M, N) ? forced : (int)FAM_STREAM;
    if (forced >= 0) return forced;
    // 256 x 256 tiles in ping-pong wherever both output dimensions exceed one
    // 128-wide tile (measured on MI355X: 1.1-1.5x the streaming family on
    // the products of the layer, weight gradients included); the streaming
    // family for skinny outputs.
    (void)tag;
    return bf16_wide_ok(M, N) ? (int)FAM_PP : (int)FAM_STREAM;
}

hipError_t launch_gemm_bf16_pair(const GemmArgs& a0, const GemmArgs& a1, hipStream_t s) {
    const bool pp = gemm_family(a0.M, a0.N, a0.tag) == FAM_PP && gemm_family(a1.M, a1.N, a1.tag) == FAM_PP &&
                    big_operands_ok(a0) && big_operands_ok(a1);
    if (pp) return launch_gemm_pp_pair(a0, a1, s);
    hipError_t e = launch_gemm_bf16(a0, s);
    return e == hipSuccess ? launch_gemm_bf16(a1, s) : e;
}

hipError_t launch_gemm_bf16(const GemmArgs& a, hipStream_t s) {
    switch (gemm_family(a.M, a.N, a.tag)) {
        case FAM_WIDE: return launch_gemm_wide(a, s);
        case FAM_BIG: return big_operands_ok(a) ? launch_gemm_big(a, s) : launch_gemm_stream(a, s);
        case FAM_PP: return big_operands_ok(a) ? launch_gemm_pp(a, s) : launch_gemm_stream(a, s);
        case FAM_STREAM: return launch_gemm_stream(a, s);
        default: return launch_gemm_reg(a, s);
    }
}

hipError_t launch_gemm_reg(const GemmArgs& a, hipStream_t s) {
    switch (a.tag) {
        case TAG_FWD_Z: return launch_layout<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_Z>(a, s);
        case TAG_INFER_H: return launch_layout<KMAJ, KMAJ, EPI_H, TAG_INFER_H>(a, s);
        case TAG_FWD_Y: return launch_layout<KMAJ, KMAJ, EPI_STORE, TAG_FWD_Y>(a, s);
        case TAG_FWD_YP: return launch_layout<KMAJ, KMAJ, EPI_Z_H, TAG_FWD_YP>(a, s);
        case TAG_BWD_DZ: return launch_layout<KMAJ, MNMAJ, EPI_DZ, TAG_BWD_DZ>(a, s);
        case TAG_BWD_DX: return launch_layout<KMAJ, MNMAJ, EPI_STORE, TAG_BWD_DX>(a, s);
        case TAG_BWD_DA: return launch_layout<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_BWD_DA>(a, s);
        case TAG_BWD_DB: return launch_layout<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_BWD_DB>(a, s);
        case TAG_DENSE_FWD: return launch_layout<KMAJ, KMAJ, EPI_STORE, TAG_DENSE_FWD>(a, s);
        case TAG_DENSE_DX: return launch_layout<KMAJ, MNMAJ, EPI_STORE, TAG_DENSE_DX>(a, s);
        case TAG_DENSE_DW: return launch_layout<MNMAJ, MNMAJ, EPI_STORE_F32, TAG_DENSE_DW>(a, s);
        default: return hipErrorNotSupported;
    }
}

}  // namespace cola
