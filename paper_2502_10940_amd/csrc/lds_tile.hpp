// lds_tile.hpp -- 256-row operand tiles in LDS for the bf16 MFMA GEMM
// families with 64-deep K tiles (gemm_big.hip, gemm_pp.hip): direct-to-LDS
// buffer loads of whole 128-byte lines, XOR-swizzled layouts, fragment reads
// for v_mfma_f32_32x32x16_bf16, and the scheduling and wait helpers.
//
// Layouts.  k-contiguous operands: [256 rows][BK k], 16-byte chunks
// XOR-swizzled by row, read with ds_read_b128; m-contiguous operands (the
// weight-gradient operands, the weights of the backward products):
// [BK k][256 m], chunks swizzled by 4 (k & 3), read with the transposing
// ds_read_b64_tr_b16.  With gfx950's 64 LDS banks neither read conflicts.
// Each 1 KB block of a tile is one direct-to-LDS instruction (64 lanes x 16
// bytes); four loader waves fill a tile.
#pragma once

#include "internal.hpp"

namespace cola {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef const __attribute__((address_space(1))) void* gptr_t;
typedef __attribute__((address_space(3))) void* lptr_t;
typedef __attribute__((address_space(3))) s16x4* lptr4_t;


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
// The same with a wave-uniform part of the offset in the instruction's scalar
// offset operand.
__device__ __forceinline__ void dtl16s(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, char* lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lptr_t)lds, 16, voff, soff, 0, 0);
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
    static constexpr int DPW = BYTES / 1024 / 4;      // direct-to-LDS instructions per loader wave (4)
    static constexpr int FRAG_READS = 1;              // LDS reads per fragment
    static_assert(CR == 4 || CR == 8, "BK of 32 or 64");

    // chunk c of row r sits at chunk c ^ swz(r): the 16 rows a quarter-wave
    // reads cover all 64 banks once
    __device__ static __forceinline__ int swz(int row) { return (row / (16 / CR)) & (CR - 1); }
    __device__ static __forceinline__ int off(int row, int c) { return row * (2 * BK) + ((c ^ swz(row)) << 4); }

    // Per-lane byte offset of 1 KB block blk of the tile (one direct-to-LDS
    // instruction), relative to the K tile's first element (row0, k0).  Rows
    // past the edge re-read the last row.
    __device__ static __forceinline__ uint32_t voff(int blk, int64_t ld, int64_t row0, int64_t rows) {
        return voff_l(blk, ld, row0, rows, threadIdx.x & 63);
    }
    // the same for an explicit lane (32-bit arithmetic: the tile's rows
    // past the edge are clamped to rows - 1 - row0, which fits an int)
    __device__ static __forceinline__ uint32_t voff_l(int blk, int64_t ld, int64_t row0, int64_t rows, int lane) {
        const int row = RPI * blk + lane / CR;
        const int lc = (lane % CR) ^ swz(row);
        const int64_t lim64 = rows - 1 - row0;
        const int lim = lim64 < 255 ? (int)lim64 : 255;
        const int lrow = row < lim ? row : lim;
        return 2u * ((uint32_t)lrow * (uint32_t)ld + 8u * (uint32_t)lc);
    }
    __device__ static __forceinline__ const char* gbase(const uint16_t* base, int64_t ld, int64_t row0, int64_t k0) {
        return reinterpret_cast<const char*>(base + row0 * ld + k0);
    }

    // voff of an interior tile (every row in range) split in two: a per-lane
    // part that depends on the block only through its parity (the swizzle
    // term repeats every two blocks) and a wave-uniform part.
    __device__ static __forceinline__ bool interior(int64_t row0, int64_t rows) { return row0 + 256 <= rows; }
    __device__ static __forceinline__ uint32_t lane_part(int par, int64_t ld, int lane) {
        const int row = RPI * par + lane / CR;
        return 2u * ((uint32_t)(lane / CR) * (uint32_t)ld + 8u * (uint32_t)((lane % CR) ^ swz(row)));
    }
    __device__ static __forceinline__ uint32_t uniform_part(int blk, int64_t ld) {
        return 2u * (uint32_t)(RPI * blk) * (uint32_t)ld;
    }

    // Guarded register path (partial K tile), NTHR threads: zeros past kend.
    template <int NTHR>
    __device__ static __forceinline__ void load_store(char* lds, const uint16_t* base, int64_t ld, int64_t row0,
                                                      int64_t rows, int64_t k0, int64_t kend) {
#pragma unroll
        for (int i = 0; i < 256 * CR / NTHR; ++i) {
            const int id = threadIdx.x + NTHR * i;
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

    // The same read with its address split into a per-lane part that depends
    // only on the k step s (computed once per kernel) and a wave-uniform part:
    // with row0 a multiple of 32, the swizzle depends on the lane alone, so
    // off(row0 + r, c) = 2 BK row0 + lane_off(s).
    __device__ static __forceinline__ uint32_t lane_off(int s, int lane) {
        const int r = lane & 31;
        return (uint32_t)(r * (2 * BK) + (((2 * s + (lane >> 5)) ^ swz(r)) << 4));
    }
    __device__ static __forceinline__ bf16x8 frag_at(const char* lds, int row0, uint32_t loff) {
        return *reinterpret_cast<const bf16x8*>(lds + row0 * (2 * BK) + loff);
    }
};

// ---- m-contiguous operand: LDS [BK k][256 m] (512-byte rows) ----
template <int BK>
struct BTile<MNMAJ, BK> {
    static constexpr int BYTES = BK * 256 * 2;
    static constexpr int DPW = BYTES / 1024 / 4;
    static constexpr int FRAG_READS = 2;

    __device__ static __forceinline__ int off(int k, int c) { return k * 512 + ((c ^ ((k & 3) << 2)) << 4); }

    // 1 KB block blk fills k rows 2 blk, 2 blk + 1; chunks that start past
    // the last column re-read the last chunk.
    __device__ static __forceinline__ uint32_t voff(int blk, int64_t ld, int64_t m0, int64_t rows) {
        return voff_l(blk, ld, m0, rows, threadIdx.x & 63);
    }
    __device__ static __forceinline__ uint32_t voff_l(int blk, int64_t ld, int64_t m0, int64_t rows, int lane) {
        const int64_t lim64 = (((rows - 1) >> 3) << 3) - m0;       // last chunk, relative to m0
        const int lim = lim64 < 255 * 8 ? (int)lim64 : 255 * 8;
        const int k = 2 * blk + (lane >> 5);
        const int lc = (lane & 31) ^ ((k & 3) << 2);
        const int lm = 8 * lc <= lim ? 8 * lc : lim;
        return 2u * ((uint32_t)k * (uint32_t)ld + (uint32_t)lm);
    }
    __device__ static __forceinline__ const char* gbase(const uint16_t* base, int64_t ld, int64_t m0, int64_t k0) {
        return reinterpret_cast<const char*>(base + k0 * ld + m0);
    }

    // voff of an interior tile (all 256 columns in range, no chunk clamped)
    // split in two: per lane (through the parity of the block, which fixes
    // k & 3 of the lane's row) and wave-uniform.
    __device__ static __forceinline__ bool interior(int64_t m0, int64_t rows) {
        return m0 + 248 <= (((rows - 1) >> 3) << 3);
    }
    __device__ static __forceinline__ uint32_t lane_part(int par, int64_t ld, int lane) {
        const int k = 2 * par + (lane >> 5);
        return 2u * ((uint32_t)(lane >> 5) * (uint32_t)ld + 8u * (uint32_t)((lane & 31) ^ ((k & 3) << 2)));
    }
    __device__ static __forceinline__ uint32_t uniform_part(int blk, int64_t ld) {
        return 2u * (uint32_t)(2 * blk) * (uint32_t)ld;
    }

    template <int NTHR>
    __device__ static __forceinline__ void load_store(char* lds, const uint16_t* base, int64_t ld, int64_t m0,
                                                      int64_t rows, int64_t k0, int64_t kend) {
#pragma unroll
        for (int i = 0; i < BK * 32 / NTHR; ++i) {
            const int id = threadIdx.x + NTHR * i;
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

    // The same read with its address split into a per-lane part for the
    // 32-column block t = m0 / 32 (computed once per kernel) and the k step:
    // with lanes i = lane % 16, g = lane / 16, the byte offset of frag(m0, s)
    // is 8192 s (16 k rows of 512 bytes per k step) plus
    // (8 (g >> 1) + (i >> 2)) 512 + 16 (4 (t ^ y) + x) + 8 (i & 1), with
    // x = 2 (g & 1) + ((i & 3) >> 1) and y = (i >> 2) & 3 (the swizzle term,
    // since 16 s + 8 (g >> 1) is a multiple of 4).
    __device__ static __forceinline__ uint32_t lane_off(int t, int lane) {
        const int g = lane >> 4;
        const int i = lane & 15;
        const int x = 2 * (g & 1) + ((i & 3) >> 1);
        const int y = (i >> 2) & 3;
        return (uint32_t)((8 * (g >> 1) + (i >> 2)) * 512 + 16 * (4 * (t ^ y) + x) + 8 * (i & 1));
    }
    __device__ static __forceinline__ bf16x8 frag_at(const char* lds, int s, uint32_t loff) {
        const char* p = lds + 8192 * s + loff;
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lptr4_t)p);
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lptr4_t)(p + 2048));
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


}  // namespace
}  // namespace cola
