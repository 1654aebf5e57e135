// epilogue.hpp -- the fused GEMM epilogues shared by the bf16 MFMA kernels.
//
// The pointwise part of the layer (rounding, sigma, sigma', the CoLA-M
// recompute of H) happens here, straight from the accumulator registers: no
// LDS staging, so the epilogue neither waits on LDS nor on the global stores
// still in flight, and its stores drain while the CU runs other MFMAs.
//
// Accumulator layout of v_mfma_f32_32x32x16_bf16: lane l, register v holds
// row 8 (v / 4) + 4 (l / 32) + v % 4, column l % 32 of the 32 x 32 tile.  For
// each group of four registers (v = 4g .. 4g+3) the four lanes of a quad hold
// a 4 x 4 block (lane = column, register = row); a two-stage exchange inside
// the quad (DPP quad permutations) transposes it, so that lane 4q + b then
// holds row 8g + 4 (l / 32) + b, columns 4q .. 4q+3: four consecutive outputs
// of one row, written with one 8-byte (bf16) or 16-byte (fp32) store.  One
// store instruction covers 8 rows x 64 contiguous bytes (bf16).
//
// Plain (not non-temporal) stores: on MI355X they sustain more bandwidth,
// 6.5 against 5.5 TB/s for a 128 MB write in this tile pattern.
#pragma once

#include "internal.hpp"
#include "device_math.hpp"

namespace cola {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// DPP quad permutations: lane 4q + i reads lane 4q + p[i].
constexpr int kQuadSwap2 = 0x4E;   // p = [2, 3, 0, 1]
constexpr int kQuadSwap1 = 0xB1;   // p = [1, 0, 3, 2]

template <int CTRL>
__device__ __forceinline__ uint32_t quad_perm(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float quad_perm(float v) {
    return __uint_as_float(quad_perm<CTRL>(__float_as_uint(v)));
}

// Per-lane byte selectors (v_perm_b32) of the 16-bit exchange.
struct QuadSel {
    bool hi2;          // lane bit 1
    uint32_t send, q0, q1;
    __device__ __forceinline__ explicit QuadSel(int lane) {
        hi2 = (lane & 2) != 0;
        const bool odd = (lane & 1) != 0;
        send = odd ? 0x05040100u : 0x07060302u;   // odd lanes send the low halves, even the high
        q0 = odd ? 0x03020504u : 0x05040100u;
        q1 = odd ? 0x03020706u : 0x07060100u;
    }
};

// Transpose of a quad's 4 x 4 block of bf16.  In: p01 = rows 0,1 and p23 =
// rows 2,3 of this lane's column (low half = lower row).  Out: row (lane & 3),
// columns 0,1 in q0 and 2,3 in q1 (low half = lower column).
__device__ __forceinline__ void transpose_bf16(const QuadSel& s, uint32_t p01, uint32_t p23,
                                               uint32_t& q0, uint32_t& q1) {
    // stage 1: lanes b and b^2 swap row pairs
    const uint32_t r = quad_perm<kQuadSwap2>(s.hi2 ? p01 : p23);
    const uint32_t d0 = s.hi2 ? r : p01;
    const uint32_t d1 = s.hi2 ? p23 : r;
    // stage 2: lanes b and b^1 swap 16-bit halves
    const uint32_t t = quad_perm<kQuadSwap1>(__builtin_amdgcn_perm(d1, d0, s.send));
    q0 = __builtin_amdgcn_perm(t, d0, s.q0);
    q1 = __builtin_amdgcn_perm(t, d1, s.q1);
}

// Transpose of a quad's 4 x 4 block of floats: in x[k] = row k of this lane's
// column; out y[k] = column k of this lane's row.
__device__ __forceinline__ void transpose_f32(int lane, const float x[4], float y[4]) {
    const bool hi2 = (lane & 2) != 0;
    const bool odd = (lane & 1) != 0;
    const float r0 = quad_perm<kQuadSwap2>(hi2 ? x[0] : x[2]);
    const float r1 = quad_perm<kQuadSwap2>(hi2 ? x[1] : x[3]);
    const float z0 = hi2 ? r0 : x[0];
    const float z1 = hi2 ? r1 : x[1];
    const float z2 = hi2 ? x[2] : r0;
    const float z3 = hi2 ? x[3] : r1;
    const float s0 = quad_perm<kQuadSwap1>(odd ? z0 : z1);
    const float s1 = quad_perm<kQuadSwap1>(odd ? z2 : z3);
    y[0] = odd ? s0 : z0;
    y[1] = odd ? z1 : s0;
    y[2] = odd ? s1 : z2;
    y[3] = odd ? z3 : s1;
}

// Lanes l and l ^ 4 (quads q and q ^ 1 of a 16-lane DPP row) exchange one
// dword: the lane with bit 2 clear receives its partner's v from lane l + 4
// (row_shl:4), the other from lane l - 4 (row_shr:4).
__device__ __forceinline__ uint32_t swap_pair(uint32_t v, bool odd) {
    const uint32_t up = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x104, 0xF, 0xF, false);
    const uint32_t dn = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);
    return odd ? dn : up;
}

// Two horizontally adjacent 32 x 32 tiles (j, j + 1) after the quad
// transposes: lane 4q + b holds columns 4q .. 4q+3 of tile j in a0, a1 and of
// tile j + 1 in b0, b1.  Quad pairs (q, q ^ 1) trade halves so that the even
// quad holds columns 8m .. 8m+7 of tile j and the odd one those of tile j + 1
// (m = q / 2): 16 bytes per lane, and one store instruction writes 8 whole
// rows of 128 contiguous bytes (the two tiles' 64 columns).  Returns the
// column (relative to tile j) of the lane's first element.
__device__ __forceinline__ int pair_tiles(int lane, uint32_t a0, uint32_t a1, uint32_t b0, uint32_t b1,
                                          u32x4_t& out) {
    const int q = (lane & 31) >> 2;
    const bool odd = (q & 1) != 0;
    const uint32_t r0 = swap_pair(odd ? a0 : b0, odd);
    const uint32_t r1 = swap_pair(odd ? a1 : b1, odd);
    out = odd ? u32x4_t{r0, r1, b0, b1} : u32x4_t{a0, a1, r0, r1};
    return 32 * (q & 1) + 8 * (q >> 1);
}

// Four bf16 (q0 = columns 0,1, q1 = columns 2,3) to p: one 8-byte store when
// vec, else the first `valid` elements one by one.
__device__ __forceinline__ void store_bf16x4(uint16_t* p, uint32_t q0, uint32_t q1, bool vec, int valid) {
    if (vec) {
        *reinterpret_cast<u32x2_t*>(p) = u32x2_t{q0, q1};
    } else {
        if (valid > 0) p[0] = (uint16_t)(q0 & 0xffffu);
        if (valid > 1) p[1] = (uint16_t)(q0 >> 16);
        if (valid > 2) p[2] = (uint16_t)(q1 & 0xffffu);
        if (valid > 3) p[3] = (uint16_t)(q1 >> 16);
    }
}

// Z (bf16) at 4 consecutive columns gn .. gn+3 of row gm, packed as two
// bf16 pairs; columns past the edge read as 0.  (EPI_DZ)
__device__ __forceinline__ u32x2_t load_z4(const GemmArgs& a, int64_t gm, int64_t gn) {
    if (gm >= a.M || gn >= a.N) return u32x2_t{0u, 0u};
    const int valid = (int)((a.N - gn) < 4 ? (a.N - gn) : 4);
    const uint16_t* zp = reinterpret_cast<const uint16_t*>(a.zin) + gm * a.ldzin + gn;
    if (valid == 4 && (reinterpret_cast<uintptr_t>(zp) & 7u) == 0) return *reinterpret_cast<const u32x2_t*>(zp);
    uint32_t e[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) e[k] = k < valid ? (uint32_t)zp[k] : 0u;
    return u32x2_t{e[0] | (e[1] << 16), e[2] | (e[3] << 16)};
}

// Epilogue of 4 consecutive columns (gn .. gn+3) of output row gm; zz: the
// matching Z values (EPI_DZ only).  FAST: the 4 columns exist and every
// pointer is aligned for one vector access (checked once per block).  ACT:
// the activation (a.act, fixed per instantiation).
template <int EPI, bool FAST, int ACT>
__device__ __forceinline__ void epilogue4(const GemmArgs& a, int64_t gm, int64_t gn, const float v[4], int split,
                                          u32x2_t zz = u32x2_t{0u, 0u}) {
    if (!FAST && (gm >= a.M || gn >= a.N)) return;
    const int valid = FAST ? 4 : (int)((a.N - gn) < 4 ? (a.N - gn) : 4);
    if constexpr (EPI == EPI_STORE_F32) {
        float* c = reinterpret_cast<float*>(a.c) + (int64_t)split * a.split_stride + gm * a.ldc + gn;
        if (FAST || (valid == 4 && (reinterpret_cast<uintptr_t>(c) & 15u) == 0)) {
            *reinterpret_cast<f32x4_t*>(c) = f32x4_t{v[0], v[1], v[2], v[3]};
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (e < valid) c[e] = v[e];
        }
    } else {
        uint16_t* c = reinterpret_cast<uint16_t*>(a.c) + gm * a.ldc + gn;
        float out[4], h[4];
        if constexpr (EPI == EPI_STORE) {
#pragma unroll
            for (int e = 0; e < 4; ++e) out[e] = v[e];
        } else if constexpr (EPI == EPI_Z_H) {
            // Z is stored rounded to bf16; H = sigma of that rounded Z
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                out[e] = round_bf16(v[e]);
                h[e] = act_sigma_c<ACT, true>(out[e]);
            }
        } else if constexpr (EPI == EPI_H) {
            // the H of EPI_Z_H: sigma of Z rounded to bf16
#pragma unroll
            for (int e = 0; e < 4; ++e) out[e] = act_sigma_c<ACT, true>(round_bf16(v[e]));
        } else if constexpr (EPI == EPI_DZ) {
            const float z[4] = {bf16_to_f32(zz[0] & 0xffffu), bf16_to_f32(zz[0] >> 16),
                                bf16_to_f32(zz[1] & 0xffffu), bf16_to_f32(zz[1] >> 16)};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float sp;
                act_sigma_both_c<ACT, true>(z[e], h[e], sp);
                out[e] = ACT == 0 ? v[e] : v[e] * sp;
            }
        }
        const bool vec = FAST || (valid == 4 && (reinterpret_cast<uintptr_t>(c) & 7u) == 0);
        store_bf16x4(c, pack_bf16x2(out[0], out[1]), pack_bf16x2(out[2], out[3]), vec, valid);
        if constexpr (EPI == EPI_Z_H || EPI == EPI_DZ) {
            if (a.aux) {
                uint16_t* hp = reinterpret_cast<uint16_t*>(a.aux) + gm * a.ldaux + gn;
                const bool hvec = FAST || (valid == 4 && (reinterpret_cast<uintptr_t>(hp) & 7u) == 0);
                store_bf16x4(hp, pack_bf16x2(h[0], h[1]), pack_bf16x2(h[2], h[3]), hvec, valid);
            }
        }
    }
}

// Z for the lane's 4 columns of row gm (FAST: one unguarded vector load).
template <bool FAST>
__device__ __forceinline__ u32x2_t z4(const GemmArgs& a, int64_t gm, int64_t gn) {
    if constexpr (FAST)
        return *reinterpret_cast<const u32x2_t*>(reinterpret_cast<const uint16_t*>(a.zin) + gm * a.ldzin + gn);
    else
        return load_z4(a, gm, gn);
}

// Interior blocks with 16-byte aligned rows (bf16 outputs): the quad
// transposes of tile pairs, then whole 128-byte row segments per store.
// Bitwise the values of the 8-byte path (same roundings, same sigma).
template <int EPI, int ACT, int TM, int TN>
__device__ __forceinline__ void epilogue_lines(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int64_t row0,
                                               int64_t col0, int lane) {
    static_assert(TN % 2 == 0, "tile pairs");
    static_assert(EPI == EPI_STORE || EPI == EPI_H || EPI == EPI_Z_H, "bf16 stores without an input");
    const int64_t lrow = 4 * (lane >> 5) + (lane & 3);
    const QuadSel sel(lane);
    uint16_t* C = reinterpret_cast<uint16_t*>(a.c);
    uint16_t* Hp = reinterpret_cast<uint16_t*>(a.aux);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int jp = 0; jp < TN / 2; ++jp) {
                const int64_t gm = row0 + 32 * i + 8 * g + lrow;
                uint32_t c[2][2], h[2][2];
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    const f32x16& v = acc[i][2 * jp + t];
                    float x[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        x[e] = v[4 * g + e];
                        if constexpr (EPI == EPI_H) x[e] = act_sigma_c<ACT, true>(round_bf16(x[e]));
                    }
                    transpose_bf16(sel, pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), c[t][0], c[t][1]);
                    if constexpr (EPI == EPI_Z_H) {
                        float y[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) y[e] = act_sigma_c<ACT, true>(round_bf16(x[e]));
                        transpose_bf16(sel, pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]), h[t][0], h[t][1]);
                    }
                }
                u32x4_t o;
                const int dc = pair_tiles(lane, c[0][0], c[0][1], c[1][0], c[1][1], o);
                const int64_t gn = col0 + 64 * jp + dc;
                *reinterpret_cast<u32x4_t*>(C + gm * a.ldc + gn) = o;
                if constexpr (EPI == EPI_Z_H) {
                    if (Hp) {
                        pair_tiles(lane, h[0][0], h[0][1], h[1][0], h[1][1], o);
                        *reinterpret_cast<u32x4_t*>(Hp + gm * a.ldaux + gn) = o;
                    }
                }
            }
}

template <int EPI, bool FAST, int ACT, int TM, int TN>
__device__ __forceinline__ void epilogue_block_impl(const GemmArgs& a, const f32x16 (&acc)[TM][TN],
                                                    int64_t row0, int64_t col0, int lane, int split) {
    const int64_t lrow = 4 * (lane >> 5) + (lane & 3);     // this lane's row within a group of 8
    const int64_t lcol = 4 * ((lane & 31) >> 2);           // its first column within a tile
    if constexpr (EPI == EPI_STORE || EPI == EPI_H) {
        // round to bf16 first, then transpose 16-bit pairs (half the exchange
        // work); sigma is elementwise, so EPI_H applies it before the transpose
        const QuadSel sel(lane);
        auto f = [&](float v) { return EPI == EPI_H ? act_sigma_c<ACT, true>(round_bf16(v)) : v; };
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    uint32_t q0, q1;
                    transpose_bf16(sel, pack_bf16x2(f(acc[i][j][4 * g]), f(acc[i][j][4 * g + 1])),
                                   pack_bf16x2(f(acc[i][j][4 * g + 2]), f(acc[i][j][4 * g + 3])), q0, q1);
                    const int64_t gm = row0 + 32 * i + 8 * g + lrow;
                    const int64_t gn = col0 + 32 * j + lcol;
                    uint16_t* c = reinterpret_cast<uint16_t*>(a.c) + gm * a.ldc + gn;
                    if (FAST) {
                        *reinterpret_cast<u32x2_t*>(c) = u32x2_t{q0, q1};
                    } else if (gm < a.M && gn < a.N) {
                        const int valid = (int)((a.N - gn) < 4 ? (a.N - gn) : 4);
                        store_bf16x4(c, q0, q1, valid == 4 && (reinterpret_cast<uintptr_t>(c) & 7u) == 0, valid);
                    }
                }
    } else if constexpr (EPI == EPI_DZ) {
        // Z for row tile i+1 is loaded before row tile i's stores: loads and
        // stores share one wait counter, so waiting for a Z load issued after
        // a store would also wait for that store.
        u32x2_t zb[2][4][TN];
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int j = 0; j < TN; ++j) zb[0][g][j] = z4<FAST>(a, row0 + 8 * g + lrow, col0 + 32 * j + lcol);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            if (i + 1 < TM) {
#pragma unroll
                for (int g = 0; g < 4; ++g)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        zb[(i + 1) & 1][g][j] = z4<FAST>(a, row0 + 32 * (i + 1) + 8 * g + lrow, col0 + 32 * j + lcol);
            }
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const float x[4] = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                                        acc[i][j][4 * g + 3]};
                    float y[4];
                    transpose_f32(lane, x, y);
                    epilogue4<EPI, FAST, ACT>(a, row0 + 32 * i + 8 * g + lrow, col0 + 32 * j + lcol, y, split,
                                              zb[i & 1][g][j]);
                }
        }
    } else {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const float x[4] = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                                        acc[i][j][4 * g + 3]};
                    float y[4];
                    transpose_f32(lane, x, y);
                    epilogue4<EPI, FAST, ACT>(a, row0 + 32 * i + 8 * g + lrow, col0 + 32 * j + lcol, y, split);
                }
    }
}

// The whole epilogue of one wave's block of TM x TN MFMA tiles, whose first
// output row and column are row0, col0, for activation ACT.  Blocks wholly
// inside the output with aligned pointers (the common case) take the
// unguarded vector path.
template <int EPI, int ACT, int TM, int TN>
__device__ __forceinline__ void epilogue_block_act(const GemmArgs& a, const f32x16 (&acc)[TM][TN],
                                               int64_t row0, int64_t col0, int lane, int split) {
    auto al = [](const void* p, int64_t ld, int64_t elems) {   // rows of elems-element vectors
        return p != nullptr && (reinterpret_cast<uintptr_t>(p) % (2 * elems)) == 0 && ld % elems == 0;
    };
    bool fast = row0 + 32 * TM <= a.M && col0 + 32 * TN <= a.N;
    if constexpr (EPI == EPI_STORE_F32) {
        const float* c = reinterpret_cast<const float*>(a.c) + (int64_t)split * a.split_stride;
        fast = fast && (reinterpret_cast<uintptr_t>(c) & 15u) == 0 && a.ldc % 4 == 0;
    } else {
        fast = fast && al(a.c, a.ldc, 4);
    }
    if constexpr (EPI == EPI_Z_H || EPI == EPI_DZ) fast = fast && (a.aux == nullptr || al(a.aux, a.ldaux, 4));
    if constexpr (EPI == EPI_DZ) fast = fast && al(a.zin, a.ldzin, 4);
    if constexpr ((EPI == EPI_STORE || EPI == EPI_H || EPI == EPI_Z_H) && TN % 2 == 0) {
        // 16-byte rows: whole 128-byte row segments per store
        bool line = fast && al(a.c, a.ldc, 8);
        if constexpr (EPI == EPI_Z_H) line = line && (a.aux == nullptr || al(a.aux, a.ldaux, 8));
        if (line) {
            epilogue_lines<EPI, ACT>(a, acc, row0, col0, lane);
            return;
        }
    }
    if (fast) epilogue_block_impl<EPI, true, ACT>(a, acc, row0, col0, lane, split);
    else epilogue_block_impl<EPI, false, ACT>(a, acc, row0, col0, lane, split);
}

// The epilogue of a wave's block with the activation a.act chosen once here
// (epilogues without sigma ignore it).
template <int EPI, int TM, int TN>
__device__ __forceinline__ void epilogue_block(const GemmArgs& a, const f32x16 (&acc)[TM][TN],
                                               int64_t row0, int64_t col0, int lane, int split) {
    if constexpr (EPI == EPI_STORE || EPI == EPI_STORE_F32) {
        epilogue_block_act<EPI, 0>(a, acc, row0, col0, lane, split);
    } else {
        if (a.act == 0) epilogue_block_act<EPI, 0>(a, acc, row0, col0, lane, split);
        else if (a.act == 2) epilogue_block_act<EPI, 2>(a, acc, row0, col0, lane, split);
        else epilogue_block_act<EPI, 1>(a, acc, row0, col0, lane, split);
    }
}

// ---------------------------------------------------------------------------
// Transposed accumulators.  A kernel that gives the MFMA the Q fragment as its
// first operand holds the tiles of C^T: lane l, register v of tile (i, j) is
// element (32 i + l % 32, 32 j + 8 (v / 4) + 4 (l / 32) + v % 4) of the
// wave's block, so every group of four registers is four consecutive columns
// of one row.  Two lane exchanges (no transposes) make the stores wide:
//  1. v_permlane32_swap (lanes 32-63 of one register with lanes 0-31 of
//     another) on the register groups 2p and 2p + 1 leaves lane l with the
//     eight columns 16 p + 8 (l / 32) + 0..7 of row l % 32;
//  2. v_permlane16_swap (lanes 16-31 / 48-63 of one register with lanes
//     0-15 / 32-47 of another) on the pieces p = 0 and p = 1 leaves lane l
//     with columns 16 ((l / 16) % 2) + 8 (l / 32) + 0..7 of row l % 16 (piece
//     X) and of row 16 + l % 16 (piece Y).
// One 16-byte store (bf16) per piece then writes 16 rows x 64 contiguous
// bytes, which sustains the full store rate of a CU (as 8 rows x 128 bytes
// does; 32 rows x 32 bytes is slower).  fp32 outputs take a third exchange
// and two stores per piece, again 16 rows x 64 contiguous bytes each.  Same roundings and sigma as the epilogues above, so the values are
// bitwise those of the other families.

// x (lanes 32-63) <-> y (lanes 0-31)
__device__ __forceinline__ void swap_halves(uint32_t& x, uint32_t& y) {
    const auto r = __builtin_amdgcn_permlane32_swap(x, y, false, false);
    x = r[0];
    y = r[1];
}
// x (lanes 16-31, 48-63) <-> y (lanes 0-15, 32-47)
__device__ __forceinline__ void swap_rows16(uint32_t& x, uint32_t& y) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, y, false, false);
    x = r[0];
    y = r[1];
}

// Eight bf16 (packed pairs w[0..3], lower column in the low half) to row gm,
// columns gn .. gn+7 of a bf16 matrix; FAST: in bounds and 16-byte aligned.
template <bool FAST>
__device__ __forceinline__ void store_bf16x8(uint16_t* base, int64_t ld, int64_t M, int64_t N, int64_t gm,
                                             int64_t gn, const uint32_t w[4]) {
    uint16_t* p = base + gm * ld + gn;
    if constexpr (FAST) {
        *reinterpret_cast<u32x4_t*>(p) = u32x4_t{w[0], w[1], w[2], w[3]};
    } else {
        if (gm >= M) return;
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (gn + e < N) p[e] = (uint16_t)((w[e >> 1] >> (16 * (e & 1))) & 0xffffu);
    }
}

// Four fp32 (bit patterns) to row gm, columns gn .. gn+3; FAST as above.
template <bool FAST>
__device__ __forceinline__ void store_f32x4(float* base, int64_t ld, int64_t M, int64_t N, int64_t gm, int64_t gn,
                                            const uint32_t* w) {
    float* p = base + gm * ld + gn;
    if constexpr (FAST) {
        *reinterpret_cast<u32x4_t*>(p) = u32x4_t{w[0], w[1], w[2], w[3]};
    } else {
        if (gm >= M) return;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (gn + e < N) p[e] = __uint_as_float(w[e]);
    }
}

// Eight bf16 of row gm, columns gn .. gn+7 (packed pairs); past the edges 0.
template <bool FAST>
__device__ __forceinline__ u32x4_t load_bf16x8(const uint16_t* base, int64_t ld, int64_t M, int64_t N, int64_t gm,
                                               int64_t gn) {
    const uint16_t* p = base + gm * ld + gn;
    if constexpr (FAST) {
        return *reinterpret_cast<const u32x4_t*>(p);
    } else {
        uint32_t e[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) e[k] = (gm < M && gn + k < N) ? (uint32_t)p[k] : 0u;
        return u32x4_t{e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16), e[6] | (e[7] << 16)};
    }
}

template <int EPI, int ACT, bool FAST, int TM, int TN>
__device__ __forceinline__ void epilogue_t_impl(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int64_t row0,
                                                int64_t col0, int lane, int split) {
    // after exchange 1: row l % 32, columns 16 p + h1 ..
    const int r1 = lane & 31;
    const int h1 = 8 * (lane >> 5);
    // after exchange 2: rows l % 16 (X) and 16 + l % 16 (Y), columns c2 ..
    const int r2 = lane & 15;
    const int c2 = 16 * ((lane >> 4) & 1) + 8 * (lane >> 5);
    uint16_t* C = reinterpret_cast<uint16_t*>(a.c);
    uint16_t* Hp = reinterpret_cast<uint16_t*>(a.aux);
    const uint16_t* Zp = reinterpret_cast<const uint16_t*>(a.zin);
    // EPI_DZ (Z), EPI_GATE (g): the input (in the layout after exchange 1) of
    // tile row i + 1 is loaded before the stores of tile row i (loads and
    // stores share one wait counter, so waiting for a load issued after a
    // store also waits for that store)
    constexpr bool kIn = EPI == EPI_DZ || EPI == EPI_GATE;
    u32x4_t zb[2][TN][2];
    auto zload = [&](int i, u32x4_t (&z)[TN][2]) {
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int p = 0; p < 2; ++p)
                z[j][p] = load_bf16x8<FAST>(Zp, a.ldzin, a.M, a.N, row0 + 32 * i + r1, col0 + 32 * j + 16 * p + h1);
    };
    if constexpr (kIn) zload(0, zb[0]);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        if constexpr (kIn) {
            if (i + 1 < TM) zload(i + 1, zb[(i + 1) & 1]);
        }
        const int64_t gx = row0 + 32 * i + r2;     // row of piece X (Y: gx + 16)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const f32x16& v = acc[i][j];
            if constexpr (EPI == EPI_STORE_F32) {
                uint32_t w[2][8];
#pragma unroll
                for (int p = 0; p < 2; ++p)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        w[p][e] = __float_as_uint(v[8 * p + e]);
                        w[p][4 + e] = __float_as_uint(v[8 * p + 4 + e]);
                        swap_halves(w[p][e], w[p][4 + e]);
                    }
#pragma unroll
                for (int e = 0; e < 8; ++e) swap_rows16(w[0][e], w[1][e]);
                // exchange 3 (fp32 only): within each piece, lanes l and l + 16
                // trade columns 4..7 and 16..19 of their eight, so that lane l
                // holds columns 4 (l / 16) + 0..3 and 16 + 4 (l / 16) + 0..3:
                // each 16-byte store then writes 16 rows x 64 contiguous bytes
#pragma unroll
                for (int p = 0; p < 2; ++p)
#pragma unroll
                    for (int e = 0; e < 4; ++e) swap_rows16(w[p][e], w[p][4 + e]);
                float* c = reinterpret_cast<float*>(a.c) + (int64_t)split * a.split_stride;
                const int64_t gf = col0 + 32 * j + 4 * (lane >> 4);
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    store_f32x4<FAST>(c, a.ldc, a.M, a.N, gx + 16 * p, gf, &w[p][0]);
                    store_f32x4<FAST>(c, a.ldc, a.M, a.N, gx + 16 * p, gf + 16, &w[p][4]);
                }
            } else {
                const int64_t gn = col0 + 32 * j + c2;
                uint32_t o[2][4], h[2][4];
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    if constexpr (EPI == EPI_DZ) {
                        // exchange 1 on the fp32 values, then sigma' of the
                        // matching Z
                        uint32_t w[8];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            w[e] = __float_as_uint(v[8 * p + e]);
                            w[4 + e] = __float_as_uint(v[8 * p + 4 + e]);
                            swap_halves(w[e], w[4 + e]);
                        }
                        const u32x4_t z = zb[i & 1][j][p];
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            float ov[2], hv[2];
#pragma unroll
                            for (int e = 0; e < 2; ++e) {
                                const float ze = bf16_to_f32(e == 0 ? (z[q] & 0xffffu) : (z[q] >> 16));
                                float sp;
                                act_sigma_both_c<ACT, true>(ze, hv[e], sp);
                                const float x = __uint_as_float(w[2 * q + e]);
                                ov[e] = ACT == 0 ? x : x * sp;
                            }
                            o[p][q] = pack_bf16x2(ov[0], ov[1]);
                            h[p][q] = pack_bf16x2(hv[0], hv[1]);
                        }
                    } else {
                        // elementwise: round and pack first, then exchange 1
                        // on the packed pairs (half the exchanges)
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const int r = 8 * p + 2 * q;        // registers r, r + 1
                            const uint32_t zz = pack_bf16x2(v[r], v[r + 1]);
                            if constexpr (EPI == EPI_STORE || EPI == EPI_GATE) {
                                o[p][q] = zz;
                            } else {
                                // sigma of the rounded values
                                const float z0 = __uint_as_float(zz << 16);
                                const float z1 = __uint_as_float(zz & 0xffff0000u);
                                const uint32_t hh =
                                    pack_bf16x2(act_sigma_c<ACT, true>(z0), act_sigma_c<ACT, true>(z1));
                                if constexpr (EPI == EPI_H) {
                                    o[p][q] = hh;
                                } else {
                                    o[p][q] = zz;
                                    h[p][q] = hh;
                                }
                            }
                        }
                        swap_halves(o[p][0], o[p][2]);
                        swap_halves(o[p][1], o[p][3]);
                        if constexpr (EPI == EPI_Z_H) {
                            swap_halves(h[p][0], h[p][2]);
                            swap_halves(h[p][1], h[p][3]);
                        }
                        if constexpr (EPI == EPI_GATE) {
                            // m = g u of the rounded u (o after exchange 1
                            // matches the layout of g)
                            const u32x4_t g = zb[i & 1][j][p];
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                const float y0 = __uint_as_float(o[p][q] << 16);
                                const float y1 = __uint_as_float(o[p][q] & 0xffff0000u);
                                const float g0 = __uint_as_float(g[q] << 16);
                                const float g1 = __uint_as_float(g[q] & 0xffff0000u);
                                h[p][q] = pack_bf16x2(g0 * y0, g1 * y1);
                            }
                        }
                    }
                }
                // exchange 2, then one store per piece (EPI_GATE without a
                // first output stores only m)
                if (EPI != EPI_GATE || C != nullptr) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) swap_rows16(o[0][q], o[1][q]);
                    store_bf16x8<FAST>(C, a.ldc, a.M, a.N, gx, gn, o[0]);
                    store_bf16x8<FAST>(C, a.ldc, a.M, a.N, gx + 16, gn, o[1]);
                }
                if constexpr (EPI == EPI_Z_H || EPI == EPI_DZ || EPI == EPI_GATE) {
                    if (Hp) {
#pragma unroll
                        for (int q = 0; q < 4; ++q) swap_rows16(h[0][q], h[1][q]);
                        store_bf16x8<FAST>(Hp, a.ldaux, a.M, a.N, gx, gn, h[0]);
                        store_bf16x8<FAST>(Hp, a.ldaux, a.M, a.N, gx + 16, gn, h[1]);
                    }
                }
            }
        }
    }
}

// EPI_DGATE: with dm = round(acc), c = round(dm u) and aux = round(dm g).
// Same exchanges and stores as the elementwise epilogues above; the inputs
// g and u of one 32 x 32 tile are loaded a tile ahead (a whole tile row
// ahead, as EPI_DZ does, would need twice the registers for two inputs).
template <bool FAST, int TM, int TN>
__device__ __forceinline__ void epilogue_t_dgate(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int64_t row0,
                                                 int64_t col0, int lane) {
    const int r1 = lane & 31;
    const int h1 = 8 * (lane >> 5);
    const int r2 = lane & 15;
    const int c2 = 16 * ((lane >> 4) & 1) + 8 * (lane >> 5);
    uint16_t* C = reinterpret_cast<uint16_t*>(a.c);
    uint16_t* Dp = reinterpret_cast<uint16_t*>(a.aux);
    const uint16_t* Gp = reinterpret_cast<const uint16_t*>(a.zin);
    const uint16_t* Up = reinterpret_cast<const uint16_t*>(a.zin2);
    u32x4_t gb[2][2], ub[2][2];              // [tile parity][piece p]
    auto load = [&](int t, int buf) {
        const int i = t / TN, j = t % TN;
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            gb[buf][p] = load_bf16x8<FAST>(Gp, a.ldzin, a.M, a.N, row0 + 32 * i + r1, col0 + 32 * j + 16 * p + h1);
            ub[buf][p] = load_bf16x8<FAST>(Up, a.ldzin2, a.M, a.N, row0 + 32 * i + r1, col0 + 32 * j + 16 * p + h1);
        }
    };
    load(0, 0);
#pragma unroll
    for (int t = 0; t < TM * TN; ++t) {
        const int i = t / TN, j = t % TN;
        if (t + 1 < TM * TN) load(t + 1, (t + 1) & 1);
        const f32x16& v = acc[i][j];
        uint32_t o[2][4], h[2][4];
#pragma unroll
        for (int p = 0; p < 2; ++p) {
#pragma unroll
            for (int q = 0; q < 4; ++q) o[p][q] = pack_bf16x2(v[8 * p + 2 * q], v[8 * p + 2 * q + 1]);
            swap_halves(o[p][0], o[p][2]);
            swap_halves(o[p][1], o[p][3]);
            const u32x4_t g = gb[t & 1][p], u = ub[t & 1][p];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float y0 = __uint_as_float(o[p][q] << 16);
                const float y1 = __uint_as_float(o[p][q] & 0xffff0000u);
                h[p][q] = pack_bf16x2(y0 * __uint_as_float(g[q] << 16), y1 * __uint_as_float(g[q] & 0xffff0000u));
                o[p][q] = pack_bf16x2(y0 * __uint_as_float(u[q] << 16), y1 * __uint_as_float(u[q] & 0xffff0000u));
            }
        }
        const int64_t gx = row0 + 32 * i + r2;
        const int64_t gn = col0 + 32 * j + c2;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            swap_rows16(o[0][q], o[1][q]);
            swap_rows16(h[0][q], h[1][q]);
        }
        store_bf16x8<FAST>(C, a.ldc, a.M, a.N, gx, gn, o[0]);
        store_bf16x8<FAST>(C, a.ldc, a.M, a.N, gx + 16, gn, o[1]);
        store_bf16x8<FAST>(Dp, a.ldaux, a.M, a.N, gx, gn, h[0]);
        store_bf16x8<FAST>(Dp, a.ldaux, a.M, a.N, gx + 16, gn, h[1]);
    }
}

// The epilogue of a wave's block of transposed accumulators (rows row0 ..,
// columns col0 ..).  Blocks wholly inside the output with 16-byte aligned
// rows take the unguarded vector path.
template <int EPI, int ACT, int TM, int TN>
__device__ __forceinline__ void epilogue_t_act(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int64_t row0,
                                               int64_t col0, int lane, int split) {
    auto al = [](const void* p, int64_t ld, int64_t elems) {   // rows of elems-element vectors
        return p != nullptr && (reinterpret_cast<uintptr_t>(p) % (2 * elems)) == 0 && ld % elems == 0;
    };
    bool fast = row0 + 32 * TM <= a.M && col0 + 32 * TN <= a.N;
    if constexpr (EPI == EPI_STORE_F32) {
        const float* c = reinterpret_cast<const float*>(a.c) + (int64_t)split * a.split_stride;
        fast = fast && (reinterpret_cast<uintptr_t>(c) & 15u) == 0 && a.ldc % 4 == 0;
    } else {
        fast = fast && ((EPI == EPI_GATE && a.c == nullptr) || al(a.c, a.ldc, 8));
    }
    if constexpr (EPI == EPI_Z_H || EPI == EPI_DZ || EPI == EPI_GATE || EPI == EPI_DGATE)
        fast = fast && (a.aux == nullptr || al(a.aux, a.ldaux, 8));
    if constexpr (EPI == EPI_DZ || EPI == EPI_GATE || EPI == EPI_DGATE) fast = fast && al(a.zin, a.ldzin, 8);
    if constexpr (EPI == EPI_DGATE) fast = fast && al(a.zin2, a.ldzin2, 8);
    if constexpr (EPI == EPI_DGATE) {
        if (fast) epilogue_t_dgate<true>(a, acc, row0, col0, lane);
        else epilogue_t_dgate<false>(a, acc, row0, col0, lane);
    } else {
        if (fast) epilogue_t_impl<EPI, ACT, true>(a, acc, row0, col0, lane, split);
        else epilogue_t_impl<EPI, ACT, false>(a, acc, row0, col0, lane, split);
    }
}

template <int EPI, int TM, int TN>
__device__ __forceinline__ void epilogue_block_t(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int64_t row0,
                                                 int64_t col0, int lane, int split) {
    if constexpr (EPI == EPI_STORE || EPI == EPI_STORE_F32 || EPI == EPI_GATE || EPI == EPI_DGATE) {
        epilogue_t_act<EPI, 0>(a, acc, row0, col0, lane, split);
    } else {
        if (a.act == 0) epilogue_t_act<EPI, 0>(a, acc, row0, col0, lane, split);
        else if (a.act == 2) epilogue_t_act<EPI, 2>(a, acc, row0, col0, lane, split);
        else epilogue_t_act<EPI, 1>(a, acc, row0, col0, lane, split);
    }
}

}  // namespace cola
