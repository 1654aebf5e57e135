// epilogue.hpp -- the fused GEMM epilogues shared by the bf16 MFMA kernels:
// accumulators are staged through LDS in 16-row half slabs so that every
// global access is a coalesced 16-byte vector, and the pointwise part of the
// layer (rounding, sigma, sigma', the CoLA-M recompute of H) happens here.
// Large outputs are written with non-temporal stores so that the streaming
// output does not evict the operand tiles other workgroups are still reading
// from L2.
#pragma once

#include "internal.hpp"
#include "device_math.hpp"

namespace cola {

typedef float f32x16 __attribute__((ext_vector_type(16)));

// Orders one wave's LDS accesses (lanes exchange data through the wave's own
// staging region; LDS operations of a wave complete in order, so a
// wavefront-scope fence and a scheduling barrier suffice).
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void store_stream(uint4* p, const uint4& v) {
    const u32x4_t x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<u32x4_t*>(p));
}
__device__ __forceinline__ void store_stream(float4* p, const float4& v) {
    const f32x4_t x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<f32x4_t*>(p));
}

// ---------------------------------------------------------------------------
// epilogue: 8 consecutive columns of one output row
// ---------------------------------------------------------------------------
template <int EPI>
__device__ __forceinline__ void epilogue8(const GemmArgs& a, int64_t gm, int64_t gn,
                                          const float* acc, int split) {
    if (gm >= a.M || gn >= a.N) return;
    const bool full = gn + 8 <= a.N;
    if constexpr (EPI == EPI_STORE_F32) {
        float* c = reinterpret_cast<float*>(a.c) + (int64_t)split * a.split_stride + gm * a.ldc + gn;
        const bool vec = full && ((reinterpret_cast<uintptr_t>(c) & 15u) == 0);
        if (vec) {
            store_stream(reinterpret_cast<float4*>(c), make_float4(acc[0], acc[1], acc[2], acc[3]));
            store_stream(reinterpret_cast<float4*>(c) + 1, make_float4(acc[4], acc[5], acc[6], acc[7]));
        } else {
            #pragma unroll
            for (int e = 0; e < 8; ++e)
                if (gn + e < a.N) c[e] = acc[e];
        }
        return;
    } else {
        uint16_t* c = reinterpret_cast<uint16_t*>(a.c) + gm * a.ldc + gn;
        float out[8];
        float h[8];
        if constexpr (EPI == EPI_STORE) {
#pragma unroll
            for (int e = 0; e < 8; ++e) out[e] = acc[e];
        } else if constexpr (EPI == EPI_Z_H) {
            // Z is stored rounded to bf16; H = sigma of that rounded Z
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                out[e] = bf16_to_f32(f32_to_bf16(acc[e]));
                h[e] = act_sigma<true>(a.act, out[e]);
            }
        } else if constexpr (EPI == EPI_DZ) {
            const uint16_t* zp = reinterpret_cast<const uint16_t*>(a.zin) + gm * a.ldzin + gn;
            float z[8];
            if (full && ((reinterpret_cast<uintptr_t>(zp) & 15u) == 0)) {
                const uint4 zz = *reinterpret_cast<const uint4*>(zp);
                const uint32_t w[4] = {zz.x, zz.y, zz.z, zz.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    z[2 * e] = bf16_to_f32(w[e] & 0xffffu);
                    z[2 * e + 1] = bf16_to_f32(w[e] >> 16);
                }
            } else {
                #pragma unroll
                for (int e = 0; e < 8; ++e) z[e] = (gn + e < a.N) ? bf16_to_f32(zp[e]) : 0.0f;
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                if (a.act == 0) {
                    out[e] = acc[e];
                    h[e] = z[e];
                } else {
                    const float s = logistic_fast(z[e]);
                    out[e] = acc[e] * (s * (1.0f + z[e] * (1.0f - s)));
                    h[e] = z[e] * s;
                }
            }
        }
        const bool vec = full && ((reinterpret_cast<uintptr_t>(c) & 15u) == 0);
        if (vec) {
            store_stream(reinterpret_cast<uint4*>(c),
                         make_uint4(pack_bf16x2(out[0], out[1]), pack_bf16x2(out[2], out[3]),
                                    pack_bf16x2(out[4], out[5]), pack_bf16x2(out[6], out[7])));
        } else {
            #pragma unroll
            for (int e = 0; e < 8; ++e)
                if (gn + e < a.N) c[e] = (uint16_t)f32_to_bf16(out[e]);
        }
        if constexpr (EPI == EPI_Z_H || EPI == EPI_DZ) {
            if (a.aux) {
                uint16_t* hp = reinterpret_cast<uint16_t*>(a.aux) + gm * a.ldaux + gn;
                if (full && ((reinterpret_cast<uintptr_t>(hp) & 15u) == 0)) {
                    store_stream(reinterpret_cast<uint4*>(hp),
                                 make_uint4(pack_bf16x2(h[0], h[1]), pack_bf16x2(h[2], h[3]),
                                            pack_bf16x2(h[4], h[5]), pack_bf16x2(h[6], h[7])));
                } else {
                    #pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (gn + e < a.N) hp[e] = (uint16_t)f32_to_bf16(h[e]);
                }
            }
        }
    }
}

// Half of MFMA row tile I (16 rows: accumulator registers 8H..8H+7) of a
// wave's accumulators: staged through LDS as fp32 in [row][col] order, then
// each lane handles 8 consecutive columns of a row, so global accesses are
// 16-byte vectors.
template <int I, int H, int BM, int BN, int EPI, int TM, int TN>
__device__ __forceinline__ void epi_half(const GemmArgs& a, const f32x16 (&acc)[TM][TN], float* stg,
                                         int64_t m0, int64_t n0, int wm, int wn, int lane, int split) {
    constexpr int WC = BN / 2;            // wave columns
    constexpr int SP = WC + 4;            // staging pitch (floats)
    constexpr int LPR = WC / 8;           // lanes per row in the read-back
    constexpr int RPP = 64 / LPR;         // rows per pass
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int vv = 0; vv < 8; ++vv) {
            const int v = 8 * H + vv;
            const int row = 8 * (vv >> 2) + 4 * (lane >> 5) + (v & 3);   // row within the half
            const int col = 32 * j + (lane & 31);
            stg[row * SP + col] = acc[I][j][v];
        }
    wave_sync();
    const int cc = lane % LPR;
    const int rr = lane / LPR;
#pragma unroll
    for (int pass = 0; pass < 16 / RPP; ++pass) {
        const int lr = pass * RPP + rr;
        const float4 x0 = *reinterpret_cast<const float4*>(stg + lr * SP + cc * 8);
        const float4 x1 = *reinterpret_cast<const float4*>(stg + lr * SP + cc * 8 + 4);
        const float vals[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
        const int64_t gm = m0 + wm * (BM / 2) + 32 * I + 16 * H + lr;
        const int64_t gn = n0 + wn * WC + cc * 8;
        epilogue8<EPI>(a, gm, gn, vals, split);
    }
    wave_sync();
}

template <int I, int BM, int BN, int EPI, int TM, int TN>
__device__ __forceinline__ void epi_slab(const GemmArgs& a, const f32x16 (&acc)[TM][TN], float* stg,
                                         int64_t m0, int64_t n0, int wm, int wn, int lane, int split) {
    epi_half<I, 0, BM, BN, EPI>(a, acc, stg, m0, n0, wm, wn, lane, split);
    epi_half<I, 1, BM, BN, EPI>(a, acc, stg, m0, n0, wm, wn, lane, split);
}


}  // namespace cola
