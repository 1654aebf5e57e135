// block_ops.hip -- the pointwise and row-wise steps of the CoLA decoder block
// (Sec. 3.2, Fig. "block"): RMSNorm with the residual sum folded in, its
// backward with the residual gradient folded in, the gated product of the MLP
// and its backward, a residual add, and sigma of a saved pre-activation (the
// H that CoLA-M recomputes, App. C).  All HBM-bound: one pass over the
// operands, 16-byte accesses on aligned interior chunks.
#include "internal.hpp"
#include "block.hpp"
#include "device_math.hpp"

namespace cola {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = 256;          // threads per workgroup
constexpr int NWAVE = NT / 64;

__device__ __forceinline__ void unpack8(u32x4 v, float (&f)[8]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = bf16_to_f32(v[i] & 0xffffu);
        f[2 * i + 1] = bf16_to_f32(v[i] >> 16);
    }
}

__device__ __forceinline__ u32x4 pack8(const float (&f)[8]) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = pack_bf16x2(f[2 * i], f[2 * i + 1]);
    return v;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

__device__ __forceinline__ u32x4 ld16(const void* p, int64_t off) {
    return *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(p) + off);
}
__device__ __forceinline__ void st16(void* p, int64_t off, u32x4 v) {
    *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(p) + off) = v;
}

// ---------------------------------------------------------------------------
// RMSNorm forward: one wave per row, the row's chunks cached in registers.
// Lane j owns chunks j, j + 64, ... (NC of them).  d is a multiple of 8.
// ---------------------------------------------------------------------------
template <int NC, bool ADD>
__global__ __launch_bounds__(NT) void rmsnorm_fwd_kernel(const uint16_t* x, const uint16_t* res, uint16_t* xsum,
                                                         const uint16_t* g, uint16_t* y, int64_t T, int d,
                                                         int64_t ld, float eps) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * NWAVE + (threadIdx.x >> 6);
    if (row >= T) return;
    const int nch = d / 8;
    float v[NC][8];
    float ss = 0.0f;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
        const int c = lane + 64 * i;
        if (c < nch) {
            unpack8(ld16(x, row * ld + 8 * c), v[i]);
            if constexpr (ADD) {
                float r[8];
                unpack8(ld16(res, row * ld + 8 * c), r);
#pragma unroll
                for (int e = 0; e < 8; ++e) v[i][e] = round_bf16(v[i][e] + r[e]);
                st16(xsum, row * ld + 8 * c, pack8(v[i]));
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) ss += v[i][e] * v[i][e];
        }
    }
    ss = wave_sum(ss);
    const float rs = rsqrtf(ss / (float)d + eps);
#pragma unroll
    for (int i = 0; i < NC; ++i) {
        const int c = lane + 64 * i;
        if (c < nch) {
            float gg[8], o[8];
            unpack8(ld16(g, 8 * c), gg);
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = v[i][e] * rs * gg[e];
            st16(y, row * ld + 8 * c, pack8(o));
        }
    }
}

// ---------------------------------------------------------------------------
// RMSNorm backward: one wave per row; each workgroup takes a contiguous run
// of rows (rows_per_wg) and leaves its gain-gradient partial sums (fixed
// order: rows in order per wave, waves in order) in partials[blockIdx][d].
// ---------------------------------------------------------------------------
template <int NC>
__global__ __launch_bounds__(NT) void rmsnorm_bwd_kernel(const uint16_t* x, const uint16_t* g, const uint16_t* dy,
                                                         const uint16_t* res_grad, uint16_t* out, float* partials,
                                                         int64_t T, int d, int64_t ld, float eps,
                                                         int64_t rows_per_wg) {
    __shared__ float xfer[NWAVE][64 * 8];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int nch = d / 8;
    // gain (packed bf16) and this lane's gain-gradient sums
    u32x4 gp[NC];
    float dg[NC][8];
#pragma unroll
    for (int i = 0; i < NC; ++i) {
        const int c = lane + 64 * i;
        gp[i] = c < nch ? ld16(g, 8 * c) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int e = 0; e < 8; ++e) dg[i][e] = 0.0f;
    }
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_wg;
    const int64_t r1 = min(T, r0 + rows_per_wg);
    for (int64_t row = r0 + wave; row < r1; row += NWAVE) {
        // s = 1 / sqrt(mean(x^2) + eps), u = dy * g, dot = u . x
        u32x4 xp[NC], dp[NC];
        float ss = 0.0f, dot = 0.0f;
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            const int c = lane + 64 * i;
            if (c < nch) {
                xp[i] = ld16(x, row * ld + 8 * c);
                dp[i] = ld16(dy, row * ld + 8 * c);
                float xv[8], dv[8], gv[8];
                unpack8(xp[i], xv);
                unpack8(dp[i], dv);
                unpack8(gp[i], gv);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    ss += xv[e] * xv[e];
                    dot += dv[e] * gv[e] * xv[e];
                }
            }
        }
        ss = wave_sum(ss);
        dot = wave_sum(dot);
        const float rs = rsqrtf(ss / (float)d + eps);
        const float k3 = rs * rs * rs * dot / (float)d;
        // out = res_grad + s u - x s^3 dot / d;  dg += dy x s
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            const int c = lane + 64 * i;
            if (c < nch) {
                float xv[8], dv[8], gv[8], rg[8], o[8];
                unpack8(xp[i], xv);
                unpack8(dp[i], dv);
                unpack8(gp[i], gv);
                unpack8(ld16(res_grad, row * ld + 8 * c), rg);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    o[e] = rg[e] + (rs * (dv[e] * gv[e]) - xv[e] * k3);
                    dg[i][e] += dv[e] * (xv[e] * rs);
                }
                st16(out, row * ld + 8 * c, pack8(o));
            }
        }
    }
    // waves 1..3 hand their sums to wave 0 through LDS, one chunk slot at a
    // time; wave 0 adds them in wave order and writes the workgroup's partial
#pragma unroll
    for (int i = 0; i < NC; ++i) {
        __syncthreads();
#pragma unroll
        for (int e = 0; e < 8; ++e) xfer[wave][lane * 8 + e] = dg[i][e];
        __syncthreads();
        const int c = lane + 64 * i;
        if (wave == 0 && c < nch) {
            float s8[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                float t = xfer[0][lane * 8 + e];
#pragma unroll
                for (int w = 1; w < NWAVE; ++w) t += xfer[w][lane * 8 + e];
                s8[e] = t;
            }
            float* p = partials + (int64_t)blockIdx.x * d + 8 * c;
            *reinterpret_cast<float4*>(p) = make_float4(s8[0], s8[1], s8[2], s8[3]);
            *reinterpret_cast<float4*>(p + 4) = make_float4(s8[4], s8[5], s8[6], s8[7]);
        }
    }
}

// First stage of the gain-gradient sum: out1[g][c] = sum of partial rows
// g * GROUP .. g * GROUP + GROUP - 1 of column c, in row order (one thread
// per column, coalesced rows); the second stage sums the groups in order.
constexpr int GROUP = 64;
__global__ __launch_bounds__(NT) void colsum_kernel(const float* __restrict__ part, int64_t S, int64_t d,
                                                    float* __restrict__ out1) {
    const int64_t col = (int64_t)blockIdx.x * NT + threadIdx.x;
    if (col >= d) return;
    const int64_t s0 = (int64_t)blockIdx.y * GROUP;
    const int64_t s1 = min(S, s0 + GROUP);
    float acc = 0.0f;
    for (int64_t r = s0; r < s1; ++r) acc += part[r * d + col];
    out1[(int64_t)blockIdx.y * d + col] = acc;
}

int64_t rows_per_workgroup(int64_t T) {
    // at most 4096 partial rows (enough workgroups to keep every CU's loads
    // in flight); whole waves of rows per workgroup
    int64_t r = (T + 4095) / 4096;
    r = (r + NWAVE - 1) / NWAVE * NWAVE;
    return r < NWAVE ? NWAVE : r;
}

// ---------------------------------------------------------------------------
// elementwise ops over [T][width]; one thread per 8-element chunk, a chunk
// that straddles the row end handled element by element.
// ---------------------------------------------------------------------------
template <int OP, int ACT>
__global__ __launch_bounds__(NT) void elementwise_kernel(EwArgs e) {
    const int64_t nch = (e.width + 7) / 8;
    const int64_t total = e.T * nch;
    for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < total; i += (int64_t)gridDim.x * NT) {
        const int64_t row = i / nch;
        const int64_t c0 = (i - row * nch) * 8;
        const int n = (int)min((int64_t)8, e.width - c0);
        float a[8] = {}, b[8] = {}, g[8] = {};
        auto get = [&](const void* p, int64_t ld, float (&f)[8]) {
            const uint16_t* q = reinterpret_cast<const uint16_t*>(p) + row * ld + c0;
            if (n == 8) {
                unpack8(*reinterpret_cast<const u32x4*>(q), f);
            } else {
                for (int k = 0; k < n; ++k) f[k] = bf16_to_f32(q[k]);
            }
        };
        auto put = [&](void* p, int64_t ld, const float (&f)[8]) {
            uint16_t* q = reinterpret_cast<uint16_t*>(p) + row * ld + c0;
            if (n == 8) {
                *reinterpret_cast<u32x4*>(q) = pack8(f);
            } else {
                for (int k = 0; k < n; ++k) q[k] = (uint16_t)f32_to_bf16(f[k]);
            }
        };
        get(e.a, e.lda, a);
        if constexpr (OP == EW_MUL || OP == EW_ADD || OP == EW_DMUL) get(e.b, e.ldb, b);
        if constexpr (OP == EW_DMUL) get(e.g, e.ldg, g);
        float c[8], c2[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            if constexpr (OP == EW_MUL) c[k] = a[k] * b[k];
            else if constexpr (OP == EW_ADD) c[k] = a[k] + b[k];
            else if constexpr (OP == EW_DMUL) {
                c[k] = g[k] * b[k];
                c2[k] = g[k] * a[k];
            } else {
                c[k] = act_sigma_c<ACT, true>(a[k]);
            }
        }
        put(e.c, e.ldc, c);
        if constexpr (OP == EW_DMUL) put(e.c2, e.ldc2, c2);
    }
}

template <int OP, int ACT>
hipError_t ew_launch(const EwArgs& e, hipStream_t s) {
    const int64_t total = e.T * ((e.width + 7) / 8);
    int64_t grid = (total + NT - 1) / NT;
    if (grid > 65536) grid = 65536;
    hipLaunchKernelGGL((elementwise_kernel<OP, ACT>), dim3((unsigned)grid), dim3(NT), 0, s, e);
    return hipGetLastError();
}

template <int NC>
hipError_t rms_fwd_nc(const void* x, const void* res, void* xsum, const void* g, void* y, int64_t T, int64_t d,
                      int64_t ld, float eps, hipStream_t s) {
    const dim3 grid((unsigned)((T + NWAVE - 1) / NWAVE));
    const uint16_t* xx = static_cast<const uint16_t*>(x);
    if (res)
        hipLaunchKernelGGL((rmsnorm_fwd_kernel<NC, true>), grid, dim3(NT), 0, s, xx,
                           static_cast<const uint16_t*>(res), static_cast<uint16_t*>(xsum),
                           static_cast<const uint16_t*>(g), static_cast<uint16_t*>(y), T, (int)d, ld, eps);
    else
        hipLaunchKernelGGL((rmsnorm_fwd_kernel<NC, false>), grid, dim3(NT), 0, s, xx, nullptr, nullptr,
                           static_cast<const uint16_t*>(g), static_cast<uint16_t*>(y), T, (int)d, ld, eps);
    return hipGetLastError();
}

template <int NC>
hipError_t rms_bwd_nc(const void* x, const void* g, const void* dy, const void* res_grad, void* out, float* dg,
                      float* partials, int64_t T, int64_t d, int64_t ld, float eps, hipStream_t s) {
    const int64_t rpw = rows_per_workgroup(T);
    const int64_t nwg = (T + rpw - 1) / rpw;
    hipLaunchKernelGGL((rmsnorm_bwd_kernel<NC>), dim3((unsigned)nwg), dim3(NT), 0, s,
                       static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(g),
                       static_cast<const uint16_t*>(dy), static_cast<const uint16_t*>(res_grad),
                       static_cast<uint16_t*>(out), partials, T, (int)d, ld, eps, rpw);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // dg = sum over the nwg partial rows: groups of GROUP rows, then the groups
    const int64_t ng = (nwg + GROUP - 1) / GROUP;
    float* groups = partials + nwg * d;
    hipLaunchKernelGGL(colsum_kernel, dim3((unsigned)((d + NT - 1) / NT), (unsigned)ng), dim3(NT), 0, s, partials,
                       nwg, d, groups);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_reduce_splits(groups, (int)ng, d, dg, d, s);
}

}  // namespace

hipError_t launch_rmsnorm_fwd(const void* x, const void* res, void* xsum, const void* g, void* y, int64_t T,
                              int64_t d, int64_t ld, float eps, hipStream_t s) {
    if (T <= 0) return hipSuccess;
    const int64_t nc = (d / 8 + 63) / 64;
    if (nc <= 1) return rms_fwd_nc<1>(x, res, xsum, g, y, T, d, ld, eps, s);
    if (nc <= 2) return rms_fwd_nc<2>(x, res, xsum, g, y, T, d, ld, eps, s);
    if (nc <= 4) return rms_fwd_nc<4>(x, res, xsum, g, y, T, d, ld, eps, s);
    if (nc <= 8) return rms_fwd_nc<8>(x, res, xsum, g, y, T, d, ld, eps, s);
    if (nc <= 16) return rms_fwd_nc<16>(x, res, xsum, g, y, T, d, ld, eps, s);
    return hipErrorInvalidValue;
}

int64_t rmsnorm_bwd_partials(int64_t T, int64_t d) {
    if (T <= 0) return 0;
    const int64_t rpw = rows_per_workgroup(T);
    const int64_t nwg = (T + rpw - 1) / rpw;
    return (nwg + (nwg + GROUP - 1) / GROUP) * d;       // the workgroups' rows, then the group sums
}

hipError_t launch_rmsnorm_bwd(const void* x, const void* g, const void* dy, const void* res_grad, void* out,
                              float* dg, float* partials, int64_t T, int64_t d, int64_t ld, float eps,
                              hipStream_t s) {
    if (T <= 0) return launch_fill_zero(dg, d, s);
    const int64_t nc = (d / 8 + 63) / 64;
    if (nc <= 1) return rms_bwd_nc<1>(x, g, dy, res_grad, out, dg, partials, T, d, ld, eps, s);
    if (nc <= 2) return rms_bwd_nc<2>(x, g, dy, res_grad, out, dg, partials, T, d, ld, eps, s);
    if (nc <= 4) return rms_bwd_nc<4>(x, g, dy, res_grad, out, dg, partials, T, d, ld, eps, s);
    if (nc <= 8) return rms_bwd_nc<8>(x, g, dy, res_grad, out, dg, partials, T, d, ld, eps, s);
    if (nc <= 16) return rms_bwd_nc<16>(x, g, dy, res_grad, out, dg, partials, T, d, ld, eps, s);
    return hipErrorInvalidValue;
}

hipError_t launch_elementwise(const EwArgs& e, hipStream_t s) {
    if (e.T <= 0 || e.width <= 0) return hipSuccess;
    switch (e.op) {
        case EW_MUL: return ew_launch<EW_MUL, 0>(e, s);
        case EW_ADD: return ew_launch<EW_ADD, 0>(e, s);
        case EW_DMUL: return ew_launch<EW_DMUL, 0>(e, s);
        case EW_SIGMA:
            if (e.act == 0) return ew_launch<EW_SIGMA, 0>(e, s);
            if (e.act == 1) return ew_launch<EW_SIGMA, 1>(e, s);
            if (e.act == 2) return ew_launch<EW_SIGMA, 2>(e, s);
            return hipErrorInvalidValue;
        default: return hipErrorInvalidValue;
    }
}

}  // namespace cola
