// gemm_f32.hip -- fp32 storage path: C[M][N] = sum_k P(m, k) Q(n, k) with
// true fp32 fused multiply-adds on the vector ALUs (no reduced-precision
// matrix shortcut), the same operand layouts and epilogues as the bf16 MFMA
// kernel.  Tiles of 64 x 64 outputs, K tiles of 16, 256 threads each owning a
// 4 x 4 block; every access is guarded, so any shape and pitch is accepted.
#include "internal.hpp"
#include "device_math.hpp"

namespace cola {
namespace {

constexpr int TB = 64;
constexpr int KT = 16;

template <int LAYOUT>
__device__ __forceinline__ float load_op(const float* base, int64_t ld, int64_t row, int64_t rows,
                                         int64_t k, int64_t kend) {
    if (row >= rows || k >= kend) return 0.0f;
    return LAYOUT == KMAJ ? base[row * ld + k] : base[k * ld + row];
}

template <int PL, int QL, int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
    __shared__ float Ps[KT][TB + 4];
    __shared__ float Qs[KT][TB + 4];
    const int64_t tiles_n = (a.N + TB - 1) / TB;
    const int64_t tiles_m = (a.M + TB - 1) / TB;
    const int64_t per_split = tiles_m * tiles_n;
    const int64_t b = blockIdx.x;
    const int split = (int)(b / per_split);
    const int64_t rem = b - (int64_t)split * per_split;
    const int64_t m0 = (rem / tiles_n) * TB;
    const int64_t n0 = (rem % tiles_n) * TB;
    const int64_t kbeg = (int64_t)split * a.k_chunk;
    const int64_t kend = min(a.K, kbeg + a.k_chunk);
    const float* P = reinterpret_cast<const float*>(a.p);
    const float* Q = reinterpret_cast<const float*>(a.q);
    const int tid = threadIdx.x;
    const int tx = tid & 15;
    const int ty = tid >> 4;

    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.0f;

    for (int64_t k0 = kbeg; k0 < kend; k0 += KT) {
        // 64 rows x 16 k per operand = 1024 values, 4 per thread; the index
        // order follows the contiguous dimension so loads coalesce.
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int idx = tid + 256 * e;
            int rp, kp, rq, kq;
            if (PL == KMAJ) { rp = idx >> 4; kp = idx & 15; } else { kp = idx >> 6; rp = idx & 63; }
            if (QL == KMAJ) { rq = idx >> 4; kq = idx & 15; } else { kq = idx >> 6; rq = idx & 63; }
            Ps[kp][rp] = load_op<PL>(P, a.ldp, m0 + rp, a.M, k0 + kp, kend);
            Qs[kq][rq] = load_op<QL>(Q, a.ldq, n0 + rq, a.N, k0 + kq, kend);
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < KT; ++kk) {
            float pv[4], qv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) pv[i] = Ps[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) qv[j] = Qs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(pv[i], qv[j], acc[i][j]);
        }
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t gm = m0 + ty * 4 + i;
        if (gm >= a.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t gn = n0 + tx * 4 + j;
            if (gn >= a.N) continue;
            const float v = acc[i][j];
            if constexpr (EPI == EPI_STORE || EPI == EPI_STORE_F32) {
                reinterpret_cast<float*>(a.c)[(int64_t)split * a.split_stride + gm * a.ldc + gn] = v;
            } else if constexpr (EPI == EPI_Z_H) {
                reinterpret_cast<float*>(a.c)[gm * a.ldc + gn] = v;
                if (a.aux) reinterpret_cast<float*>(a.aux)[gm * a.ldaux + gn] = act_sigma<false>(a.act, v);
            } else if constexpr (EPI == EPI_H) {
                reinterpret_cast<float*>(a.c)[gm * a.ldc + gn] = act_sigma<false>(a.act, v);
            } else if constexpr (EPI == EPI_DZ) {
                const float z = reinterpret_cast<const float*>(a.zin)[gm * a.ldzin + gn];
                reinterpret_cast<float*>(a.c)[gm * a.ldc + gn] = v * act_sigma_prime<false>(a.act, z);
                if (a.aux) reinterpret_cast<float*>(a.aux)[gm * a.ldaux + gn] = act_sigma<false>(a.act, z);
            }
        }
    }
}

template <int PL, int QL, int EPI>
hipError_t launch_t(const GemmArgs& a, hipStream_t s) {
    const int64_t tiles = ((a.M + TB - 1) / TB) * ((a.N + TB - 1) / TB) * (int64_t)a.splits;
    if (tiles <= 0) return hipSuccess;
    if (tiles > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((gemm_f32_kernel<PL, QL, EPI>), dim3((unsigned)tiles), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s) {
    const int pl = a.p_layout, ql = a.q_layout;
    switch (a.epi) {
        case EPI_Z_H:
            if (pl == KMAJ && ql == KMAJ) return launch_t<KMAJ, KMAJ, EPI_Z_H>(a, s);
            break;
        case EPI_H:
            if (pl == KMAJ && ql == KMAJ) return launch_t<KMAJ, KMAJ, EPI_H>(a, s);
            break;
        case EPI_STORE:
            if (pl == KMAJ && ql == KMAJ) return launch_t<KMAJ, KMAJ, EPI_STORE>(a, s);
            if (pl == KMAJ && ql == MNMAJ) return launch_t<KMAJ, MNMAJ, EPI_STORE>(a, s);
            break;
        case EPI_DZ:
            if (pl == KMAJ && ql == MNMAJ) return launch_t<KMAJ, MNMAJ, EPI_DZ>(a, s);
            break;
        case EPI_STORE_F32:
            if (pl == MNMAJ && ql == MNMAJ) return launch_t<MNMAJ, MNMAJ, EPI_STORE_F32>(a, s);
            break;
        default:
            break;
    }
    return hipErrorNotSupported;
}

// ---------------------------------------------------------------------------
// split-K reduction, zero fill, and row repacking of 16-bit weights
// ---------------------------------------------------------------------------
namespace {

// The split reduction's fixed order, which depends only on the split count:
// the partials in chunks of kChunk in split order, each chunk summed in
// order, then the chunk sums in order (up to kChunk splits: the plain sum in
// split order).  Two kernels follow it: one thread per output group summing
// every chunk in turn, and, for split counts above kChunk, kChunkLanes
// threads per output group summing chunks side by side and combining them in
// LDS, which keeps several times as many loads in flight when the output is
// small.
constexpr int kChunk = 8;
constexpr int kChunkLanes = 4;
constexpr int kMaxChunks = 32;

__device__ __forceinline__ float4 add4(float4 a, float4 b) {
    return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}
__device__ __forceinline__ float add4(float a, float b) { return a + b; }

// Sum of partials k0 .. k1-1 (k1 > k0) of element i; V = float4 (stride in
// float4 units) or float.
// (All of a chunk's loads are issued before its sums.)
template <class V>
__device__ __forceinline__ V chunk_sum(const V* __restrict__ part, int64_t stride, int64_t i, int k0, int k1) {
    V v[kChunk];
#pragma unroll
    for (int u = 0; u < kChunk; ++u)
        if (k0 + u < k1) v[u] = part[(int64_t)(k0 + u) * stride + i];
    V s = v[0];
#pragma unroll
    for (int u = 1; u < kChunk; ++u)
        if (k0 + u < k1) s = add4(s, v[u]);
    return s;
}

template <class V>
__device__ __forceinline__ V ordered_sum(const V* __restrict__ part, int64_t stride, int64_t i, int splits) {
    V s = chunk_sum(part, stride, i, 0, min(kChunk, splits));
    for (int k0 = kChunk; k0 < splits; k0 += kChunk) s = add4(s, chunk_sum(part, stride, i, k0, min(k0 + kChunk, splits)));
    return s;
}

bool reduce_vec_ok(const float* part, int64_t stride, const float* out) {
    return (stride & 3) == 0 && (reinterpret_cast<uintptr_t>(part) & 15u) == 0 &&
           (reinterpret_cast<uintptr_t>(out) & 15u) == 0;
}

// One thread per output group, block blk of nblk (grid-stride over float4
// groups, scalar tail).
__device__ __forceinline__ void reduce_splits_range(const float* __restrict__ part, int splits, int64_t stride,
                                                    float* __restrict__ out, int64_t n, int64_t blk,
                                                    int64_t nblk) {
    const int64_t n4 = n >> 2;
    const bool vec = ((stride & 3) == 0) && ((reinterpret_cast<uintptr_t>(part) & 15u) == 0) &&
                     ((reinterpret_cast<uintptr_t>(out) & 15u) == 0);
    const int64_t step = nblk * blockDim.x;
    int64_t i = blk * blockDim.x + threadIdx.x;
    if (vec) {
        const float4* p4 = reinterpret_cast<const float4*>(part);
        for (; i < n4; i += step) reinterpret_cast<float4*>(out)[i] = ordered_sum(p4, stride >> 2, i, splits);
        // scalar tail
        i = n4 * 4 + blk * blockDim.x + threadIdx.x;
    }
    for (; i < n; i += step) out[i] = ordered_sum(part, stride, i, splits);
}

// kChunkLanes threads per float4 output group (n a multiple of 4, 16-byte
// aligned rows): 256 / kChunkLanes groups per block.
__device__ __forceinline__ void reduce_chunks_range(const float* __restrict__ part, int splits, int64_t stride,
                                                    float* __restrict__ out, int64_t n, int64_t blk) {
    constexpr int OPB = 256 / kChunkLanes;
    __shared__ float4 sums[kMaxChunks][OPB];
    const int j = threadIdx.x / OPB, o = threadIdx.x % OPB;
    const int64_t i = blk * OPB + o, n4 = n >> 2;
    const int chunks = (splits + kChunk - 1) / kChunk;
    const float4* p4 = reinterpret_cast<const float4*>(part);
    if (i < n4)
        for (int c = j; c < chunks; c += kChunkLanes)
            sums[c][o] = chunk_sum(p4, stride >> 2, i, kChunk * c, min(kChunk * c + kChunk, splits));
    __syncthreads();
    if (j == 0 && i < n4) {
        float4 s = sums[0][o];
        for (int c = 1; c < chunks; ++c) s = add4(s, sums[c][o]);
        reinterpret_cast<float4*>(out)[i] = s;
    }
}

__global__ __launch_bounds__(256) void reduce_chunks_kernel(const float* __restrict__ p0, int64_t st0,
                                                            float* __restrict__ o0, int64_t n0, int64_t g0,
                                                            const float* __restrict__ p1, int64_t st1,
                                                            float* __restrict__ o1, int64_t n1, int splits) {
    if ((int64_t)blockIdx.x < g0) reduce_chunks_range(p0, splits, st0, o0, n0, blockIdx.x);
    else reduce_chunks_range(p1, splits, st1, o1, n1, (int64_t)blockIdx.x - g0);
}

__global__ __launch_bounds__(256) void reduce_splits_kernel(const float* __restrict__ part, int splits,
                                                            int64_t stride, float* __restrict__ out,
                                                            int64_t n) {
    reduce_splits_range(part, splits, stride, out, n, blockIdx.x, gridDim.x);
}

// Two reductions with the same split count in one launch: blocks [0, g0) sum
// the partials of output 0, the rest those of output 1 (same order, so the
// same bits as two launches).
__global__ __launch_bounds__(256) void reduce_splits2_kernel(const float* __restrict__ p0, int64_t st0,
                                                             float* __restrict__ o0, int64_t n0, int64_t g0,
                                                             const float* __restrict__ p1, int64_t st1,
                                                             float* __restrict__ o1, int64_t n1, int splits) {
    if ((int64_t)blockIdx.x < g0) reduce_splits_range(p0, splits, st0, o0, n0, blockIdx.x, g0);
    else reduce_splits_range(p1, splits, st1, o1, n1, (int64_t)blockIdx.x - g0, (int64_t)gridDim.x - g0);
}

__global__ __launch_bounds__(256) void fill_zero_kernel(float* __restrict__ out, int64_t n) {
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += step) out[i] = 0.0f;
}

__global__ __launch_bounds__(256) void pack_rows_kernel(const uint16_t* __restrict__ src, int64_t rows,
                                                        int64_t width, uint16_t* __restrict__ dst,
                                                        int64_t ld) {
    const int64_t n = rows * ld;
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += step) {
        const int64_t r = i / ld;
        const int64_t c = i - r * ld;
        dst[i] = c < width ? src[r * width + c] : (uint16_t)0;
    }
}

// dP = dY (.) sigma'(P) (the both-sigma variant's backward through its outer
// sigma).  One thread per group of V consecutive elements of a row (V = 8 for
// bf16, 4 for fp32: one 16-byte access per operand when every row start is
// 16-byte aligned), grid-stride over the groups.  bf16 products are taken in
// fp32 and rounded to nearest even.
template <bool BF16>
__global__ __launch_bounds__(256) void outer_grad_kernel(const void* __restrict__ dy, int64_t lddy,
                                                         const void* __restrict__ p, int64_t ldp,
                                                         void* __restrict__ out, int64_t ldo, int64_t T,
                                                         int64_t n, int act, int vec) {
    constexpr int V = BF16 ? 8 : 4;
    const int64_t groups = (n + V - 1) / V;
    const int64_t total = T * groups;
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < total; g += step) {
        const int64_t t = g / groups;
        const int64_t c0 = (g - t * groups) * V;
        const int valid = (int)(n - c0 < V ? n - c0 : V);
        if constexpr (BF16) {
            const uint16_t* a = reinterpret_cast<const uint16_t*>(dy) + t * lddy + c0;
            const uint16_t* b = reinterpret_cast<const uint16_t*>(p) + t * ldp + c0;
            uint16_t* o = reinterpret_cast<uint16_t*>(out) + t * ldo + c0;
            if (vec && valid == V) {
                const uint4 av = *reinterpret_cast<const uint4*>(a);
                const uint4 bv = *reinterpret_cast<const uint4*>(b);
                const uint32_t aw[4] = {av.x, av.y, av.z, av.w};
                const uint32_t bw[4] = {bv.x, bv.y, bv.z, bv.w};
                uint32_t ow[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const float lo = bf16_to_f32(aw[k] & 0xffffu) * act_sigma_prime<true>(act, bf16_to_f32(bw[k] & 0xffffu));
                    const float hi = bf16_to_f32(aw[k] >> 16) * act_sigma_prime<true>(act, bf16_to_f32(bw[k] >> 16));
                    ow[k] = pack_bf16x2(lo, hi);
                }
                *reinterpret_cast<uint4*>(o) = make_uint4(ow[0], ow[1], ow[2], ow[3]);
            } else {
                for (int e = 0; e < valid; ++e)
                    o[e] = (uint16_t)f32_to_bf16(bf16_to_f32(a[e]) * act_sigma_prime<true>(act, bf16_to_f32(b[e])));
            }
        } else {
            const float* a = reinterpret_cast<const float*>(dy) + t * lddy + c0;
            const float* b = reinterpret_cast<const float*>(p) + t * ldp + c0;
            float* o = reinterpret_cast<float*>(out) + t * ldo + c0;
            if (vec && valid == V) {
                const float4 av = *reinterpret_cast<const float4*>(a);
                const float4 bv = *reinterpret_cast<const float4*>(b);
                *reinterpret_cast<float4*>(o) =
                    make_float4(av.x * act_sigma_prime<false>(act, bv.x), av.y * act_sigma_prime<false>(act, bv.y),
                                av.z * act_sigma_prime<false>(act, bv.z), av.w * act_sigma_prime<false>(act, bv.w));
            } else {
                for (int e = 0; e < valid; ++e) o[e] = a[e] * act_sigma_prime<false>(act, b[e]);
            }
        }
    }
}

unsigned grid_for(int64_t work) {
    int64_t g = (work + 255) / 256;
    if (g < 1) g = 1;
    if (g > 4096) g = 4096;
    return (unsigned)g;
}

}  // namespace

// Whether the chunk-parallel kernel takes a reduction (the same order, so
// the same bits, as the one-thread-per-group kernel).
static bool chunks_ok(const float* part, int64_t stride, const float* out, int64_t n, int splits) {
    return splits > kChunk && splits <= kChunk * kMaxChunks && n % 4 == 0 && reduce_vec_ok(part, stride, out);
}
static int64_t chunk_blocks(int64_t n) { return (n / 4 + 256 / kChunkLanes - 1) / (256 / kChunkLanes); }

hipError_t launch_reduce_splits2(const float* p0, int64_t st0, float* o0, int64_t n0, const float* p1, int64_t st1,
                                 float* o1, int64_t n1, int splits, hipStream_t s) {
    if (n0 <= 0) return launch_reduce_splits(p1, splits, st1, o1, n1, s);
    if (n1 <= 0) return launch_reduce_splits(p0, splits, st0, o0, n0, s);
    if (chunks_ok(p0, st0, o0, n0, splits) && chunks_ok(p1, st1, o1, n1, splits)) {
        const int64_t b0 = chunk_blocks(n0), b1 = chunk_blocks(n1);
        if (b0 + b1 > 0x7fffffffLL) return hipErrorInvalidConfiguration;
        hipLaunchKernelGGL(reduce_chunks_kernel, dim3((unsigned)(b0 + b1)), dim3(256), 0, s, p0, st0, o0, n0, b0, p1,
                           st1, o1, n1, splits);
        return hipGetLastError();
    }
    const unsigned g0 = grid_for((n0 + 3) / 4), g1 = grid_for((n1 + 3) / 4);
    hipLaunchKernelGGL(reduce_splits2_kernel, dim3(g0 + g1), dim3(256), 0, s, p0, st0, o0, n0, (int64_t)g0, p1, st1,
                       o1, n1, splits);
    return hipGetLastError();
}

hipError_t launch_reduce_splits(const float* part, int splits, int64_t stride, float* out, int64_t n,
                                hipStream_t s) {
    if (n <= 0) return hipSuccess;
    if (chunks_ok(part, stride, out, n, splits)) {
        const int64_t b = chunk_blocks(n);
        if (b > 0x7fffffffLL) return hipErrorInvalidConfiguration;
        hipLaunchKernelGGL(reduce_chunks_kernel, dim3((unsigned)b), dim3(256), 0, s, part, stride, out, n, b, part,
                           stride, out, (int64_t)0, splits);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(reduce_splits_kernel, dim3(grid_for((n + 3) / 4)), dim3(256), 0, s, part, splits,
                       stride, out, n);
    return hipGetLastError();
}

hipError_t launch_pack_rows(const void* src, int64_t rows, int64_t width, void* dst, int64_t ld,
                            hipStream_t s) {
    if (rows <= 0) return hipSuccess;
    hipLaunchKernelGGL(pack_rows_kernel, dim3(grid_for(rows * ld)), dim3(256), 0, s,
                       reinterpret_cast<const uint16_t*>(src), rows, width, reinterpret_cast<uint16_t*>(dst), ld);
    return hipGetLastError();
}

hipError_t launch_outer_grad(bool bf16, const void* dy, int64_t lddy, const void* p, int64_t ldp, void* out,
                             int64_t ldo, int64_t T, int64_t n, int act, hipStream_t s) {
    if (T <= 0 || n <= 0) return hipSuccess;
    const int64_t V = bf16 ? 8 : 4;
    auto al = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15u) == 0; };
    const int vec = al(dy) && al(p) && al(out) && lddy % V == 0 && ldp % V == 0 && ldo % V == 0;
    const unsigned grid = grid_for(T * ((n + V - 1) / V));
    if (bf16)
        hipLaunchKernelGGL(outer_grad_kernel<true>, dim3(grid), dim3(256), 0, s, dy, lddy, p, ldp, out, ldo, T, n,
                           act, vec);
    else
        hipLaunchKernelGGL(outer_grad_kernel<false>, dim3(grid), dim3(256), 0, s, dy, lddy, p, ldp, out, ldo, T, n,
                           act, vec);
    return hipGetLastError();
}

hipError_t launch_fill_zero(float* out, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_for(n)), dim3(256), 0, s, out, n);
    return hipGetLastError();
}

}  // namespace cola
