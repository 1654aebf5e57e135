// attention.hip -- causal multi-head self-attention with rotary position
// embeddings, the scaled dot product that the CoLA decoder block keeps
// unchanged (Sec. 3.2, Fig. "block"; App. C counts it as 4 n^2 d per
// sequence), forward and backward, for the block path.
//
// Layout: q, k, v, att and their gradients are [T][ld] bf16, token-major,
// sequence s in rows s*L .. s*L + L - 1, head h in columns h*HD .. h*HD+HD-1
// (HD = 64 or 128).  lse and D are [heads][T] fp32.  RoPE pairs element i of
// a head with i + HD/2 (rotate-half) at angle pos * base^(-2i/HD), pos = the
// token's index within its sequence; it is applied to q and k as they are
// loaded (fp32 rotation of the bf16 values from a (cos, sin) table computed
// once per call, rounded to bf16 for the MFMA), and its transpose to dq and
// dk before they are stored.
//
// Kernels (CDNA4, wave64, v_mfma_f32_32x32x16_bf16; lane l, register v of a
// 32 x 32 accumulator holds row 8 (v / 4) + 4 (l / 32) + v % 4, column l % 32).
// Head size 64 and sequences of at most 256 tokens (the paper's LLaMA shapes)
// run in two whole-sequence kernels; other shapes in three staged kernels.
//  * whole-sequence forward: one workgroup of 4 waves per (sequence, head)
//    loads the sequence's rotated keys and its values into LDS once; each
//    wave then takes 32-query blocks in a snake order that balances the
//    causal work and sweeps 32-key blocks up to its diagonal with an online
//    softmax (scores in the exp2 domain).  The score tile is computed
//    transposed, S^T = K Q^T, so that each lane holds one query's scores: its
//    row statistics need one exchange with lane l ^ 32, and the
//    probabilities feed O^T += V^T P^T directly from the accumulator
//    registers (the 32 keys of a block sit in the lane in an order that the
//    V^T fragment's transposing LDS reads, ds_read_b64_tr_b16 on the
//    row-major V tile, follow).  Stores att and the log2-sum-exp of the
//    scaled scores.
//  * whole-sequence backward: one workgroup of 8 waves per (sequence, head)
//    loads rotated q and k, v and dO into LDS once and forms
//    D = rowsum(dO * O) and the log-sum-exp per query there; wave w then
//    computes dk, dv of key block w (S = Q K^T, dP = dO V^T,
//    dS = P (dP - D), dV^T += dO^T P, dK^T += Q^T dS over the query blocks
//    from the diagonal on) and dq of query block w (dQ^T += K^T dS^T over the
//    key blocks up to the diagonal): nqb + 1 blocks of work on every wave.
//    Both write their output blocks through a per-wave LDS stage so that a
//    store instruction covers 16 rows x 64 contiguous bytes.
//  * staged kernels: forward, backward dq (which also forms D) and backward
//    dk, dv, one workgroup of 4 waves per (sequence, head, 128 queries or
//    keys), 64 rows staged in LDS per barrier pair (the forward loads the
//    next stage during the current one), the same block arithmetic.
// The whole-sequence kernels evaluate the causal mask only on blocks on the
// diagonal or holding rows past the sequence end.  Every LDS tile is
// row-major; transposed operands come from the transposing reads.
// No atomics: each output element is written by one lane, in a fixed order
// of summation (bitwise reproducible).
#include <math.h>

#include "internal.hpp"
#include "block.hpp"
#include "device_math.hpp"

namespace cola {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s16x4* lptr4_t;

constexpr int NW = 4;            // waves per workgroup
constexpr int WB = 32;           // queries (keys) per wave
constexpr int CHUNK = NW * WB;   // queries (keys) per workgroup
constexpr int STG = 64;          // rows (keys or queries) staged in LDS per barrier pair: two 32-row sub-blocks
constexpr float kLog2e = 1.4426950408889634f;
// 1 / sqrt(HD), the scale of the scores
template <int HD>
constexpr float kScale = HD == 64 ? 0.125f : 0.08838834764831845f;

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_frag(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// exp2 by the hardware instruction alone (no range reduction for denormal
// results): its arguments here are scores minus their running maximum or
// minus the log-sum-exp, so a result it flushes to zero is below 2^-126 and
// far below the bf16 resolution of the probabilities it feeds.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

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

// The rotation table: rope[pos][i] = (cos, sin) of pos * base^(-2i/HD),
// i < HD/2, fp32 pairs, computed once per call (rope_table_kernel).
// Rotate the pairs (i0 + e, i0 + e + HD/2), e < 8, of one token at position
// pos: lo[e] = element i0 + e, hi[e] = element i0 + e + HD/2.
template <int HD>
__device__ __forceinline__ void rope8(float (&lo)[8], float (&hi)[8], int i0, int pos, const float* rope) {
    const float4* t = reinterpret_cast<const float4*>(rope + 2 * ((int64_t)pos * (HD / 2) + i0));
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
        const float4 cs = t[e2];                // (cos, sin) of elements i0 + 2 e2 and i0 + 2 e2 + 1
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int e = 2 * e2 + h;
            const float c = h ? cs.z : cs.x, sn = h ? cs.w : cs.y;
            const float a = lo[e], b = hi[e];
            lo[e] = a * c - b * sn;
            hi[e] = b * c + a * sn;
        }
    }
}

__global__ void rope_table_kernel(float* rope, int L, int half, float nl2b) {
    const int64_t n = (int64_t)L * half;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int pos = (int)(i / half), j = (int)(i % half);
        float sn, cs;
        sincosf((float)pos * exp2f((float)j * nl2b), &sn, &cs);
        rope[2 * i] = cs;
        rope[2 * i + 1] = sn;
    }
}

// 16 bytes (8 bf16) of row `row` (0 if the row is past the sequence end).
__device__ __forceinline__ u32x4 load8(const uint16_t* base, int64_t ld, int64_t row, bool ok, int col) {
    if (!ok) return u32x4{0u, 0u, 0u, 0u};
    return *reinterpret_cast<const u32x4*>(base + row * ld + col);
}

// Fragment registers of one wave-owned row (query or key) of a head: step s
// (HD / 16 steps of 16 elements) holds elements 16 s + 8 (lane / 32) .. + 7,
// the layout of both MFMA operands.  load_row_raw issues the loads,
// row_frags rotates them (ROT: by the row's position) into fragments.
template <int HD>
__device__ __forceinline__ void load_row_raw(u32x4 (&raw)[HD / 16], const uint16_t* base, int64_t ld, int64_t row,
                                             bool ok, int col0, int hh) {
#pragma unroll
    for (int s = 0; s < HD / 16; ++s) raw[s] = load8(base, ld, row, ok, col0 + 16 * s + 8 * hh);
}

template <int HD, bool ROT>
__device__ __forceinline__ void row_frags(bf16x8 (&f)[HD / 16], u32x4 (&raw)[HD / 16], int pos, const float* rope,
                                          int hh) {
    constexpr int NS = HD / 16;
    if constexpr (ROT) {
#pragma unroll
        for (int s = 0; s < NS / 2; ++s) {
            float lo[8], hi[8];
            unpack8(raw[s], lo);
            unpack8(raw[s + NS / 2], hi);
            rope8<HD>(lo, hi, 16 * s + 8 * hh, pos, rope);
            raw[s] = pack8(lo);
            raw[s + NS / 2] = pack8(hi);
        }
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) f[s] = as_frag(raw[s]);
}

template <int HD, bool ROT>
__device__ __forceinline__ void load_row_frags(bf16x8 (&f)[HD / 16], const uint16_t* base, int64_t ld, int64_t row,
                                               bool ok, int col0, int pos, const float* rope, int hh) {
    u32x4 raw[HD / 16];
    load_row_raw<HD>(raw, base, ld, row, ok, col0, hh);
    row_frags<HD, ROT>(f, raw, pos, rope, hh);
}

// LDS tile of STG rows x HD, row-major, 16-byte chunks XOR-swizzled by the
// row (conflict-free fragment reads of both kinds below).
template <int HD>
struct RowTile {
    static constexpr int BYTES = STG * HD * 2;
    __device__ static __forceinline__ int off(int row, int chunk) { return row * (HD * 2) + ((chunk ^ (row & 7)) << 4); }
    // A-operand fragment of step s (HD elements 16 s ..) for rows r0 .. r0 + 31
    // (lane: row r0 + lane % 32)
    __device__ static __forceinline__ bf16x8 frag(const char* t, int r0, int s, int lane) {
        const int row = r0 + (lane & 31);
        return *reinterpret_cast<const bf16x8*>(t + off(row, 2 * s + (lane >> 5)));
    }
    // A-operand fragment of the transpose: 32 HD elements (tile nt) x 16 rows
    // (step s of the 32-row sub-block at r0), by two transposing reads.  Lane
    // (n = 32 nt + lane % 32, hh = lane / 32) receives rows
    // r0 + 16 s + 4 hh + 0..3 and r0 + 16 s + 8 + 4 hh + 0..3 at element n --
    // the order in which the transposed score tile leaves those rows in a
    // lane's accumulator registers 8 s .. 8 s + 7.  (In each 16-lane group,
    // lanes 4q .. 4q + 3 point at row q of a 4 x 16 block, four consecutive
    // elements each, and lane i receives element i of the block.)
    __device__ static __forceinline__ bf16x8 frag_tr(const char* t, int r0, int nt, int s, int lane) {
        const int g = lane >> 4, i = lane & 15;
        const int m = 32 * nt + 16 * (g & 1) + 4 * (i & 3);
        const int k = r0 + 16 * s + 4 * (g >> 1) + (i >> 2);
        const int byte = (m & 7) * 2;
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lptr4_t)(t + off(k, m >> 3) + byte));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lptr4_t)(t + off(k + 8, m >> 3) + byte));
        const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        return __builtin_bit_cast(bf16x8, v);
    }
};

// STG rows (sequence positions p0 .. p0 + STG - 1, zeros from L on) of one
// head on their way into a row-major LDS tile: load() brings this thread's
// share into registers (issued a stage ahead, so the loads fly during the
// current stage's MFMAs), put() rotates them by position when ROT and writes
// them to LDS.  Each thread moves pairs of chunks (c, c + HD / 16):
// elements i and i + HD/2.
template <int HD>
struct Stage {
    static constexpr int HC = HD / 16;                 // chunk pairs per row
    static constexpr int NI = STG * HC / (NW * 64);    // pairs per thread
    u32x4 a[NI], b[NI];
    int p0;

    __device__ __forceinline__ void load(const uint16_t* base, int64_t ld, int64_t seq_row0, int p, int L,
                                         int col0) {
        p0 = p;
#pragma unroll
        for (int it = 0; it < NI; ++it) {
            const int i = threadIdx.x + NW * 64 * it;
            const int row = i / HC, c = i % HC;
            const int pos = p0 + row;
            const bool ok = pos < L;
            a[it] = load8(base, ld, seq_row0 + pos, ok, col0 + 8 * c);
            b[it] = load8(base, ld, seq_row0 + pos, ok, col0 + 8 * (c + HC));
        }
    }

    template <bool ROT>
    __device__ __forceinline__ void put(char* rt, int L, const float* rope) {
#pragma unroll
        for (int it = 0; it < NI; ++it) {
            const int i = threadIdx.x + NW * 64 * it;
            const int row = i / HC, c = i % HC;
            const int pos = p0 + row;
            u32x4 x = a[it], y = b[it];
            if constexpr (ROT) {
                if (pos < L) {
                    float lo[8], hi[8];
                    unpack8(x, lo);
                    unpack8(y, hi);
                    rope8<HD>(lo, hi, 8 * c, pos, rope);
                    x = pack8(lo);
                    y = pack8(hi);
                }
            }
            *reinterpret_cast<u32x4*>(rt + RowTile<HD>::off(row, c)) = x;
            *reinterpret_cast<u32x4*>(rt + RowTile<HD>::off(row, c + HC)) = y;
        }
    }
};

// Row (key or query) of register v of a 32 x 32 accumulator, within its tile.
__device__ __forceinline__ int acc_row(int v, int hh) { return 8 * (v >> 2) + 4 * hh + (v & 3); }

// Store a [HD rows x 32 columns] accumulator set (tiles nt = 0 .. HD/32 - 1,
// transposed output: column = this lane's token, rows = head elements) as
// bf16 into the token's row, scaled, with RoPE's transpose when ROT.
template <int HD, bool ROT>
__device__ __forceinline__ void store_rows(const f32x16 (&acc)[HD / 32], float scale, uint16_t* out, int64_t ld,
                                           int64_t row, bool ok, int col0, int pos, const float* rope, int hh) {
    constexpr int NT = HD / 32;
    if (!ok) return;
    float x[NT][16];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) x[t][v] = acc[t][v] * scale;
    if constexpr (ROT) {
        // element n = 32 t + acc_row(v) pairs with n + HD/2: tile t + NT/2, same v;
        // groups of four consecutive n read their (cos, sin) as two float4
#pragma unroll
        for (int t = 0; t < NT / 2; ++t)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n0 = 32 * t + 8 * g + 4 * hh;
                const float4* tb = reinterpret_cast<const float4*>(rope + 2 * ((int64_t)pos * (HD / 2) + n0));
                const float4 c01 = tb[0], c23 = tb[1];
                const float cs[4] = {c01.x, c01.z, c23.x, c23.z}, sn[4] = {c01.y, c01.w, c23.y, c23.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int v = 4 * g + e;
                    const float a = x[t][v], b = x[t + NT / 2][v];
                    // transpose of the rotation: angle -ang
                    x[t][v] = a * cs[e] + b * sn[e];
                    x[t + NT / 2][v] = b * cs[e] - a * sn[e];
                }
            }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int n = 32 * t + 8 * g + 4 * hh;
            u32x2 w;
            w[0] = pack_bf16x2(x[t][4 * g], x[t][4 * g + 1]);
            w[1] = pack_bf16x2(x[t][4 * g + 2], x[t][4 * g + 3]);
            *reinterpret_cast<u32x2*>(out + row * ld + col0 + n) = w;
        }
}

// Max with lane l ^ 32 (the other half of a query's scores) by one
// v_permlane32_swap.
__device__ __forceinline__ float xor32_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Probabilities may reach 2^kSlack against a stale softmax reference.
constexpr float kSlack = 8.0f;

// One 32-key block of the online softmax of this lane's query: p holds the
// block's raw scores (-inf where masked), mb their maximum over this lane's
// half of them, c > 0 the factor to the exp2 domain (1/sqrt(HD) log2 e).  The
// reference m (exp2 domain) moves, and l and the output accumulators are
// rescaled, only when some query of the wave sees a block maximum above
// m + kSlack; otherwise the probabilities are taken against the old
// reference (at most 2^kSlack), which changes the result only by rounding
// and skips the rescale for the whole wave.  p leaves holding the
// probabilities exp2(c p - m).
template <int NT>
__device__ __forceinline__ void softmax_block(float (&p)[16], float mb, float c, float& m, float& l,
                                              f32x16 (&o)[NT]) {
    mb = xor32_max(mb) * c;
    if (__ballot(mb > m + kSlack) != 0) {
        const float mn = fmaxf(m, mb);
        const float alpha = m == mn ? 1.0f : exp2_hw(m - mn);
        l *= alpha;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) o[t][v] *= alpha;
        m = mn;
    }
    float ls = 0.0f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        p[v] = exp2_hw(fmaf(p[v], c, -m));
        ls += p[v];
    }
    l += ls;
}

// Output block [32 rows x HD] of one wave written through a per-wave LDS
// stage (32 rows x 32 bf16, 2 KB, 16-byte chunks XOR-swizzled by row / 4),
// one 32-element tile at a time: written from the accumulator layout (each
// lane one row, four elements per write), read back as 16 rows x 64
// contiguous bytes per instruction and stored that way.  The same wave reads
// what it wrote and LDS executes one wave's accesses in order, so no barrier
// is needed.
constexpr int kStageBytes = 32 * 64;

__device__ __forceinline__ int stage_off(int r, int c) { return r * 64 + ((c ^ ((r >> 2) & 3)) << 4); }

// acc[t][v]: head element 32 t + acc_row(v, hh) of this lane's row (lane % 32
// of the block starting at row_base; nrows of them are stored), scaled, with
// RoPE's transpose (ROT) at position pos.
template <int HD, bool ROT>
__device__ __forceinline__ void store_block(const f32x16 (&acc)[HD / 32], float scale, uint16_t* out, int64_t ld,
                                            int64_t row_base, int nrows, int col0, int pos, const float* rope,
                                            char* stage, int lane) {
    constexpr int NT = HD / 32;
    const int hh = lane >> 5, r = lane & 31;
    float x[NT][16];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) x[t][v] = acc[t][v] * scale;
    if constexpr (ROT) {
#pragma unroll
        for (int t = 0; t < NT / 2; ++t)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n0 = 32 * t + 8 * g + 4 * hh;
                const float4* tb = reinterpret_cast<const float4*>(rope + 2 * ((int64_t)pos * (HD / 2) + n0));
                const float4 c01 = tb[0], c23 = tb[1];
                const float cs[4] = {c01.x, c01.z, c23.x, c23.z}, sn[4] = {c01.y, c01.w, c23.y, c23.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int v = 4 * g + e;
                    const float a = x[t][v], b = x[t + NT / 2][v];
                    x[t][v] = a * cs[e] + b * sn[e];
                    x[t + NT / 2][v] = b * cs[e] - a * sn[e];
                }
            }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            u32x2 w;
            w[0] = pack_bf16x2(x[t][4 * g], x[t][4 * g + 1]);
            w[1] = pack_bf16x2(x[t][4 * g + 2], x[t][4 * g + 3]);
            *reinterpret_cast<u32x2*>(stage + stage_off(r, g) + 8 * hh) = w;
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int rr = (lane >> 2) + 16 * i, cc = lane & 3;
            const u32x4 v = *reinterpret_cast<const u32x4*>(stage + stage_off(rr, cc));
            if (rr < nrows) *reinterpret_cast<u32x4*>(out + (row_base + rr) * ld + col0 + 32 * t + 8 * cc) = v;
        }
    }
}

struct AttnArgs {
    const uint16_t *q, *k, *v, *o, *dO;
    uint16_t *att, *dq, *dk, *dv;
    float *lse, *D;          // [heads][T]
    const float* rope;       // [L][HD/2] (cos, sin)
    int64_t ld;              // row pitch of every [T][ld] tensor
    int64_t T;
    int L, heads;
};

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
template <int HD>
__global__ __launch_bounds__(NW * 64) void attn_fwd_kernel(AttnArgs a) {
    constexpr int NS = HD / 16, NT = HD / 32;
    __shared__ __attribute__((aligned(16))) char kt[RowTile<HD>::BYTES];
    __shared__ __attribute__((aligned(16))) char vt[RowTile<HD>::BYTES];
    const int chunk = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
    const int L = a.L;
    const int64_t row0 = (int64_t)s * L;
    const int col0 = h * HD;
    const int qw0 = chunk * CHUNK + WB * wave;           // first query of the wave
    const int qp = qw0 + (lane & 31);                      // this lane's query
    const bool qok = qp < L;
    const int qm = qok ? qp : L - 1;                       // masking position (rows past L are dropped)
    const float c = kLog2e * kScale<HD>;                   // scores to the exp2 domain

    bf16x8 qf[NS];
    load_row_frags<HD, true>(qf, a.q, a.ld, row0 + qp, qok, col0, qm, a.rope, hh);
    f32x16 o[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) o[t] = f32x16{};
    float m = -INFINITY, l = 0.0f;

    const int kend = min(L, chunk * CHUNK + CHUNK);       // keys any query of the workgroup sees
    Stage<HD> sk, sv;
    sk.load(a.k, a.ld, row0, 0, L, col0);
    sv.load(a.v, a.ld, row0, 0, L, col0);
    for (int k0 = 0; k0 < kend; k0 += STG) {
        __syncthreads();                                   // the previous tiles are consumed
        sk.template put<true>(kt, L, a.rope);
        sv.template put<false>(vt, L, a.rope);
        __syncthreads();
        if (k0 + STG < kend) {                             // the next stage's rows fly during this one
            sk.load(a.k, a.ld, row0, k0 + STG, L, col0);
            sv.load(a.v, a.ld, row0, k0 + STG, L, col0);
        }
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
            const int kb = k0 + 32 * sub;
            if (kb > qw0 + WB - 1 || kb >= kend || qw0 >= L) continue;   // after all of the wave's queries
            f32x16 st = f32x16{};
#pragma unroll
            for (int i = 0; i < NS; ++i) st = mfma(RowTile<HD>::frag(kt, 32 * sub, i, lane), qf[i], st);
            float p[16];
            float mb = -INFINITY;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int kp = kb + acc_row(v, hh);
                p[v] = (kp <= qm) ? st[v] : -INFINITY;
                mb = fmaxf(mb, p[v]);
            }
            softmax_block<NT>(p, mb, c, m, l, o);          // the first block holds key 0: m becomes finite
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                float pf[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) pf[e] = p[8 * t2 + e];
                const bf16x8 pb = as_frag(pack8(pf));
#pragma unroll
                for (int t = 0; t < NT; ++t) o[t] = mfma(RowTile<HD>::frag_tr(vt, 32 * sub, t, t2, lane), pb, o[t]);
            }
        }
    }
    l += __shfl_xor(l, 32);
    store_rows<HD, false>(o, 1.0f / l, a.att, a.ld, row0 + qp, qok, col0, qm, a.rope, hh);
    if (qok && hh == 0) a.lse[(int64_t)h * a.T + row0 + qp] = m + log2f(l);
}

// ---------------------------------------------------------------------------
// backward: dq (and D = rowsum(dO * O))
// ---------------------------------------------------------------------------
template <int HD>
__global__ __launch_bounds__(NW * 64) void attn_bwd_dq_kernel(AttnArgs a) {
    constexpr int NS = HD / 16, NT = HD / 32;
    __shared__ __attribute__((aligned(16))) char kt[RowTile<HD>::BYTES];
    __shared__ __attribute__((aligned(16))) char vt[RowTile<HD>::BYTES];
    const int chunk = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
    const int L = a.L;
    const int64_t row0 = (int64_t)s * L;
    const int col0 = h * HD;
    const int qw0 = chunk * CHUNK + WB * wave;
    const int qp = qw0 + (lane & 31);
    const bool qok = qp < L;
    const int qm = qok ? qp : L - 1;
    const float c = kLog2e * kScale<HD>;

    bf16x8 qf[NS], df[NS], of[NS];
    load_row_frags<HD, true>(qf, a.q, a.ld, row0 + qp, qok, col0, qm, a.rope, hh);
    load_row_frags<HD, false>(df, a.dO, a.ld, row0 + qp, qok, col0, qm, a.rope, hh);
    load_row_frags<HD, false>(of, a.o, a.ld, row0 + qp, qok, col0, qm, a.rope, hh);
    // D = rowsum(dO * O) over the head (this lane's half, then lane ^ 32's)
    float D = 0.0f;
#pragma unroll
    for (int i = 0; i < NS; ++i) {
        float x[8], y[8];
        unpack8(__builtin_bit_cast(u32x4, df[i]), x);
        unpack8(__builtin_bit_cast(u32x4, of[i]), y);
#pragma unroll
        for (int e = 0; e < 8; ++e) D += x[e] * y[e];
    }
    D += __shfl_xor(D, 32);
    const float lse = qok ? a.lse[(int64_t)h * a.T + row0 + qp] : 0.0f;
    if (qok && hh == 0) a.D[(int64_t)h * a.T + row0 + qp] = D;

    f32x16 dq[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) dq[t] = f32x16{};
    const int kend = min(L, chunk * CHUNK + CHUNK);
    // (no prefetch of the next stage here: its registers would cost occupancy)
    for (int k0 = 0; k0 < kend; k0 += STG) {
        __syncthreads();
        {
            Stage<HD> sk, sv;
            sk.load(a.k, a.ld, row0, k0, L, col0);
            sv.load(a.v, a.ld, row0, k0, L, col0);
            sk.template put<true>(kt, L, a.rope);
            sv.template put<false>(vt, L, a.rope);
        }
        __syncthreads();
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
            const int kb = k0 + 32 * sub;
            if (kb > qw0 + WB - 1 || kb >= kend || qw0 >= L) continue;
            f32x16 st = f32x16{}, dpt = f32x16{};
#pragma unroll
            for (int i = 0; i < NS; ++i) {
                st = mfma(RowTile<HD>::frag(kt, 32 * sub, i, lane), qf[i], st);
                dpt = mfma(RowTile<HD>::frag(vt, 32 * sub, i, lane), df[i], dpt);
            }
            float ds[16];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int kp = kb + acc_row(v, hh);
                const float p = (kp <= qm && qok) ? exp2_hw(st[v] * c - lse) : 0.0f;
                ds[v] = p * (dpt[v] - D);
            }
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                float f[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) f[e] = ds[8 * t2 + e];
                const bf16x8 db = as_frag(pack8(f));
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    dq[t] = mfma(RowTile<HD>::frag_tr(kt, 32 * sub, t, t2, lane), db, dq[t]);
            }
        }
    }
    store_rows<HD, true>(dq, kScale<HD>, a.dq, a.ld, row0 + qp, qok, col0, qm, a.rope, hh);
}

// ---------------------------------------------------------------------------
// backward: dk, dv
// ---------------------------------------------------------------------------
template <int HD>
__global__ __launch_bounds__(NW * 64) void attn_bwd_dkdv_kernel(AttnArgs a) {
    constexpr int NS = HD / 16, NT = HD / 32;
    __shared__ __attribute__((aligned(16))) char qt[RowTile<HD>::BYTES];
    __shared__ __attribute__((aligned(16))) char dt[RowTile<HD>::BYTES];
    __shared__ float slse[STG], sD[STG];
    const int chunk = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
    const int L = a.L;
    const int64_t row0 = (int64_t)s * L;
    const int col0 = h * HD;
    const int kw0 = chunk * CHUNK + WB * wave;             // first key of the wave
    const int kp = kw0 + (lane & 31);                      // this lane's key
    const bool kok = kp < L;
    const int km = kok ? kp : L - 1;
    const float c = kLog2e * kScale<HD>;

    bf16x8 kf[NS], vf[NS];
    load_row_frags<HD, true>(kf, a.k, a.ld, row0 + kp, kok, col0, km, a.rope, hh);
    load_row_frags<HD, false>(vf, a.v, a.ld, row0 + kp, kok, col0, km, a.rope, hh);
    f32x16 dk[NT], dv[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        dk[t] = f32x16{};
        dv[t] = f32x16{};
    }
    // query blocks from the workgroup's first key (rounded down to a stage) to the sequence end
    // (no prefetch of the next stage here: its registers would cost occupancy)
    for (int q0 = (chunk * CHUNK) / STG * STG; q0 < L; q0 += STG) {
        __syncthreads();
        {
            Stage<HD> sq, sd;
            sq.load(a.q, a.ld, row0, q0, L, col0);
            sd.load(a.dO, a.ld, row0, q0, L, col0);
            sq.template put<true>(qt, L, a.rope);
            sd.template put<false>(dt, L, a.rope);
        }
        if (threadIdx.x < STG) {
            const int qpos = q0 + threadIdx.x;
            const bool ok = qpos < L;
            slse[threadIdx.x] = ok ? a.lse[(int64_t)h * a.T + row0 + qpos] : 0.0f;
            sD[threadIdx.x] = ok ? a.D[(int64_t)h * a.T + row0 + qpos] : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
            const int qb = q0 + 32 * sub;
            // every query of the sub-block is before the wave's keys, or past the end
            if (qb + 31 < kw0 || qb >= L || kw0 >= L) continue;
            f32x16 st = f32x16{}, dp = f32x16{};
#pragma unroll
            for (int i = 0; i < NS; ++i) {
                st = mfma(RowTile<HD>::frag(qt, 32 * sub, i, lane), kf[i], st);
                dp = mfma(RowTile<HD>::frag(dt, 32 * sub, i, lane), vf[i], dp);
            }
            float p[16], ds[16];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int r = 32 * sub + acc_row(v, hh);
                const int qpos = q0 + r;
                const bool ok = qpos < L && km <= qpos && kok;
                p[v] = ok ? exp2_hw(st[v] * c - slse[r]) : 0.0f;
                ds[v] = p[v] * (dp[v] - sD[r]);
            }
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                float fp[8], fd[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    fp[e] = p[8 * t2 + e];
                    fd[e] = ds[8 * t2 + e];
                }
                const bf16x8 pb = as_frag(pack8(fp));
                const bf16x8 db = as_frag(pack8(fd));
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    dv[t] = mfma(RowTile<HD>::frag_tr(dt, 32 * sub, t, t2, lane), pb, dv[t]);
                    dk[t] = mfma(RowTile<HD>::frag_tr(qt, 32 * sub, t, t2, lane), db, dk[t]);
                }
            }
        }
    }
    store_rows<HD, true>(dk, kScale<HD>, a.dk, a.ld, row0 + kp, kok, col0, km, a.rope, hh);
    store_rows<HD, false>(dv, 1.0f, a.dv, a.ld, row0 + kp, kok, col0, km, a.rope, hh);
}

// ---------------------------------------------------------------------------
// whole-sequence kernels (seq_len <= LMAX, HD = 64): one workgroup per
// (sequence, head) keeps the whole sequence's rotated keys and values (and,
// backward, queries and output gradients) in LDS, loaded and rotated once,
// with one barrier; every wave then works on its own 32-row blocks with no
// further synchronisation.  Causal work is balanced by handing out query
// blocks in a snake order (forward: blocks i and 2 NW - 1 - i of every
// 2 NW to the same wave) and, backward, by pairing key block w (its dk, dv:
// nqb - w query blocks) with query block w (its dq: w + 1 key blocks) on
// wave w.  Only the blocks on the diagonal, or holding rows past the
// sequence end, are masked.
// ---------------------------------------------------------------------------
constexpr int LMAX = 256;

// Rows 0 .. L-1 of one head (zeros from L to the next multiple of 32) into a
// row-major LDS tile, NB chunk pairs (elements i, i + HD/2) per thread of NTHR:
// load() issues every load first, put() rotates (ROT, by the row's position)
// and writes.
template <int HD, int NTHR, int NB>
struct SeqRows {
    static constexpr int HC = HD / 16;
    u32x4 a[NB], b[NB];

    __device__ __forceinline__ void load(const uint16_t* base, int64_t ld, int64_t seq_row0, int L, int col0) {
#pragma unroll
        for (int it = 0; it < NB; ++it) {
            const int i = threadIdx.x + NTHR * it;
            const int row = i / HC, c = i % HC;
            const bool ok = row < L;
            a[it] = load8(base, ld, seq_row0 + row, ok, col0 + 8 * c);
            b[it] = load8(base, ld, seq_row0 + row, ok, col0 + 8 * (c + HC));
        }
    }

    template <bool ROT>
    __device__ __forceinline__ void put(char* t, int L, int LB, const float* rope) {
#pragma unroll
        for (int it = 0; it < NB; ++it) {
            const int i = threadIdx.x + NTHR * it;
            const int row = i / HC, c = i % HC;
            if (row >= LB) continue;
            u32x4 x = a[it], y = b[it];
            if constexpr (ROT) {
                if (row < L) {
                    float lo[8], hi[8];
                    unpack8(x, lo);
                    unpack8(y, hi);
                    rope8<HD>(lo, hi, 8 * c, row, rope);
                    x = pack8(lo);
                    y = pack8(hi);
                }
            }
            *reinterpret_cast<u32x4*>(t + RowTile<HD>::off(row, c)) = x;
            *reinterpret_cast<u32x4*>(t + RowTile<HD>::off(row, c + HC)) = y;
        }
    }
};

template <int HD>
__global__ __launch_bounds__(NW * 64) void attn_fwd_seq_kernel(AttnArgs a) {
    constexpr int NS = HD / 16, NT = HD / 32;
    constexpr int NB = LMAX * (HD / 16) / (NW * 64);
    __shared__ __attribute__((aligned(16))) char kt[LMAX * HD * 2];
    __shared__ __attribute__((aligned(16))) char vt[LMAX * HD * 2];
    __shared__ __attribute__((aligned(16))) char stg[NW][kStageBytes];
    const int h = blockIdx.x, s = blockIdx.y;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
    const int L = a.L;
    const int nqb = (L + 31) >> 5, LB = 32 * nqb;
    const int64_t row0 = (int64_t)s * L;
    const int col0 = h * HD;
    const float c = kLog2e * kScale<HD>;
    // the wave's j-th query block: 2 NW (j / 2) + (w or 2 NW - 1 - w), increasing in j
    auto qblock = [&](int j) { return 2 * NW * (j >> 1) + ((j & 1) ? 2 * NW - 1 - wave : wave); };

    int j = 0, qb = qblock(0);
    u32x4 raw[NS];                                         // the next query block's rows, loaded ahead
    {
        const int qp = 32 * qb + (lane & 31);
        load_row_raw<HD>(raw, a.q, a.ld, row0 + qp, qb < nqb && qp < L, col0, hh);
        SeqRows<HD, NW * 64, NB> rk, rv;
        rk.load(a.k, a.ld, row0, L, col0);
        rv.load(a.v, a.ld, row0, L, col0);
        rk.template put<true>(kt, L, LB, a.rope);
        rv.template put<false>(vt, L, LB, a.rope);
    }
    __syncthreads();
    while (qb < nqb) {
        const int qp = 32 * qb + (lane & 31);
        const bool qok = qp < L;
        const int qm = qok ? qp : L - 1;                   // masking position (rows past L are dropped)
        bf16x8 qf[NS];
        row_frags<HD, true>(qf, raw, qm, a.rope, hh);
        const int qn = qblock(++j);
        if (qn < nqb) {
            const int qpn = 32 * qn + (lane & 31);
            load_row_raw<HD>(raw, a.q, a.ld, row0 + qpn, qpn < L, col0, hh);
        }
        f32x16 o[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) o[t] = f32x16{};
        float m = -INFINITY, l = 0.0f;
        for (int kb = 0; kb <= qb; ++kb) {
            f32x16 st = f32x16{};
#pragma unroll
            for (int i = 0; i < NS; ++i) st = mfma(RowTile<HD>::frag(kt, 32 * kb, i, lane), qf[i], st);
            float p[16];
            float mb = -INFINITY;
            if (kb == qb) {                                // the diagonal: keys after the query (or past L) drop out
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    p[v] = (32 * kb + acc_row(v, hh) <= qm) ? st[v] : -INFINITY;
                    mb = fmaxf(mb, p[v]);
                }
            } else {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    p[v] = st[v];
                    mb = fmaxf(mb, p[v]);
                }
            }
            softmax_block<NT>(p, mb, c, m, l, o);          // the first block holds key 0: m becomes finite
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                float pf[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) pf[e] = p[8 * t2 + e];
                const bf16x8 pb = as_frag(pack8(pf));
#pragma unroll
                for (int t = 0; t < NT; ++t) o[t] = mfma(RowTile<HD>::frag_tr(vt, 32 * kb, t, t2, lane), pb, o[t]);
            }
        }
        l += __shfl_xor(l, 32);
        store_block<HD, false>(o, 1.0f / l, a.att, a.ld, row0 + 32 * qb, L - 32 * qb, col0, qm, a.rope, stg[wave],
                               lane);
        if (qok && hh == 0) a.lse[(int64_t)h * a.T + row0 + qp] = m + log2f(l);
        qb = qn;
    }
}

template <int HD>
__global__ __launch_bounds__(2 * NW * 64) void attn_bwd_seq_kernel(AttnArgs a) {
    constexpr int NTH = 2 * NW * 64;                       // 8 waves: one per 32-row block of a 256-row sequence
    constexpr int NS = HD / 16, NT = HD / 32;
    constexpr int NB = LMAX * (HD / 16) / NTH;
    __shared__ __attribute__((aligned(16))) char qt[LMAX * HD * 2];
    __shared__ __attribute__((aligned(16))) char kt[LMAX * HD * 2];
    __shared__ __attribute__((aligned(16))) char vt[LMAX * HD * 2];
    __shared__ __attribute__((aligned(16))) char dt[LMAX * HD * 2];
    __shared__ float slse[LMAX], sD[LMAX];
    __shared__ __attribute__((aligned(16))) char stg[2 * NW][kStageBytes];
    const int h = blockIdx.x, s = blockIdx.y;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
    const int L = a.L;
    const int nqb = (L + 31) >> 5, LB = 32 * nqb;
    const int64_t row0 = (int64_t)s * L;
    const int col0 = h * HD;
    const float c = kLog2e * kScale<HD>;
    {
        SeqRows<HD, NTH, NB> rq, rk, rv, rd;
        rq.load(a.q, a.ld, row0, L, col0);
        rk.load(a.k, a.ld, row0, L, col0);
        rv.load(a.v, a.ld, row0, L, col0);
        rd.load(a.dO, a.ld, row0, L, col0);
        // D = rowsum(dO * O) and the log-sum-exp of this wave's 32 queries
        const int qd = 32 * wave + (lane & 31);
        const bool dok = wave < nqb && qd < L;
        u32x4 ro[NS], rdo[NS];
        load_row_raw<HD>(ro, a.o, a.ld, row0 + qd, dok, col0, hh);
        load_row_raw<HD>(rdo, a.dO, a.ld, row0 + qd, dok, col0, hh);
        const float lse = dok ? a.lse[(int64_t)h * a.T + row0 + qd] : 0.0f;
        rq.template put<true>(qt, L, LB, a.rope);
        rk.template put<true>(kt, L, LB, a.rope);
        rv.template put<false>(vt, L, LB, a.rope);
        rd.template put<false>(dt, L, LB, a.rope);
        float D = 0.0f;
#pragma unroll
        for (int i = 0; i < NS; ++i) {
            float x[8], y[8];
            unpack8(rdo[i], x);
            unpack8(ro[i], y);
#pragma unroll
            for (int e = 0; e < 8; ++e) D += x[e] * y[e];
        }
        D += __shfl_xor(D, 32);
        if (wave < nqb && hh == 0) {
            sD[qd] = D;
            slse[qd] = lse;
        }
    }
    __syncthreads();
    if (wave >= nqb) return;                               // no barrier follows

    // key block wave: dk, dv over the query blocks from the diagonal on
    {
        const int kb = wave;
        const int kp = 32 * kb + (lane & 31);
        const bool kok = kp < L;
        const int km = kok ? kp : L - 1;
        bf16x8 kf[NS], vf[NS];
#pragma unroll
        for (int i = 0; i < NS; ++i) {
            kf[i] = RowTile<HD>::frag(kt, 32 * kb, i, lane);
            vf[i] = RowTile<HD>::frag(vt, 32 * kb, i, lane);
        }
        f32x16 dk[NT], dv[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            dk[t] = f32x16{};
            dv[t] = f32x16{};
        }
        for (int qb = kb; qb < nqb; ++qb) {
            f32x16 st = f32x16{}, dp = f32x16{};
#pragma unroll
            for (int i = 0; i < NS; ++i) {
                st = mfma(RowTile<HD>::frag(qt, 32 * qb, i, lane), kf[i], st);
                dp = mfma(RowTile<HD>::frag(dt, 32 * qb, i, lane), vf[i], dp);
            }
            float p[16], ds[16];
            if (qb == kb || 32 * qb + 32 > L) {            // the diagonal, or queries past the end
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int r = 32 * qb + acc_row(v, hh);    // < 32 nqb <= LMAX: in bounds either way
                    const bool ok = r < L && km <= r && kok;
                    const float e = exp2_hw(st[v] * c - slse[r]);
                    p[v] = ok ? e : 0.0f;
                    ds[v] = p[v] * (dp[v] - sD[r]);
                }
            } else {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int r = 32 * qb + acc_row(v, hh);
                    p[v] = exp2_hw(st[v] * c - slse[r]);
                    ds[v] = p[v] * (dp[v] - sD[r]);
                }
            }
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                float fp[8], fd[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    fp[e] = p[8 * t2 + e];
                    fd[e] = ds[8 * t2 + e];
                }
                const bf16x8 pb = as_frag(pack8(fp));
                const bf16x8 db = as_frag(pack8(fd));
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    dv[t] = mfma(RowTile<HD>::frag_tr(dt, 32 * qb, t, t2, lane), pb, dv[t]);
                    dk[t] = mfma(RowTile<HD>::frag_tr(qt, 32 * qb, t, t2, lane), db, dk[t]);
                }
            }
        }
        store_block<HD, true>(dk, kScale<HD>, a.dk, a.ld, row0 + 32 * kb, L - 32 * kb, col0, km, a.rope, stg[wave],
                              lane);
        store_block<HD, false>(dv, 1.0f, a.dv, a.ld, row0 + 32 * kb, L - 32 * kb, col0, km, a.rope, stg[wave], lane);
    }

    // query block wave: dq over the key blocks up to the diagonal
    {
        const int qb = wave;
        const int qp = 32 * qb + (lane & 31);
        const bool qok = qp < L;
        const int qm = qok ? qp : L - 1;
        bf16x8 qf[NS], df[NS];
#pragma unroll
        for (int i = 0; i < NS; ++i) {
            qf[i] = RowTile<HD>::frag(qt, 32 * qb, i, lane);
            df[i] = RowTile<HD>::frag(dt, 32 * qb, i, lane);
        }
        const float lse = slse[qp], D = sD[qp];
        f32x16 dq[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) dq[t] = f32x16{};
        for (int kb = 0; kb <= qb; ++kb) {
            f32x16 st = f32x16{}, dpt = f32x16{};
#pragma unroll
            for (int i = 0; i < NS; ++i) {
                st = mfma(RowTile<HD>::frag(kt, 32 * kb, i, lane), qf[i], st);
                dpt = mfma(RowTile<HD>::frag(vt, 32 * kb, i, lane), df[i], dpt);
            }
            float ds[16];
            if (kb == qb) {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const bool ok = 32 * kb + acc_row(v, hh) <= qm && qok;
                    const float p = ok ? exp2_hw(st[v] * c - lse) : 0.0f;
                    ds[v] = p * (dpt[v] - D);
                }
            } else {
                // rows past L (zero q, dO, lse and D) give p = 1 and ds = 0 here, and are not stored
#pragma unroll
                for (int v = 0; v < 16; ++v) ds[v] = exp2_hw(st[v] * c - lse) * (dpt[v] - D);
            }
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                float f[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) f[e] = ds[8 * t2 + e];
                const bf16x8 db = as_frag(pack8(f));
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    dq[t] = mfma(RowTile<HD>::frag_tr(kt, 32 * kb, t, t2, lane), db, dq[t]);
            }
        }
        store_block<HD, true>(dq, kScale<HD>, a.dq, a.ld, row0 + 32 * qb, L - 32 * qb, col0, qm, a.rope, stg[wave],
                              lane);
    }
}

template <int HD>
hipError_t launch_all(int which, const AttnArgs& a, int n_seq, hipStream_t s) {
    const dim3 grid((unsigned)((a.L + CHUNK - 1) / CHUNK), (unsigned)a.heads, (unsigned)n_seq);
    if (which == 0) hipLaunchKernelGGL(attn_fwd_kernel<HD>, grid, dim3(NW * 64), 0, s, a);
    else if (which == 1) hipLaunchKernelGGL(attn_bwd_dq_kernel<HD>, grid, dim3(NW * 64), 0, s, a);
    else hipLaunchKernelGGL(attn_bwd_dkdv_kernel<HD>, grid, dim3(NW * 64), 0, s, a);
    return hipGetLastError();
}

hipError_t launch(int which, const AttnArgs& a, int hd, int n_seq, hipStream_t s) {
    if (n_seq <= 0 || a.L <= 0 || a.heads <= 0) return hipSuccess;
    if (hd == 64) return launch_all<64>(which, a, n_seq, s);
    if (hd == 128) return launch_all<128>(which, a, n_seq, s);
    return hipErrorInvalidValue;
}

// The whole-sequence kernels take HD = 64 and sequences of at most LMAX
// tokens (four 32 KB tiles of LDS backward); the rest runs in the staged
// kernels above.
bool whole_sequence(int hd, int L) { return hd == 64 && L <= LMAX; }

hipError_t launch_seq(int which, const AttnArgs& a, int n_seq, hipStream_t s) {
    if (n_seq <= 0 || a.L <= 0 || a.heads <= 0) return hipSuccess;
    const dim3 grid((unsigned)a.heads, (unsigned)n_seq);
    if (which == 0) hipLaunchKernelGGL(attn_fwd_seq_kernel<64>, grid, dim3(NW * 64), 0, s, a);
    else hipLaunchKernelGGL(attn_bwd_seq_kernel<64>, grid, dim3(2 * NW * 64), 0, s, a);
    return hipGetLastError();
}

AttnArgs make(const AttnShape& sh) {
    AttnArgs a{};
    a.ld = sh.ld;
    a.T = (int64_t)sh.n_seq * sh.seq_len;
    a.L = sh.seq_len;
    a.heads = sh.heads;
    a.rope = sh.rope;
    return a;
}

}  // namespace

int64_t attn_rope_table_floats(int seq_len, int head_dim) { return (int64_t)seq_len * head_dim; }

hipError_t launch_attn_rope_table(const AttnShape& sh, float* rope, hipStream_t s) {
    const int half = sh.head_dim / 2;
    const int64_t n = (int64_t)sh.seq_len * half;
    if (n <= 0) return hipSuccess;
    const float nl2b = -2.0f * log2f(sh.rope_base) / (float)sh.head_dim;
    const int64_t grid = (n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024;
    hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)grid), dim3(256), 0, s, rope, sh.seq_len, half, nl2b);
    return hipGetLastError();
}

hipError_t launch_attn_fwd(const AttnShape& sh, const void* q, const void* k, const void* v, void* att, float* lse,
                           hipStream_t s) {
    AttnArgs a = make(sh);
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.att = static_cast<uint16_t*>(att);
    a.lse = lse;
    if (whole_sequence(sh.head_dim, sh.seq_len)) return launch_seq(0, a, sh.n_seq, s);
    return launch(0, a, sh.head_dim, sh.n_seq, s);
}

hipError_t launch_attn_bwd(const AttnShape& sh, const void* q, const void* k, const void* v, const void* att,
                           const float* lse, const void* dO, void* dq, void* dk, void* dv, float* D, hipStream_t s) {
    AttnArgs a = make(sh);
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.o = static_cast<const uint16_t*>(att);
    a.dO = static_cast<const uint16_t*>(dO);
    a.dq = static_cast<uint16_t*>(dq);
    a.dk = static_cast<uint16_t*>(dk);
    a.dv = static_cast<uint16_t*>(dv);
    a.lse = const_cast<float*>(lse);
    a.D = D;
    if (whole_sequence(sh.head_dim, sh.seq_len)) return launch_seq(1, a, sh.n_seq, s);
    hipError_t e = launch(1, a, sh.head_dim, sh.n_seq, s);        // dq, and D for the next kernel
    if (e != hipSuccess) return e;
    return launch(2, a, sh.head_dim, sh.n_seq, s);
}

}  // namespace cola
