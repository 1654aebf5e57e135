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
// 32 x 32 accumulator holds row 8 (v / 4) + 4 (l / 32) + v % 4, column l % 32):
//  * forward: one workgroup of 4 waves per (sequence, head, 128 queries);
//    each wave owns 32 queries and sweeps 32-key blocks up to its diagonal
//    (staged 64 keys per barrier pair) with an online softmax (scores in the
//    exp2 domain).  The score tile is
//    computed transposed, S^T = K Q^T, so that each lane holds one query's
//    scores: its row statistics need one exchange with lane l ^ 32, and the
//    probabilities feed O^T += V^T P^T directly from the accumulator
//    registers (the 32 keys of a block sit in the lane in an order that the
//    V^T fragment's transposing LDS reads, ds_read_b64_tr_b16 on the
//    row-major V tile, follow).  Stores att and the log2-sum-exp of the
//    scaled scores.  Every LDS tile is row-major; transposed operands come
//    from the transposing reads.
//  * backward dq: the same sweep, recomputing P from lse, with dP^T = V dO^T,
//    dS = P (dP - D), dQ^T += K^T dS^T; it also forms D = rowsum(dO * O).
//  * backward dk, dv: one workgroup per (sequence, head, 128 keys), each wave
//    32 keys, sweeping 32-query blocks from its diagonal: S = Q K^T,
//    dP = dO V^T, dV^T += dO^T P, dK^T += Q^T dS.
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
// the layout of both MFMA operands.  ROT: rotated by the row's position.
template <int HD, bool ROT>
__device__ __forceinline__ void load_row_frags(bf16x8 (&f)[HD / 16], const uint16_t* base, int64_t ld, int64_t row,
                                               bool ok, int col0, int pos, const float* rope, int hh) {
    constexpr int NS = HD / 16;
    u32x4 raw[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) raw[s] = load8(base, ld, row, ok, col0 + 16 * s + 8 * hh);
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
                p[v] = (kp <= qm) ? st[v] * c : -INFINITY;
                mb = fmaxf(mb, p[v]);
            }
            mb = fmaxf(mb, __shfl_xor(mb, 32));
            const float mn = fmaxf(m, mb);                // finite: key 0 is in the first sub-block
            const float alpha = exp2f(m - mn);
            float ls = 0.0f;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                p[v] = exp2f(p[v] - mn);
                ls += p[v];
            }
            l = l * alpha + ls;
            m = mn;
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int v = 0; v < 16; ++v) o[t][v] *= alpha;
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
                const float p = (kp <= qm && qok) ? exp2f(st[v] * c - lse) : 0.0f;
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
                p[v] = ok ? exp2f(st[v] * c - slse[r]) : 0.0f;
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
    hipError_t e = launch(1, a, sh.head_dim, sh.n_seq, s);        // dq, and D for the next kernel
    if (e != hipSuccess) return e;
    return launch(2, a, sh.head_dim, sh.n_seq, s);
}

}  // namespace cola
