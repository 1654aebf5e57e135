// block.hpp -- declarations of the decoder-block path shared by attention.hip,
// block_ops.hip, block_abi.hip and (for the hooks) cola_abi.hip.  Not part
// of the public ABI (that is include/cola.h).
#pragma once

#include "../../include/cola.h"
#include "internal.hpp"

namespace cola {

// ---- the decoder-block path (attention.hip, block_ops.hip) ----

// Causal multi-head attention over n_seq sequences of seq_len tokens: q, k,
// v, att, dO, dq, dk, dv are [n_seq * seq_len][ld] bf16 (head h in columns
// h * head_dim ..), lse and D [heads][T] fp32.  head_dim 64 or 128; rotary
// embedding of q and k with base rope_base inside the kernels.
struct AttnShape {
    int n_seq, seq_len, heads, head_dim;
    int64_t ld;
    float rope_base;
    const float* rope;    // the (cos, sin) table of launch_attn_rope_table
};
// The rotation table [seq_len][head_dim / 2] of (cos, sin) pairs that the
// attention kernels read: attn_rope_table_floats floats, filled by
// launch_attn_rope_table before them on the same stream.
int64_t attn_rope_table_floats(int seq_len, int head_dim);
hipError_t launch_attn_rope_table(const AttnShape& sh, float* rope, hipStream_t s);
// att = softmax(rope(q) rope(k)^T / sqrt(hd), causal) v; lse = log2-sum-exp
// of the scores scaled by log2(e) / sqrt(hd).
hipError_t launch_attn_fwd(const AttnShape& sh, const void* q, const void* k, const void* v, void* att, float* lse,
                           hipStream_t s);
// dq, dk, dv (gradients of the projections' outputs q, k, v) from dO and the
// forward's att and lse; D = rowsum(dO * att) per head is written on the way.
hipError_t launch_attn_bwd(const AttnShape& sh, const void* q, const void* k, const void* v, const void* att,
                           const float* lse, const void* dO, void* dq, void* dk, void* dv, float* D, hipStream_t s);

// RMSNorm over rows of d elements (bf16, row pitch ld): y = x g / sqrt(mean(x^2) + eps).
// With res != NULL the normalised input is x + res, rounded to bf16 and
// stored to xsum (the residual sum of the block).
hipError_t launch_rmsnorm_fwd(const void* x, const void* res, void* xsum, const void* g, void* y, int64_t T,
                              int64_t d, int64_t ld, float eps, hipStream_t s);
// Its backward for the upstream dy: out = res_grad + dx (bf16), and the gain
// gradient dg (fp32 [d]) as per-workgroup partial sums reduced in a fixed
// order; partials needs rmsnorm_bwd_partials(T, d) floats.
int64_t rmsnorm_bwd_partials(int64_t T, int64_t d);
hipError_t launch_rmsnorm_bwd(const void* x, const void* g, const void* dy, const void* res_grad, void* out,
                              float* dg, float* partials, int64_t T, int64_t d, int64_t ld, float eps,
                              hipStream_t s);
// Elementwise over [T][width] bf16 with row pitch ld (each operand its own):
//   MUL:  c = a * b          (the gated product)
//   ADD:  c = a + b          (a residual sum)
//   DMUL: c = g * b, c2 = g * a   for g = the gradient (the gated product's backward)
//   SIGMA: c = sigma(a)      (H of a saved pre-activation; act)
enum EwOp : int { EW_MUL = 0, EW_ADD = 1, EW_DMUL = 2, EW_SIGMA = 3 };
struct EwArgs {
    int op, act;
    int64_t T, width;
    const void* a; int64_t lda;
    const void* b; int64_t ldb;
    const void* g; int64_t ldg;
    void* c; int64_t ldc;
    void* c2; int64_t ldc2;
};
hipError_t launch_elementwise(const EwArgs& e, hipStream_t s);

// Hooks of cola_abi.hip for the block path: one launch bracketed by the
// timing events of class kc (when timing is on); the text behind
// COLA_ERR_HIP (returns COLA_ERR_HIP); and the up projection
// Y = H B^T (bf16, K2 of the layer) from a given H, B [d_out][r] contiguous
// with r a multiple of 8.
hipError_t timed_call(int kc, double flops, double bytes, hipStream_t s, hipError_t (*fn)(void*), void* ctx);
template <class F>
hipError_t timed_fn(int kc, double flops, double bytes, hipStream_t s, F f) {
    return timed_call(kc, flops, bytes, s, [](void* c) { return (*static_cast<F*>(c))(); }, &f);
}
int set_hip_error(hipError_t e, const char* where);
// Y = H B^T (bf16, B [d_out][r] with pitch r).  With `fused` non-NULL the
// gated product is tried in its epilogue: Y = u and m = g u (g, m with
// Y's pitch); *fused tells whether it ran (else the caller forms m).
hipError_t launch_up_projection(int64_t T, int64_t d_out, int64_t r, const void* H, int64_t ldh, const void* B,
                                void* Y, int64_t ldy, hipStream_t s, const void* g = nullptr, void* m = nullptr,
                                bool* fused = nullptr);
// cola_group_fwd whose last projection also stores m = g u (g the group's
// first output; g, u, m with pitch ld), and cola_bwd whose dX = dm GEMM
// stores dg = dm u and du = dm g instead (g, u, dg, du with pitch ld); each
// sets *fused to whether the fused epilogue ran (the ping-pong family takes
// the product and the fusion option is on), else the caller forms the
// products with the elementwise kernels.  keep_u false: a fused forward
// stores m only, leaving the last projection's Y unwritten.
int group_fwd_gated(const cola_group_desc* desc, const void* X, const void* A_all, const void* const* B,
                    void* const* Y, void* Z_all, void* H_all, void* ws, size_t ws_bytes, cola_stream_t stream,
                    const void* g, int64_t ld, void* m, bool* fused, bool keep_u);
int layer_bwd_gated(const cola_desc* desc, const void* dY, const void* X, const void* Z, const void* H,
                    const void* A, const void* B, void* dX, float* dA, float* dB, void* ws, size_t ws_bytes,
                    cola_stream_t stream, const void* g, const void* u, int64_t ld, void* dg, void* du,
                    bool* fused);

}  // namespace cola
