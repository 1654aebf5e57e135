/*
 * cola.h -- C ABI of libcola.so, the MI355X (gfx950) CoLA layer.
 *
 * The CoLA layer replaces a full-size linear projection h = W x by the
 * low-rank auto-encoder h = B sigma(A x), with A in R^{r x d_in},
 * B in R^{d_out x r} and sigma a pointwise nonlinearity
 * (arXiv 2502.10940, Sec. 3.2, Eq. main-fwd; the same layer replaces the
 * attention projections, Eq. full-rank-linear).  Its gradients follow the
 * paper's 2x rule, two GEMMs per forward GEMM (Sec. 3.4):
 *   dH = dY B,  dZ = dH (.) sigma'(Z),  dX = dZ A,  dA = dZ^T X,  dB = dY^T H.
 * CoLA-M (Sec. 4.2, App. C) saves only the r-wide pre-activation Z = A x and
 * recomputes H = sigma(Z) in backward; its outputs are bitwise those of CoLA.
 *
 * Layout.  Every tensor is row-major and token-major (one token per row; the
 * paper's X in R^{d_in x n} is stored transposed):
 *   X, dX  [T][ldx]  (d_in used per row)      A   [r][d_in]   contiguous
 *   Y, dY  [T][ldy]  (d_out used per row)     B   [d_out][r]  contiguous
 *   Z, H   [T][ldz]  (r used per row)         dA  [r][d_in]   fp32, contiguous
 *                                             dB  [d_out][r]  fp32, contiguous
 * A leading dimension of 0 means "contiguous" (ld = width).  Row padding
 * (ld > width) is never written.  It may be read up to the first multiple of
 * 8 elements past the width (bf16) -- values read there only reach outputs
 * that are discarded -- so a padded tensor must be allocated as rows x ld
 * elements.
 *
 * Precision.  COLA_BF16: activations and weights are bf16, every product is
 * accumulated in fp32, Z/H/dZ are rounded to bf16 (round to nearest even)
 * when stored, and H = bf16(sigma(Z_bf16)) in both modes; dA, dB are fp32.
 * COLA_F32: fp32 storage, fp32 arithmetic throughout (no reduced-precision
 * shortcut).
 *
 * Ownership and streams.  The caller allocates every buffer, including the
 * workspace sized by cola_workspace_bytes().  The library never allocates
 * device memory, never frees, never synchronises: all work is enqueued on the
 * given stream (a hipStream_t; NULL = the null stream), and the call returns
 * once it is enqueued.  Buffers must stay valid until that work completes.
 * Calls that share a workspace must be ordered on one stream.
 *
 * Errors.  Every entry point validates all of its arguments before it
 * enqueues anything; on any error nothing is enqueued and the outputs are
 * untouched.  No C++ exception crosses this boundary.
 *
 * Alignment.  Base pointers that are 16-byte aligned with ld a multiple of
 * 16 bytes take the vector path; anything else is accepted and takes a
 * per-element path (same results, slower).
 *
 * Determinism.  Results are bitwise reproducible run to run: the T-long
 * weight-gradient sums are split into a fixed number of chunks whose fp32
 * partials are added in a fixed order.
 */
#ifndef COLA_H
#define COLA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define COLA_ABI_VERSION 2

/* A hipStream_t, kept opaque so this header needs no HIP headers. */
typedef void* cola_stream_t;

typedef enum { COLA_F32 = 0, COLA_BF16 = 1 } cola_dtype;

/* sigma: identity (the conventional low-rank product B A x, Sec. 3.3),
 * SiLU z * logistic(z) (Swish, the activation of the paper's LLaMA runs), or
 * GeLU z * Phi(z) with Phi the standard normal CDF (the exact form; the
 * paper names GeLU for its BERT runs without saying which form). */
typedef enum { COLA_ACT_IDENTITY = 0, COLA_ACT_SILU = 1, COLA_ACT_GELU = 2 } cola_act;

/* Largest row pitch, in elements, of any activation or weight (and so of
 * any width): 2^22.  Wider descriptors are refused with COLA_ERR_BAD_SHAPE. */
#define COLA_MAX_PITCH (1LL << 22)

typedef enum {
    COLA_OK = 0,
    COLA_ERR_INVALID_ARG = 1,      /* NULL desc/pointer, bad enum, H vs recompute mismatch */
    COLA_ERR_BAD_SHAPE = 2,        /* d_in, d_out or r < 1, T < 0, ld < width, a row pitch above
                                      COLA_MAX_PITCH, size overflow */
    COLA_ERR_WORKSPACE = 3,        /* ws_bytes below the size cola_workspace_bytes() returns */
    COLA_ERR_HIP = 4,              /* a launch failed; cola_strerror() returns HIP's text */
    COLA_ERR_UNSUPPORTED = 5,      /* combination not compiled in */
    COLA_ERR_SCRATCH = 6           /* cola_bwd_scratch: needs more than COLA_SCRATCH_BYTES */
} cola_status;

typedef struct {
    int64_t T;          /* tokens (rows); T = 0 is an empty batch */
    int64_t d_in;       /* input width  (>= 1) */
    int64_t d_out;      /* output width (>= 1) */
    int64_t r;          /* rank (>= 1); r >= min(d_in, d_out) is accepted */
    int64_t ldx;        /* row pitch of X and dX in elements, 0 = d_in  */
    int64_t ldy;        /* row pitch of Y and dY in elements, 0 = d_out */
    int64_t ldz;        /* row pitch of Z and H in elements, 0 = r      */
    int32_t dtype;      /* cola_dtype */
    int32_t act;        /* cola_act */
    int32_t recompute;  /* 0 = CoLA (H stored), 1 = CoLA-M (only Z stored) */
} cola_desc;

int cola_abi_version(void);

/* Text for a status code; for COLA_ERR_HIP the text of the last failure. */
const char* cola_strerror(int status);

/* Workspace bytes for phase 0 (cola_fwd, cola_fwd_outer), 1 (cola_bwd),
 * 2 (cola_infer) or 3 (cola_bwd_outer); 0 on an invalid descriptor or phase.
 * Forward needs T*r elements when recompute = 1 (H lives only there), else
 * nothing.  Backward needs dZ (T*r elements), H again when recompute = 1, and
 * the fp32 partial sums of dA and dB.  Inference needs T*r elements for H
 * whatever recompute says.  The both-sigma backward needs the backward's
 * workspace plus T*d_out elements for dP.  Weights whose row length is not a
 * multiple of 8 (bf16) add a padded copy.  Buffers the library lays out
 * itself get row pitches of whole 128-byte cache lines.
 *
 * Layout advice for the caller's activations (X, Y, Z, H, dX, dY): rows must
 * be 16-byte aligned for the vector path (else a slower guarded path runs);
 * rows that start on 128-byte cache lines (pitch a multiple of 64 bf16 or 32
 * fp32 elements) are faster still -- up to 1.4x on a GEMM whose K-contiguous
 * operand would otherwise straddle lines (measured on MI355X). */
size_t cola_workspace_bytes(const cola_desc* desc, int phase);

/* Forward (Eq. main-fwd): Z = X A^T, H = sigma(Z), Y = H B^T.
 * Writes Z and Y; writes H when recompute = 0 (H must then be non-NULL unless
 * T = 0) and keeps H in the workspace when recompute = 1 (H must then be
 * NULL).  With T = 0 nothing is enqueued and activation pointers may be NULL. */
int cola_fwd(const cola_desc* desc,
             const void* X, const void* A, const void* B,
             void* Y, void* Z, void* H,
             void* ws, size_t ws_bytes, cola_stream_t stream);

/* Backward (Sec. 3.4, 2x rule; CoLA-M recompute per Sec. 4.2):
 *   dZ = (dY B) (.) sigma'(Z)   [and H = sigma(Z) into the workspace if recompute = 1]
 *   dX = dZ A,  dA = dZ^T X,  dB = dY^T H.
 * Reads the saved Z (and H when recompute = 0; H must be NULL when
 * recompute = 1).  dX is overwritten in the storage dtype; dA and dB are
 * overwritten in fp32 (not accumulated).  T = 0 writes dA = dB = 0. */
int cola_bwd(const cola_desc* desc,
             const void* dY, const void* X, const void* Z, const void* H,
             const void* A, const void* B,
             void* dX, float* dA, float* dB,
             void* ws, size_t ws_bytes, cola_stream_t stream);

/* Backward for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same computation and results as cola_bwd (bitwise), with its workspace in a
 * static device array of the library instead of a caller buffer.  Nothing is
 * allocated or freed by the call; the array (COLA_SCRATCH_BYTES per GPU) is
 * placed when the library's code object is loaded on a GPU and held until the
 * process ends.  Each GPU has its own array, shared by every call on that
 * GPU: calls that overlap on one GPU (concurrent streams, threads or graph
 * replays in flight) race on it and must be ordered by the caller.  A call
 * whose workspace (cola_workspace_bytes(desc, 1)) exceeds COLA_SCRATCH_BYTES
 * returns COLA_ERR_SCRATCH and enqueues nothing.  Arguments, ownership,
 * errors and T = 0 as cola_bwd. */
#define COLA_SCRATCH_BYTES ((size_t)64 << 20)
int cola_bwd_scratch(const cola_desc* desc,
                     const void* dY, const void* X, const void* Z, const void* H,
                     const void* A, const void* B,
                     void* dX, float* dA, float* dB, cola_stream_t stream);

/* The "both sigma" variant of the ablation (App. ablation, Table
 * "ablation"): the nonlinearity that followed the original linear layer is
 * kept on top of the layer, Y = sigma_out(B sigma(A x)), sigma_out given by
 * outer_act (a cola_act).
 * Forward: as cola_fwd, and K2 stores both P = H B^T (the output before
 * sigma_out, which the backward needs) and Y = sigma_out(P); P and Y are
 * [T][ldy] in the storage dtype, Y computed from P rounded to that dtype.
 * Backward: dP = dY (.) sigma_out'(P), rounded to the storage dtype, then the
 * backward of cola_bwd with dP in place of dY.  Workspace: phase 0 forward,
 * phase 3 backward.  Ownership, errors and the H/recompute rule as in
 * cola_fwd / cola_bwd; an invalid outer_act is COLA_ERR_INVALID_ARG. */
int cola_fwd_outer(const cola_desc* desc, int outer_act,
                   const void* X, const void* A, const void* B,
                   void* Y, void* P, void* Z, void* H,
                   void* ws, size_t ws_bytes, cola_stream_t stream);

int cola_bwd_outer(const cola_desc* desc, int outer_act,
                   const void* dY, const void* P, const void* X, const void* Z, const void* H,
                   const void* A, const void* B,
                   void* dX, float* dA, float* dB,
                   void* ws, size_t ws_bytes, cola_stream_t stream);

/* Inference forward (Eq. main-fwd with nothing kept for a backward pass; the
 * paper's inference comparison, App. "Inference Efficiency"):
 *   Y = sigma(X A^T) B^T
 * H lives only in the workspace (phase 2) and Z is never stored.  Y is
 * bitwise the Y of cola_fwd on the same inputs.  desc->recompute is ignored;
 * X, A, B, Y as in cola_fwd.  T = 0 enqueues nothing. */
int cola_infer(const cola_desc* desc,
               const void* X, const void* A, const void* B, void* Y,
               void* ws, size_t ws_bytes, cola_stream_t stream);

/* ------------------------------------------------------------------------
 * Grouped projections that read the same input (Sec. 3.2 applied to every
 * projection of a block: q, k, v of attention read the same X, and so do
 * gate and up of the MLP).  Projection p is its own CoLA layer
 * (A_p [r_p][d_in], B_p [d_out_p][r_p], one sigma for the group); the group
 * runs the shared-input products once:
 *   forward:  Z_all = X [A_1; ..; A_n]^T           one GEMM, N = R = sum r_p
 *             H_p = sigma(Z_p),  Y_p = H_p B_p^T    per projection
 *   backward: dZ_p = (dY_p B_p) (.) sigma'(Z_p)     per projection
 *             dX = sum_p dZ_p A_p                  one GEMM, K = R
 *             [dA_1; ..; dA_n] = dZ_all^T X         one GEMM, M = R
 *             dB_p = dY_p^T H_p                     per projection
 * The results are those of cola_fwd / cola_bwd run on each projection, except
 * that dX is the sum of the projections' input gradients (the gradient of
 * the shared input).  X is read once instead of n times in each direction.
 *
 * Layout: A_all [R][d_in] and dA_all [R][d_in] (fp32) contiguous, projection
 * p in rows R_p .. R_p + r_p - 1 with R_p = r_0 + .. + r_{p-1};
 * Z_all, H_all [T][ldz], projection p in columns R_p ..; per projection
 * B_p [d_out_p][r_p] and dB_p (fp32) contiguous, Y_p / dY_p [T][ldy_p];
 * X, dX [T][ldx].  B, Y, dY, dB are arrays of n pointers.  Ownership,
 * streams, padding, precision, errors and CoLA-M (recompute = 1: H_all NULL,
 * kept in the workspace) follow cola_fwd / cola_bwd.  n is 1 .. 8.
 * ------------------------------------------------------------------------ */
#define COLA_GROUP_MAX 8

typedef struct {
    int64_t T;                        /* tokens (rows); T = 0 is an empty batch */
    int64_t d_in;                     /* shared input width (>= 1) */
    int32_t n;                        /* projections, 1 .. COLA_GROUP_MAX */
    int32_t dtype;                    /* cola_dtype */
    int32_t act;                      /* cola_act */
    int32_t recompute;                /* 0 = CoLA, 1 = CoLA-M */
    int64_t r[COLA_GROUP_MAX];        /* ranks (>= 1); R = r[0] + .. + r[n-1] */
    int64_t d_out[COLA_GROUP_MAX];    /* output widths (>= 1) */
    int64_t ldy[COLA_GROUP_MAX];      /* row pitch of Y_p and dY_p, 0 = d_out[p] */
    int64_t ldx;                      /* row pitch of X and dX, 0 = d_in */
    int64_t ldz;                      /* row pitch of Z_all and H_all, 0 = R */
} cola_group_desc;

/* Workspace bytes for phase 0 (forward), 1 (backward) or 2 (inference); 0
 * on an invalid descriptor or phase. */
size_t cola_group_workspace_bytes(const cola_group_desc* desc, int phase);

int cola_group_fwd(const cola_group_desc* desc,
                   const void* X, const void* A_all, const void* const* B,
                   void* const* Y, void* Z_all, void* H_all,
                   void* ws, size_t ws_bytes, cola_stream_t stream);

/* Inference forward of the group (cola_infer per projection, with the
 * shared-input GEMM run once): Y_p = sigma(X A_p^T) B_p^T, H_all only in
 * the workspace (phase 2), no Z.  desc->recompute and desc->ldz are ignored;
 * each Y_p is bitwise that of cola_group_fwd. */
int cola_group_infer(const cola_group_desc* desc,
                     const void* X, const void* A_all, const void* const* B,
                     void* const* Y, void* ws, size_t ws_bytes, cola_stream_t stream);

/* dX is overwritten with sum_p dZ_p A_p; dA_all and every dB_p are
 * overwritten (fp32).  T = 0 writes dA_all = 0 and dB_p = 0. */
int cola_group_bwd(const cola_group_desc* desc,
                   const void* const* dY, const void* X, const void* Z_all, const void* H_all,
                   const void* A_all, const void* const* B,
                   void* dX, float* dA_all, float* const* dB,
                   void* ws, size_t ws_bytes, cola_stream_t stream);

/* Dense full-rank baseline on the same kernels (Eq. full-rank-linear and
 * the 2x rule of Sec. 3.4): Y = X W^T, dX = dY W, dW = dY^T X, with
 * W [d_out][d_in] contiguous and dW fp32 contiguous. */
typedef struct {
    int64_t T, d_in, d_out;
    int64_t ldx, ldy;   /* 0 = contiguous */
    int32_t dtype;      /* cola_dtype */
} dense_desc;

size_t dense_workspace_bytes(const dense_desc* desc, int phase);
int dense_fwd(const dense_desc* desc, const void* X, const void* W, void* Y,
              void* ws, size_t ws_bytes, cola_stream_t stream);
int dense_bwd(const dense_desc* desc, const void* dY, const void* X, const void* W,
              void* dX, float* dW, void* ws, size_t ws_bytes, cola_stream_t stream);

/* ------------------------------------------------------------------------
 * Decoder block: a LLaMA-style pre-norm block whose seven linear projections
 * are CoLA layers (Sec. 3.2, Fig. "block"), in CoLA or block-level CoLA-M
 * (Sec. 4.2, App. C).  The self-attention's scaled dot product, the residual
 * connections and the gated product of the MLP are the usual ones; with only
 * the low-rank sigma (the paper's 1B/7B setting, App. ablation) the MLP is
 * down(gate(b) (.) up(b)) without the original SiLU:
 *   a   = rmsnorm(x0) (.) g1
 *   q, k, v = CoLA_q(a), CoLA_k(a), CoLA_v(a)                    (one group)
 *   att = per sequence and head, softmax(rope(q) rope(k)^T / sqrt(hd),
 *         causal) v       (hd = d / heads; RoPE pairs element i of a head
 *         with i + hd/2, angle pos * rope_base^(-2i/hd), pos = the token's
 *         index in its sequence)
 *   x1  = x0 + CoLA_o(att)
 *   b   = rmsnorm(x1) (.) g2,   rmsnorm(x) = x / sqrt(mean(x^2) + eps)
 *   gt, u = CoLA_gate(b), CoLA_up(b)                             (one group)
 *   x2  = x1 + CoLA_down(gt (.) u)
 * CoLA keeps every activation the backward reads in `saved` (and the
 * log2-sum-exp of the attention scores).  CoLA-M keeps x1 and the seven
 * r-wide pre-activations Z only (with the caller's x0: 2nd + 7nr values,
 * App. C); its backward recomputes the norms, the up projections
 * B sigma(Z) of q, k, v, gate and up, the gated product and the attention,
 * then runs the same backward.  Both modes give bitwise the same outputs.
 *
 * Tensors: x0, x2, dx2, dx0 are [T][d] bf16 contiguous, T = n_seq * seq_len,
 * sequence s in rows s*seq_len ..; weights bf16 contiguous, gradients fp32
 * contiguous (overwritten), in the shapes of cola_block_weights.  The layout
 * of `saved` is the library's (cola_block_saved_slot gives each tensor's
 * offset and pitch).  bf16 only; head_dim 64 or 128; d and r multiples of 8;
 * 3r and ffn, rounded up to multiples of 64, at most COLA_MAX_PITCH;
 * x0, x2, dx2, dx0, g1, g2, saved and ws 16-byte aligned (else
 * COLA_ERR_INVALID_ARG); n_seq and heads at most 65535.
 * Ownership, streams and errors as for cola_fwd; T = 0 enqueues nothing in
 * the forward and zero-fills the gradients in the backward.
 * ------------------------------------------------------------------------ */
typedef struct {
    int64_t n_seq, seq_len;   /* sequences and tokens per sequence (>= 1) */
    int64_t d, ffn, heads;    /* model width, MLP width, attention heads */
    int64_t r;                /* rank of all seven projections */
    int32_t act;              /* cola_act of the CoLA layers */
    int32_t recompute;        /* 0 = CoLA, 1 = CoLA-M */
    float rope_base;          /* rotary base, e.g. 10000 */
    float eps;                /* RMSNorm epsilon, e.g. 1e-6 */
} cola_block_desc;

typedef struct {
    const void *g1, *g2;              /* [d] RMSNorm gains */
    const void *A_qkv;                /* [3r][d]: A_q, A_k, A_v stacked */
    const void *B_q, *B_k, *B_v;      /* [d][r] each */
    const void *A_o, *B_o;            /* [r][d], [d][r] */
    const void *A_gu;                 /* [2r][d]: A_gate, A_up stacked */
    const void *B_g, *B_u;            /* [ffn][r] each */
    const void *A_d, *B_d;            /* [r][ffn], [d][r] */
} cola_block_weights;

typedef struct {                      /* fp32, shapes as cola_block_weights */
    float *g1, *g2, *A_qkv, *B_q, *B_k, *B_v, *A_o, *B_o, *A_gu, *B_g, *B_u, *A_d, *B_d;
} cola_block_grads;

/* Tensors in `saved` (cola_block_saved_slot): x1, the pre-activations Z of
 * q,k,v [T][3r], o [T][r], gate,up [T][2r], down [T][r] (both modes); CoLA
 * also a, H_qkv, q, k, v, att, the attention's log2-sum-exp (fp32
 * [heads][T], scores scaled by log2(e)/sqrt(hd)), H_o, b, H_gu, gt, u, m =
 * gt (.) u, H_down. */
typedef enum {
    COLA_BLK_X1 = 0, COLA_BLK_Z_QKV, COLA_BLK_Z_O, COLA_BLK_Z_GU, COLA_BLK_Z_DOWN,
    COLA_BLK_A, COLA_BLK_H_QKV, COLA_BLK_Q, COLA_BLK_K, COLA_BLK_V, COLA_BLK_ATT, COLA_BLK_LSE,
    COLA_BLK_H_O, COLA_BLK_B, COLA_BLK_H_GU, COLA_BLK_GATE, COLA_BLK_UP, COLA_BLK_M, COLA_BLK_H_DOWN,
    COLA_BLK_SLOTS
} cola_block_slot;

/* Bytes of `saved` for the descriptor's mode; 0 on an invalid descriptor. */
size_t cola_block_saved_bytes(const cola_block_desc* desc);
/* Byte offset and row pitch (elements) of a slot in `saved`; returns
 * COLA_ERR_INVALID_ARG for a slot the mode does not keep. */
int cola_block_saved_slot(const cola_block_desc* desc, int slot, size_t* offset, int64_t* ld);
/* Workspace bytes for phase 0 (forward) or 1 (backward); 0 if invalid. */
size_t cola_block_workspace_bytes(const cola_block_desc* desc, int phase);

int cola_block_fwd(const cola_block_desc* desc, const cola_block_weights* w, const void* x0, void* x2,
                   void* saved, size_t saved_bytes, void* ws, size_t ws_bytes, cola_stream_t stream);
/* x0: the forward's input (the caller keeps it); dx0 is overwritten. */
int cola_block_bwd(const cola_block_desc* desc, const cola_block_weights* w, const void* x0,
                   const void* saved, size_t saved_bytes, const void* dx2, void* dx0,
                   const cola_block_grads* grads, void* ws, size_t ws_bytes, cola_stream_t stream);

/* Tuning options, process-wide (every GPU and thread of the process), read
 * at each call; for tuning, comparisons and tests, not needed for correct
 * results.  Every setting gives results within the stated tolerances;
 * settings differ at most in the last bits of fp32 sums.
 *   COLA_OPT_STREAM_ONLY (default 0): 1 sends every bf16 product to the
 *     streaming kernel family (BM x 128 tiles) instead of the 256 x 256
 *     ping-pong family.
 *   COLA_OPT_WGRAD_PAIR (default 1): 0 launches the two weight gradients of a
 *     layer (and of a group) one by one instead of in one launch.
 *   COLA_OPT_FUSE_GATE (default 1): 0 keeps the decoder block's gated
 *     product (m = gate * up) and its backward in separate elementwise
 *     kernels instead of the epilogues of the up projection's Y = H B^T and
 *     the down projection's dX = dZ A (same roundings, so the same bits).
 * Workspace sizes depend on the settings: size the workspace after setting
 * them (a call whose workspace is too small returns COLA_ERR_WORKSPACE).
 * cola_set_option returns COLA_ERR_INVALID_ARG for an unknown option or a
 * value other than 0 or 1; cola_get_option returns the value, or -1. */
typedef enum { COLA_OPT_STREAM_ONLY = 0, COLA_OPT_WGRAD_PAIR = 1, COLA_OPT_FUSE_GATE = 2 } cola_option;
int cola_set_option(int option, int value);
int cola_get_option(int option);

/* Kernel timing (profiling aid).  While enabled, every kernel the library
 * launches is bracketed by two HIP events on its stream; reading sums the
 * elapsed times per kernel class and waits for the recorded events.
 * Kernel classes: */
typedef enum {
    COLA_KC_FWD_Z = 0,     /* Z = X A^T with the sigma epilogue        */
    COLA_KC_FWD_Y = 1,     /* Y = H B^T                                */
    COLA_KC_BWD_DZ = 2,    /* dZ = (dY B) (.) sigma'(Z) [+ H recompute] */
    COLA_KC_BWD_DX = 3,    /* dX = dZ A                                */
    COLA_KC_BWD_DA = 4,    /* dA = dZ^T X (split over tokens)          */
    COLA_KC_BWD_DB = 5,    /* dB = dY^T H (split over tokens)          */
    COLA_KC_REDUCE = 6,    /* fixed-order sum of the dA/dB partials    */
    COLA_KC_DENSE_FWD = 7, /* Y = X W^T                                */
    COLA_KC_DENSE_DX = 8,  /* dX = dY W                                */
    COLA_KC_DENSE_DW = 9,  /* dW = dY^T X                              */
    COLA_KC_FILL = 10,     /* zero fill (empty batches)                */
    COLA_KC_INFER_H = 11,  /* H = sigma(X A^T), Z not kept (inference) */
    COLA_KC_OUTER_GRAD = 12, /* dP = dY (.) sigma_out'(P), both-sigma variant */
    COLA_KC_BWD_DADB = 13, /* dA and dB in one launch (bf16, both outputs
                              wider than 128): the two token-split weight
                              gradients share the launch and the split    */
    COLA_KC_ATTN_FWD = 14, /* block: causal attention forward             */
    COLA_KC_ATTN_BWD = 15, /* block: attention backward (dq, then dk dv)  */
    COLA_KC_NORM = 16,     /* block: RMSNorm forward (+ residual sum)     */
    COLA_KC_NORM_BWD = 17, /* block: RMSNorm backward (+ residual grad)   */
    COLA_KC_POINTWISE = 18,/* block: gated product, residual add, sigma   */
    COLA_KC_COUNT = 19
} cola_kernel_class;

/* Per-class totals since the last reset: launches, elapsed milliseconds,
 * algorithmic flops (2 M N K per GEMM) and algorithmic bytes (each operand
 * read once, each output written once).  Returns COLA_ERR_INVALID_ARG for a
 * bad class or NULL pointers, COLA_ERR_HIP if an event failed. */
int cola_timing_enable(int on);
int cola_timing_reset(void);
int cola_timing_read(int kernel_class, int64_t* launches, double* ms,
                     double* flops, double* bytes);
const char* cola_kernel_name(int kernel_class);

#ifdef __cplusplus
}
#endif

#endif /* COLA_H */
