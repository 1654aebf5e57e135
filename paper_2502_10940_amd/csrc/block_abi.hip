// block_abi.hip -- the decoder-block entry points of libcola.so (include/cola.h,
// cola_block_*): a LLaMA-style pre-norm block whose seven linear projections
// are CoLA layers (Sec. 3.2, Fig. "block"), forward and backward, in CoLA or
// block-level CoLA-M (Sec. 4.2, App. C: keep x1 and the seven r-wide
// pre-activations, recompute the up projections and the attention).
//
// The projections run through the layer entry points (q, k, v and gate, up as
// same-input groups); the rest is attention.hip and block_ops.hip.  The gated
// product and its backward run in GEMM epilogues where the ping-pong family
// takes the product (else, and with COLA_OPT_FUSE_GATE = 0, in elementwise
// kernels: same roundings, same bits).  Launch order, one stream:
//   forward : a = norm(x0); Z,H,q,k,v (group); att, lse; Z,H,o; x1 = x0 + o and
//             b = norm(x1) (one pass); Z,H,gt,u (group) with m = gt u (in
//             up's GEMM epilogue); Z,H,y (down); x2 = x1 + y
//   backward: [CoLA-M: b = norm(x1); H_gu = sigma(Z_gu); gt, u = H B^T, m]
//             down bwd with dgt, du = dm u, dm gt (in its dX GEMM epilogue);
//             gate/up bwd -> db;
//             dx1 = dx2 + norm_bwd(db) (+ dg2);
//             [CoLA-M: a = norm(x0); H_qkv = sigma(Z_qkv); q, k, v = H B^T; att, lse]
//             o bwd -> datt; attention bwd -> dq, dk, dv; q/k/v bwd -> da;
//             dx0 = dx1 + norm_bwd(da) (+ dg1)
#include <math.h>
#include <string.h>

#include <new>

#include "../../include/cola.h"
#include "internal.hpp"
#include "block.hpp"

using namespace cola;

namespace {

constexpr int64_t kMaxDim = int64_t(1) << 32;

size_t a256(size_t x) { return (x + 255) & ~size_t(255); }
int64_t lp64(int64_t w) { return (w + 63) / 64 * 64; }   // a whole number of 128-byte lines (bf16)

struct Blk {
    int64_t n_seq, L, T, d, ffn, heads, hd, r;
    int act;
    bool m;                 // CoLA-M
    float base, eps;
    int64_t ld3, ld2, ld1, ldf;   // pitches of [T][3r], [T][2r], [T][r], [T][ffn]
};

int check_block(const cola_block_desc* dsc, Blk* out) {
    if (!dsc) return COLA_ERR_INVALID_ARG;
    if (dsc->act != COLA_ACT_IDENTITY && dsc->act != COLA_ACT_SILU && dsc->act != COLA_ACT_GELU)
        return COLA_ERR_INVALID_ARG;
    if (dsc->recompute != 0 && dsc->recompute != 1) return COLA_ERR_INVALID_ARG;
    if (!(dsc->rope_base > 0.0f) || !isfinite(dsc->rope_base) || !(dsc->eps >= 0.0f) || !isfinite(dsc->eps))
        return COLA_ERR_INVALID_ARG;
    if (dsc->n_seq < 0 || dsc->seq_len < 1 || dsc->d < 8 || dsc->ffn < 1 || dsc->heads < 1 || dsc->r < 1)
        return COLA_ERR_BAD_SHAPE;
    if (dsc->n_seq > 65535 || dsc->heads > 65535) return COLA_ERR_BAD_SHAPE;   // attention grid dimensions
    if (dsc->n_seq > kMaxDim || dsc->seq_len > kMaxDim || dsc->d > 8192 || dsc->ffn > kMaxDim || dsc->r > kMaxDim)
        return COLA_ERR_BAD_SHAPE;
    if (dsc->d % 8 != 0 || dsc->r % 8 != 0 || dsc->d % dsc->heads != 0) return COLA_ERR_BAD_SHAPE;
    const int64_t hd = dsc->d / dsc->heads;
    if (hd != 64 && hd != 128) return COLA_ERR_UNSUPPORTED;
    Blk b;
    b.n_seq = dsc->n_seq; b.L = dsc->seq_len; b.T = dsc->n_seq * dsc->seq_len;
    b.d = dsc->d; b.ffn = dsc->ffn; b.heads = dsc->heads; b.hd = hd; b.r = dsc->r;
    b.act = dsc->act; b.m = dsc->recompute == 1; b.base = dsc->rope_base; b.eps = dsc->eps;
    if ((double)b.T * (double)(b.ffn > b.d ? b.ffn : b.d) > 4.0e15) return COLA_ERR_BAD_SHAPE;
    if (b.T > (int64_t(1) << 31)) return COLA_ERR_BAD_SHAPE;
    b.ld3 = lp64(3 * b.r); b.ld2 = lp64(2 * b.r); b.ld1 = lp64(b.r); b.ldf = lp64(b.ffn);
    if (b.ld3 > kMaxPitch || b.ldf > kMaxPitch) return COLA_ERR_BAD_SHAPE;
    *out = b;
    return COLA_OK;
}

// ---- layout of `saved` ----
struct Saved {
    size_t off[COLA_BLK_SLOTS];
    int64_t ld[COLA_BLK_SLOTS];
    bool kept[COLA_BLK_SLOTS];
    size_t total;
};

Saved plan_saved(const Blk& b) {
    Saved s{};
    size_t at = 0;
    auto put = [&](int slot, int64_t ld, size_t esz, int64_t rows) {
        s.off[slot] = at;
        s.ld[slot] = ld;
        s.kept[slot] = true;
        at += a256((size_t)rows * (size_t)ld * esz);
    };
    put(COLA_BLK_X1, b.d, 2, b.T);
    put(COLA_BLK_Z_QKV, b.ld3, 2, b.T);
    put(COLA_BLK_Z_O, b.ld1, 2, b.T);
    put(COLA_BLK_Z_GU, b.ld2, 2, b.T);
    put(COLA_BLK_Z_DOWN, b.ld1, 2, b.T);
    if (!b.m) {
        put(COLA_BLK_A, b.d, 2, b.T);
        put(COLA_BLK_H_QKV, b.ld3, 2, b.T);
        put(COLA_BLK_Q, b.d, 2, b.T);
        put(COLA_BLK_K, b.d, 2, b.T);
        put(COLA_BLK_V, b.d, 2, b.T);
        put(COLA_BLK_ATT, b.d, 2, b.T);
        put(COLA_BLK_LSE, b.T, 4, b.heads);
        put(COLA_BLK_H_O, b.ld1, 2, b.T);
        put(COLA_BLK_B, b.d, 2, b.T);
        put(COLA_BLK_H_GU, b.ld2, 2, b.T);
        put(COLA_BLK_GATE, b.ldf, 2, b.T);
        put(COLA_BLK_UP, b.ldf, 2, b.T);
        put(COLA_BLK_M, b.ldf, 2, b.T);
        put(COLA_BLK_H_DOWN, b.ld1, 2, b.T);
    }
    s.total = b.T == 0 ? 0 : at;
    return s;
}

// ---- the sub-calls' descriptors ----
cola_group_desc qkv_desc(const Blk& b, int recompute) {
    cola_group_desc g{};
    g.T = b.T; g.d_in = b.d; g.n = 3; g.dtype = COLA_BF16; g.act = b.act; g.recompute = recompute;
    for (int p = 0; p < 3; ++p) { g.r[p] = b.r; g.d_out[p] = b.d; g.ldy[p] = b.d; }
    g.ldx = b.d; g.ldz = b.ld3;
    return g;
}
cola_group_desc gu_desc(const Blk& b, int recompute) {
    cola_group_desc g{};
    g.T = b.T; g.d_in = b.d; g.n = 2; g.dtype = COLA_BF16; g.act = b.act; g.recompute = recompute;
    for (int p = 0; p < 2; ++p) { g.r[p] = b.r; g.d_out[p] = b.ffn; g.ldy[p] = b.ldf; }
    g.ldx = b.d; g.ldz = b.ld2;
    return g;
}
cola_desc o_desc(const Blk& b, int recompute) {
    cola_desc c{};
    c.T = b.T; c.d_in = b.d; c.d_out = b.d; c.r = b.r; c.ldx = b.d; c.ldy = b.d; c.ldz = b.ld1;
    c.dtype = COLA_BF16; c.act = b.act; c.recompute = recompute;
    return c;
}
cola_desc down_desc(const Blk& b, int recompute) {
    cola_desc c{};
    c.T = b.T; c.d_in = b.ffn; c.d_out = b.d; c.r = b.r; c.ldx = b.ldf; c.ldy = b.d; c.ldz = b.ld1;
    c.dtype = COLA_BF16; c.act = b.act; c.recompute = recompute;
    return c;
}

size_t smax(size_t a, size_t b) { return a > b ? a : b; }

// ---- workspace layouts ----
struct Ws {
    size_t sub, sub_bytes;                 // the sub-calls' workspace
    size_t rope;                           // the attention's rotation table
    size_t tmp;                            // forward: o and y before their residual sums  [T][d]
    // transients of CoLA-M (forward: everything CoLA would keep; backward: the recomputes)
    size_t a, q, k, v, att, lse, b, hqkv, hgu, gt, up, m;
    // backward
    size_t dx1, datt, dq, dk, dv, db, da, dm, dgt, du, D, part;
    size_t total;
};

Ws plan_ws(const Blk& b, int phase) {
    Ws w{};
    size_t at = 0;
    auto take = [&](size_t bytes) {
        const size_t o = at;
        at += a256(bytes);
        return o;
    };
    const size_t nd = (size_t)b.T * (size_t)b.d * 2, nf = (size_t)b.T * (size_t)b.ldf * 2;
    const size_t nl = (size_t)b.T * (size_t)b.heads * 4;
    const int rc = b.m ? 1 : 0;
    if (phase == 0) {
        const cola_group_desc g1 = qkv_desc(b, rc), g2 = gu_desc(b, rc);
        const cola_desc c1 = o_desc(b, rc), c2 = down_desc(b, rc);
        w.sub_bytes = smax(smax(cola_group_workspace_bytes(&g1, 0), cola_group_workspace_bytes(&g2, 0)),
                           smax(cola_workspace_bytes(&c1, 0), cola_workspace_bytes(&c2, 0)));
        w.sub = take(w.sub_bytes);
        w.rope = take((size_t)attn_rope_table_floats((int)b.L, (int)b.hd) * 4);
        w.tmp = take(nd);
        if (b.m) {
            w.a = take(nd); w.q = take(nd); w.k = take(nd); w.v = take(nd); w.att = take(nd); w.lse = take(nl);
            w.b = take(nd); w.gt = take(nf); w.up = take(nf); w.m = take(nf);
        }
    } else {
        // the groups take H (kept or recomputed), the single layers regenerate it in CoLA-M
        const cola_group_desc g1 = qkv_desc(b, 0), g2 = gu_desc(b, 0);
        const cola_desc c1 = o_desc(b, rc), c2 = down_desc(b, rc);
        w.sub_bytes = smax(smax(cola_group_workspace_bytes(&g1, 1), cola_group_workspace_bytes(&g2, 1)),
                           smax(cola_workspace_bytes(&c1, 1), cola_workspace_bytes(&c2, 1)));
        w.sub = take(w.sub_bytes);
        w.rope = take((size_t)attn_rope_table_floats((int)b.L, (int)b.hd) * 4);
        w.dx1 = take(nd); w.datt = take(nd); w.dq = take(nd); w.dk = take(nd); w.dv = take(nd);
        w.db = take(nd); w.da = take(nd); w.dm = take(nf); w.dgt = take(nf); w.du = take(nf);
        w.D = take(nl);
        w.part = take((size_t)rmsnorm_bwd_partials(b.T, b.d) * 4);
        if (b.m) {
            w.a = take(nd); w.q = take(nd); w.k = take(nd); w.v = take(nd); w.att = take(nd); w.lse = take(nl);
            w.b = take(nd); w.gt = take(nf); w.up = take(nf); w.m = take(nf);
            w.hqkv = take((size_t)b.T * (size_t)b.ld3 * 2);
            w.hgu = take((size_t)b.T * (size_t)b.ld2 * 2);
        }
    }
    w.total = b.T == 0 ? 0 : at;
    return w;
}

// ---- launches with their timing classes ----
struct Ctx {
    const Blk& b;
    hipStream_t s;
    const float* rope;      // the rotation table in the workspace
};

int chk(hipError_t e, const char* where) { return e == hipSuccess ? COLA_OK : set_hip_error(e, where); }

// causal (query, key) pairs per sequence and head: the attention's algorithmic work
double causal_pairs(const Blk& b) { return (double)b.L * (double)(b.L + 1) / 2.0; }

int norm_fwd(const Ctx& c, const void* x, const void* res, void* xsum, const void* g, void* y) {
    const Blk& b = c.b;
    const double bytes = 2.0 * (double)b.T * b.d * (res ? 4.0 : 2.0);
    return chk(timed_fn(COLA_KC_NORM, 0.0, bytes, c.s, [&] {
                   return launch_rmsnorm_fwd(x, res, xsum, g, y, b.T, b.d, b.d, b.eps, c.s);
               }), "rmsnorm");
}

int norm_bwd(const Ctx& c, const void* x, const void* g, const void* dy, const void* res_grad, void* out, float* dg,
             float* part) {
    const Blk& b = c.b;
    const double bytes = 2.0 * (double)b.T * b.d * 4.0;
    return chk(timed_fn(COLA_KC_NORM_BWD, 0.0, bytes, c.s, [&] {
                   return launch_rmsnorm_bwd(x, g, dy, res_grad, out, dg, part, b.T, b.d, b.d, b.eps, c.s);
               }), "rmsnorm_bwd");
}

int ew(const Ctx& c, int op, int64_t width, const void* a, int64_t lda, const void* bb, int64_t ldb, const void* g,
       int64_t ldg, void* out, int64_t ldc, void* out2, int64_t ldc2) {
    const Blk& b = c.b;
    EwArgs e{};
    e.op = op; e.act = b.act; e.T = b.T; e.width = width;
    e.a = a; e.lda = lda; e.b = bb; e.ldb = ldb; e.g = g; e.ldg = ldg; e.c = out; e.ldc = ldc; e.c2 = out2; e.ldc2 = ldc2;
    const double nops = op == EW_SIGMA ? 2.0 : (op == EW_DMUL ? 5.0 : 3.0);
    const double bytes = 2.0 * (double)b.T * width * nops;
    return chk(timed_fn(COLA_KC_POINTWISE, 0.0, bytes, c.s, [&] { return launch_elementwise(e, c.s); }),
               "pointwise");
}

AttnShape attn_shape(const Blk& b, const float* rope) {
    AttnShape a{};
    a.n_seq = (int)b.n_seq; a.seq_len = (int)b.L; a.heads = (int)b.heads; a.head_dim = (int)b.hd;
    a.ld = b.d; a.rope_base = b.base; a.rope = rope;
    return a;
}

int rope_table(const Ctx& c, float* rope) {
    const AttnShape sh = attn_shape(c.b, rope);
    return chk(timed_fn(COLA_KC_POINTWISE, 0.0, 8.0 * (double)c.b.L * c.b.hd / 2.0, c.s,
                        [&] { return launch_attn_rope_table(sh, rope, c.s); }), "rope_table");
}

int attn_fwd(const Ctx& c, const void* q, const void* k, const void* v, void* att, float* lse) {
    const Blk& b = c.b;
    const double flops = 4.0 * causal_pairs(b) * (double)b.hd * (double)b.heads * (double)b.n_seq;
    const double bytes = 2.0 * (double)b.T * b.d * 4.0 + 4.0 * (double)b.T * b.heads;
    const AttnShape sh = attn_shape(b, c.rope);
    return chk(timed_fn(COLA_KC_ATTN_FWD, flops, bytes, c.s, [&] { return launch_attn_fwd(sh, q, k, v, att, lse, c.s); }),
               "attn_fwd");
}

int attn_bwd(const Ctx& c, const void* q, const void* k, const void* v, const void* att, const float* lse,
             const void* dO, void* dq, void* dk, void* dv, float* D) {
    const Blk& b = c.b;
    const double flops = 8.0 * causal_pairs(b) * (double)b.hd * (double)b.heads * (double)b.n_seq;
    const double bytes = 2.0 * (double)b.T * b.d * 8.0 + 8.0 * (double)b.T * b.heads;
    const AttnShape sh = attn_shape(b, c.rope);
    return chk(timed_fn(COLA_KC_ATTN_BWD, flops, bytes, c.s,
                        [&] { return launch_attn_bwd(sh, q, k, v, att, lse, dO, dq, dk, dv, D, c.s); }),
               "attn_bwd");
}

int up(const Ctx& c, int64_t d_out, const void* H, int64_t ldh, const void* B, void* Y, int64_t ldy) {
    return chk(launch_up_projection(c.b.T, d_out, c.b.r, H, ldh, B, Y, ldy, c.s), "up_projection");
}

template <class F>
int guarded(F&& f) {
    try {
        return f();
    } catch (...) {
        return set_hip_error(hipErrorUnknown, "unexpected host exception");
    }
}

bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool weights_ok(const cola_block_weights* w) {
    return w && w->g1 && w->g2 && w->A_qkv && w->B_q && w->B_k && w->B_v && w->A_o && w->B_o && w->A_gu && w->B_g &&
           w->B_u && w->A_d && w->B_d && al16(w->g1) && al16(w->g2);
}
bool grads_ok(const cola_block_grads* g) {
    return g && g->g1 && g->g2 && g->A_qkv && g->B_q && g->B_k && g->B_v && g->A_o && g->B_o && g->A_gu && g->B_g &&
           g->B_u && g->A_d && g->B_d;
}

}  // namespace

extern "C" {

size_t cola_block_saved_bytes(const cola_block_desc* desc) {
    Blk b;
    if (check_block(desc, &b) != COLA_OK) return 0;
    return plan_saved(b).total;
}

int cola_block_saved_slot(const cola_block_desc* desc, int slot, size_t* offset, int64_t* ld) {
    Blk b;
    const int st = check_block(desc, &b);
    if (st != COLA_OK) return st;
    if (slot < 0 || slot >= COLA_BLK_SLOTS || !offset || !ld) return COLA_ERR_INVALID_ARG;
    const Saved s = plan_saved(b);
    if (!s.kept[slot]) return COLA_ERR_INVALID_ARG;
    *offset = s.off[slot];
    *ld = s.ld[slot];
    return COLA_OK;
}

size_t cola_block_workspace_bytes(const cola_block_desc* desc, int phase) {
    Blk b;
    if (check_block(desc, &b) != COLA_OK || (phase != 0 && phase != 1)) return 0;
    return plan_ws(b, phase).total;
}

int cola_block_fwd(const cola_block_desc* desc, const cola_block_weights* w, const void* x0, void* x2, void* saved,
                   size_t saved_bytes, void* ws, size_t ws_bytes, cola_stream_t stream) {
    return guarded([&]() -> int {
        Blk b;
        int st = check_block(desc, &b);
        if (st != COLA_OK) return st;
        if (!weights_ok(w)) return COLA_ERR_INVALID_ARG;
        if (b.T == 0) return COLA_OK;
        if (!x0 || !x2 || !saved || !al16(x0) || !al16(x2) || !al16(saved) || (ws && !al16(ws)))
            return COLA_ERR_INVALID_ARG;
        const Saved S = plan_saved(b);
        const Ws W = plan_ws(b, 0);
        if (saved_bytes < S.total) return COLA_ERR_WORKSPACE;
        if (W.total > 0 && (!ws || ws_bytes < W.total)) return COLA_ERR_WORKSPACE;
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        char* sv = static_cast<char*>(saved);
        char* wk = static_cast<char*>(ws);
        const Ctx c{b, s, reinterpret_cast<const float*>(wk + W.rope)};
        if ((st = rope_table(c, reinterpret_cast<float*>(wk + W.rope))) != COLA_OK) return st;
        auto SV = [&](int slot) -> char* { return sv + S.off[slot]; };
        // where each activation lives: `saved` (CoLA) or the workspace (CoLA-M)
        char* a = b.m ? wk + W.a : SV(COLA_BLK_A);
        char* q = b.m ? wk + W.q : SV(COLA_BLK_Q);
        char* k = b.m ? wk + W.k : SV(COLA_BLK_K);
        char* v = b.m ? wk + W.v : SV(COLA_BLK_V);
        char* att = b.m ? wk + W.att : SV(COLA_BLK_ATT);
        float* lse = reinterpret_cast<float*>(b.m ? wk + W.lse : SV(COLA_BLK_LSE));
        char* bn = b.m ? wk + W.b : SV(COLA_BLK_B);
        char* gt = b.m ? wk + W.gt : SV(COLA_BLK_GATE);
        char* u = b.m ? wk + W.up : SV(COLA_BLK_UP);
        char* m = b.m ? wk + W.m : SV(COLA_BLK_M);
        char* tmp = wk + W.tmp;
        void* sub = wk + W.sub;
        const int rc = b.m ? 1 : 0;

        if ((st = norm_fwd(c, x0, nullptr, nullptr, w->g1, a)) != COLA_OK) return st;
        {
            const cola_group_desc g = qkv_desc(b, rc);
            const void* B3[3] = {w->B_q, w->B_k, w->B_v};
            void* Y3[3] = {q, k, v};
            st = cola_group_fwd(&g, a, w->A_qkv, B3, Y3, SV(COLA_BLK_Z_QKV), b.m ? nullptr : SV(COLA_BLK_H_QKV), sub,
                                W.sub_bytes, stream);
            if (st != COLA_OK) return st;
        }
        if ((st = attn_fwd(c, q, k, v, att, lse)) != COLA_OK) return st;
        {
            const cola_desc o = o_desc(b, rc);
            st = cola_fwd(&o, att, w->A_o, w->B_o, tmp, SV(COLA_BLK_Z_O), b.m ? nullptr : SV(COLA_BLK_H_O), sub,
                          W.sub_bytes, stream);
            if (st != COLA_OK) return st;
        }
        if ((st = norm_fwd(c, x0, tmp, SV(COLA_BLK_X1), w->g2, bn)) != COLA_OK) return st;
        {
            // gate and up as a group; m = gate * up in up's Y = H B^T epilogue
            // where the ping-pong family runs it, else elementwise
            const cola_group_desc g = gu_desc(b, rc);
            const void* B2[2] = {w->B_g, w->B_u};
            void* Y2[2] = {gt, u};
            bool fused = false;
            // CoLA-M reads up again only after recomputing it, so the
            // fused epilogue stores m alone there
            st = group_fwd_gated(&g, bn, w->A_gu, B2, Y2, SV(COLA_BLK_Z_GU), b.m ? nullptr : SV(COLA_BLK_H_GU), sub,
                                 W.sub_bytes, stream, gt, b.ldf, m, &fused, !b.m);
            if (st != COLA_OK) return st;
            if (!fused && (st = ew(c, EW_MUL, b.ffn, gt, b.ldf, u, b.ldf, nullptr, 0, m, b.ldf, nullptr, 0)) != COLA_OK)
                return st;
        }
        {
            const cola_desc dn = down_desc(b, rc);
            st = cola_fwd(&dn, m, w->A_d, w->B_d, tmp, SV(COLA_BLK_Z_DOWN), b.m ? nullptr : SV(COLA_BLK_H_DOWN), sub,
                          W.sub_bytes, stream);
            if (st != COLA_OK) return st;
        }
        return ew(c, EW_ADD, b.d, SV(COLA_BLK_X1), b.d, tmp, b.d, nullptr, 0, x2, b.d, nullptr, 0);
    });
}

int cola_block_bwd(const cola_block_desc* desc, const cola_block_weights* w, const void* x0, const void* saved,
                   size_t saved_bytes, const void* dx2, void* dx0, const cola_block_grads* gr, void* ws,
                   size_t ws_bytes, cola_stream_t stream) {
    return guarded([&]() -> int {
        Blk b;
        int st = check_block(desc, &b);
        if (st != COLA_OK) return st;
        if (!weights_ok(w) || !grads_ok(gr)) return COLA_ERR_INVALID_ARG;
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        if (b.T == 0) {
            // empty batch: every gradient is an empty sum
            const int64_t n[13] = {b.d, b.d, 3 * b.r * b.d, b.d * b.r, b.d * b.r, b.d * b.r, b.r * b.d, b.d * b.r,
                                   2 * b.r * b.d, b.ffn * b.r, b.ffn * b.r, b.r * b.ffn, b.d * b.r};
            float* p[13] = {gr->g1, gr->g2, gr->A_qkv, gr->B_q, gr->B_k, gr->B_v, gr->A_o, gr->B_o, gr->A_gu,
                            gr->B_g, gr->B_u, gr->A_d, gr->B_d};
            for (int i = 0; i < 13; ++i) {
                hipError_t e = launch_fill_zero(p[i], n[i], s);
                if (e != hipSuccess) return set_hip_error(e, "fill_zero");
            }
            return COLA_OK;
        }
        if (!x0 || !saved || !dx2 || !dx0 || !al16(x0) || !al16(saved) || !al16(dx2) || !al16(dx0) ||
            (ws && !al16(ws)))
            return COLA_ERR_INVALID_ARG;
        const Saved S = plan_saved(b);
        const Ws W = plan_ws(b, 1);
        if (saved_bytes < S.total) return COLA_ERR_WORKSPACE;
        if (!ws || ws_bytes < W.total) return COLA_ERR_WORKSPACE;
        const char* sv = static_cast<const char*>(saved);
        char* wk = static_cast<char*>(ws);
        const Ctx c{b, s, reinterpret_cast<const float*>(wk + W.rope)};
        if ((st = rope_table(c, reinterpret_cast<float*>(wk + W.rope))) != COLA_OK) return st;
        auto SV = [&](int slot) -> const char* { return sv + S.off[slot]; };
        const char* x1 = SV(COLA_BLK_X1);
        const char* Zqkv = SV(COLA_BLK_Z_QKV);
        const char* Zgu = SV(COLA_BLK_Z_GU);
        // kept (CoLA) or recomputed into the workspace (CoLA-M)
        const char* a = b.m ? wk + W.a : SV(COLA_BLK_A);
        const char* q = b.m ? wk + W.q : SV(COLA_BLK_Q);
        const char* k = b.m ? wk + W.k : SV(COLA_BLK_K);
        const char* v = b.m ? wk + W.v : SV(COLA_BLK_V);
        const char* att = b.m ? wk + W.att : SV(COLA_BLK_ATT);
        const float* lse = reinterpret_cast<const float*>(b.m ? wk + W.lse : SV(COLA_BLK_LSE));
        const char* bn = b.m ? wk + W.b : SV(COLA_BLK_B);
        const char* gt = b.m ? wk + W.gt : SV(COLA_BLK_GATE);
        const char* u = b.m ? wk + W.up : SV(COLA_BLK_UP);
        const char* m = b.m ? wk + W.m : SV(COLA_BLK_M);
        const char* Hqkv = b.m ? wk + W.hqkv : SV(COLA_BLK_H_QKV);
        const char* Hgu = b.m ? wk + W.hgu : SV(COLA_BLK_H_GU);
        void* sub = wk + W.sub;
        char *dx1 = wk + W.dx1, *datt = wk + W.datt, *dq = wk + W.dq, *dk = wk + W.dk, *dv = wk + W.dv;
        char *db = wk + W.db, *da = wk + W.da, *dm = wk + W.dm, *dgt = wk + W.dgt, *du = wk + W.du;
        float* D = reinterpret_cast<float*>(wk + W.D);
        float* part = reinterpret_cast<float*>(wk + W.part);
        const int rc = b.m ? 1 : 0;

        if (b.m) {
            // the MLP side: b, H_gu = sigma(Z_gu), gt and u = H B^T, m = gt u
            if ((st = norm_fwd(c, x1, nullptr, nullptr, w->g2, wk + W.b)) != COLA_OK) return st;
            if ((st = ew(c, EW_SIGMA, 2 * b.r, Zgu, b.ld2, nullptr, 0, nullptr, 0, wk + W.hgu, b.ld2, nullptr, 0)) !=
                COLA_OK)
                return st;
            if ((st = up(c, b.ffn, wk + W.hgu, b.ld2, w->B_g, wk + W.gt, b.ldf)) != COLA_OK) return st;
            bool fused = false;
            if ((st = chk(launch_up_projection(b.T, b.ffn, b.r, wk + W.hgu + b.r * 2, b.ld2, w->B_u, wk + W.up, b.ldf,
                                               s, gt, wk + W.m, &fused),
                          "up_projection")) != COLA_OK)
                return st;
            if (!fused &&
                (st = ew(c, EW_MUL, b.ffn, gt, b.ldf, u, b.ldf, nullptr, 0, wk + W.m, b.ldf, nullptr, 0)) != COLA_OK)
                return st;
        }
        {
            // down's backward; dgt = dm u and du = dm gt in its dX = dm
            // epilogue where the ping-pong family runs it, else elementwise
            const cola_desc dn = down_desc(b, rc);
            bool fused = false;
            st = layer_bwd_gated(&dn, dx2, m, SV(COLA_BLK_Z_DOWN), b.m ? nullptr : SV(COLA_BLK_H_DOWN), w->A_d, w->B_d,
                                 dm, gr->A_d, gr->B_d, sub, W.sub_bytes, stream, gt, u, b.ldf, dgt, du, &fused);
            if (st != COLA_OK) return st;
            if (!fused &&
                (st = ew(c, EW_DMUL, b.ffn, gt, b.ldf, u, b.ldf, dm, b.ldf, dgt, b.ldf, du, b.ldf)) != COLA_OK)
                return st;
        }
        {
            const cola_group_desc g = gu_desc(b, 0);
            const void* dY2[2] = {dgt, du};
            const void* B2[2] = {w->B_g, w->B_u};
            float* dB2[2] = {gr->B_g, gr->B_u};
            st = cola_group_bwd(&g, dY2, bn, Zgu, Hgu, w->A_gu, B2, db, gr->A_gu, dB2, sub, W.sub_bytes, stream);
            if (st != COLA_OK) return st;
        }
        if ((st = norm_bwd(c, x1, w->g2, db, dx2, dx1, gr->g2, part)) != COLA_OK) return st;
        if (b.m) {
            // the attention side: a, H_qkv = sigma(Z_qkv), q, k, v = H B^T, att and lse
            if ((st = norm_fwd(c, x0, nullptr, nullptr, w->g1, wk + W.a)) != COLA_OK) return st;
            if ((st = ew(c, EW_SIGMA, 3 * b.r, Zqkv, b.ld3, nullptr, 0, nullptr, 0, wk + W.hqkv, b.ld3, nullptr, 0)) !=
                COLA_OK)
                return st;
            const void* Bp[3] = {w->B_q, w->B_k, w->B_v};
            char* Yp[3] = {wk + W.q, wk + W.k, wk + W.v};
            for (int p = 0; p < 3; ++p)
                if ((st = up(c, b.d, wk + W.hqkv + (size_t)p * b.r * 2, b.ld3, Bp[p], Yp[p], b.d)) != COLA_OK)
                    return st;
            if ((st = attn_fwd(c, q, k, v, wk + W.att, reinterpret_cast<float*>(wk + W.lse))) != COLA_OK) return st;
        }
        {
            const cola_desc o = o_desc(b, rc);
            st = cola_bwd(&o, dx1, att, SV(COLA_BLK_Z_O), b.m ? nullptr : SV(COLA_BLK_H_O), w->A_o, w->B_o, datt,
                          gr->A_o, gr->B_o, sub, W.sub_bytes, stream);
            if (st != COLA_OK) return st;
        }
        if ((st = attn_bwd(c, q, k, v, att, lse, datt, dq, dk, dv, D)) != COLA_OK) return st;
        {
            const cola_group_desc g = qkv_desc(b, 0);
            const void* dY3[3] = {dq, dk, dv};
            const void* B3[3] = {w->B_q, w->B_k, w->B_v};
            float* dB3[3] = {gr->B_q, gr->B_k, gr->B_v};
            st = cola_group_bwd(&g, dY3, a, Zqkv, Hqkv, w->A_qkv, B3, da, gr->A_qkv, dB3, sub, W.sub_bytes, stream);
            if (st != COLA_OK) return st;
        }
        return norm_bwd(c, x0, w->g1, da, dx1, dx0, gr->g1, part);
    });
}

}  // extern "C"
