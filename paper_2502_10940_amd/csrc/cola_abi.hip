// cola_abi.hip -- the C ABI of libcola.so (include/cola.h): argument
// validation, workspace planning, the launch sequence of each call, and the
// optional per-kernel event timing.
//
// Launch sequences (one stream, no host synchronisation):
//   cola_fwd : K1  Z = X A^T, H = sigma(Z)          (epilogue writes Z and H)
//              K2  Y = H B^T
//   cola_bwd : K3  dZ = (dY B) (.) sigma'(Z)        (CoLA-M: also H = sigma(Z))
//              K4  dX = dZ A
//              K5  dA partials = dZ^T X             (split over tokens)
//              K6  dB partials = dY^T H             (split over tokens)
//                  (bf16 with both outputs wider than 128: K5 and K6 in one
//                  launch, one split of T for both)
//              K7  dA, dB = fixed-order sums of the partials
//   dense    : Y = X W^T ; dX = dY W ; dW = dY^T X (split over tokens + K7)
#include <mutex>
#include <new>
#include <stdio.h>
#include <string.h>
#include <vector>

#include "../../include/cola.h"
#include "internal.hpp"
#include "block.hpp"

using namespace cola;

namespace {

thread_local char g_err[256] = "";

int hip_fail(hipError_t e, const char* where) {
    snprintf(g_err, sizeof(g_err), "%s: %s", where, hipGetErrorString(e));
    return COLA_ERR_HIP;
}

// ---------------------------------------------------------------------------
// timing
// ---------------------------------------------------------------------------
struct Timed {
    hipEvent_t start, stop;
    int kc;
    double flops, bytes;
};

struct TimingState {
    std::mutex mu;
    bool on = false;
    std::vector<Timed> pending;
    std::vector<hipEvent_t> free_events;
    int64_t launches[COLA_KC_COUNT] = {};
    double ms[COLA_KC_COUNT] = {};
    double flops[COLA_KC_COUNT] = {};
    double bytes[COLA_KC_COUNT] = {};
};

TimingState& timing() {
    static TimingState* t = new TimingState();   // never destroyed: events may outlive static dtors
    return *t;
}

hipError_t get_event(TimingState& t, hipEvent_t* e) {
    if (!t.free_events.empty()) {
        *e = t.free_events.back();
        t.free_events.pop_back();
        return hipSuccess;
    }
    return hipEventCreate(e);
}

// Drain recorded events into the totals (waits for them).
hipError_t drain(TimingState& t) {
    for (const Timed& x : t.pending) {
        hipError_t e = hipEventSynchronize(x.stop);
        if (e != hipSuccess) return e;
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, x.start, x.stop);
        if (e != hipSuccess) return e;
        t.launches[x.kc] += 1;
        t.ms[x.kc] += ms;
        t.flops[x.kc] += x.flops;
        t.bytes[x.kc] += x.bytes;
        t.free_events.push_back(x.start);
        t.free_events.push_back(x.stop);
    }
    t.pending.clear();
    return hipSuccess;
}

// Run one launch, bracketed by events when timing is on.
template <class F>
hipError_t timed(int kc, double flops, double bytes, hipStream_t s, F&& launch) {
    TimingState& t = timing();
    if (!t.on) return launch();
    std::lock_guard<std::mutex> lock(t.mu);
    if (t.pending.size() >= 8192) {
        hipError_t e = drain(t);
        if (e != hipSuccess) return e;
    }
    Timed x{};
    x.kc = kc; x.flops = flops; x.bytes = bytes;
    hipError_t e = get_event(t, &x.start);
    if (e == hipSuccess) e = get_event(t, &x.stop);
    if (e == hipSuccess) e = hipEventRecord(x.start, s);
    if (e != hipSuccess) return e;
    e = launch();
    if (e != hipSuccess) return e;
    e = hipEventRecord(x.stop, s);
    if (e != hipSuccess) return e;
    t.pending.push_back(x);
    return hipSuccess;
}

// ---------------------------------------------------------------------------
// shapes and plans
// ---------------------------------------------------------------------------
constexpr int64_t kMaxDim = int64_t(1) << 40;   // keeps every byte count far from overflow
static_assert(COLA_MAX_PITCH == kMaxPitch, "the public pitch limit is the kernels' limit");

struct Dims {
    int64_t T, d_in, d_out, r, ldx, ldy, ldz;
    bool bf16;
    size_t esize;
};

bool valid_act(int act) { return act == COLA_ACT_IDENTITY || act == COLA_ACT_SILU || act == COLA_ACT_GELU; }

int check_desc(const cola_desc* d, Dims* out) {
    if (!d) return COLA_ERR_INVALID_ARG;
    if (d->dtype != COLA_F32 && d->dtype != COLA_BF16) return COLA_ERR_INVALID_ARG;
    if (!valid_act(d->act)) return COLA_ERR_INVALID_ARG;
    if (d->recompute != 0 && d->recompute != 1) return COLA_ERR_INVALID_ARG;
    if (d->T < 0 || d->d_in < 1 || d->d_out < 1 || d->r < 1) return COLA_ERR_BAD_SHAPE;
    if (d->T > kMaxDim || d->d_in > kMaxDim || d->d_out > kMaxDim || d->r > kMaxDim)
        return COLA_ERR_BAD_SHAPE;
    Dims x;
    x.T = d->T; x.d_in = d->d_in; x.d_out = d->d_out; x.r = d->r;
    x.ldx = d->ldx ? d->ldx : d->d_in;
    x.ldy = d->ldy ? d->ldy : d->d_out;
    x.ldz = d->ldz ? d->ldz : d->r;
    if (x.ldx < x.d_in || x.ldy < x.d_out || x.ldz < x.r) return COLA_ERR_BAD_SHAPE;
    if (x.ldx > kMaxPitch || x.ldy > kMaxPitch || x.ldz > kMaxPitch) return COLA_ERR_BAD_SHAPE;
    // element counts of the largest operands must stay below 2^62
    const double big = (double)x.T * (double)(x.ldx > x.ldy ? x.ldx : x.ldy);
    if (big > 4.0e18 || (double)x.r * (double)(x.d_in > x.d_out ? x.d_in : x.d_out) > 4.0e18)
        return COLA_ERR_BAD_SHAPE;
    x.bf16 = d->dtype == COLA_BF16;
    x.esize = x.bf16 ? 2 : 4;
    *out = x;
    return COLA_OK;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Split of a token-long (K = T) weight-gradient GEMM into chunks of whole K
// tiles (at least four per chunk).  Depends only on the shape, so results are
// reproducible run to run.
struct Split {
    int splits;
    int64_t k_chunk;
};

// The split count S minimises a modelled time: rounds(S) * ceil(ktiles / S)
// K-tile steps of about 2 us each, where rounds(S) = ceil(tiles * S / slots)
// and slots is the number of workgroups the chip runs at once -- a split that
// leaves a few workgroups for a second round costs a whole round -- plus
// writing and re-reading the S fp32 partials at about 4 TB/s.
// Split of K for `tiles` output tiles (workgroups) on `slots` resident
// workgroups, whose fp32 partials total `elems` values per split.
Split plan_split_tiles(bool bf16, int64_t tiles, int64_t slots, int64_t K, double elems) {
    const int64_t bk = bf16 ? BF16_BK : F32_BK;
    const int64_t ktiles = (K + bk - 1) / bk;
    if (ktiles < 1) return Split{1, bk};                       // empty batch: nothing to split
    const double step_us = 2.0;
    const double partial_us_per_split = elems * 8.0 / 4.0e6;
    int64_t maxs = ktiles / 4;
    if (maxs < 1) maxs = 1;
    if (maxs > 64) maxs = 64;
    int64_t best_s = 1;
    double best_cost = -1.0;
    for (int64_t s = 1; s <= maxs; ++s) {
        const int64_t chunk = (ktiles + s - 1) / s;
        const int64_t eff_s = (ktiles + chunk - 1) / chunk;   // splits actually used
        const int64_t rounds = (tiles * eff_s + slots - 1) / slots;
        const double cost = (double)(rounds * chunk) * step_us +
                            (eff_s > 1 ? (double)eff_s * partial_us_per_split : 0.0);
        if (best_cost < 0 || cost < best_cost) {
            best_cost = cost;
            best_s = s;
        }
    }
    const int64_t chunk_tiles = (ktiles + best_s - 1) / best_s;
    Split s;
    s.k_chunk = chunk_tiles * bk;
    s.splits = (int)((K + s.k_chunk - 1) / s.k_chunk);
    if (s.splits < 1) s.splits = 1;
    return s;
}

Split plan_split(bool bf16, int64_t M, int64_t N, int64_t K, int tag) {
    return plan_split_tiles(bf16, gemm_tiles(bf16, M, N, tag), gemm_slots(bf16, M, N, tag), K,
                            (double)M * (double)N);
}

// The two weight gradients of a layer in one launch (bf16, both in the PP
// family): their tiles share the slots and one split of K = T.  The option
// COLA_OPT_WGRAD_PAIR = 0 launches them one by one (tuning, comparisons).
bool wgrad_pairing_on() { return get_option(OPT_WGRAD_PAIR) == 1; }
bool pair_wgrads(bool bf16, int64_t r, int64_t d_in, int64_t d_out) {
    return wgrad_pairing_on() && bf16 && gemm_family(r, d_in, TAG_BWD_DA) == FAM_PP &&
           gemm_family(d_out, r, TAG_BWD_DB) == FAM_PP;
}
Split plan_split_pair(int64_t r, int64_t d_in, int64_t d_out, int64_t T) {
    const int64_t tiles = gemm_tiles(true, r, d_in, TAG_BWD_DA) + gemm_tiles(true, d_out, r, TAG_BWD_DB);
    return plan_split_tiles(true, tiles, gemm_slots(true, r, d_in, TAG_BWD_DA), T,
                            (double)r * (double)d_in + (double)d_out * (double)r);
}

// Row pitch (elements) of a buffer the library lays out itself: a whole
// number of 128-byte cache lines, so every K tile of a row starts on a line
// (rows that straddle lines cost up to 1.4x on MI355X, measured).
int64_t line_pitch(bool bf16, int64_t width) {
    const int64_t per = bf16 ? 64 : 32;
    return (width + per - 1) / per * per;
}

// A bf16 weight whose rows are not a whole number of 16-byte chunks (width
// not a multiple of 8) is copied to the workspace with a line-aligned pitch,
// so the MFMA kernel keeps its vector loads.  Depends only on the shape.
struct Pack {
    bool on;
    int64_t ld;     // pitch to use for the weight
    size_t off, bytes;
};

Pack plan_pack(bool bf16, int64_t rows, int64_t width, size_t off) {
    Pack p;
    p.off = off;
    p.on = bf16 && (width % 8) != 0;
    p.ld = p.on ? line_pitch(true, width) : width;
    p.bytes = p.on ? align256((size_t)rows * (size_t)p.ld * 2) : 0;
    return p;
}

// Resolve a weight to (pointer, pitch), enqueueing its repack if planned.
hipError_t use_weight(const Pack& pk, const void* w, int64_t rows, int64_t width, char* ws,
                      const void** out, int64_t* ld, hipStream_t s) {
    if (!pk.on) {
        *out = w;
        *ld = width;
        return hipSuccess;
    }
    *out = ws + pk.off;
    *ld = pk.ld;
    return launch_pack_rows(w, rows, width, ws + pk.off, pk.ld, s);
}

struct FwdPlan {
    int64_t ldw;          // pitch of the workspace copy of H (CoLA-M)
    size_t off_h, total;
    Pack pa, pb;          // repacked A [r][d_in] and B [d_out][r]
};

FwdPlan plan_fwd(const Dims& x, bool recompute) {
    FwdPlan p;
    p.ldw = line_pitch(x.bf16, x.r);
    p.off_h = 0;
    const size_t hbytes = recompute ? align256((size_t)x.T * (size_t)p.ldw * x.esize) : 0;
    p.pa = plan_pack(x.bf16, x.r, x.d_in, hbytes);
    p.pb = plan_pack(x.bf16, x.d_out, x.r, p.pa.off + p.pa.bytes);
    p.total = p.pb.off + p.pb.bytes;
    if (x.T == 0) p.total = 0;
    return p;
}

struct BwdPlan {
    int64_t ldw;          // pitch of dZ (and recomputed H) in the workspace
    size_t off_dz, off_h, off_pa, off_pb, total;
    Split sa, sb;         // the same split for both when pair
    bool pair;            // dA and dB in one launch
    Pack wa, wb;          // repacked A and B
};

BwdPlan plan_bwd(const Dims& x, bool recompute) {
    BwdPlan p;
    p.ldw = line_pitch(x.bf16, x.r);
    const size_t zbytes = align256((size_t)x.T * (size_t)p.ldw * x.esize);
    p.pair = pair_wgrads(x.bf16, x.r, x.d_in, x.d_out);
    if (p.pair) {
        p.sa = p.sb = plan_split_pair(x.r, x.d_in, x.d_out, x.T);
    } else {
        p.sa = plan_split(x.bf16, x.r, x.d_in, x.T, TAG_BWD_DA);
        p.sb = plan_split(x.bf16, x.d_out, x.r, x.T, TAG_BWD_DB);
    }
    p.off_dz = 0;
    p.off_h = zbytes;
    p.off_pa = p.off_h + (recompute ? zbytes : 0);
    const size_t pa = p.sa.splits > 1 ? align256((size_t)p.sa.splits * (size_t)(x.r * x.d_in) * 4) : 0;
    p.off_pb = p.off_pa + pa;
    const size_t pb = p.sb.splits > 1 ? align256((size_t)p.sb.splits * (size_t)(x.d_out * x.r) * 4) : 0;
    p.wa = plan_pack(x.bf16, x.r, x.d_in, p.off_pb + pb);
    p.wb = plan_pack(x.bf16, x.d_out, x.r, p.wa.off + p.wa.bytes);
    p.total = p.wb.off + p.wb.bytes;
    if (x.T == 0) p.total = 0;
    return p;
}

size_t fwd_ws(const Dims& x, bool recompute) { return plan_fwd(x, recompute).total; }

hipError_t gemm(const GemmArgs& a, bool bf16, hipStream_t s) {
    return bf16 ? launch_gemm_bf16(a, s) : launch_gemm_f32(a, s);
}

GemmArgs make_args(int tag, int64_t M, int64_t N, int64_t K, const void* p, int64_t ldp, int pl,
                   const void* q, int64_t ldq, int ql, void* c, int64_t ldc, int epi, int act) {
    GemmArgs a{};
    a.tag = tag;
    a.M = M; a.N = N; a.K = K;
    a.p = p; a.ldp = ldp; a.p_layout = pl;
    a.q = q; a.ldq = ldq; a.q_layout = ql;
    a.c = c; a.ldc = ldc;
    a.epi = epi; a.act = act;
    a.splits = 1;
    a.k_chunk = K > 0 ? K : 1;
    a.split_stride = 0;
    return a;
}

double gemm_flops(int64_t M, int64_t N, int64_t K) { return 2.0 * (double)M * (double)N * (double)K; }

// Weight gradient C[M][N] = sum_t P[t][m] Q[t][n] with K = T split into
// chunks whose partials are summed in a fixed order.
int wgrad(bool bf16, int64_t M, int64_t N, int64_t T, const void* P, int64_t ldp, const void* Q,
          int64_t ldq, float* C, const Split& sp, float* partials, int kc, double bytes_in,
          hipStream_t s) {
    GemmArgs a = make_args(kc, M, N, T, P, ldp, MNMAJ, Q, ldq, MNMAJ, C, N, EPI_STORE_F32, 0);
    a.splits = sp.splits;
    a.k_chunk = sp.k_chunk;
    if (sp.splits > 1) {
        a.c = partials;
        a.split_stride = M * N;
    }
    const double out_bytes = (double)M * (double)N * 4.0 * (sp.splits > 1 ? sp.splits : 1);
    hipError_t e = timed(kc, gemm_flops(M, N, T), bytes_in + out_bytes, s, [&] { return gemm(a, bf16, s); });
    if (e != hipSuccess) return hip_fail(e, cola_kernel_name(kc));
    if (sp.splits > 1) {
        const double rb = (double)M * (double)N * 4.0 * (sp.splits + 1);
        e = timed(COLA_KC_REDUCE, 0.0, rb, s,
                  [&] { return launch_reduce_splits(partials, sp.splits, M * N, C, M * N, s); });
        if (e != hipSuccess) return hip_fail(e, "reduce");
    }
    return COLA_OK;
}

// Both weight gradients of a layer, C0[M0][N0] = sum_t P0[t][m] Q0[t][n] and
// C1 likewise, in one launch with one split of K = T (bf16 PP family), then
// the fixed-order reductions of their partials.
int wgrad_pair(int64_t T, const Split& sp, int64_t M0, int64_t N0, const void* P0, int64_t ldp0, const void* Q0,
               int64_t ldq0, float* C0, float* part0, int64_t M1, int64_t N1, const void* P1, int64_t ldp1,
               const void* Q1, int64_t ldq1, float* C1, float* part1, double bytes_in, hipStream_t s) {
    GemmArgs a0 = make_args(TAG_BWD_DA, M0, N0, T, P0, ldp0, MNMAJ, Q0, ldq0, MNMAJ, C0, N0, EPI_STORE_F32, 0);
    GemmArgs a1 = make_args(TAG_BWD_DB, M1, N1, T, P1, ldp1, MNMAJ, Q1, ldq1, MNMAJ, C1, N1, EPI_STORE_F32, 0);
    for (GemmArgs* a : {&a0, &a1}) {
        a->splits = sp.splits;
        a->k_chunk = sp.k_chunk;
    }
    if (sp.splits > 1) {
        a0.c = part0;
        a0.split_stride = M0 * N0;
        a1.c = part1;
        a1.split_stride = M1 * N1;
    }
    const double elems = (double)M0 * (double)N0 + (double)M1 * (double)N1;
    const double out_bytes = elems * 4.0 * (sp.splits > 1 ? sp.splits : 1);
    hipError_t e = timed(COLA_KC_BWD_DADB, gemm_flops(M0, N0, T) + gemm_flops(M1, N1, T), bytes_in + out_bytes, s,
                         [&] { return launch_gemm_bf16_pair(a0, a1, s); });
    if (e != hipSuccess) return hip_fail(e, cola_kernel_name(COLA_KC_BWD_DADB));
    if (sp.splits > 1) {
        e = timed(COLA_KC_REDUCE, 0.0, elems * 4.0 * (sp.splits + 1), s, [&] {
            return launch_reduce_splits2(part0, M0 * N0, C0, M0 * N0, part1, M1 * N1, C1, M1 * N1, sp.splits, s);
        });
        if (e != hipSuccess) return hip_fail(e, "reduce");
    }
    return COLA_OK;
}

template <class F>
int guarded(F&& f) {
    try {
        return f();
    } catch (const std::bad_alloc&) {
        snprintf(g_err, sizeof(g_err), "host allocation failed");
        return COLA_ERR_HIP;
    } catch (...) {
        snprintf(g_err, sizeof(g_err), "unexpected host exception");
        return COLA_ERR_HIP;
    }
}

// The gated product of the decoder block's MLP fused into a GEMM epilogue
// (ping-pong family only; the caller runs the elementwise kernels when
// *fused comes back false): forward, the last projection of a group stores
// u and m = g u, g being the group's first output; backward, the layer's
// dX = dm GEMM stores dg = dm u and du = dm g instead.  g, u, m, dg and du
// share the row pitch ld.
struct Gate {
    const void* g;
    const void* u;
    int64_t ld;
    void* out;       // m (forward) or dg (backward)
    void* out2;      // du (backward)
    bool* fused;
    bool keep_u;     // forward: the fused epilogue also stores u (else only m)
};

bool gate_fusion_on() { return get_option(OPT_FUSE_GATE) == 1; }

// Forward of one validated layer with its pointers and workspace checked.
// outer >= 0: the both-sigma variant (K2 stores P and Y = sigma_out(P)).
int layer_forward(const Dims& x, int act, bool recompute, const void* X, const void* A, const void* B, void* Y,
                  void* Z, void* H, int outer, void* P, char* w, hipStream_t s) {
    const FwdPlan p = plan_fwd(x, recompute);
    void* Hbuf = recompute ? (void*)(w + p.off_h) : H;
    const int64_t ldh = recompute ? p.ldw : x.ldz;
    const double es = (double)x.esize;
    const void* Aw;
    const void* Bw;
    int64_t lda, ldb;
    hipError_t e = use_weight(p.pa, A, x.r, x.d_in, w, &Aw, &lda, s);
    if (e == hipSuccess) e = use_weight(p.pb, B, x.d_out, x.r, w, &Bw, &ldb, s);
    if (e != hipSuccess) return hip_fail(e, "pack_rows");

    // K1: Z = X A^T, H = sigma(Z)
    GemmArgs k1 = make_args(TAG_FWD_Z, x.T, x.r, x.d_in, X, x.ldx, KMAJ, Aw, lda, KMAJ, Z, x.ldz, EPI_Z_H,
                            act);
    k1.aux = Hbuf;
    k1.ldaux = ldh;
    const double b1 = es * ((double)x.T * x.d_in + (double)x.r * x.d_in + 2.0 * x.T * x.r);
    e = timed(COLA_KC_FWD_Z, gemm_flops(x.T, x.r, x.d_in), b1, s, [&] { return gemm(k1, x.bf16, s); });
    if (e != hipSuccess) return hip_fail(e, "fwd_z_sigma");

    // K2: Y = H B^T; with an outer sigma (outer >= 0) K2 stores P = H B^T
    // and Y = sigma_out(P)
    GemmArgs k2 = make_args(TAG_FWD_Y, x.T, x.d_out, x.r, Hbuf, ldh, KMAJ, Bw, ldb, KMAJ, Y, x.ldy, EPI_STORE,
                            act);
    if (outer >= 0) {
        k2 = make_args(TAG_FWD_YP, x.T, x.d_out, x.r, Hbuf, ldh, KMAJ, Bw, ldb, KMAJ, P, x.ldy, EPI_Z_H, outer);
        k2.aux = Y;
        k2.ldaux = x.ldy;
    }
    const double b2 = es * ((double)x.T * x.r + (double)x.d_out * x.r + (double)x.T * x.d_out *
                            (outer >= 0 ? 2.0 : 1.0));
    e = timed(COLA_KC_FWD_Y, gemm_flops(x.T, x.d_out, x.r), b2, s, [&] { return gemm(k2, x.bf16, s); });
    if (e != hipSuccess) return hip_fail(e, "fwd_y");
    return COLA_OK;
}

// Backward of one validated layer with a non-empty batch, its pointers and
// workspace checked; dY has row pitch ldy.
int layer_backward(const Dims& x, int act, bool recompute, const void* dY, int64_t ldy, const void* X,
                   const void* Z, const void* H, const void* A, const void* B, void* dX, float* dA, float* dB,
                   char* w, hipStream_t s, const Gate* gate = nullptr) {
    const BwdPlan p = plan_bwd(x, recompute);
    void* dZ = w + p.off_dz;
    const void* Hbuf = recompute ? (const void*)(w + p.off_h) : H;
    const int64_t ldh = recompute ? p.ldw : x.ldz;
    const double es = (double)x.esize;
    const void* Aw;
    const void* Bw;
    int64_t lda, ldb;
    hipError_t e = use_weight(p.wa, A, x.r, x.d_in, w, &Aw, &lda, s);
    if (e == hipSuccess) e = use_weight(p.wb, B, x.d_out, x.r, w, &Bw, &ldb, s);
    if (e != hipSuccess) return hip_fail(e, "pack_rows");

    // K3: dZ = (dY B) (.) sigma'(Z); CoLA-M regenerates H = sigma(Z) here
    GemmArgs k3 = make_args(TAG_BWD_DZ, x.T, x.r, x.d_out, dY, ldy, KMAJ, Bw, ldb, MNMAJ, dZ, p.ldw, EPI_DZ,
                            act);
    k3.zin = Z;
    k3.ldzin = x.ldz;
    k3.aux = recompute ? (void*)(w + p.off_h) : nullptr;
    k3.ldaux = p.ldw;
    const double b3 = es * ((double)x.T * x.d_out + (double)x.d_out * x.r +
                            (double)x.T * x.r * (recompute ? 3.0 : 2.0));
    e = timed(COLA_KC_BWD_DZ, gemm_flops(x.T, x.r, x.d_out), b3, s, [&] { return gemm(k3, x.bf16, s); });
    if (e != hipSuccess) return hip_fail(e, "bwd_dz");

    // K4: dX = dZ A (or, gated, dg = dm u and du = dm g with dm = dZ A)
    GemmArgs k4 = make_args(TAG_BWD_DX, x.T, x.d_in, x.r, dZ, p.ldw, KMAJ, Aw, lda, MNMAJ, dX, x.ldx, EPI_STORE,
                            act);
    double b4 = es * ((double)x.T * x.r + (double)x.r * x.d_in + (double)x.T * x.d_in);
    if (gate) {
        GemmArgs kg = make_args(TAG_BWD_DXG, x.T, x.d_in, x.r, dZ, p.ldw, KMAJ, Aw, lda, MNMAJ, gate->out, gate->ld,
                                EPI_DGATE, act);
        kg.zin = gate->g;
        kg.ldzin = gate->ld;
        kg.zin2 = gate->u;
        kg.ldzin2 = gate->ld;
        kg.aux = gate->out2;
        kg.ldaux = gate->ld;
        *gate->fused = x.bf16 && gate_fusion_on() && pp_takes(kg);
        if (*gate->fused) {
            k4 = kg;
            b4 = es * ((double)x.T * x.r + (double)x.r * x.d_in + 4.0 * x.T * x.d_in);
        }
    }
    e = timed(COLA_KC_BWD_DX, gemm_flops(x.T, x.d_in, x.r), b4, s, [&] { return gemm(k4, x.bf16, s); });
    if (e != hipSuccess) return hip_fail(e, "bwd_dx");

    // K5: dA = dZ^T X ; K6: dB = dY^T H  (+ K7 fixed-order reductions);
    // one launch for both when they share the PP family
    if (p.pair)
        return wgrad_pair(x.T, p.sa, x.r, x.d_in, dZ, p.ldw, X, x.ldx, dA, reinterpret_cast<float*>(w + p.off_pa),
                          x.d_out, x.r, dY, ldy, Hbuf, ldh, dB, reinterpret_cast<float*>(w + p.off_pb),
                          es * ((double)x.T * x.r + (double)x.T * x.d_in + (double)x.T * x.d_out +
                                (double)x.T * x.r),
                          s);
    int st = wgrad(x.bf16, x.r, x.d_in, x.T, dZ, p.ldw, X, x.ldx, dA, p.sa,
               reinterpret_cast<float*>(w + p.off_pa), COLA_KC_BWD_DA,
               es * ((double)x.T * x.r + (double)x.T * x.d_in), s);
    if (st != COLA_OK) return st;
    st = wgrad(x.bf16, x.d_out, x.r, x.T, dY, ldy, Hbuf, ldh, dB, p.sb,
               reinterpret_cast<float*>(w + p.off_pb), COLA_KC_BWD_DB,
               es * ((double)x.T * x.d_out + (double)x.T * x.r), s);
    return st;
}

// dA = dB = 0 for an empty batch (the token sums are empty).
int zero_weight_grads(const Dims& x, float* dA, float* dB, hipStream_t s) {
    hipError_t e = timed(COLA_KC_FILL, 0.0, 4.0 * x.r * x.d_in, s,
                         [&] { return launch_fill_zero(dA, x.r * x.d_in, s); });
    if (e == hipSuccess)
        e = timed(COLA_KC_FILL, 0.0, 4.0 * x.d_out * x.r, s, [&] { return launch_fill_zero(dB, x.d_out * x.r, s); });
    return e == hipSuccess ? COLA_OK : hip_fail(e, "fill_zero");
}

int bwd_checked(const cola_desc* desc, const void* dY, const void* X, const void* Z, const void* H, const void* A,
                const void* B, void* dX, float* dA, float* dB, void* ws, size_t ws_bytes, cola_stream_t stream,
                const Gate* gate) {
    Dims x;
    int st = check_desc(desc, &x);
    if (st != COLA_OK) return st;
    const bool recompute = desc->recompute == 1;
    if (recompute ? (H != nullptr) : (H == nullptr && x.T > 0)) return COLA_ERR_INVALID_ARG;
    if (!dA || !dB) return COLA_ERR_INVALID_ARG;
    if (gate) *gate->fused = false;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (x.T == 0) return zero_weight_grads(x, dA, dB, s);
    if (!dY || !X || !Z || !A || !B || !dX) return COLA_ERR_INVALID_ARG;
    const BwdPlan p = plan_bwd(x, recompute);
    if (!ws || ws_bytes < p.total) return COLA_ERR_WORKSPACE;
    return layer_backward(x, desc->act, recompute, dY, x.ldy, X, Z, H, A, B, dX, dA, dB,
                          reinterpret_cast<char*>(ws), s, gate);
}

// Workspace of the both-sigma backward: the layer's, then dP = dY sigma_out'(P).
struct OuterPlan {
    int64_t ldg;
    size_t off_g, total;
};

OuterPlan plan_outer_bwd(const Dims& x, bool recompute) {
    OuterPlan o;
    o.ldg = line_pitch(x.bf16, x.d_out);
    o.off_g = plan_bwd(x, recompute).total;
    o.total = x.T == 0 ? 0 : o.off_g + align256((size_t)x.T * (size_t)o.ldg * x.esize);
    return o;
}

}  // namespace

// ---- hooks for the other translation units (the block path) ----
namespace cola {

hipError_t timed_call(int kc, double flops, double bytes, hipStream_t s, hipError_t (*fn)(void*), void* ctx) {
    return timed(kc, flops, bytes, s, [&] { return fn(ctx); });
}

int set_hip_error(hipError_t e, const char* where) { return hip_fail(e, where); }

hipError_t launch_up_projection(int64_t T, int64_t d_out, int64_t r, const void* H, int64_t ldh, const void* B,
                                void* Y, int64_t ldy, hipStream_t s, const void* g, void* m, bool* fused) {
    GemmArgs k2 = make_args(TAG_FWD_Y, T, d_out, r, H, ldh, KMAJ, B, r, KMAJ, Y, ldy, EPI_STORE, 0);
    double bytes = 2.0 * ((double)T * r + (double)d_out * r + (double)T * d_out);
    if (fused) {
        GemmArgs kg = make_args(TAG_FWD_YG, T, d_out, r, H, ldh, KMAJ, B, r, KMAJ, Y, ldy, EPI_GATE, 0);
        kg.zin = g;
        kg.ldzin = ldy;
        kg.aux = m;
        kg.ldaux = ldy;
        *fused = gate_fusion_on() && pp_takes(kg);
        if (*fused) {
            k2 = kg;
            bytes = 2.0 * ((double)T * r + (double)d_out * r + 3.0 * T * d_out);
        }
    }
    return timed(COLA_KC_FWD_Y, gemm_flops(T, d_out, r), bytes, s, [&] { return gemm(k2, true, s); });
}

}  // namespace cola

extern "C" {

int cola_abi_version(void) { return COLA_ABI_VERSION; }

int cola_set_option(int option, int value) {
    static_assert((int)COLA_OPT_STREAM_ONLY == (int)OPT_STREAM_ONLY && (int)COLA_OPT_WGRAD_PAIR == (int)OPT_WGRAD_PAIR,
                  "option numbering");
    return set_option(option, value) == 0 ? COLA_OK : COLA_ERR_INVALID_ARG;
}

int cola_get_option(int option) { return get_option(option); }

const char* cola_strerror(int status) {
    switch (status) {
        case COLA_OK: return "success";
        case COLA_ERR_INVALID_ARG: return "invalid argument (NULL pointer, bad enum, or H/recompute mismatch)";
        case COLA_ERR_BAD_SHAPE: return "bad shape (dimension < 1, T < 0, ld < width, or size overflow)";
        case COLA_ERR_WORKSPACE: return "workspace too small";
        case COLA_ERR_HIP: return g_err[0] ? g_err : "HIP error";
        case COLA_ERR_UNSUPPORTED: return "unsupported combination";
        case COLA_ERR_SCRATCH: return "the call needs more than the library's static scratch (COLA_SCRATCH_BYTES)";
        default: return "unknown status";
    }
}

const char* cola_kernel_name(int kc) {
    static const char* names[COLA_KC_COUNT] = {
        "fwd_z_sigma", "fwd_y", "bwd_dz", "bwd_dx", "bwd_da", "bwd_db",
        "reduce_splits", "dense_fwd", "dense_dx", "dense_dw", "fill_zero", "infer_h", "outer_grad",
        "bwd_da_db", "attn_fwd", "attn_bwd", "norm", "norm_bwd", "pointwise"};
    if (kc < 0 || kc >= COLA_KC_COUNT) return "invalid";
    return names[kc];
}

size_t cola_workspace_bytes(const cola_desc* desc, int phase) {
    Dims x;
    if (check_desc(desc, &x) != COLA_OK) return 0;
    if (phase == 0) return fwd_ws(x, desc->recompute == 1);
    if (phase == 1) return plan_bwd(x, desc->recompute == 1).total;
    if (phase == 2) return fwd_ws(x, true);     // inference: H in the workspace, as CoLA-M's forward
    if (phase == 3) return plan_outer_bwd(x, desc->recompute == 1).total;
    return 0;
}

int cola_fwd(const cola_desc* desc, const void* X, const void* A, const void* B, void* Y, void* Z,
             void* H, void* ws, size_t ws_bytes, cola_stream_t stream) {
    return guarded([&]() -> int {
        Dims x;
        int st = check_desc(desc, &x);
        if (st != COLA_OK) return st;
        const bool recompute = desc->recompute == 1;
        // CoLA-M never takes H; CoLA needs it unless the batch is empty
        if (recompute ? (H != nullptr) : (H == nullptr && x.T > 0)) return COLA_ERR_INVALID_ARG;
        if (x.T == 0) return COLA_OK;
        if (!X || !A || !B || !Y || !Z) return COLA_ERR_INVALID_ARG;
        const FwdPlan p = plan_fwd(x, recompute);
        if (p.total > 0 && (!ws || ws_bytes < p.total)) return COLA_ERR_WORKSPACE;
        return layer_forward(x, desc->act, recompute, X, A, B, Y, Z, H, -1, nullptr, reinterpret_cast<char*>(ws),
                             reinterpret_cast<hipStream_t>(stream));
    });
}

int cola_fwd_outer(const cola_desc* desc, int outer_act, const void* X, const void* A, const void* B, void* Y,
                   void* P, void* Z, void* H, void* ws, size_t ws_bytes, cola_stream_t stream) {
    return guarded([&]() -> int {
        Dims x;
        int st = check_desc(desc, &x);
        if (st != COLA_OK) return st;
        if (!valid_act(outer_act)) return COLA_ERR_INVALID_ARG;
        const bool recompute = desc->recompute == 1;
        if (recompute ? (H != nullptr) : (H == nullptr && x.T > 0)) return COLA_ERR_INVALID_ARG;
        if (x.T == 0) return COLA_OK;
        if (!X || !A || !B || !Y || !P || !Z) return COLA_ERR_INVALID_ARG;
        const FwdPlan p = plan_fwd(x, recompute);
        if (p.total > 0 && (!ws || ws_bytes < p.total)) return COLA_ERR_WORKSPACE;
        return layer_forward(x, desc->act, recompute, X, A, B, Y, Z, H, outer_act, P, reinterpret_cast<char*>(ws),
                             reinterpret_cast<hipStream_t>(stream));
    });
}

int cola_bwd(const cola_desc* desc, const void* dY, const void* X, const void* Z, const void* H,
             const void* A, const void* B, void* dX, float* dA, float* dB, void* ws, size_t ws_bytes,
             cola_stream_t stream) {
    return guarded([&]() -> int { return bwd_checked(desc, dY, X, Z, H, A, B, dX, dA, dB, ws, ws_bytes, stream, nullptr); });
}

// ---------------------------------------------------------------------------
// backward without a caller workspace: the library's static device scratch
// ---------------------------------------------------------------------------
}  // extern "C"

namespace {

// The workspace of cola_bwd_scratch: one array per GPU, placed by the code
// object loader and held until the process ends.  In host code `scratch` is
// a host-side stand-in, not a device address: kernels get the address that
// hipGetSymbolAddress returns for the current device, kept per device.
static __device__ __align__(256) unsigned char scratch[COLA_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

struct ScratchPtrs {
    std::mutex mu;
    void* ptr[kMaxDevices] = {};
};

ScratchPtrs& scratch_ptrs() {
    static ScratchPtrs* s = new ScratchPtrs();   // never destroyed
    return *s;
}

// Device address of this device's scratch (looked up once per device, with
// that device current).
int scratch_of_current_device(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) {
        snprintf(g_err, sizeof(g_err), "device %d beyond the %d the scratch table holds", dev, kMaxDevices);
        return COLA_ERR_HIP;
    }
    ScratchPtrs& t = scratch_ptrs();
    std::lock_guard<std::mutex> lock(t.mu);
    if (!t.ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) {
            snprintf(g_err, sizeof(g_err), "hipGetSymbolAddress(scratch) returned NULL");
            return COLA_ERR_HIP;
        }
        t.ptr[dev] = p;
    }
    *out = t.ptr[dev];
    return COLA_OK;
}

}  // namespace

extern "C" {

int cola_bwd_scratch(const cola_desc* desc, const void* dY, const void* X, const void* Z, const void* H,
                     const void* A, const void* B, void* dX, float* dA, float* dB, cola_stream_t stream) {
    return guarded([&]() -> int {
        Dims x;
        int st = check_desc(desc, &x);
        if (st != COLA_OK) return st;
        const bool recompute = desc->recompute == 1;
        if (recompute ? (H != nullptr) : (H == nullptr && x.T > 0)) return COLA_ERR_INVALID_ARG;
        if (!dA || !dB) return COLA_ERR_INVALID_ARG;
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        if (x.T == 0) return zero_weight_grads(x, dA, dB, s);
        if (!dY || !X || !Z || !A || !B || !dX) return COLA_ERR_INVALID_ARG;
        const BwdPlan p = plan_bwd(x, recompute);
        if (p.total > COLA_SCRATCH_BYTES) return COLA_ERR_SCRATCH;
        void* w = nullptr;
        st = scratch_of_current_device(&w);
        if (st != COLA_OK) return st;
        return layer_backward(x, desc->act, recompute, dY, x.ldy, X, Z, H, A, B, dX, dA, dB,
                              reinterpret_cast<char*>(w), s);
    });
}

int cola_bwd_outer(const cola_desc* desc, int outer_act, const void* dY, const void* P, const void* X,
                   const void* Z, const void* H, const void* A, const void* B, void* dX, float* dA, float* dB,
                   void* ws, size_t ws_bytes, cola_stream_t stream) {
    return guarded([&]() -> int {
        Dims x;
        int st = check_desc(desc, &x);
        if (st != COLA_OK) return st;
        if (!valid_act(outer_act)) return COLA_ERR_INVALID_ARG;
        const bool recompute = desc->recompute == 1;
        if (recompute ? (H != nullptr) : (H == nullptr && x.T > 0)) return COLA_ERR_INVALID_ARG;
        if (!dA || !dB) return COLA_ERR_INVALID_ARG;
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        if (x.T == 0) return zero_weight_grads(x, dA, dB, s);
        if (!dY || !P || !X || !Z || !A || !B || !dX) return COLA_ERR_INVALID_ARG;
        const OuterPlan o = plan_outer_bwd(x, recompute);
        if (!ws || ws_bytes < o.total) return COLA_ERR_WORKSPACE;
        char* w = reinterpret_cast<char*>(ws);
        // dP = dY (.) sigma_out'(P), rounded to the storage dtype like dZ
        void* dP = w + o.off_g;
        const double bytes = (double)x.esize * 3.0 * (double)x.T * (double)x.d_out;
        hipError_t e = timed(COLA_KC_OUTER_GRAD, 0.0, bytes, s, [&] {
            return launch_outer_grad(x.bf16, dY, x.ldy, P, x.ldy, dP, o.ldg, x.T, x.d_out, outer_act, s);
        });
        if (e != hipSuccess) return hip_fail(e, "outer_grad");
        return layer_backward(x, desc->act, recompute, dP, o.ldg, X, Z, H, A, B, dX, dA, dB, w, s);
    });
}

// ---------------------------------------------------------------------------
// dense baseline
// ---------------------------------------------------------------------------
static int check_dense(const dense_desc* d, Dims* out) {
    if (!d) return COLA_ERR_INVALID_ARG;
    cola_desc c{};
    c.T = d->T; c.d_in = d->d_in; c.d_out = d->d_out; c.r = 1;
    c.ldx = d->ldx; c.ldy = d->ldy; c.ldz = 0;
    c.dtype = d->dtype; c.act = COLA_ACT_IDENTITY; c.recompute = 0;
    return check_desc(&c, out);
}

// Workspace of the dense path: [split-K partials of dW (phase 1)] [W repack].
struct DensePlan {
    Split sp;
    size_t parts;
    Pack pw;
    size_t total;
};

static DensePlan plan_dense(const Dims& x, int phase) {
    DensePlan p;
    p.sp = plan_split(x.bf16, x.d_out, x.d_in, x.T, TAG_DENSE_DW);
    p.parts = (phase == 1 && p.sp.splits > 1) ? align256((size_t)p.sp.splits * (size_t)(x.d_out * x.d_in) * 4) : 0;
    p.pw = plan_pack(x.bf16, x.d_out, x.d_in, p.parts);
    p.total = p.pw.off + p.pw.bytes;
    if (x.T == 0) p.total = 0;
    return p;
}

size_t dense_workspace_bytes(const dense_desc* desc, int phase) {
    Dims x;
    if (check_dense(desc, &x) != COLA_OK) return 0;
    if (phase != 0 && phase != 1) return 0;
    return plan_dense(x, phase).total;
}

int dense_fwd(const dense_desc* desc, const void* X, const void* W, void* Y, void* ws, size_t ws_bytes,
              cola_stream_t stream) {
    return guarded([&]() -> int {
        Dims x;
        int st = check_dense(desc, &x);
        if (st != COLA_OK) return st;
        if (x.T == 0) return COLA_OK;
        if (!X || !W || !Y) return COLA_ERR_INVALID_ARG;
        const DensePlan p = plan_dense(x, 0);
        if (p.total > 0 && (!ws || ws_bytes < p.total)) return COLA_ERR_WORKSPACE;
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        const void* Ww;
        int64_t ldw;
        hipError_t e = use_weight(p.pw, W, x.d_out, x.d_in, reinterpret_cast<char*>(ws), &Ww, &ldw, s);
        if (e != hipSuccess) return hip_fail(e, "pack_rows");
        GemmArgs a = make_args(TAG_DENSE_FWD, x.T, x.d_out, x.d_in, X, x.ldx, KMAJ, Ww, ldw, KMAJ, Y, x.ldy, EPI_STORE, 0);
        const double b = (double)x.esize * ((double)x.T * x.d_in + (double)x.d_out * x.d_in + (double)x.T * x.d_out);
        e = timed(COLA_KC_DENSE_FWD, gemm_flops(x.T, x.d_out, x.d_in), b, s, [&] { return gemm(a, x.bf16, s); });
        return e == hipSuccess ? COLA_OK : hip_fail(e, "dense_fwd");
    });
}

int dense_bwd(const dense_desc* desc, const void* dY, const void* X, const void* W, void* dX, float* dW,
              void* ws, size_t ws_bytes, cola_stream_t stream) {
    return guarded([&]() -> int {
        Dims x;
        int st = check_dense(desc, &x);
        if (st != COLA_OK) return st;
        if (!dW) return COLA_ERR_INVALID_ARG;
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        if (x.T == 0) {
            hipError_t e = timed(COLA_KC_FILL, 0.0, 4.0 * x.d_out * x.d_in, s,
                                 [&] { return launch_fill_zero(dW, x.d_out * x.d_in, s); });
            return e == hipSuccess ? COLA_OK : hip_fail(e, "fill_zero");
        }
        if (!dY || !X || !W || !dX) return COLA_ERR_INVALID_ARG;
        const DensePlan p = plan_dense(x, 1);
        if (p.total > 0 && (!ws || ws_bytes < p.total)) return COLA_ERR_WORKSPACE;
        char* w = reinterpret_cast<char*>(ws);
        const void* Ww;
        int64_t ldw;
        hipError_t e = use_weight(p.pw, W, x.d_out, x.d_in, w, &Ww, &ldw, s);
        if (e != hipSuccess) return hip_fail(e, "pack_rows");
        GemmArgs a = make_args(TAG_DENSE_DX, x.T, x.d_in, x.d_out, dY, x.ldy, KMAJ, Ww, ldw, MNMAJ, dX, x.ldx, EPI_STORE, 0);
        const double b = (double)x.esize * ((double)x.T * x.d_out + (double)x.d_out * x.d_in + (double)x.T * x.d_in);
        e = timed(COLA_KC_DENSE_DX, gemm_flops(x.T, x.d_in, x.d_out), b, s, [&] { return gemm(a, x.bf16, s); });
        if (e != hipSuccess) return hip_fail(e, "dense_dx");
        return wgrad(x.bf16, x.d_out, x.d_in, x.T, dY, x.ldy, X, x.ldx, dW, p.sp, reinterpret_cast<float*>(w),
                     COLA_KC_DENSE_DW, (double)x.esize * ((double)x.T * x.d_out + (double)x.T * x.d_in), s);
    });
}

// ---------------------------------------------------------------------------
// timing API
// ---------------------------------------------------------------------------
int cola_timing_enable(int on) {
    return guarded([&]() -> int {
        TimingState& t = timing();
        std::lock_guard<std::mutex> lock(t.mu);
        t.on = on != 0;
        return COLA_OK;
    });
}

int cola_timing_reset(void) {
    return guarded([&]() -> int {
        TimingState& t = timing();
        std::lock_guard<std::mutex> lock(t.mu);
        hipError_t e = drain(t);
        for (int k = 0; k < COLA_KC_COUNT; ++k) {
            t.launches[k] = 0; t.ms[k] = 0; t.flops[k] = 0; t.bytes[k] = 0;
        }
        return e == hipSuccess ? COLA_OK : hip_fail(e, "timing_reset");
    });
}

int cola_timing_read(int kc, int64_t* launches, double* ms, double* flops, double* bytes) {
    if (kc < 0 || kc >= COLA_KC_COUNT || !launches || !ms || !flops || !bytes) return COLA_ERR_INVALID_ARG;
    return guarded([&]() -> int {
        TimingState& t = timing();
        std::lock_guard<std::mutex> lock(t.mu);
        hipError_t e = drain(t);
        if (e != hipSuccess) return hip_fail(e, "timing_read");
        *launches = t.launches[kc];
        *ms = t.ms[kc];
        *flops = t.flops[kc];
        *bytes = t.bytes[kc];
        return COLA_OK;
    });
}

}  // extern "C"

// ---------------------------------------------------------------------------
// grouped projections that read the same input
// ---------------------------------------------------------------------------
namespace {

struct GDims {
    int64_t T, d_in, ldx, ldz, R;
    int n;
    int64_t r[COLA_GROUP_MAX], d_out[COLA_GROUP_MAX], ldy[COLA_GROUP_MAX], off[COLA_GROUP_MAX];
    bool bf16;
    size_t esize;
};

int check_group(const cola_group_desc* d, GDims* out) {
    if (!d) return COLA_ERR_INVALID_ARG;
    if (d->n < 1 || d->n > COLA_GROUP_MAX) return COLA_ERR_INVALID_ARG;
    GDims g{};
    g.n = d->n;
    g.R = 0;
    for (int p = 0; p < g.n; ++p) {
        // each projection must be a valid single layer (enums, shapes, pitches)
        cola_desc c{};
        c.T = d->T; c.d_in = d->d_in; c.d_out = d->d_out[p]; c.r = d->r[p];
        c.ldx = d->ldx; c.ldy = d->ldy[p]; c.ldz = 0;
        c.dtype = d->dtype; c.act = d->act; c.recompute = d->recompute;
        Dims x;
        const int st = check_desc(&c, &x);
        if (st != COLA_OK) return st;
        g.r[p] = x.r; g.d_out[p] = x.d_out; g.ldy[p] = x.ldy; g.off[p] = g.R;
        g.R += x.r;
        g.T = x.T; g.d_in = x.d_in; g.ldx = x.ldx; g.bf16 = x.bf16; g.esize = x.esize;
    }
    if (g.R > kMaxDim) return COLA_ERR_BAD_SHAPE;
    g.ldz = d->ldz ? d->ldz : g.R;
    if (g.ldz < g.R || g.ldz > kMaxPitch) return COLA_ERR_BAD_SHAPE;
    if ((double)g.T * (double)g.ldz > 4.0e18 || (double)g.R * (double)g.d_in > 4.0e18) return COLA_ERR_BAD_SHAPE;
    *out = g;
    return COLA_OK;
}

// Workspace: [H_all copy (CoLA-M)] [repacked A_all] [repacked B_p ...]
struct GFwdPlan {
    int64_t ldw;
    size_t off_h, total;
    Pack pa, pb[COLA_GROUP_MAX];
};

GFwdPlan plan_group_fwd(const GDims& g, bool recompute) {
    GFwdPlan p;
    p.ldw = line_pitch(g.bf16, g.R);
    p.off_h = 0;
    const size_t hbytes = recompute ? align256((size_t)g.T * (size_t)p.ldw * g.esize) : 0;
    p.pa = plan_pack(g.bf16, g.R, g.d_in, hbytes);
    size_t next = p.pa.off + p.pa.bytes;
    for (int q = 0; q < g.n; ++q) {
        p.pb[q] = plan_pack(g.bf16, g.d_out[q], g.r[q], next);
        next = p.pb[q].off + p.pb[q].bytes;
    }
    p.total = g.T == 0 ? 0 : next;
    return p;
}

// The weight gradients of a group are the products w = 0 (dA_all, R x d_in)
// and w = 1 + p (dB_p, d_out_p x r_p), all over K = T.  They run in pairs
// (0, 1), (2, 3), ...: one launch with one split for a pair whose members
// both go to the PP family (bf16, both output dimensions above 128), else one
// launch each.  Workspace: [dZ_all] [H_all (CoLA-M)] [partials of the first
// member of a pair] [of the second], both reused pair after pair,
// [repacked A_all] [repacked B_p ...].
struct GBwdPlan {
    int64_t ldw;
    size_t off_dz, off_h, off_p0, off_p1, total;
    int nw;                                // 1 + number of projections
    Split sp[COLA_GROUP_MAX + 1];          // split of each product (shared within a launched pair)
    bool paired[COLA_GROUP_MAX + 1];       // pair starting at an even w launched together
    Pack wa, wb[COLA_GROUP_MAX];
};

// Shape (M, N) and kernel tag of weight-gradient product w of a group.
void group_wgrad_shape(const GDims& g, int w, int64_t* M, int64_t* N, int* tag) {
    if (w == 0) {
        *M = g.R;
        *N = g.d_in;
        *tag = TAG_BWD_DA;
    } else {
        *M = g.d_out[w - 1];
        *N = g.r[w - 1];
        *tag = TAG_BWD_DB;
    }
}

GBwdPlan plan_group_bwd(const GDims& g, bool recompute) {
    GBwdPlan p;
    p.ldw = line_pitch(g.bf16, g.R);
    const size_t zbytes = align256((size_t)g.T * (size_t)p.ldw * g.esize);
    p.off_dz = 0;
    p.off_h = zbytes;
    p.off_p0 = p.off_h + (recompute ? zbytes : 0);
    p.nw = g.n + 1;
    size_t pb[2] = {0, 0};
    for (int w0 = 0; w0 < p.nw; w0 += 2) {
        int64_t M[2], N[2];
        int tag[2];
        const int cnt = w0 + 1 < p.nw ? 2 : 1;
        for (int k = 0; k < cnt; ++k) group_wgrad_shape(g, w0 + k, &M[k], &N[k], &tag[k]);
        p.paired[w0] = cnt == 2 && wgrad_pairing_on() && g.bf16 && gemm_family(M[0], N[0], tag[0]) == FAM_PP &&
                       gemm_family(M[1], N[1], tag[1]) == FAM_PP;
        if (p.paired[w0]) {
            const int64_t tiles = gemm_tiles(true, M[0], N[0], tag[0]) + gemm_tiles(true, M[1], N[1], tag[1]);
            p.sp[w0] = p.sp[w0 + 1] = plan_split_tiles(true, tiles, gemm_slots(true, M[0], N[0], tag[0]), g.T,
                                                       (double)M[0] * N[0] + (double)M[1] * N[1]);
        } else {
            for (int k = 0; k < cnt; ++k) p.sp[w0 + k] = plan_split(g.bf16, M[k], N[k], g.T, tag[k]);
        }
        for (int k = 0; k < cnt; ++k) {
            const Split& sp = p.sp[w0 + k];
            const size_t b = sp.splits > 1 ? align256((size_t)sp.splits * (size_t)(M[k] * N[k]) * 4) : 0;
            if (b > pb[k]) pb[k] = b;
        }
    }
    p.off_p1 = p.off_p0 + pb[0];
    p.wa = plan_pack(g.bf16, g.R, g.d_in, p.off_p1 + pb[1]);
    size_t next = p.wa.off + p.wa.bytes;
    for (int q = 0; q < g.n; ++q) {
        p.wb[q] = plan_pack(g.bf16, g.d_out[q], g.r[q], next);
        next = p.wb[q].off + p.wb[q].bytes;
    }
    p.total = g.T == 0 ? 0 : next;
    return p;
}

}  // namespace

extern "C" {

size_t cola_group_workspace_bytes(const cola_group_desc* desc, int phase) {
    GDims g;
    if (check_group(desc, &g) != COLA_OK) return 0;
    if (phase == 0) return plan_group_fwd(g, desc->recompute == 1).total;
    if (phase == 1) return plan_group_bwd(g, desc->recompute == 1).total;
    if (phase == 2) return plan_group_fwd(g, true).total;
    return 0;
}

}  // extern "C"

namespace {

// Forward of a validated group with the pointers checked.  Z_all == NULL is
// the inference forward: K1 stores only H (into the workspace), nothing is
// kept for a backward pass.
int group_forward(const GDims& g, int act, const void* X, const void* A_all, const void* const* B,
                  void* const* Y, void* Z_all, void* H_all, bool h_in_ws, char* w, hipStream_t s,
                  const Gate* gate = nullptr) {
    const GFwdPlan p = plan_group_fwd(g, h_in_ws);
    char* Hbuf = h_in_ws ? w + p.off_h : reinterpret_cast<char*>(H_all);
    const int64_t ldh = h_in_ws ? p.ldw : g.ldz;
    const double es = (double)g.esize;

    const void* Aw;
    int64_t lda;
    hipError_t e = use_weight(p.pa, A_all, g.R, g.d_in, w, &Aw, &lda, s);
    if (e != hipSuccess) return hip_fail(e, "pack_rows");

    // K1 for every projection at once: Z_all = X A_all^T, H_all = sigma(Z_all)
    if (Z_all) {
        GemmArgs k1 = make_args(TAG_FWD_Z, g.T, g.R, g.d_in, X, g.ldx, KMAJ, Aw, lda, KMAJ, Z_all, g.ldz, EPI_Z_H,
                                act);
        k1.aux = Hbuf;
        k1.ldaux = ldh;
        const double b1 = es * ((double)g.T * g.d_in + (double)g.R * g.d_in + 2.0 * g.T * g.R);
        e = timed(COLA_KC_FWD_Z, gemm_flops(g.T, g.R, g.d_in), b1, s, [&] { return gemm(k1, g.bf16, s); });
        if (e != hipSuccess) return hip_fail(e, "fwd_z_sigma");
    } else {
        GemmArgs k1 = make_args(TAG_INFER_H, g.T, g.R, g.d_in, X, g.ldx, KMAJ, Aw, lda, KMAJ, Hbuf, ldh, EPI_H, act);
        const double b1 = es * ((double)g.T * g.d_in + (double)g.R * g.d_in + (double)g.T * g.R);
        e = timed(COLA_KC_INFER_H, gemm_flops(g.T, g.R, g.d_in), b1, s, [&] { return gemm(k1, g.bf16, s); });
        if (e != hipSuccess) return hip_fail(e, "infer_h");
    }

    // K2 per projection: Y_p = H_p B_p^T
    for (int q = 0; q < g.n; ++q) {
        const void* Bw;
        int64_t ldb;
        e = use_weight(p.pb[q], B[q], g.d_out[q], g.r[q], w, &Bw, &ldb, s);
        if (e != hipSuccess) return hip_fail(e, "pack_rows");
        GemmArgs k2 = make_args(TAG_FWD_Y, g.T, g.d_out[q], g.r[q], Hbuf + g.off[q] * g.esize, ldh, KMAJ, Bw,
                                ldb, KMAJ, Y[q], g.ldy[q], EPI_STORE, act);
        double b2 = es * ((double)g.T * g.r[q] + (double)g.d_out[q] * g.r[q] + (double)g.T * g.d_out[q]);
        if (gate && q == g.n - 1) {
            // the last projection also stores m = g u (g: the group's first output)
            GemmArgs kg = make_args(TAG_FWD_YG, g.T, g.d_out[q], g.r[q], Hbuf + g.off[q] * g.esize, ldh, KMAJ, Bw,
                                    ldb, KMAJ, Y[q], gate->ld, EPI_GATE, act);
            kg.zin = gate->g;
            kg.ldzin = gate->ld;
            kg.aux = gate->out;
            kg.ldaux = gate->ld;
            *gate->fused = g.bf16 && gate_fusion_on() && g.ldy[q] == gate->ld && pp_takes(kg);
            if (*gate->fused) {
                k2 = kg;
                if (!gate->keep_u) k2.c = nullptr;
                b2 = es * ((double)g.T * g.r[q] + (double)g.d_out[q] * g.r[q] +
                           (gate->keep_u ? 3.0 : 2.0) * g.T * g.d_out[q]);
            }
        }
        e = timed(COLA_KC_FWD_Y, gemm_flops(g.T, g.d_out[q], g.r[q]), b2, s, [&] { return gemm(k2, g.bf16, s); });
        if (e != hipSuccess) return hip_fail(e, "fwd_y");
    }
    return COLA_OK;
}

// The group of one projection that a single-layer descriptor describes.
GDims single_group(const Dims& x) {
    GDims g{};
    g.T = x.T; g.d_in = x.d_in; g.ldx = x.ldx; g.ldz = x.ldz; g.R = x.r; g.n = 1;
    g.r[0] = x.r; g.d_out[0] = x.d_out; g.ldy[0] = x.ldy; g.off[0] = 0;
    g.bf16 = x.bf16; g.esize = x.esize;
    return g;
}

int group_fwd_checked(const cola_group_desc* desc, const void* X, const void* A_all, const void* const* B,
                      void* const* Y, void* Z_all, void* H_all, void* ws, size_t ws_bytes, cola_stream_t stream,
                      const Gate* gate) {
    GDims g;
    int st = check_group(desc, &g);
    if (st != COLA_OK) return st;
    const bool recompute = desc->recompute == 1;
    if (recompute ? (H_all != nullptr) : (H_all == nullptr && g.T > 0)) return COLA_ERR_INVALID_ARG;
    if (gate) *gate->fused = false;
    if (g.T == 0) return COLA_OK;
    if (!X || !A_all || !B || !Y || !Z_all) return COLA_ERR_INVALID_ARG;
    for (int q = 0; q < g.n; ++q)
        if (!B[q] || !Y[q]) return COLA_ERR_INVALID_ARG;
    const GFwdPlan p = plan_group_fwd(g, recompute);
    if (p.total > 0 && (!ws || ws_bytes < p.total)) return COLA_ERR_WORKSPACE;
    return group_forward(g, desc->act, X, A_all, B, Y, Z_all, H_all, recompute, reinterpret_cast<char*>(ws),
                         reinterpret_cast<hipStream_t>(stream), gate);
}

int infer_checked(const GDims& g, int act, const void* X, const void* A_all, const void* const* B, void* const* Y,
                  void* ws, size_t ws_bytes, cola_stream_t stream) {
    if (g.T == 0) return COLA_OK;
    if (!X || !A_all || !B || !Y) return COLA_ERR_INVALID_ARG;
    for (int q = 0; q < g.n; ++q)
        if (!B[q] || !Y[q]) return COLA_ERR_INVALID_ARG;
    const size_t need = plan_group_fwd(g, true).total;
    if (need > 0 && (!ws || ws_bytes < need)) return COLA_ERR_WORKSPACE;
    return group_forward(g, act, X, A_all, B, Y, nullptr, nullptr, true, reinterpret_cast<char*>(ws),
                         reinterpret_cast<hipStream_t>(stream));
}

}  // namespace

extern "C" {

int cola_group_fwd(const cola_group_desc* desc, const void* X, const void* A_all, const void* const* B,
                   void* const* Y, void* Z_all, void* H_all, void* ws, size_t ws_bytes, cola_stream_t stream) {
    return guarded([&]() -> int {
        return group_fwd_checked(desc, X, A_all, B, Y, Z_all, H_all, ws, ws_bytes, stream, nullptr);
    });
}

int cola_group_infer(const cola_group_desc* desc, const void* X, const void* A_all, const void* const* B,
                     void* const* Y, void* ws, size_t ws_bytes, cola_stream_t stream) {
    return guarded([&]() -> int {
        GDims g;
        const int st = check_group(desc, &g);
        if (st != COLA_OK) return st;
        return infer_checked(g, desc->act, X, A_all, B, Y, ws, ws_bytes, stream);
    });
}

int cola_infer(const cola_desc* desc, const void* X, const void* A, const void* B, void* Y, void* ws,
               size_t ws_bytes, cola_stream_t stream) {
    return guarded([&]() -> int {
        Dims x;
        const int st = check_desc(desc, &x);
        if (st != COLA_OK) return st;
        const void* Bs[1] = {B};
        void* Ys[1] = {Y};
        return infer_checked(single_group(x), desc->act, X, A, Bs, Ys, ws, ws_bytes, stream);
    });
}

int cola_group_bwd(const cola_group_desc* desc, const void* const* dY, const void* X, const void* Z_all,
                   const void* H_all, const void* A_all, const void* const* B, void* dX, float* dA_all,
                   float* const* dB, void* ws, size_t ws_bytes, cola_stream_t stream) {
    return guarded([&]() -> int {
        GDims g;
        int st = check_group(desc, &g);
        if (st != COLA_OK) return st;
        const bool recompute = desc->recompute == 1;
        if (recompute ? (H_all != nullptr) : (H_all == nullptr && g.T > 0)) return COLA_ERR_INVALID_ARG;
        if (!dA_all || !dB) return COLA_ERR_INVALID_ARG;
        for (int q = 0; q < g.n; ++q)
            if (!dB[q]) return COLA_ERR_INVALID_ARG;
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        if (g.T == 0) {
            // empty batch: the token sums are empty
            hipError_t e = timed(COLA_KC_FILL, 0.0, 4.0 * g.R * g.d_in, s,
                                 [&] { return launch_fill_zero(dA_all, g.R * g.d_in, s); });
            for (int q = 0; q < g.n && e == hipSuccess; ++q)
                e = timed(COLA_KC_FILL, 0.0, 4.0 * g.d_out[q] * g.r[q], s,
                          [&] { return launch_fill_zero(dB[q], g.d_out[q] * g.r[q], s); });
            return e == hipSuccess ? COLA_OK : hip_fail(e, "fill_zero");
        }
        if (!dY || !X || !Z_all || !A_all || !B || !dX) return COLA_ERR_INVALID_ARG;
        for (int q = 0; q < g.n; ++q)
            if (!dY[q] || !B[q]) return COLA_ERR_INVALID_ARG;
        const GBwdPlan p = plan_group_bwd(g, recompute);
        if (!ws || ws_bytes < p.total) return COLA_ERR_WORKSPACE;

        char* w = reinterpret_cast<char*>(ws);
        char* dZ = w + p.off_dz;
        const char* Hbuf = recompute ? w + p.off_h : reinterpret_cast<const char*>(H_all);
        const int64_t ldh = recompute ? p.ldw : g.ldz;
        const double es = (double)g.esize;
        const void* Aw;
        int64_t lda;
        hipError_t e = use_weight(p.wa, A_all, g.R, g.d_in, w, &Aw, &lda, s);
        if (e != hipSuccess) return hip_fail(e, "pack_rows");

        // K3 per projection: dZ_p = (dY_p B_p) (.) sigma'(Z_p)  [+ H_p for CoLA-M]
        for (int q = 0; q < g.n; ++q) {
            const void* Bw;
            int64_t ldb;
            e = use_weight(p.wb[q], B[q], g.d_out[q], g.r[q], w, &Bw, &ldb, s);
            if (e != hipSuccess) return hip_fail(e, "pack_rows");
            GemmArgs k3 = make_args(TAG_BWD_DZ, g.T, g.r[q], g.d_out[q], dY[q], g.ldy[q], KMAJ, Bw, ldb, MNMAJ,
                                    dZ + g.off[q] * g.esize, p.ldw, EPI_DZ, desc->act);
            k3.zin = reinterpret_cast<const char*>(Z_all) + g.off[q] * g.esize;
            k3.ldzin = g.ldz;
            k3.aux = recompute ? (void*)(w + p.off_h + g.off[q] * g.esize) : nullptr;
            k3.ldaux = p.ldw;
            const double b3 = es * ((double)g.T * g.d_out[q] + (double)g.d_out[q] * g.r[q] +
                                    (double)g.T * g.r[q] * (recompute ? 3.0 : 2.0));
            e = timed(COLA_KC_BWD_DZ, gemm_flops(g.T, g.r[q], g.d_out[q]), b3, s, [&] { return gemm(k3, g.bf16, s); });
            if (e != hipSuccess) return hip_fail(e, "bwd_dz");
        }

        // K4 for every projection at once: dX = dZ_all A_all = sum_p dZ_p A_p
        GemmArgs k4 = make_args(TAG_BWD_DX, g.T, g.d_in, g.R, dZ, p.ldw, KMAJ, Aw, lda, MNMAJ, dX, g.ldx, EPI_STORE,
                                desc->act);
        const double b4 = es * ((double)g.T * g.R + (double)g.R * g.d_in + (double)g.T * g.d_in);
        e = timed(COLA_KC_BWD_DX, gemm_flops(g.T, g.d_in, g.R), b4, s, [&] { return gemm(k4, g.bf16, s); });
        if (e != hipSuccess) return hip_fail(e, "bwd_dx");

        // K5 for every projection at once, dA_all = dZ_all^T X (product 0),
        // and K6 per projection, dB_p = dY_p^T H_p (product 1 + p), in pairs
        struct Prod {
            int64_t M, N;
            const void *P, *Q;
            int64_t ldp, ldq;
            float* C;
            int kc;
        };
        Prod pr[COLA_GROUP_MAX + 1];
        pr[0] = Prod{g.R, g.d_in, dZ, X, p.ldw, g.ldx, dA_all, COLA_KC_BWD_DA};
        for (int q = 0; q < g.n; ++q)
            pr[q + 1] = Prod{g.d_out[q], g.r[q], dY[q], Hbuf + g.off[q] * g.esize, g.ldy[q], ldh, dB[q],
                             COLA_KC_BWD_DB};
        float* part[2] = {reinterpret_cast<float*>(w + p.off_p0), reinterpret_cast<float*>(w + p.off_p1)};
        auto in_bytes = [&](const Prod& a) { return es * ((double)g.T * a.M + (double)g.T * a.N); };
        for (int w0 = 0; w0 < p.nw; w0 += 2) {
            const int cnt = w0 + 1 < p.nw ? 2 : 1;
            if (p.paired[w0]) {
                const Prod &a = pr[w0], &b = pr[w0 + 1];
                st = wgrad_pair(g.T, p.sp[w0], a.M, a.N, a.P, a.ldp, a.Q, a.ldq, a.C, part[0], b.M, b.N, b.P, b.ldp,
                                b.Q, b.ldq, b.C, part[1], in_bytes(a) + in_bytes(b), s);
                if (st != COLA_OK) return st;
                continue;
            }
            for (int k = 0; k < cnt; ++k) {
                const Prod& a = pr[w0 + k];
                st = wgrad(g.bf16, a.M, a.N, g.T, a.P, a.ldp, a.Q, a.ldq, a.C, p.sp[w0 + k], part[k], a.kc,
                           in_bytes(a), s);
                if (st != COLA_OK) return st;
            }
        }
        return COLA_OK;
    });
}

}  // extern "C"

// ---- the block's gated-product hooks (block.hpp) ----
namespace cola {

int group_fwd_gated(const cola_group_desc* desc, const void* X, const void* A_all, const void* const* B,
                    void* const* Y, void* Z_all, void* H_all, void* ws, size_t ws_bytes, cola_stream_t stream,
                    const void* g, int64_t ld, void* m, bool* fused, bool keep_u) {
    if (!fused) return COLA_ERR_INVALID_ARG;
    *fused = false;
    const Gate gate{g, nullptr, ld, m, nullptr, fused, keep_u};
    return guarded([&]() -> int {
        return group_fwd_checked(desc, X, A_all, B, Y, Z_all, H_all, ws, ws_bytes, stream, &gate);
    });
}

int layer_bwd_gated(const cola_desc* desc, const void* dY, const void* X, const void* Z, const void* H,
                    const void* A, const void* B, void* dX, float* dA, float* dB, void* ws, size_t ws_bytes,
                    cola_stream_t stream, const void* g, const void* u, int64_t ld, void* dg, void* du,
                    bool* fused) {
    if (!fused) return COLA_ERR_INVALID_ARG;
    *fused = false;
    const Gate gate{g, u, ld, dg, du, fused, true};
    return guarded([&]() -> int {
        return bwd_checked(desc, dY, X, Z, H, A, B, dX, dA, dB, ws, ws_bytes, stream, &gate);
    });
}

}  // namespace cola
