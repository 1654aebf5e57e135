// gemm_dispatch.hip -- which bf16 MFMA kernel family runs each GEMM
// C[M][N] = sum_k P(m, k) Q(n, k) of the layer, and the library's tuning
// options.
//
//  * PP (gemm_pp.hip): 256 x 256 tiles, two wave groups in ping-pong, for
//    every product whose output exceeds one 128-wide tile in both dimensions
//    (weight gradients: at least 128 in both) and whose operands have
//    16-byte aligned rows (measured on MI355X:
//    1.1-1.5x the streaming family on the products of the layer, weight
//    gradients included).
//  * STREAM (gemm_stream.hip): BM x 128 tiles, two workgroups per CU, for
//    skinny outputs, unaligned operands and K tails of any shape.
#include <atomic>

#include "internal.hpp"

namespace cola {

namespace {
// process-wide tuning options (cola_set_option)
std::atomic<int> g_force_stream{0};
std::atomic<int> g_wgrad_pair{1};
std::atomic<int> g_fuse_gate{1};
}  // namespace

int set_option(int option, int value) {
    if (value != 0 && value != 1) return -1;
    switch (option) {
        case OPT_STREAM_ONLY: g_force_stream.store(value); return 0;
        case OPT_WGRAD_PAIR: g_wgrad_pair.store(value); return 0;
        case OPT_FUSE_GATE: g_fuse_gate.store(value); return 0;
        default: return -1;
    }
}

int get_option(int option) {
    switch (option) {
        case OPT_STREAM_ONLY: return g_force_stream.load();
        case OPT_WGRAD_PAIR: return g_wgrad_pair.load();
        case OPT_FUSE_GATE: return g_fuse_gate.load();
        default: return -1;
    }
}

// The PP family takes only operands with 16-byte aligned rows whose tile
// offsets fit its 32-bit per-lane offsets.
bool pp_operands_ok(const GemmArgs& a) {
    auto al = [](const void* p, int64_t ld) {
        return (reinterpret_cast<uintptr_t>(p) & 15u) == 0 && (ld & 7) == 0 && ld < (int64_t(1) << 22);
    };
    return al(a.p, a.ldp) && al(a.q, a.ldq);
}

int gemm_family(int64_t M, int64_t N, int tag) {
    if (g_force_stream.load(std::memory_order_relaxed)) return FAM_STREAM;
    // weight gradients take PP down to 128 x 128 outputs: half-empty 256-row
    // tiles, but the pair of dA and dB in one launch over the whole chip
    // (measured on MI355X at rank 128: the 60M-shaped step 1.479 -> 1.394 ms)
    if ((tag == TAG_BWD_DA || tag == TAG_BWD_DB) && M >= 128 && N >= 128) return FAM_PP;
    return bf16_wide_ok(M, N) ? (int)FAM_PP : (int)FAM_STREAM;
}

bool pp_takes(const GemmArgs& a) { return gemm_family(a.M, a.N, a.tag) == FAM_PP && pp_operands_ok(a); }

hipError_t launch_gemm_bf16_pair(const GemmArgs& a0, const GemmArgs& a1, hipStream_t s) {
    const bool pp = gemm_family(a0.M, a0.N, a0.tag) == FAM_PP && gemm_family(a1.M, a1.N, a1.tag) == FAM_PP &&
                    pp_operands_ok(a0) && pp_operands_ok(a1);
    if (pp) return launch_gemm_pp_pair(a0, a1, s);
    hipError_t e = launch_gemm_bf16(a0, s);
    return e == hipSuccess ? launch_gemm_bf16(a1, s) : e;
}

hipError_t launch_gemm_bf16(const GemmArgs& a, hipStream_t s) {
    if (gemm_family(a.M, a.N, a.tag) == FAM_PP && pp_operands_ok(a)) return launch_gemm_pp(a, s);
    return launch_gemm_stream(a, s);
}

}  // namespace cola
