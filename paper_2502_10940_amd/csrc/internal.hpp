// internal.hpp -- declarations shared by the translation units of libcola.so.
// Not part of the public ABI (that is include/cola.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cola {

// Operand layout of a GEMM C[M][N] = sum_k P(m, k) Q(n, k):
//   KMAJ : element (m, k) at ptr[m * ld + k]   (k contiguous)
//   MNMAJ: element (m, k) at ptr[k * ld + m]   (m contiguous, k strided)
enum Layout : int { KMAJ = 0, MNMAJ = 1 };

// Epilogue applied to the fp32 accumulator tile.
enum Epilogue : int {
    EPI_STORE = 0,     // c = acc, in the output dtype (bf16 / fp32 for GEMMs in fp32 storage)
    EPI_STORE_F32 = 1, // c = acc as fp32 (weight gradients, split-K partials)
    EPI_Z_H = 2,       // c = Z = round(acc); aux = H = round(sigma(Z))
    EPI_DZ = 3,        // c = dZ = round(acc * sigma'(Z)), Z read from zin; aux = H if non-NULL
    EPI_H = 4,         // c = H = round(sigma(round(acc))): H of EPI_Z_H without storing Z (inference)
    // the gated MLP of the decoder block (ping-pong family only):
    EPI_GATE = 5,      // c = u = round(acc) (not stored when c is NULL); aux = m = round(g u), g read from zin
    EPI_DGATE = 6,     // with dm = round(acc): c = round(dm u), aux = round(dm g); g from zin, u from zin2
};

// Which step of the layer a GEMM is (same numbering as the kernel classes of
// the public timing API).
enum Tag : int {
    TAG_FWD_Z = 0, TAG_FWD_Y = 1, TAG_BWD_DZ = 2, TAG_BWD_DX = 3, TAG_BWD_DA = 4,
    TAG_BWD_DB = 5, TAG_DENSE_FWD = 7, TAG_DENSE_DX = 8, TAG_DENSE_DW = 9, TAG_INFER_H = 11,
    TAG_FWD_YP = 12,    // K2 of the both-sigma variant: EPI_Z_H storing P and sigma_out(P)
    TAG_FWD_YG = 13,    // K2 of the up projection with the gated product (EPI_GATE)
    TAG_BWD_DXG = 14    // K4 of the down projection with the gated product's backward (EPI_DGATE)
};

struct GemmArgs {
    int64_t M, N, K;
    const void* p; int64_t ldp; int p_layout;    // left operand P
    const void* q; int64_t ldq; int q_layout;    // right operand Q (C = P Q^T)
    void* c; int64_t ldc;                        // output
    void* aux; int64_t ldaux;                    // second output (H) or NULL
    const void* zin; int64_t ldzin;              // Z read by EPI_DZ, g by EPI_GATE / EPI_DGATE
    const void* zin2; int64_t ldzin2;            // u read by EPI_DGATE
    int epi;
    int tag;                                     // Tag
    int act;                                     // 0 identity, 1 SiLU
    int splits;                                  // split-K count (>= 1)
    int64_t k_chunk;                             // K range per split (multiple of the K tile)
    int64_t split_stride;                        // elements between partial slices of c
};

// Enqueue one GEMM.  Return hipSuccess or the launch error.
hipError_t launch_gemm_bf16(const GemmArgs& a, hipStream_t s);
// The kernel families behind launch_gemm_bf16:
//   STREAM -- BM x 128 tiles, direct-to-LDS loads, three K stages, two per CU
//   PP     -- 256 x 256 tiles, two wave groups per workgroup in ping-pong
hipError_t launch_gemm_stream(const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_pp(const GemmArgs& a, hipStream_t s);
// Two weight-gradient products (both operands m-contiguous, fp32 output) in
// one PP grid: a0's tiles and splits, then a1's.  Operands as for PP.
hipError_t launch_gemm_pp_pair(const GemmArgs& a0, const GemmArgs& a1, hipStream_t s);
// a0 and a1 in one launch when both go to the PP family with operands it
// takes (else one launch each, as launch_gemm_bf16).
hipError_t launch_gemm_bf16_pair(const GemmArgs& a0, const GemmArgs& a1, hipStream_t s);

enum Family : int { FAM_STREAM = 1, FAM_PP = 4 };
// Family used for a GEMM (also used by the split planner): PP where both
// output dimensions exceed 128, else STREAM; the option OPT_STREAM_ONLY
// sends every product to STREAM.
int gemm_family(int64_t M, int64_t N, int tag);
// Whether the PP family runs this GEMM (family and operand alignment): the
// gated epilogues exist only there.
bool pp_takes(const GemmArgs& a);

// Process-wide tuning options (the public cola_set_option): the values of
// cola_option in include/cola.h.  set_option returns 0, or -1 for an unknown
// option or a value other than 0 / 1.
enum Option : int { OPT_STREAM_ONLY = 0, OPT_WGRAD_PAIR = 1, OPT_FUSE_GATE = 2 };
int set_option(int option, int value);
int get_option(int option);

// fp32 storage: the VALU GEMM of gemm_f32.hip (true fp32 FMAs).
hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s);

// out[i] = sum_{s < splits} part[s * stride + i], s in increasing order (fp32).
hipError_t launch_reduce_splits(const float* part, int splits, int64_t stride,
                                float* out, int64_t n, hipStream_t s);
// Both at once for two outputs with the same split count (one launch).
hipError_t launch_reduce_splits2(const float* p0, int64_t st0, float* o0, int64_t n0, const float* p1, int64_t st1,
                                 float* o1, int64_t n1, int splits, hipStream_t s);
// dst[r][c] = src[r][c] for c < width, 0 for width <= c < ld (16-bit
// elements; src rows are contiguous).  Gives weights with odd widths a
// 16-byte aligned row pitch.
hipError_t launch_pack_rows(const void* src, int64_t rows, int64_t width, void* dst, int64_t ld,
                            hipStream_t s);
// out[i] = 0 for i < n (fp32 words).
hipError_t launch_fill_zero(float* out, int64_t n, hipStream_t s);

// out[t][o] = dy[t][o] * sigma_act'(p[t][o]) over T rows of n elements, in
// the storage dtype (bf16 rounded to nearest even, or fp32).
hipError_t launch_outer_grad(bool bf16, const void* dy, int64_t lddy, const void* p, int64_t ldp, void* out,
                             int64_t ldo, int64_t T, int64_t n, int act, hipStream_t s);

// Largest row pitch (elements) of any operand: the 256 x 256 family reads a
// K tile of a k-contiguous operand through a buffer descriptor whose range is
// 2^31 bytes from the tile's first row, and 255 rows of this pitch fit it.
// Descriptors with wider pitches are refused (COLA_ERR_BAD_SHAPE).
constexpr int64_t kMaxPitch = int64_t(1) << 22;

// K tile of the bf16 kernel: split-K chunks are multiples of it.
constexpr int BF16_BK = 64;
// K tile of the fp32 kernel.
constexpr int F32_BK = 16;

// Tile geometry of the launchers (mirrored here for planning): the PP family
// uses 256 x 256 (only when M > 128 and N > 128), STREAM BM x 128 with
// BM = 256 (128 when M <= 128); fp32 uses 64 x 64.
inline bool bf16_wide_ok(int64_t M, int64_t N) { return M > 128 && N > 128; }
inline int64_t gemm_tiles(bool bf16, int64_t M, int64_t N, int tag) {
    const bool wide = bf16 && gemm_family(M, N, tag) == FAM_PP;
    const int64_t tm = bf16 ? (M > 128 ? 256 : 128) : 64;
    const int64_t tn = bf16 ? (wide ? 256 : 128) : 64;
    return ((M + tm - 1) / tm) * ((N + tn - 1) / tn);
}
// Workgroups the chip holds at once (256 CUs).
inline int64_t gemm_slots(bool bf16, int64_t M, int64_t N, int tag) {
    if (!bf16) return 1024;
    return gemm_family(M, N, tag) == FAM_PP ? 256 : 512;
}

}  // namespace cola
