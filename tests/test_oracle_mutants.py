"""The pins are strong enough: copies of the oracle with one planted mistake
each (a dropped term, a wrong sign, a wrong operand, an off-by-one) must fail
at least one pin.  Mistakes are planted in a temporary copy of the oracle's
source on the CPU; the real oracle is untouched."""
import subprocess

import pytest

import oracle
from oracle.build import SRC
import test_oracle_pins as pins

MUTANTS = {
    "sigma_prime_drops_z_term": ("return s * (1.0 + z * (1.0 - s));", "return s;"),
    "logistic_wrong_sign": ("return 1.0 / (1.0 + exp(-z));", "return 1.0 / (1.0 + exp(z));"),
    "dA_from_H_not_dZ": ("gemm_tn(r, d_in, T, dZ, X, dA);", "gemm_tn(r, d_in, T, H, X, dA);"),
    "dB_from_Z_not_H": ("gemm_tn(d_out, r, T, dY, H, dB);", "gemm_tn(d_out, r, T, dY, Z, dB);"),
    "no_sigma_prime_in_dZ": ("dZ[i] *= oracle_sigma_prime(act, Z[i]);", "dZ[i] *= 1.0;"),
    "gemm_nt_drops_last_k": ("for (int64_t k = 0; k < K; ++k) s += P[m * K + k] * Q[n * K + k];",
                             "for (int64_t k = 0; k + 1 < K; ++k) s += P[m * K + k] * Q[n * K + k];"),
    "rows_sigma_prime_of_H": ("dz[j] = s * oracle_sigma_prime(act, z[j]);",
                              "dz[j] = s * oracle_sigma_prime(act, h[j]);"),
    "wgrad_dB_uses_dZ": ("for (int64_t t = 0; t < T; ++t) s += dY[t * d_out + o] * H[t];",
                         "for (int64_t t = 0; t < T; ++t) s += dY[t * d_out + o] * dZ[t];"),
    "H_skips_sigma": ("H[i] = oracle_sigma(act, Z[i]);\n    gemm_nt", "H[i] = Z[i];\n    gemm_nt"),
    "gelu_prime_drops_pdf_term": ("if (act == 2) return normal_cdf(z) + z * normal_pdf(z);",
                                  "if (act == 2) return normal_cdf(z);"),
    "gelu_cdf_wrong_sign": ("return 0.5 * erfc(-z * 0.70710678118654752440);",
                            "return 0.5 * erfc(z * 0.70710678118654752440);"),
    "gelu_pdf_wrong_scale": ("exp(-0.5 * z * z)", "exp(-z * z)"),
    "outer_backward_drops_sigma_prime": ("dP[i] = dY[i] * oracle_sigma_prime(outer, P[i]);", "dP[i] = dY[i];"),
    "outer_sigma_prime_of_Y": ("dP[i] = dY[i] * oracle_sigma_prime(outer, P[i]);",
                               "dP[i] = dY[i] * oracle_sigma_prime(outer, oracle_sigma(outer, P[i]));"),
    "outer_forward_skips_sigma": ("Y[i] = oracle_sigma(outer, P[i]);", "Y[i] = P[i];"),
    "outer_uses_inner_act": ("dP[i] = dY[i] * oracle_sigma_prime(outer, P[i]);",
                             "dP[i] = dY[i] * oracle_sigma_prime(act, P[i]);"),
    "dense_dW_transposed": ("gemm_tn(d_out, d_in, T, dY, X, dW);", "gemm_tn(d_in, d_out, T, X, dY, dW);"),
    "dense_dX_reads_W_transposed": ("gemm_nn(T, d_in, d_out, dY, W, dX);", "gemm_nt(T, d_in, d_out, dY, W, dX);"),
    "dense_fwd_reads_W_transposed": ("gemm_nt(T, d_out, d_in, X, W, Y);", "gemm_nn(T, d_out, d_in, X, W, Y);"),
    "mac_counter_fwd_only_one_gemm": ("static void gemm_nt(int64_t M, int64_t N, int64_t K,\n                    const double* P, const double* Q, double* C) {\n    g_mac_count += M * N * K;",
                                      "static void gemm_nt(int64_t M, int64_t N, int64_t K,\n                    const double* P, const double* Q, double* C) {\n    g_mac_count += M * N;"),
}


def battery():
    """Run a selection of pins; return the names of those that failed."""
    checks = [
        ("silu_values", pins.test_silu_special_values, ()),
        ("silu_fd", pins.test_silu_derivative_by_central_difference, (1.0,)),
        ("silu_expit", pins.test_silu_against_scipy_expit, ()),
        ("identity", pins.test_identity_sigma_is_low_rank_product, ((7, 5, 4, 3),)),
        ("fd_grads", pins.test_gradients_by_central_differences, ((3, 5, 4, 2), "silu")),
        ("torch", pins.test_against_torch_fp64_autograd, ((16, 32, 24, 8), "silu")),
        ("gelu_values", pins.test_gelu_special_values, ()),
        ("gelu_ndtr", pins.test_gelu_against_scipy_ndtr, ()),
        ("gelu_fd", pins.test_gelu_derivative_by_central_difference, (-0.75,)),
        ("fd_grads_gelu", pins.test_gradients_by_central_differences, ((3, 5, 4, 2), "gelu")),
        ("prop1", pins.test_prop1_limit_construction, ()),
        ("lemma", pins.test_lemma_esigma_zero_construction, ()),
        ("sampled", pins.test_sampled_rows_and_columns_match_full, ()),
        ("flops", pins.test_layer_flop_count, ((3, 8, 5, 2),)),
        ("outer_identity", pins.test_outer_identity_is_the_plain_layer, ("silu",)),
        ("outer_fd", pins.test_outer_gradients_by_central_differences, ((3, 5, 4, 2), "identity", "silu")),
        ("outer_torch", pins.test_outer_against_torch_fp64_autograd, ("silu", "gelu")),
        ("dense_fd", pins.test_dense_gradients_by_central_differences, ((4, 2, 7),)),
        ("dense_cross", pins.test_dense_backward_cross_pinned_to_cola, ((9, 7, 5, 3),)),
    ]
    failed = []
    for name, fn, args in checks:
        try:
            fn(*args)
        except AssertionError:
            failed.append(name)
    return failed


def test_real_oracle_passes_battery():
    oracle.use_library(None)
    assert battery() == []


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_mutant_is_caught(mutant, tmp_path):
    old, new = MUTANTS[mutant]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation site not found exactly once"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                    str(path), "-o", str(lib), "-lm"], check=True)
    try:
        oracle.use_library(str(lib))
        failed = battery()
    finally:
        oracle.use_library(None)
    assert failed, f"mutant {mutant} passed every pin"
