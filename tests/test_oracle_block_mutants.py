"""The block oracle's pins are strong enough: copies of oracle/block.py with one
planted mistake each (a dropped term, a wrong sign, a wrong operand, an
off-by-one mask, a recompute from the wrong saved tensor) must fail at least
one pin.  Mistakes are planted in a temporary copy on the CPU; the real
oracle is untouched."""
import importlib.util

import pytest

import test_oracle_block as pins
from oracle import block as real_block

SRC = real_block.__file__

MUTANTS = {
    "rmsnorm_drops_eps": ("return x * g[None, :] / np.sqrt(ms + eps)", "return x * g[None, :] / np.sqrt(ms)"),
    "rmsnorm_bwd_drops_projection": ("dx = s * u - x * (s ** 3) * np.sum(u * x, axis=1, keepdims=True) / d",
                                     "dx = s * u"),
    "rmsnorm_bwd_gain_grad_unnormalised": ("dg = np.sum(dy * x * s, axis=0)", "dg = np.sum(dy * x, axis=0)"),
    "rope_wrong_sign": ("= lo * c - hi * s", "= lo * c + hi * s"),
    "rope_angle_exponent": ("inv = base ** (-np.arange(0, hd // 2, dtype=np.float64) * 2.0 / hd)",
                            "inv = base ** (-np.arange(0, hd // 2, dtype=np.float64) * 1.0 / hd)"),
    "attention_no_scale": ("S = qr[rows, cols] @ kr[rows, cols].T / np.sqrt(hd)",
                           "S = qr[rows, cols] @ kr[rows, cols].T"),
    "attention_mask_leaks_next_token": ("future = np.triu(np.ones((seq_len, seq_len), dtype=bool), 1)",
                                         "future = np.triu(np.ones((seq_len, seq_len), dtype=bool), 2)"),
    "softmax_bwd_drops_row_term": ("dS = P * (dP - np.sum(dP * P, axis=1, keepdims=True))", "dS = P * dP"),
    "attention_bwd_no_inverse_rope": ("return (rope(dqr, n_seq, seq_len, heads, base, inverse=True),",
                                      "return (rope(dqr, n_seq, seq_len, heads, base, inverse=False),"),
    "attention_bwd_dk_from_dS": ("dkr[rows, cols] = dS.T @ qr[rows, cols] / np.sqrt(hd)",
                                 "dkr[rows, cols] = dS @ qr[rows, cols] / np.sqrt(hd)"),
    "gated_bwd_swaps_factors": ('dgt = dm * s["up"]', 'dgt = dm * s["gate"]'),
    "mid_residual_gradient_dropped": ("dx1 = dx2 + dx1_n", "dx1 = dx1_n"),
    "input_residual_gradient_dropped": ("dx0 = dx1 + dx0_n", "dx0 = dx0_n"),
    "recompute_norm_from_block_input": ('out["b"] = rmsnorm(saved["x1"], w["g2"], c.eps)',
                                        'out["b"] = rmsnorm(x0, w["g2"], c.eps)'),
    "recompute_q_from_k": ('_, out["q"] = oracle.cola_up_from_z(Z["q"], w["B_q"], act)',
                           '_, out["q"] = oracle.cola_up_from_z(Z["k"], w["B_q"], act)'),
    "cola_m_keeps_extra": ('saved = {"x1": x1, "Z": Z}\n', 'saved = {"x1": x1, "Z": Z, "a": a}\n'),
}


def battery():
    checks = [
        ("rms_torch", pins.test_rmsnorm_against_torch_and_autograd, ()),
        ("rms_const", pins.test_rmsnorm_constant_row_closed_form, ()),
        ("rms_fd", pins.test_rmsnorm_backward_by_central_differences, ()),
        ("rope_complex", pins.test_rope_complex_form_and_angles, ()),
        ("rope_props", pins.test_rope_inverse_norms_and_relative_position, ()),
        ("attn_torch", pins.test_attention_against_torch_sdpa_and_autograd, ((2, 7, 3, 4),)),
        ("attn_closed", pins.test_attention_causal_closed_forms, ()),
        ("block_torch", pins.test_block_against_torch_autograd, ("silu", False)),
        ("block_torch_m", pins.test_block_against_torch_autograd, ("silu", True)),
        ("cola_m_eq", pins.test_block_cola_m_equals_cola, ()),
        ("saved", pins.test_cola_m_saved_memory_is_2nd_plus_7nr, ()),
    ]
    failed = []
    for name, fn, args in checks:
        try:
            fn(*args)
        except (AssertionError, FloatingPointError, ValueError):
            failed.append(name)
    return failed


def _with_block(module):
    """Run the battery with pins.OB pointing at `module`."""
    old = pins.OB
    pins.OB = module
    try:
        return battery()
    finally:
        pins.OB = old


def test_real_block_oracle_passes_battery():
    assert _with_block(real_block) == []


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_block_mutant_is_caught(mutant, tmp_path):
    old, new = MUTANTS[mutant]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation site not found exactly once"
    path = tmp_path / "block_mutant.py"
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location(f"block_mutant_{mutant}", str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    assert _with_block(mod), f"mutant {mutant} passed every pin"
