"""GPU parity of the "both sigma" variant (App. ablation: the nonlinearity
that followed the original linear layer kept on top of the layer, Y =
sigma_out(B sigma(A x))) called through the C ABI, against the fp64 oracle:
P (the output before sigma_out), Y, Z, H, dX, dA, dB element by element; with
sigma_out = identity the variant is bitwise the plain layer.

Tolerance (relative Frobenius error per tensor): 1e-5 for fp32 storage,
1e-2 for bf16 storage with fp32 accumulation."""
import numpy as np
import pytest
import torch

import oracle
from paper_2502_10940_amd import cola
from paper_2502_10940_amd import inputs as I

from layer_runner import DEV, NAN_BITS, LayerRun, empty, relerr, to_f64

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 1e-2}

# (name, T, d_in, d_out, r, dtype, act, outer, ldy)
CASES = [
    ("gate_bf16", 600, 520, 700, 136, "bf16", "silu", "silu", None),
    ("gelu_odd_bf16", 333, 301, 77, 37, "bf16", "gelu", "gelu", 80),
    ("silu_f32", 130, 70, 90, 20, "f32", "silu", "silu", None),
    ("mixed_f32", 77, 64, 48, 16, "f32", "identity", "gelu", 53),
]


class OuterRun(LayerRun):
    def __init__(self, ins, T, d_in, d_out, r, dtype, act, outer, recompute, ldy=None):
        super().__init__(ins, T, d_in, d_out, r, dtype, act, recompute, ldy=ldy)
        self.outer = outer
        self.P = empty(T, self.ldy, dtype, NAN_BITS[dtype])
        n = max(cola.workspace_bytes(self.desc, 0), cola.workspace_bytes(self.desc, 3), 1)
        self.ws = torch.empty(n, dtype=torch.uint8, device=DEV)

    def forward(self):
        cola.fwd_outer(self.desc, self.outer, self.X, self.A, self.B, self.Y, self.P, self.Z, self.H, self.ws)

    def backward(self):
        cola.bwd_outer(self.desc, self.outer, self.dY, self.P, self.X, self.Z, self.H, self.A, self.B, self.dX,
                       self.dA, self.dB, self.ws)

    def outputs(self):
        out = super().outputs()
        out["P"] = to_f64(self.P, self.d_out)
        return out


def case_inputs(i):
    name, T, d_in, d_out, r, dtype, act, outer, ldy = CASES[i]
    return I.layer_inputs(400 + i, 0, d_in, d_out, r, T, dtype)


@pytest.mark.parametrize("recompute", [False, True], ids=["cola", "cola_m"])
@pytest.mark.parametrize("case", range(len(CASES)), ids=[c[0] for c in CASES])
def test_outer_parity(case, recompute):
    name, T, d_in, d_out, r, dtype, act, outer, ldy = CASES[case]
    ins = case_inputs(case)
    Z, H, P, Y = oracle.cola_fwd_outer(ins["X"].f64, ins["A"].f64, ins["B"].f64, act=act, outer=outer)
    _, _, dX, dA, dB = oracle.cola_bwd_outer(ins["X"].f64, Z, P, ins["A"].f64, ins["B"].f64, ins["dY"].f64,
                                            act=act, outer=outer)
    ref = {"Z": Z, "H": H, "P": P, "Y": Y, "dX": dX, "dA": dA, "dB": dB}
    run = OuterRun(ins, T, d_in, d_out, r, dtype, act, outer, recompute, ldy=ldy).run()
    got = run.outputs()
    assert run.padding_untouched()
    if ldy is not None:
        assert torch.isnan(run.P[:, d_out:].float()).all()
    for k, g in got.items():
        assert np.all(np.isfinite(g)), f"{name}: non-finite values in {k}"
        e = relerr(g, ref[k])
        assert e <= TOL[dtype], f"{name}: {k} relative Frobenius error {e:.3e} > {TOL[dtype]}"


@pytest.mark.parametrize("recompute", [False, True], ids=["cola", "cola_m"])
def test_outer_identity_is_plain_layer_bitwise(recompute):
    name, T, d_in, d_out, r, dtype, act, outer, ldy = CASES[0]
    ins = case_inputs(0)
    # dY and the workspace dP get the same 16-byte-multiple pitch, so both runs
    # load them the same way (the K order of a GEMM may depend on the operand
    # path, aligned or not; each is deterministic)
    ldy = (d_out + 7) // 8 * 8
    plain = LayerRun(ins, T, d_in, d_out, r, dtype, act, recompute, ldy=ldy).run()
    both = OuterRun(ins, T, d_in, d_out, r, dtype, act, "identity", recompute, ldy=ldy).run()
    raw_b, raw_p = both.raw(), plain.raw()
    for k in ("Y", "Z", "dX", "dA", "dB"):
        assert np.array_equal(raw_b[k], raw_p[k]), k
    assert torch.equal(both.P[:, :d_out].contiguous().view(torch.int16), plain.Y[:, :d_out].contiguous().view(torch.int16))


def test_outer_empty_batch_zeroes_weight_gradients():
    d = cola.desc(0, 32, 24, 8, "bf16")
    dA = torch.full((8, 32), float("nan"), dtype=torch.float32, device=DEV)
    dB = torch.full((24, 8), float("nan"), dtype=torch.float32, device=DEV)
    cola.fwd_outer(d, "silu", None, None, None, None, None, None, None)
    cola.bwd_outer(d, "silu", None, None, None, None, None, None, None, None, dA, dB)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dA).item() == 0 and torch.count_nonzero(dB).item() == 0
