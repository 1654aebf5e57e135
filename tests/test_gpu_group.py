"""GPU parity of the grouped projections (several CoLA layers reading the same
input X: q, k, v of attention, gate and up of the MLP) called through the C
ABI, against the fp64 oracle run projection by projection: Z_all, H_all, Y_p,
dA_all, dB_p element by element, and dX against the sum of the projections'
input gradients.  Plus: the grouped forward and the per-projection outputs
of the backward are bitwise those of the single-layer calls, CoLA-M equals
CoLA bitwise, and the empty batch.

Tolerance (relative Frobenius error per tensor): 1e-5 for fp32 storage,
1e-2 for bf16 storage with fp32 accumulation."""
import numpy as np
import pytest
import torch

import oracle
from paper_2502_10940_amd import cola
from paper_2502_10940_amd import inputs as I

from layer_runner import DEV, NAN_BITS, TORCH_DT, empty, relerr, to_device, to_f64

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 1e-2}

# (name, T, d_in, ranks, output widths, dtype, act)
CASES = [
    ("qkv_bf16", 700, 520, [136, 136, 136], [264, 264, 264], "bf16", "silu"),
    ("gate_up_bf16", 513, 256, [64, 64], [688, 688], "bf16", "silu"),
    # weight gradients dA_all with dB_gate in one launch, dB_up alone
    ("gate_up_wide_bf16", 600, 264, [136, 136], [300, 300], "bf16", "silu"),
    ("ragged_odd_bf16", 333, 301, [37, 64, 9], [100, 1, 77], "bf16", "gelu"),
    ("single_f32", 130, 70, [20], [90], "f32", "silu"),
    ("pair_f32", 77, 130, [33, 8], [65, 40], "f32", "gelu"),
]


def group_inputs(case_id, T, d_in, ranks, widths, dtype):
    """Shared X (projection 0's), and A_p, B_p, dY_p of each projection."""
    projs = [I.layer_inputs(300 + case_id, p, d_in, widths[p], ranks[p], T, dtype) for p in range(len(ranks))]
    return projs[0]["X"], [q["A"] for q in projs], [q["B"] for q in projs], [q["dY"] for q in projs]


def oracle_group(X, As, Bs, dYs, act):
    out = {"Z": [], "H": [], "Y": [], "dA": [], "dB": [], "dX": 0.0}
    for A, B, dY in zip(As, Bs, dYs):
        Z, H, Y = oracle.cola_fwd(X.f64, A.f64, B.f64, act)
        _, dX, dA, dB = oracle.cola_bwd(X.f64, Z, A.f64, B.f64, dY.f64, act)
        out["Z"].append(Z)
        out["H"].append(H)
        out["Y"].append(Y)
        out["dA"].append(dA)
        out["dB"].append(dB)
        out["dX"] = out["dX"] + dX
    return out


class GroupRun:
    def __init__(self, X, As, Bs, dYs, T, d_in, ranks, widths, dtype, act, recompute, ldz=None):
        self.T, self.d_in, self.ranks, self.widths, self.dtype = T, d_in, ranks, widths, dtype
        self.R = sum(ranks)
        self.off = np.cumsum([0] + ranks[:-1]).tolist()
        self.ldz = ldz or self.R
        self.desc = cola.group_desc(T, d_in, ranks, widths, dtype, act, recompute, ldz=self.ldz)
        nanb = NAN_BITS[dtype]
        self.X = to_device(X.store, dtype)
        self.A_all = to_device(np.concatenate([A.store for A in As], axis=0), dtype)
        self.B = [to_device(B.store, dtype) for B in Bs]
        self.dY = [to_device(dY.store, dtype) for dY in dYs]
        self.Y = [empty(T, w, dtype, nanb) for w in widths]
        self.Z = empty(T, self.ldz, dtype, nanb)
        self.H = None if recompute else empty(T, self.ldz, dtype, nanb)
        self.dX = empty(T, d_in, dtype, nanb)
        self.dA = torch.full((self.R, d_in), float("nan"), dtype=torch.float32, device=DEV)
        self.dB = [torch.full((w, r), float("nan"), dtype=torch.float32, device=DEV) for r, w in zip(ranks, widths)]
        n = max(cola.group_workspace_bytes(self.desc, 0), cola.group_workspace_bytes(self.desc, 1), 1)
        self.ws = torch.empty(n, dtype=torch.uint8, device=DEV)

    def run(self):
        cola.group_fwd(self.desc, self.X, self.A_all, self.B, self.Y, self.Z, self.H, self.ws)
        cola.group_bwd(self.desc, self.dY, self.X, self.Z, self.H, self.A_all, self.B, self.dX, self.dA,
                       self.dB, self.ws)
        torch.cuda.synchronize()
        return self

    def results(self):
        Z = to_f64(self.Z)
        out = {"Z": [Z[:, o:o + r] for o, r in zip(self.off, self.ranks)],
               "Y": [to_f64(y) for y in self.Y],
               "dX": to_f64(self.dX),
               "dA": [to_f64(self.dA)[o:o + r] for o, r in zip(self.off, self.ranks)],
               "dB": [to_f64(b) for b in self.dB]}
        if self.H is not None:
            H = to_f64(self.H)
            out["H"] = [H[:, o:o + r] for o, r in zip(self.off, self.ranks)]
        return out


def check(got, ref, dtype, label):
    tol = TOL[dtype]
    for k, g in got.items():
        gl = g if isinstance(g, list) else [g]
        rl = ref[k] if isinstance(ref[k], list) else [ref[k]]
        for p, (gp, rp) in enumerate(zip(gl, rl)):
            assert np.all(np.isfinite(gp)), f"{label}: non-finite values in {k}[{p}]"
            e = relerr(gp, rp)
            assert e <= tol, f"{label}: {k}[{p}] relative Frobenius error {e:.3e} > {tol}"


@pytest.mark.parametrize("recompute", [False, True], ids=["cola", "cola_m"])
@pytest.mark.parametrize("case", range(len(CASES)), ids=[c[0] for c in CASES])
def test_group_parity(case, recompute):
    name, T, d_in, ranks, widths, dtype, act = CASES[case]
    X, As, Bs, dYs = group_inputs(case, T, d_in, ranks, widths, dtype)
    ref = oracle_group(X, As, Bs, dYs, act)
    run = GroupRun(X, As, Bs, dYs, T, d_in, ranks, widths, dtype, act, recompute).run()
    got = run.results()
    if recompute:
        ref = {k: v for k, v in ref.items() if k != "H"}
    check(got, ref, dtype, f"{name}/{'cola_m' if recompute else 'cola'}")


def test_group_matches_single_layers_bitwise():
    """Grouped forward, dZ-dependent dB_p: bitwise the single-layer results
    (same kernels and tile sums); CoLA-M bitwise CoLA."""
    name, T, d_in, ranks, widths, dtype, act = CASES[0]
    X, As, Bs, dYs = group_inputs(0, T, d_in, ranks, widths, dtype)
    grp = GroupRun(X, As, Bs, dYs, T, d_in, ranks, widths, dtype, act, False).run()
    grp_m = GroupRun(X, As, Bs, dYs, T, d_in, ranks, widths, dtype, act, True).run()
    for p, (A, B, dY) in enumerate(zip(As, Bs, dYs)):
        r, w, o = ranks[p], widths[p], grp.off[p]
        d = cola.desc(T, d_in, w, r, dtype, act)
        Xd = grp.X
        Ad, Bd, dYd = to_device(A.store, dtype), to_device(B.store, dtype), to_device(dY.store, dtype)
        Y = torch.empty((T, w), dtype=TORCH_DT[dtype], device=DEV)
        Z = torch.empty((T, r), dtype=TORCH_DT[dtype], device=DEV)
        H = torch.empty((T, r), dtype=TORCH_DT[dtype], device=DEV)
        dX = torch.empty((T, d_in), dtype=TORCH_DT[dtype], device=DEV)
        dA = torch.empty((r, d_in), dtype=torch.float32, device=DEV)
        dB = torch.empty((w, r), dtype=torch.float32, device=DEV)
        ws = torch.empty(max(cola.workspace_bytes(d, 0), cola.workspace_bytes(d, 1), 1), dtype=torch.uint8,
                         device=DEV)
        cola.fwd(d, Xd, Ad, Bd, Y, Z, H, ws)
        cola.bwd(d, dYd, Xd, Z, H, Ad, Bd, dX, dA, dB, ws)
        torch.cuda.synchronize()
        assert torch.equal(grp.Z[:, o:o + r], Z)
        assert torch.equal(grp.H[:, o:o + r], H)
        assert torch.equal(grp.Y[p], Y)
        assert torch.equal(grp.dB[p], dB)
    for p in range(len(ranks)):
        assert torch.equal(grp.Y[p], grp_m.Y[p])
        assert torch.equal(grp.dB[p], grp_m.dB[p])
    assert torch.equal(grp.dX, grp_m.dX)
    assert torch.equal(grp.dA, grp_m.dA)


def test_group_empty_batch_zeroes_weight_gradients():
    ranks, widths = [8, 16], [32, 24]
    d = cola.group_desc(0, 32, ranks, widths, "bf16")
    dA = torch.full((24, 32), float("nan"), dtype=torch.float32, device=DEV)
    dB = [torch.full((w, r), float("nan"), dtype=torch.float32, device=DEV) for r, w in zip(ranks, widths)]
    cola.group_fwd(d, None, None, [None, None], [None, None], None, None)
    cola.group_bwd(d, [None, None], None, None, None, None, [None, None], None, dA, dB)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dA).item() == 0
    for b in dB:
        assert torch.count_nonzero(b).item() == 0


@pytest.mark.parametrize("case", range(len(CASES)), ids=[c[0] for c in CASES])
def test_group_infer(case):
    """Inference forward of the group: each Y_p against the oracle, and bitwise
    the Y_p of the training forward (the same kernels and sums; H is never
    written out, Z not at all)."""
    name, T, d_in, ranks, widths, dtype, act = CASES[case]
    X, As, Bs, dYs = group_inputs(case, T, d_in, ranks, widths, dtype)
    ref = oracle_group(X, As, Bs, dYs, act)
    run = GroupRun(X, As, Bs, dYs, T, d_in, ranks, widths, dtype, act, False)
    cola.group_fwd(run.desc, run.X, run.A_all, run.B, run.Y, run.Z, run.H, run.ws)
    nanb = NAN_BITS[dtype]
    Yi = [empty(T, w, dtype, nanb) for w in widths]
    ws = torch.empty(max(cola.group_workspace_bytes(run.desc, 2), 1), dtype=torch.uint8, device=DEV)
    cola.group_infer(run.desc, run.X, run.A_all, run.B, Yi, ws)
    torch.cuda.synchronize()
    check({"Y": [to_f64(y) for y in Yi]}, {"Y": ref["Y"]}, dtype, f"{name}/infer")
    for p in range(len(ranks)):
        assert torch.equal(Yi[p], run.Y[p]), f"{name}: inference Y[{p}] differs from the training forward"


@pytest.mark.parametrize("case", [0, 2, 4], ids=[CASES[c][0] for c in (0, 2, 4)])
def test_single_infer(case):
    """cola_infer on each projection alone: oracle parity and bitwise the Y of
    cola_fwd."""
    name, T, d_in, ranks, widths, dtype, act = CASES[case]
    X, As, Bs, dYs = group_inputs(case, T, d_in, ranks, widths, dtype)
    ref = oracle_group(X, As, Bs, dYs, act)
    Xd = to_device(X.store, dtype)
    for p, (A, B) in enumerate(zip(As, Bs)):
        r, w = ranks[p], widths[p]
        d = cola.desc(T, d_in, w, r, dtype, act)
        Ad, Bd = to_device(A.store, dtype), to_device(B.store, dtype)
        Y = torch.empty((T, w), dtype=TORCH_DT[dtype], device=DEV)
        Z = torch.empty((T, r), dtype=TORCH_DT[dtype], device=DEV)
        H = torch.empty((T, r), dtype=TORCH_DT[dtype], device=DEV)
        cola.fwd(d, Xd, Ad, Bd, Y, Z, H, torch.empty(max(cola.workspace_bytes(d, 0), 1), dtype=torch.uint8,
                                                     device=DEV))
        Yi = empty(T, w, dtype, NAN_BITS[dtype])
        cola.infer(d, Xd, Ad, Bd, Yi, torch.empty(cola.workspace_bytes(d, 2), dtype=torch.uint8, device=DEV))
        torch.cuda.synchronize()
        check({"Y": to_f64(Yi)}, {"Y": ref["Y"][p]}, dtype, f"{name}/infer[{p}]")
        assert torch.equal(Yi, Y)


def test_group_weight_gradients_unpaired_switch():
    """COLA_OPT_WGRAD_PAIR = 0 launches every weight-gradient product of a group
    on its own instead of two by two: both paths match the oracle, the fp32
    gradients agree to summation order and the rest bitwise."""
    cases = [0, 2]      # q, k, v (three products of dB and dA_all); gate, up (wide, 136-rank)
    for case in cases:
        name, T, d_in, ranks, widths, dtype, act = CASES[case]
        X, As, Bs, dYs = group_inputs(case, T, d_in, ranks, widths, dtype)
        ref = oracle_group(X, As, Bs, dYs, act)
        paired = GroupRun(X, As, Bs, dYs, T, d_in, ranks, widths, dtype, act, False).run().results()
        old = cola.get_option(cola.OPT_WGRAD_PAIR)
        cola.set_option(cola.OPT_WGRAD_PAIR, 0)
        try:
            unpaired = GroupRun(X, As, Bs, dYs, T, d_in, ranks, widths, dtype, act, False).run().results()
        finally:
            cola.set_option(cola.OPT_WGRAD_PAIR, old)
        check(paired, ref, dtype, f"{name}/paired")
        check(unpaired, ref, dtype, f"{name}/unpaired")
        for k in ("dA", "dB"):
            for p in range(len(ranks)):
                assert relerr(unpaired[k][p], paired[k][p]) <= 1e-5, f"{name}: {k}[{p}]"
        for k in ("Z", "H", "Y"):
            for p in range(len(ranks)):
                assert np.array_equal(unpaired[k][p], paired[k][p]), f"{name}: {k}[{p}]"
        assert np.array_equal(unpaired["dX"], paired["dX"]), f"{name}: dX"
