"""GPU parity: the HIP library (called through the C ABI) against the fp64
oracle on the same seeded inputs, element by element over whole tensors, at
sizes the oracle finishes in seconds -- several tiles, ragged tails, padded
and unaligned pitches, degenerate shapes -- plus the invariants the method
fixes (CoLA-M bitwise equal to CoLA, run-to-run determinism, dense baseline).

Tolerance (relative Frobenius error per tensor): 1e-5 for fp32 storage,
1e-2 for bf16 storage with fp32 accumulation."""
import numpy as np
import pytest
import torch

import oracle
from paper_2502_10940_amd import cola
from paper_2502_10940_amd import inputs as I

from layer_runner import DEV, LayerRun, relerr, to_device, to_f64

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 1e-2}

# (name, T, d_in, d_out, r, dtype, act)
CASES = [
    ("single_layer_f32_T256_512_r128", 256, 512, 512, 128, "f32", "silu"),
    ("tiles_ragged_bf16", 300, 520, 264, 136, "bf16", "silu"),
    ("mid_bf16_ffn1376", 1000, 768, 1376, 192, "bf16", "silu"),
    ("down_bf16_ragged_k", 700, 1376, 512, 128, "bf16", "silu"),
    ("identity_bf16", 260, 300, 200, 72, "bf16", "identity"),
    ("identity_f32", 130, 70, 90, 20, "f32", "identity"),
    ("ragged_f32", 77, 130, 65, 33, "f32", "silu"),
    ("long_tokens_bf16", 5000, 64, 96, 16, "bf16", "silu"),
    ("long_tokens_f32", 3000, 40, 24, 8, "f32", "silu"),
    ("tiny_bf16", 1, 1, 1, 1, "bf16", "silu"),
    ("tiny_f32", 1, 1, 1, 1, "f32", "silu"),
    ("odd_pitch_bf16", 17, 37, 29, 5, "bf16", "silu"),
    ("rank_ge_width_bf16", 40, 16, 24, 32, "bf16", "silu"),
    ("t255_bf16", 255, 264, 136, 8, "bf16", "silu"),
    ("odd_width_weight_repack_bf16", 300, 301, 263, 40, "bf16", "silu"),
    ("odd_rank_weight_repack_bf16", 200, 136, 144, 37, "bf16", "silu"),
    ("gelu_bf16", 600, 520, 264, 136, "bf16", "gelu"),
    ("gelu_f32", 256, 512, 512, 128, "f32", "gelu"),
    # more output tiles than CUs with whole K tiles: the persistent 256 x 256
    # kernel, ragged in M and N, its tiles swept in column bands of 8 + 4
    # (24 x 12 tiles of Y = H B^T here, of dX = dZ A in the next case)
    ("persistent_banded_wide_out_bf16", 6044, 300, 3000, 128, "bf16", "silu"),
    ("persistent_banded_wide_in_bf16", 6044, 3000, 300, 128, "bf16", "silu"),
    # 256 x 256 family with unaligned output rows: dX [T][301] and Y [T][263]
    # (bf16, rows not a whole number of 16-byte chunks), dA [136][301] (fp32,
    # rows not a whole number of 4 floats): the guarded stores of the
    # transposed epilogue
    ("odd_width_rank136_bf16", 600, 301, 263, 136, "bf16", "silu"),
    # odd rank above 128: Z, H [T][137] written by the sigma epilogue and Z
    # read by the dZ epilogue through the guarded paths
    ("odd_rank137_bf16", 500, 264, 300, 137, "bf16", "silu"),
]


def gen(case_id, T, d_in, d_out, r, dtype, with_dense=False):
    return I.layer_inputs(100 + case_id, 0, d_in, d_out, r, T, dtype, with_dense=with_dense)


def oracle_all(ins, act):
    X, A, B, dY = (ins[k].f64 for k in ("X", "A", "B", "dY"))
    Z, H, Y = oracle.cola_fwd(X, A, B, act)
    dZ, dX, dA, dB = oracle.cola_bwd(X, Z, A, B, dY, act)
    return {"Z": Z, "H": H, "Y": Y, "dX": dX, "dA": dA, "dB": dB}


def check(got, ref, dtype, label):
    tol = TOL[dtype]
    for k, g in got.items():
        assert np.all(np.isfinite(g)), f"{label}: non-finite values in {k}"
        e = relerr(g, ref[k])
        assert e <= tol, f"{label}: {k} relative Frobenius error {e:.3e} > {tol}"


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cola.lib()
    yield


@pytest.mark.parametrize("recompute", [False, True], ids=["cola", "cola_m"])
@pytest.mark.parametrize("case", range(len(CASES)), ids=[c[0] for c in CASES])
def test_parity_small(case, recompute):
    name, T, d_in, d_out, r, dtype, act = CASES[case]
    print(f"\n[parity] {name} recompute={recompute}", flush=True)
    ins = gen(case, T, d_in, d_out, r, dtype)
    ref = oracle_all(ins, act)
    run = LayerRun(ins, T, d_in, d_out, r, dtype, act, recompute).run()
    check(run.outputs(), ref, dtype, name)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("recompute", [False, True], ids=["cola", "cola_m"])
def test_padded_pitches_untouched(dtype, recompute):
    T, d_in, d_out, r = 200, 130, 270, 40
    ins = gen(50, T, d_in, d_out, r, dtype)
    ref = oracle_all(ins, "silu")
    run = LayerRun(ins, T, d_in, d_out, r, dtype, "silu", recompute,
                   ldx=136, ldy=280, ldz=48).run()
    check(run.outputs(), ref, dtype, "padded")
    assert run.padding_untouched()


def test_unaligned_base_pointers():
    """Row pitches and base pointers off the 16-byte grid take the per-element path."""
    T, d_in, d_out, r = 65, 72, 48, 16
    dtype = "bf16"
    ins = gen(51, T, d_in, d_out, r, dtype)
    ref = oracle_all(ins, "silu")
    run = LayerRun(ins, T, d_in, d_out, r, dtype, "silu", False)
    # shift X by one element inside a larger allocation
    big = torch.zeros(T * d_in + 1, dtype=torch.bfloat16, device=DEV)
    big[1:] = run.X.reshape(-1)
    X_view = big[1:].view(T, d_in)
    assert X_view.data_ptr() % 16 != 0
    cola.fwd(run.desc, X_view, run.A, run.B, run.Y, run.Z, run.H, run.ws)
    cola.bwd(run.desc, run.dY, X_view, run.Z, run.H, run.A, run.B, run.dX, run.dA, run.dB, run.ws)
    torch.cuda.synchronize()
    check(run.outputs(), ref, dtype, "unaligned")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_cola_m_bitwise_equals_cola(dtype):
    T, d_in, d_out, r = 600, 264, 392, 72
    ins = gen(52, T, d_in, d_out, r, dtype)
    a = LayerRun(ins, T, d_in, d_out, r, dtype, "silu", False).run().raw()
    b = LayerRun(ins, T, d_in, d_out, r, dtype, "silu", True).run().raw()
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_run_to_run_bitwise_determinism():
    T, d_in, d_out, r = 4096, 256, 384, 64
    ins = gen(53, T, d_in, d_out, r, "bf16")
    run = LayerRun(ins, T, d_in, d_out, r, "bf16", "silu", False)
    first = run.run().raw()
    for _ in range(2):
        again = run.run().raw()
        for k in first:
            assert np.array_equal(first[k], again[k]), k


@pytest.mark.parametrize("recompute", [False, True], ids=["cola", "cola_m"])
def test_empty_batch(recompute):
    d = cola.desc(0, 32, 24, 8, "bf16", "silu", recompute)
    dA = torch.full((8, 32), float("nan"), device=DEV)
    dB = torch.full((24, 8), float("nan"), device=DEV)
    cola.fwd(d, None, None, None, None, None, None, None)
    cola.bwd(d, None, None, None, None, None, None, None, dA, dB, None)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dA).item() == 0 and torch.count_nonzero(dB).item() == 0


@pytest.mark.parametrize("dtype,d_in", [("bf16", 300), ("f32", 300), ("bf16", 301)])
def test_dense_parity(dtype, d_in):
    T, d_out = 520, 264
    ins = gen(54, T, d_in, d_out, 8, dtype, with_dense=True)
    X, W, dY = ins["X"].f64, ins["W"].f64, ins["dY"].f64
    Yr = oracle.dense_fwd(X, W)
    dXr, dWr = oracle.dense_bwd(X, W, dY)
    d = cola.dense_desc(T, d_in, d_out, dtype)
    Xd = to_device(ins["X"].store, dtype)
    Wd = to_device(ins["W"].store, dtype)
    dYd = to_device(ins["dY"].store, dtype)
    Y = torch.empty((T, d_out), dtype=Xd.dtype, device=DEV)
    dX = torch.empty((T, d_in), dtype=Xd.dtype, device=DEV)
    dW = torch.empty((d_out, d_in), dtype=torch.float32, device=DEV)
    ws = torch.empty(max(1, cola.dense_workspace_bytes(d, 0), cola.dense_workspace_bytes(d, 1)),
                     dtype=torch.uint8, device=DEV)
    cola.dense_fwd(d, Xd, Wd, Y, ws)
    cola.dense_bwd(d, dYd, Xd, Wd, dX, dW, ws)
    torch.cuda.synchronize()
    for got, ref, k in ((to_f64(Y), Yr, "Y"), (to_f64(dX), dXr, "dX"), (to_f64(dW), dWr, "dW")):
        assert relerr(got, ref) <= TOL[dtype], k


def test_identity_cola_equals_dense_with_merged_weight():
    """sigma = identity: CoLA computes X (B A)^T, the dense layer with W = B A (Sec. 3.3)."""
    T, d_in, d_out, r = 384, 200, 168, 24
    dtype = "f32"
    ins = gen(55, T, d_in, d_out, r, dtype)
    run = LayerRun(ins, T, d_in, d_out, r, dtype, "identity", False)
    run.forward()
    W = (run.B.double() @ run.A.double()).float().contiguous()
    d = cola.dense_desc(T, d_in, d_out, dtype)
    Yd = torch.empty((T, d_out), dtype=torch.float32, device=DEV)
    cola.dense_fwd(d, run.X, W, Yd)
    torch.cuda.synchronize()
    assert relerr(to_f64(run.Y), to_f64(Yd)) <= 1e-5


class _option:
    """Set a library tuning option for the duration of a with-block."""

    def __init__(self, option, value):
        self.option, self.value = option, value

    def __enter__(self):
        self.old = cola.get_option(self.option)
        cola.set_option(self.option, self.value)

    def __exit__(self, *exc):
        cola.set_option(self.option, self.old)


def test_weight_gradients_unpaired_switch():
    """COLA_OPT_WGRAD_PAIR = 0 launches dA and dB one by one instead of in one
    launch: both paths match the oracle and each other."""
    T, d_in, d_out, r = 1000, 768, 1376, 192
    ins = I.layer_inputs(160, 0, d_in, d_out, r, T, "bf16")
    ref = oracle_all(ins, "silu")
    paired = LayerRun(ins, T, d_in, d_out, r, "bf16", "silu", False).run().outputs()
    check(paired, ref, "bf16", "paired")
    with _option(cola.OPT_WGRAD_PAIR, 0):
        unpaired = LayerRun(ins, T, d_in, d_out, r, "bf16", "silu", False).run().outputs()
    check(unpaired, ref, "bf16", "unpaired")
    for k in ("dA", "dB"):
        assert relerr(unpaired[k], paired[k]) <= 1e-5, k
    for k in ("Z", "H", "Y", "dX"):
        assert np.array_equal(unpaired[k], paired[k]), k


def test_streaming_family_forced():
    """COLA_OPT_STREAM_ONLY = 1 sends every bf16 product to the streaming
    family (BM x 128 tiles): against the oracle on ragged tiles, unaligned
    output rows and an odd rank above 128, CoLA and CoLA-M."""
    names = ("tiles_ragged_bf16", "odd_width_rank136_bf16", "odd_rank137_bf16")
    cases = [i for i, c in enumerate(CASES) if c[0] in names]
    assert len(cases) == len(names)
    with _option(cola.OPT_STREAM_ONLY, 1):
        for case in cases:
            name, T, d_in, d_out, r, dtype, act = CASES[case]
            ins = gen(case, T, d_in, d_out, r, dtype)
            ref = oracle_all(ins, act)
            for rc in (False, True):
                got = LayerRun(ins, T, d_in, d_out, r, dtype, act, rc).run().outputs()
                check(got, ref, dtype, f"stream/{name}/recompute={rc}")


@pytest.mark.parametrize("recompute", [False, True])
def test_library_flop_counters_equal_oracle_macs(recompute):
    """The library's per-launch flop counters (2 M N K per GEMM) summed over one
    forward + backward equal twice the oracle's counted multiply-adds for the
    same shape (Sec. 3.4), in both modes, with the weight gradients split over
    tokens."""
    T, d_in, d_out, r = 2048, 520, 264, 136
    ins = gen(60, T, d_in, d_out, r, "bf16")
    run = LayerRun(ins, T, d_in, d_out, r, "bf16", "silu", recompute)
    cola.timing_reset()
    cola.timing_enable(True)
    try:
        run.run()
    finally:
        cola.timing_enable(False)
    total = sum(cola.timing_read(k)[2] for k in range(len(cola.KERNEL_CLASSES)))
    cola.timing_reset()
    X, A, B, dY = ins["X"].f64, ins["A"].f64, ins["B"].f64, ins["dY"].f64
    oracle.reset_macs()
    Z, _, _ = oracle.cola_fwd(X, A, B)
    oracle.cola_bwd(X, Z, A, B, dY)
    assert total == 2 * oracle.macs()
