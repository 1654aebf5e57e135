"""cola_bwd_scratch, the backward whose workspace is the library's static
device scratch (for callers that cannot allocate): through the C ABI, its
outputs equal cola_bwd's on the same inputs (same kernels, same split plan:
bitwise) and match the oracle within the bf16 / fp32 tolerance, on two calls
in a row, the second with a smaller input (the scratch keeps the first call's
contents, which the second must not depend on); a call needing more than the
scratch holds is refused before anything is enqueued; and, for the callers it
is for, a forward and the scratch backward captured in a HIP graph replay
bitwise the eager result."""
import numpy as np
import pytest
import torch

import oracle
from paper_2502_10940_amd import cola
from paper_2502_10940_amd import inputs as I

from layer_runner import DEV, LayerRun, relerr, to_f64

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 1e-2}


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cola.lib()
    yield


def scratch_backward(run):
    """Backward of a LayerRun (its forward done) through cola_bwd_scratch into
    fresh NaN-filled gradient buffers."""
    dX = torch.full_like(run.dX, float("nan"))
    dA = torch.full_like(run.dA, float("nan"))
    dB = torch.full_like(run.dB, float("nan"))
    cola.bwd_scratch(run.desc, run.dY, run.X, run.Z, run.H, run.A, run.B, dX, dA, dB)
    torch.cuda.synchronize()
    return {"dX": to_f64(dX, run.d_in), "dA": to_f64(dA), "dB": to_f64(dB)}


# (T, d_in, d_out, r, dtype, recompute): each pair runs large then small
PAIRS = [
    ((3000, 1024, 1376, 256, "bf16", False), (700, 520, 264, 136, "bf16", False)),
    ((2048, 768, 768, 192, "bf16", True), (300, 264, 200, 40, "bf16", True)),
    ((1024, 512, 384, 128, "f32", False), (77, 130, 65, 33, "f32", False)),
]


@pytest.mark.parametrize("pair", PAIRS, ids=["bf16_cola", "bf16_colam", "f32_cola"])
def test_scratch_backward_matches_cola_bwd_twice(pair):
    for k, (T, d_in, d_out, r, dtype, rc) in enumerate(pair):
        print(f"\n[scratch] call {k}: T={T} {d_in}->{d_out} r={r} {dtype} recompute={rc}", flush=True)
        ins = I.layer_inputs(300 + k, 0, d_in, d_out, r, T, dtype)
        run = LayerRun(ins, T, d_in, d_out, r, dtype, "silu", rc)
        assert cola.workspace_bytes(run.desc, 1) <= cola.SCRATCH_BYTES
        run.run()
        got = scratch_backward(run)
        ref_gpu = run.outputs()
        for name in ("dX", "dA", "dB"):
            assert np.array_equal(got[name], ref_gpu[name]), name
        X, A, B, dY = ins["X"].f64, ins["A"].f64, ins["B"].f64, ins["dY"].f64
        Z, _, _ = oracle.cola_fwd(X, A, B, "silu")
        _, dXr, dAr, dBr = oracle.cola_bwd(X, Z, A, B, dY, "silu")
        for name, ref in (("dX", dXr), ("dA", dAr), ("dB", dBr)):
            assert relerr(got[name], ref) <= TOL[dtype], name


def test_scratch_backward_refuses_oversized_call():
    # 1B attention shape: the backward's workspace is far above the scratch size
    d = cola.desc(32768, 2048, 2048, 512)
    assert cola.workspace_bytes(d, 1) > cola.SCRATCH_BYTES
    fake = 0x1000        # never dereferenced: the call is refused before any launch
    dA = torch.full((512, 2048), float("nan"), device=DEV)
    dB = torch.full((2048, 512), float("nan"), device=DEV)
    with pytest.raises(cola.ColaError) as e:
        cola.bwd_scratch(d, fake, fake, fake, fake, fake, fake, fake, dA, dB)
    assert e.value.status == cola.ERR_SCRATCH
    torch.cuda.synchronize()
    assert torch.isnan(dA).all() and torch.isnan(dB).all()


def test_scratch_backward_empty_batch():
    d = cola.desc(0, 32, 24, 8)
    dA = torch.full((8, 32), float("nan"), device=DEV)
    dB = torch.full((24, 8), float("nan"), device=DEV)
    cola.bwd_scratch(d, None, None, None, None, None, None, None, dA, dB)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dA).item() == 0 and torch.count_nonzero(dB).item() == 0


def _bits(t, width):
    v = t[:, :width] if t.dim() == 2 and width is not None else t
    return v.contiguous().view(torch.int16 if v.dtype == torch.bfloat16 else torch.int32).clone()


def test_scratch_backward_replays_in_a_hip_graph():
    """A forward and the scratch backward captured in a HIP graph
    (torch.cuda.CUDAGraph) and replayed three times, with eager work between
    the replays (another layer's forward and scratch backward, which rewrite
    the shared scratch) and synchronisations; every replay bitwise the eager
    result."""
    T, d_in, d_out, r = 1500, 512, 768, 128
    run = LayerRun(I.layer_inputs(310, 0, d_in, d_out, r, T, "bf16"), T, d_in, d_out, r, "bf16", "silu", False)
    other = LayerRun(I.layer_inputs(311, 0, 384, 640, 96, 900, "bf16"), 900, 384, 640, 96, "bf16", "silu", False)
    dX = torch.full_like(run.dX, float("nan"))
    dA = torch.full_like(run.dA, float("nan"))
    dB = torch.full_like(run.dB, float("nan"))

    def step():
        run.forward()
        cola.bwd_scratch(run.desc, run.dY, run.X, run.Z, run.H, run.A, run.B, dX, dA, dB)

    step()
    torch.cuda.synchronize()
    outs = (("Y", run.Y, d_out), ("Z", run.Z, r), ("H", run.H, r), ("dX", dX, d_in), ("dA", dA, None),
            ("dB", dB, None))
    ref = {name: _bits(t, w) for name, t, w in outs}
    graph = torch.cuda.CUDAGraph()
    cs = torch.cuda.Stream()
    cs.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cs):
        with torch.cuda.graph(graph, stream=cs):
            step()
    torch.cuda.synchronize()
    for rep in range(3):
        print(f"\n[graph] replay {rep}", flush=True)
        for _, t, _ in outs:
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, t, w in outs:
            assert torch.equal(_bits(t, w), ref[name]), f"replay {rep}: {name}"
        other.forward()
        scratch_backward(other)
    del graph
