"""Concurrent use of the layer API on two HIP streams, the way the benchmark's
step runs the seven projections: each stream has one workspace that its
layers share, and the two streams' forwards and backwards overlap.  Every
output must be bitwise the one the same layer gives alone on the default
stream (the kernels and their summation orders do not depend on what else
runs), so nothing in the library is shared between calls beyond what the
caller passes in."""
import numpy as np
import pytest
import torch

from paper_2502_10940_amd import cola
from paper_2502_10940_amd import inputs as I

from layer_runner import DEV, LayerRun

pytestmark = pytest.mark.gpu

# (T, d_in, d_out, r, recompute): the two families, split weight gradients,
# the persistent walk, CoLA and CoLA-M
LAYERS = [(1000, 768, 1376, 192, False), (700, 1376, 512, 128, True), (600, 520, 264, 136, False),
          (6044, 300, 3000, 128, True), (2048, 2048, 2048, 512, False), (300, 64, 96, 16, True)]


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cola.lib()
    yield


def make_runs():
    runs = []
    for i, (T, d_in, d_out, r, rec) in enumerate(LAYERS):
        ins = I.layer_inputs(800 + i, 0, d_in, d_out, r, T, "bf16")
        runs.append(LayerRun(ins, T, d_in, d_out, r, "bf16", "silu", rec,
                             ldx=I.padded_ld(d_in, "bf16"), ldy=I.padded_ld(d_out, "bf16"),
                             ldz=I.padded_ld(r, "bf16")))
    return runs


def test_two_streams_bitwise_equal_serial():
    serial = make_runs()
    for run in serial:
        run.run()
    expect = [run.raw() for run in serial]

    runs = make_runs()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]          # default priority
    owner = [i % 2 for i in range(len(runs))]
    # one workspace per stream, shared by its layers
    for s in range(2):
        need = max(run.ws.numel() for run, o in zip(runs, owner) if o == s)
        ws = torch.empty(need, dtype=torch.uint8, device=DEV)
        for run, o in zip(runs, owner):
            if o == s:
                run.ws = ws
    torch.cuda.synchronize()
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for _ in range(2):                                             # twice: the second pass reuses everything
        for run, o in zip(runs, owner):
            with torch.cuda.stream(streams[o]):
                run.forward()
        for run, o in reversed(list(zip(runs, owner))):
            with torch.cuda.stream(streams[o]):
                run.backward()
    torch.cuda.synchronize()
    for i, (run, exp) in enumerate(zip(runs, expect)):
        got = run.raw()
        assert run.padding_untouched(), f"layer {i}: pad columns written"
        for k in exp:
            assert np.array_equal(got[k], exp[k]), f"layer {i} {LAYERS[i]}: {k} differs from the serial run"


@pytest.mark.parametrize("fill", [0x00, 0xFF], ids=["zeros", "ones"])
def test_workspace_contents_do_not_matter(fill):
    """The workspace is scratch: whatever it holds before a call (zeros, or
    all bits set, which reads as NaN in bf16 and fp32) the outputs are
    bitwise those of a fresh run, so no kernel reads workspace it has not
    written (split partials, packed weights, CoLA-M's H)."""
    reference = make_runs()
    for run in reference:
        run.run()
    runs = make_runs()
    for run in runs:
        run.ws.fill_(fill)
    torch.cuda.synchronize()
    for i, (run, ref) in enumerate(zip(runs, reference)):
        run.run()
        got, exp = run.raw(), ref.raw()
        for k in exp:
            assert np.array_equal(got[k], exp[k]), f"layer {i} {LAYERS[i]}: {k} depends on the workspace contents"


@pytest.mark.parametrize("recompute", [False, True], ids=["cola", "colam"])
def test_block_workspace_and_saved_contents_do_not_matter(recompute):
    """The decoder block's workspace and saved buffer start with all bits
    set: the forward writes every saved tensor it keeps and the backward
    reads nothing of the workspace it has not written."""
    from block_runner import BlockRun
    shape = (2, 100, 256, 270, 4, 64)
    ins = I.block_inputs(33, shape[0], shape[1], shape[2], shape[3], shape[5])
    ref = BlockRun(ins, *shape, "silu", recompute).run().raw()
    run = BlockRun(ins, *shape, "silu", recompute)
    run.ws.fill_(0xFF)
    run.saved.fill_(0xFF)
    torch.cuda.synchronize()
    got = run.run().raw()
    for k in ref:
        assert np.array_equal(got[k], ref[k]), f"{k} depends on the workspace or saved contents"
