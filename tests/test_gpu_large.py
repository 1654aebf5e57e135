"""GPU parity with activations larger than 4 GiB: a layer whose output Y and
incoming gradient dY are 65536 x 34816 bf16 (4.25 GiB each), so that rows past
the 2 GiB and 4 GiB marks are written by K2's epilogue and read by K3 (dY as
the k-contiguous operand) and K6 (dY as the m-contiguous operand of the
weight gradient).  Rank 192 keeps every product in the 256 x 256 family, and
K2 runs persistent (34816 output tiles).  Checked against the fp64 oracle:
sampled rows of Z, H, Y and dX (one token in every 256-row tile, so rows on
both sides of each mark), rows of dA and columns of dB for sampled rank
indices (sums over all 65536 tokens), and the same rows under the bf16
storage policy."""
import numpy as np
import pytest
import torch

import oracle
from paper_2502_10940_amd import cola
from paper_2502_10940_amd import inputs as I

from layer_runner import LayerRun, relerr
from test_gpu_fullsize import per_tile
from test_gpu_rounding import TOL as ROUNDED_TOL, rounded_layer

pytestmark = pytest.mark.gpu

T, D_IN, D_OUT, R = 65536, 256, 34816, 192
TOL = 1e-2


@pytest.fixture(scope="module")
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cola.lib()
    yield


@pytest.fixture(scope="module")
def data(_device):
    """Inputs and the oracle's expected values, computed once for both modes."""
    print(f"\n[large] T={T} {D_IN}->{D_OUT} r={R}: Y and dY {T * D_OUT * 2 / 2**30:.2f} GiB each", flush=True)
    assert T * D_OUT * 2 > 4 * 2**30
    ins = I.layer_inputs(900, 0, D_IN, D_OUT, R, T, "bf16")
    rows = per_tile(T, 901)
    assert rows.max() * D_OUT * 2 > 4 * 2**30        # rows past the 4 GiB mark are sampled
    X, A, B = ins["X"].f64, ins["A"].f64, ins["B"].f64
    dY_rows = I.bf16_bits_to_f64(ins["dY"].store[rows])
    ref = oracle.cola_rows(X[rows], A, B, dY_rows, np.arange(rows.size), "silu")
    rr = rounded_layer(X[rows], A, B, dY_rows, "silu")
    # weight gradients: sums over every token, so the whole of dY (18 GB in fp64)
    ranks = np.array([0, 1, 63, 64, 127, 128, 190, 191], dtype=np.int64)
    ref_dA, ref_dB = oracle.cola_wgrad_cols(X, A, B, ins["dY"].f64, ranks, "silu")
    print("[large] oracle done", flush=True)
    return ins, rows, ref, rr, ranks, ref_dA, ref_dB


@pytest.mark.parametrize("recompute", [False, True], ids=["cola", "colam"])
def test_activations_beyond_4gib(data, recompute):
    ins, rows, ref, rr, ranks, ref_dA, ref_dB = data
    print(f"\n[large] recompute={recompute}", flush=True)
    run = LayerRun(ins, T, D_IN, D_OUT, R, "bf16", "silu", recompute).run()
    for t, w in ((run.Y, D_OUT), (run.Z, R), (run.dX, D_IN), (run.dA, D_IN), (run.dB, R)):
        assert torch.isfinite(t[:, :w].float()).all()
    rows_t = torch.from_numpy(rows).to(run.X.device)

    def grab(t, width):
        return t.index_select(0, rows_t)[:, :width].float().cpu().numpy().astype(np.float64)

    got = {"Z": grab(run.Z, R), "Y": grab(run.Y, D_OUT), "dX": grab(run.dX, D_IN)}
    if run.H is not None:
        got["H"] = grab(run.H, R)
    for k, g in got.items():
        e = relerr(g, ref[k])
        assert e <= TOL, f"{k}: {e:.3e} against the oracle"
        e = relerr(g, rr[k])
        assert e <= ROUNDED_TOL, f"{k}: {e:.3e} against the storage-policy reference"
    ranks_t = torch.from_numpy(ranks).to(run.X.device)
    got_dA = run.dA.index_select(0, ranks_t).double().cpu().numpy()
    got_dB = run.dB.index_select(1, ranks_t).double().cpu().numpy().T
    assert relerr(got_dA, ref_dA) <= TOL
    assert relerr(got_dB, ref_dB) <= TOL
