"""GPU parity at the full workload sizes (LLaMA-60M/350M/1B/7B-shaped blocks),
in the launch configuration the benchmark times (row pitches padded to 16
bytes, bf16, SiLU): the oracle evaluates sampled outputs one by one -- whole
rows of Z, H, Y, dX for sampled tokens, and whole rows of dA / columns of dB
for sampled rank indices -- and the GPU must match them within the bf16
tolerance.  Unsampled outputs are checked for finiteness.  The 7B-shaped
block runs in CoLA-M mode as well as CoLA."""
import numpy as np
import pytest
import torch

import oracle
from paper_2502_10940_amd import cola
from paper_2502_10940_amd import inputs as I

from layer_runner import LayerRun, relerr

pytestmark = pytest.mark.gpu

TOL = 1e-2


def sample_rows(T):
    rows = {0, 1, 127, 128, 255, 256, T // 2, T // 2 + 1, T - 2, T - 1}
    rng = np.random.Generator(np.random.PCG64(T))
    rows |= set(int(x) for x in rng.integers(0, T, 6))
    return np.array(sorted(r for r in rows if 0 <= r < T), dtype=np.int64)


def sample_rank(r):
    return np.array(sorted({0, r // 2 + 1, r - 1}), dtype=np.int64)


# workload, projection index (0 = q: d->d, 4 = gate: d->ffn, 6 = down: ffn->d), modes
CASES = []
for cfg in (2, 3, 4, 5):
    for proj in (0, 4, 6):
        modes = (False, True) if cfg in (4, 5) else (False,)
        for m in modes:
            CASES.append((cfg, proj, m))


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cola.lib()
    yield


@pytest.mark.parametrize("cfg,proj,recompute", CASES,
                         ids=[f"w{c}-{I.PROJECTIONS[p]}-{'colam' if m else 'cola'}" for c, p, m in CASES])
def test_fullsize_sampled(cfg, proj, recompute):
    w = I.WORKLOADS[cfg]
    name, idx, d_in, d_out = I.projections(cfg)[proj]
    T, r = w["T"], w["r"]
    print(f"\n[fullsize] workload {cfg} {name} T={T} {d_in}->{d_out} r={r} recompute={recompute}",
          flush=True)
    ins = I.layer_inputs(cfg, idx, d_in, d_out, r, T, "bf16")
    run = LayerRun(ins, T, d_in, d_out, r, "bf16", "silu", recompute,
                   ldx=I.padded_ld(d_in, "bf16"), ldy=I.padded_ld(d_out, "bf16"),
                   ldz=I.padded_ld(r, "bf16")).run()

    rows = sample_rows(T)
    ranks = sample_rank(r)
    rows_t = torch.from_numpy(rows).to(run.X.device)

    def grab(t, width):
        return t.index_select(0, rows_t)[:, :width].float().cpu().numpy().astype(np.float64)

    got = {"Z": grab(run.Z, r), "Y": grab(run.Y, d_out), "dX": grab(run.dX, d_in)}
    if run.H is not None:
        got["H"] = grab(run.H, r)
    got_dA = run.dA.index_select(0, torch.from_numpy(ranks).to(run.X.device)).double().cpu().numpy()
    got_dB = run.dB.index_select(1, torch.from_numpy(ranks).to(run.X.device)).double().cpu().numpy().T

    # every output finite (within each row's logical width; the pad columns keep their NaN fill)
    for t, width in ((run.Y, d_out), (run.Z, r), (run.dX, d_in), (run.dA, d_in), (run.dB, r)):
        assert torch.isfinite(t[:, :width].float()).all()
    assert run.padding_untouched()

    X, A, B, dY = ins["X"].f64, ins["A"].f64, ins["B"].f64, ins["dY"].f64
    ref = oracle.cola_rows(X, A, B, dY, rows, "silu")
    for k, g in got.items():
        e = relerr(g, ref[k])
        assert e <= TOL, f"{k}: {e:.3e}"
    ref_dA, ref_dB = oracle.cola_wgrad_cols(X, A, B, dY, ranks, "silu")
    assert relerr(got_dA, ref_dA) <= TOL
    assert relerr(got_dB, ref_dB) <= TOL
