"""A seeded sweep of layer shapes around the kernels' decision points.

Each of T, d_in, d_out and r is drawn from one of three bands -- below one
32-wide MFMA tile, around the 128 / 256 tile edges (where the launcher
switches between the streaming and the 256 x 256 families and where the
ragged-edge paths start), and several tiles wide -- together with the storage
dtype, the activation, CoLA or CoLA-M, and tight or cache-line row pitches
(tight pitches with odd widths take the guarded, unaligned paths).  Every
draw runs forward and backward through the C ABI and is compared with the
fp64 oracle (1e-2 bf16, 1e-5 fp32); bf16 draws are also held to the
reference that applies the path's bf16 storage policy (1e-3, Z and H equal
bit for bit except for the rare element next to a rounding boundary).  Pad
columns must keep their NaN fill.  The draws are fixed by the seed, so a
failure names a reproducible shape."""
import numpy as np
import pytest
import torch

import oracle
from paper_2502_10940_amd import cola
from paper_2502_10940_amd import inputs as I

from layer_runner import LayerRun, relerr
from test_gpu_rounding import TOL as ROUNDED_TOL, rounded_layer

SEED = 25021094
N_DRAWS = 96
# oracle cost bound: T r (d_in + d_out) multiply-adds per GEMM pass
MAX_WORK = 3.0e8
TOL = {"f32": 1e-5, "bf16": 1e-2}
EDGES = (32, 64, 127, 128, 129, 255, 256, 257)


def _dim(rng, lo_band, hi_band):
    band = int(rng.integers(0, 3))
    if band == 0:
        return int(rng.integers(1, 41))
    if band == 1:
        return max(1, int(EDGES[int(rng.integers(0, len(EDGES)))] + rng.integers(-1, 2)))
    return int(rng.integers(lo_band, hi_band + 1))


def draws(seed=SEED, n=N_DRAWS):
    """The sweep's cases: (T, d_in, d_out, r, dtype, act, recompute, padded)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out = []
    while len(out) < n:
        T = _dim(rng, 300, 3000)
        d_in = _dim(rng, 300, 1500)
        d_out = _dim(rng, 300, 1500)
        r = _dim(rng, 260, 520)
        if T * r * (d_in + d_out) > MAX_WORK:
            continue
        dtype = "f32" if rng.random() < 0.2 else "bf16"
        act = ("silu", "gelu", "identity")[int(rng.choice(3, p=[0.6, 0.25, 0.15]))]
        out.append((T, d_in, d_out, r, dtype, act, bool(rng.random() < 0.5), bool(rng.random() < 0.5)))
    return out


CASES = draws()


def _id(c):
    T, d_in, d_out, r, dtype, act, rec, padded = c
    return f"T{T}-{d_in}x{d_out}-r{r}-{dtype}-{act}-{'colam' if rec else 'cola'}-{'pad' if padded else 'tight'}"


def test_draws_cover_the_bands():
    """The sweep is what it claims (no GPU): deterministic, within the oracle
    budget, and reaching both sides of the family switch (an output
    dimension of at most 128 against both above 128), ragged and exact tile
    edges, both dtypes, every activation, both modes and both pitch kinds."""
    assert draws() == CASES
    assert all(T * r * (di + do) <= MAX_WORK for T, di, do, r, *_ in CASES)
    dims = [d for T, di, do, r, *_ in CASES for d in (T, di, do, r)]
    assert min(dims) >= 1
    assert any(d <= 40 for d in dims) and any(d > 300 for d in dims)
    assert any(d % 256 == 0 for d in dims) and any(d % 128 == 0 and d % 256 for d in dims)
    assert any(d % 32 for d in dims)
    # K1 / K3 outputs are T x r, K2 / K4 outputs T x d_out / T x d_in
    assert any(c[3] <= 128 for c in CASES)
    assert any(T > 128 and r > 128 for T, _, _, r, *_ in CASES)
    assert any(T > 128 and do > 128 for T, _, do, *_ in CASES)
    assert {c[4] for c in CASES} == {"bf16", "f32"}
    assert {c[5] for c in CASES} == {"silu", "gelu", "identity"}
    assert {c[6] for c in CASES} == {False, True}
    assert {c[7] for c in CASES} == {False, True}


@pytest.fixture(scope="module")
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cola.lib()
    yield


@pytest.mark.gpu
@pytest.mark.parametrize("case", range(len(CASES)), ids=[_id(c) for c in CASES])
def test_shape_sweep(case, _device):
    T, d_in, d_out, r, dtype, act, recompute, padded = CASES[case]
    print(f"\n[sweep] case {case}: {_id(CASES[case])}", flush=True)
    ins = I.layer_inputs(500 + case, 0, d_in, d_out, r, T, dtype)
    pitch = (lambda w: I.padded_ld(w, dtype)) if padded else (lambda w: w)
    run = LayerRun(ins, T, d_in, d_out, r, dtype, act, recompute,
                   ldx=pitch(d_in), ldy=pitch(d_out), ldz=pitch(r)).run()
    got = run.outputs()
    assert run.padding_untouched()

    X, A, B, dY = (ins[k].f64 for k in ("X", "A", "B", "dY"))
    Z, H, Y = oracle.cola_fwd(X, A, B, act)
    _, dX, dA, dB = oracle.cola_bwd(X, Z, A, B, dY, act)
    ref = {"Z": Z, "H": H, "Y": Y, "dX": dX, "dA": dA, "dB": dB}
    for k, g in got.items():
        assert np.all(np.isfinite(g)), f"{k}: non-finite values"
        e = relerr(g, ref[k])
        assert e <= TOL[dtype], f"{k}: {e:.3e} against the oracle"

    if dtype == "bf16":
        rr = rounded_layer(X, A, B, dY, act)
        for k, g in got.items():
            e = relerr(g, rr[k])
            assert e <= ROUNDED_TOL, f"{k}: {e:.3e} against the storage-policy reference"
            if k in ("Z", "H"):
                differ = int(np.sum(g != rr[k]))
                assert differ <= 2 + 0.001 * g.size, f"{k}: {differ} of {g.size} elements differ"
