"""Seeded synthetic inputs and workload shapes for the CoLA layer.

This module serves both sides of every parity check (the GPU library's tests
and benchmark, and the fp64 oracle's tests).  It holds none of the layer's
arithmetic: only the workload shapes, seeded Gaussian draws, and rounding of
those draws to the storage format (fp32, or bf16 with round-to-nearest-even).

Workloads.  The paper's LLaMA shapes (rank/width pairs of Table "main results";
r = d/4 per App. D) with every linear projection of a decoder
block replaced by a CoLA layer (Sec. 3.2, Fig. "block"): q, k, v, o map
d -> d, gate and up map d -> ffn, down maps ffn -> d.  The paper prints no
FFN widths; 1376, 2736, 5461 and 11008 are the usual LLaMA widths for
d = 512, 1024, 2048 and 4096 (about 2.7 d, cf. d_ff ~ 2.5 d in App. C).

Distributions.  X ~ N(0, 1), A ~ N(0, 1/d_in), B ~ N(0, 1/r), upstream
gradient dY ~ N(0, 1), dense weight W ~ N(0, 1/d_in); the second argument is
a variance, so Z = X A^T is about N(0, 1) and SiLU works in its nonlinear
range.  Draws are float32 standard normals from numpy's PCG64; tensor seed =
1000*workload + 10*projection + tensor (tensor ids X=0, A=1, B=2, dY=3, W=4),
and each block of 4096 rows is seeded with SeedSequence([tensor seed, block]).
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

PROJECTIONS = ("q", "k", "v", "o", "gate", "up", "down")
TENSOR_IDS = {"X": 0, "A": 1, "B": 2, "dY": 3, "W": 4}

WORKLOADS = {
    1: dict(name="single CoLA layer, fp32, T=256, 512->512, r=128",
            T=256, d=512, ffn=None, r=128, dtype="f32"),
    2: dict(name="LLaMA-60M-shaped block, bf16, T=65536, d=512, ffn=1376, r=128",
            T=65536, d=512, ffn=1376, r=128, dtype="bf16"),
    3: dict(name="LLaMA-350M-shaped block, bf16, T=32768, d=1024, ffn=2736, r=256",
            T=32768, d=1024, ffn=2736, r=256, dtype="bf16"),
    4: dict(name="LLaMA-1B-shaped block, bf16, T=32768, d=2048, ffn=5461, r=512",
            T=32768, d=2048, ffn=5461, r=512, dtype="bf16"),
    5: dict(name="LLaMA-7B-shaped block, bf16, CoLA-M, T=16384, d=4096, ffn=11008, r=1024",
            T=16384, d=4096, ffn=11008, r=1024, dtype="bf16"),
}


def projections(cfg: int):
    """The projections of workload ``cfg`` as (name, index, d_in, d_out)."""
    w = WORKLOADS[cfg]
    d, ffn = w["d"], w["ffn"]
    if ffn is None:
        return [("single", 0, d, d)]
    shape = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d),
             "gate": (d, ffn), "up": (d, ffn), "down": (ffn, d)}
    return [(p, i, shape[p][0], shape[p][1]) for i, p in enumerate(PROJECTIONS)]


def seed_of(cfg: int, proj: int, tensor: str) -> int:
    return 1000 * cfg + 10 * proj + TENSOR_IDS[tensor]


ROWS_PER_BLOCK = 4096


def _pool_size() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def gaussian(seed: int, shape, std: float) -> np.ndarray:
    """float32 N(0, std^2) draws.  Rows are drawn in blocks of ROWS_PER_BLOCK;
    block b comes from PCG64(SeedSequence([seed, b])), so the values do not
    depend on how many threads fill them."""
    shape = tuple(int(s) for s in shape)
    out = np.empty(shape, dtype=np.float32)
    rows = shape[0] if shape else 1
    flat = out.reshape(rows, -1) if shape else out.reshape(1, 1)
    nblk = max(1, (rows + ROWS_PER_BLOCK - 1) // ROWS_PER_BLOCK)

    def fill(b):
        lo, hi = b * ROWS_PER_BLOCK, min(rows, (b + 1) * ROWS_PER_BLOCK)
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, b])))
        blk = flat[lo:hi]
        rng.standard_normal(blk.shape, dtype=np.float32, out=blk)
        blk *= np.float32(std)

    if nblk == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(_pool_size()) as ex:
            list(ex.map(fill, range(nblk)))
    return out


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round to nearest, ties to even); returns uint16 bits.
    The synthetic inputs are finite Gaussian draws, so no NaN/Inf handling."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.reshape(-1).view(np.uint32)
    out = np.empty(u.shape, dtype=np.uint16)
    step = 1 << 22

    def rnd(lo):
        v = u[lo:lo + step]
        t = v >> np.uint32(16)
        t &= np.uint32(1)
        t += np.uint32(0x7FFF)
        t += v
        t >>= np.uint32(16)
        out[lo:lo + step] = t

    if u.size <= step:
        rnd(0)
    else:
        with ThreadPoolExecutor(_pool_size()) as ex:
            list(ex.map(rnd, range(0, u.size, step)))
    return out.reshape(x.shape)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(bits).astype(np.float64)


class Tensor:
    """One synthetic tensor: ``store`` is what the GPU receives (float32 values
    or bf16 bits as uint16), ``f64`` the exact value of each stored element."""

    def __init__(self, store: np.ndarray, dtype: str):
        self.store = store
        self.dtype = dtype

    @property
    def f64(self) -> np.ndarray:
        if self.dtype == "bf16":
            return bf16_bits_to_f64(self.store)
        return self.store.astype(np.float64)

    @property
    def shape(self):
        return self.store.shape


def make(seed: int, shape, std: float, dtype: str) -> Tensor:
    x = gaussian(seed, shape, std)
    if dtype == "bf16":
        return Tensor(f32_to_bf16_bits(x), "bf16")
    if dtype == "f32":
        return Tensor(x, "f32")
    raise ValueError(dtype)


def layer_inputs(cfg: int, proj: int, d_in: int, d_out: int, r: int, T: int,
                 dtype: str, with_dense: bool = False) -> dict:
    """X, A, B, dY (and W for the dense baseline) of one projection."""
    out = {
        "X": make(seed_of(cfg, proj, "X"), (T, d_in), 1.0, dtype),
        "A": make(seed_of(cfg, proj, "A"), (r, d_in), 1.0 / math.sqrt(d_in), dtype),
        "B": make(seed_of(cfg, proj, "B"), (d_out, r), 1.0 / math.sqrt(r), dtype),
        "dY": make(seed_of(cfg, proj, "dY"), (T, d_out), 1.0, dtype),
    }
    if with_dense:
        out["W"] = make(seed_of(cfg, proj, "W"), (d_out, d_in), 1.0 / math.sqrt(d_in), dtype)
    return out


def padded_ld(width: int, dtype: str) -> int:
    """Row pitch (elements) that starts every row on a 128-byte cache line
    (the kernels need 16-byte aligned rows for their vector path; whole lines
    are faster still)."""
    per = 64 if dtype == "bf16" else 32
    return (width + per - 1) // per * per


def with_pitch(a: np.ndarray, ld: int, fill) -> np.ndarray:
    """Copy rows of ``a`` into a (rows, ld) array; columns >= width hold ``fill``
    (used to show that no kernel reads past a row's logical width)."""
    rows, width = a.shape
    if ld < width:
        raise ValueError("ld < width")
    out = np.full((rows, ld), fill, dtype=a.dtype)
    out[:, :width] = a
    return out


# ---------------------------------------------------------------------------
# decoder block inputs (the block-level path): the residual-stream input, the
# upstream gradient of the block output, the two RMSNorm gains and the
# weights of the seven projections
# ---------------------------------------------------------------------------

# LLaMA head counts of the workloads (head dim 64 up to the 1B shape, 128 at 7B)
HEADS = {2: 8, 3: 16, 4: 32, 5: 32}
SEQ_LEN = 256
BLOCK_TENSOR_IDS = {"x0": 0, "dx2": 1, "g1": 2, "g2": 3, "A_qkv": 4, "B_q": 5, "B_k": 6, "B_v": 7, "A_o": 8,
                    "B_o": 9, "A_gu": 10, "B_g": 11, "B_u": 12, "A_d": 13, "B_d": 14}


def block_shapes(d: int, ffn: int, r: int) -> dict:
    """Shapes of the block's parameters: A of the same-input groups stacked
    (q, k, v: [3r][d]; gate, up: [2r][d])."""
    return {"g1": (d,), "g2": (d,), "A_qkv": (3 * r, d), "B_q": (d, r), "B_k": (d, r), "B_v": (d, r),
            "A_o": (r, d), "B_o": (d, r), "A_gu": (2 * r, d), "B_g": (ffn, r), "B_u": (ffn, r),
            "A_d": (r, ffn), "B_d": (d, r)}


def block_inputs(seed: int, n_seq: int, seq_len: int, d: int, ffn: int, r: int, dtype: str = "bf16") -> dict:
    """x0, dx2 ~ N(0, 1) [T][d]; gains g = 1 + N(0, 0.1^2); A ~ N(0, 1/d_in),
    B ~ N(0, 1/r) per projection (the layer recipe).  Tensor seed =
    100000 + 1000 * seed + tensor id."""
    T = n_seq * seq_len
    base = 100000 + 1000 * seed
    out = {"x0": make(base + 0, (T, d), 1.0, dtype), "dx2": make(base + 1, (T, d), 1.0, dtype)}
    for name, shape in block_shapes(d, ffn, r).items():
        sid = base + BLOCK_TENSOR_IDS[name]
        if name in ("g1", "g2"):
            g = gaussian(sid, (1, shape[0]), 0.1).reshape(shape) + np.float32(1.0)
            out[name] = Tensor(f32_to_bf16_bits(g) if dtype == "bf16" else g, dtype)
        elif name.startswith("A"):
            out[name] = make(sid, shape, 1.0 / math.sqrt(shape[1]), dtype)
        else:
            out[name] = make(sid, shape, 1.0 / math.sqrt(r), dtype)
    return out
