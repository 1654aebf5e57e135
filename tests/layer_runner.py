"""Helpers for the GPU tests: put synthetic inputs on the device, run the
library's forward and backward through the C ABI (via the ctypes binding),
and bring the results back as fp64 numpy arrays.  No arithmetic of the layer
happens here."""
from __future__ import annotations

import numpy as np
import torch

from paper_2502_10940_amd import cola
from paper_2502_10940_amd import inputs as I

DEV = "cuda:0"
TORCH_DT = {"bf16": torch.bfloat16, "f32": torch.float32}
NAN_BITS = {"bf16": 0x7FC0, "f32": np.float32(np.nan)}


def to_device(store: np.ndarray, dtype: str, ld: int | None = None, fill=None) -> torch.Tensor:
    """Host storage (bf16 bits as uint16, or float32) -> device tensor [rows][ld]."""
    a = store
    if ld is not None and ld != a.shape[1]:
        a = I.with_pitch(a, ld, NAN_BITS[dtype] if fill is None else fill)
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(DEV)


def empty(rows, ld, dtype, fill_bits=None):
    t = torch.empty((rows, ld), dtype=TORCH_DT[dtype], device=DEV)
    if fill_bits is not None:
        if dtype == "bf16":
            t.view(torch.int16).fill_(int(np.int16(np.uint16(fill_bits).view(np.int16))))
        else:
            t.fill_(float(fill_bits))
    return t


def to_f64(t: torch.Tensor, width: int | None = None) -> np.ndarray:
    a = t.detach().float().cpu().numpy().astype(np.float64)
    if width is not None:
        a = a[:, :width]
    return a


def relerr(got: np.ndarray, ref: np.ndarray) -> float:
    nr = np.linalg.norm(ref)
    ng = np.linalg.norm(got - ref)
    if nr == 0:
        return 0.0 if np.linalg.norm(got) == 0 else float("inf")
    return float(ng / nr)


class LayerRun:
    """One CoLA layer on the GPU: inputs resident, outputs allocated with the
    requested pitches (pad columns pre-filled with NaN so stray writes show)."""

    def __init__(self, ins: dict, T, d_in, d_out, r, dtype, act="silu", recompute=False,
                 ldx=None, ldy=None, ldz=None):
        self.T, self.d_in, self.d_out, self.r = T, d_in, d_out, r
        self.dtype, self.act, self.recompute = dtype, act, recompute
        self.ldx = ldx or d_in
        self.ldy = ldy or d_out
        self.ldz = ldz or r
        self.desc = cola.desc(T, d_in, d_out, r, dtype, act, recompute,
                              self.ldx, self.ldy, self.ldz)
        nanb = NAN_BITS[dtype]
        self.X = to_device(ins["X"].store, dtype, self.ldx)
        self.A = to_device(ins["A"].store, dtype)
        self.B = to_device(ins["B"].store, dtype)
        self.dY = to_device(ins["dY"].store, dtype, self.ldy)
        self.Y = empty(T, self.ldy, dtype, nanb)
        self.Z = empty(T, self.ldz, dtype, nanb)
        self.H = None if recompute else empty(T, self.ldz, dtype, nanb)
        self.dX = empty(T, self.ldx, dtype, nanb)
        self.dA = torch.full((r, d_in), float("nan"), dtype=torch.float32, device=DEV)
        self.dB = torch.full((d_out, r), float("nan"), dtype=torch.float32, device=DEV)
        wf = cola.workspace_bytes(self.desc, 0)
        wb = cola.workspace_bytes(self.desc, 1)
        self.ws = torch.empty(max(wf, wb, 1), dtype=torch.uint8, device=DEV)

    def forward(self):
        cola.fwd(self.desc, self.X, self.A, self.B, self.Y, self.Z, self.H, self.ws)

    def backward(self):
        cola.bwd(self.desc, self.dY, self.X, self.Z, self.H, self.A, self.B, self.dX,
                 self.dA, self.dB, self.ws)

    def run(self):
        self.forward()
        self.backward()
        torch.cuda.synchronize()
        return self

    def outputs(self) -> dict:
        out = {"Y": to_f64(self.Y, self.d_out), "Z": to_f64(self.Z, self.r),
               "dX": to_f64(self.dX, self.d_in), "dA": to_f64(self.dA), "dB": to_f64(self.dB)}
        if self.H is not None:
            out["H"] = to_f64(self.H, self.r)
        return out

    def padding_untouched(self) -> bool:
        """Columns past each row's width must still hold the NaN fill."""
        for t, w in ((self.Y, self.d_out), (self.Z, self.r), (self.dX, self.d_in)) + \
                (((self.H, self.r),) if self.H is not None else ()):
            if t.shape[1] > w and not torch.isnan(t[:, w:].float()).all():
                return False
        return True

    def raw(self) -> dict:
        """Outputs as raw bits (for bitwise comparisons)."""
        def bits(t, w):
            x = t[:, :w].contiguous()
            return (x.view(torch.int16) if self.dtype == "bf16" else x.view(torch.int32)).cpu().numpy()
        out = {"Y": bits(self.Y, self.d_out), "Z": bits(self.Z, self.r), "dX": bits(self.dX, self.d_in),
               "dA": self.dA.view(torch.int32).cpu().numpy(), "dB": self.dB.view(torch.int32).cpu().numpy()}
        return out
