"""Helpers for the block GPU tests and the bench: put a block's synthetic inputs
on the device, run the library's block forward and backward through the C ABI
(via the ctypes binding), and read results and saved tensors back.  No
arithmetic of the block happens here."""
from __future__ import annotations

import numpy as np
import torch

from paper_2502_10940_amd import cola

DEV = "cuda:0"


def bf16_dev(store: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(store).view(np.int16)).view(torch.bfloat16).to(DEV)


class BlockRun:
    def __init__(self, ins: dict, n_seq, seq_len, d, ffn, heads, r, act="silu", recompute=False):
        self.n_seq, self.seq_len, self.d, self.ffn, self.heads, self.r = n_seq, seq_len, d, ffn, heads, r
        self.T = n_seq * seq_len
        self.desc = cola.block_desc(n_seq, seq_len, d, ffn, heads, r, act, recompute)
        self.w = {k: bf16_dev(ins[k].store) for k in cola.BLOCK_PARAMS}
        self.x0 = bf16_dev(ins["x0"].store)
        self.dx2 = bf16_dev(ins["dx2"].store)
        self.x2 = torch.full((self.T, d), float("nan"), dtype=torch.bfloat16, device=DEV)
        self.dx0 = torch.full((self.T, d), float("nan"), dtype=torch.bfloat16, device=DEV)
        self.grads = {k: torch.full(v.shape, float("nan"), dtype=torch.float32, device=DEV)
                      for k, v in self.w.items()}
        self.saved = torch.empty(max(1, cola.block_saved_bytes(self.desc)), dtype=torch.uint8, device=DEV)
        ws = max(cola.block_workspace_bytes(self.desc, 0), cola.block_workspace_bytes(self.desc, 1), 1)
        self.ws = torch.empty(ws, dtype=torch.uint8, device=DEV)

    def forward(self):
        cola.block_fwd(self.desc, self.w, self.x0, self.x2, self.saved, self.ws)

    def backward(self):
        cola.block_bwd(self.desc, self.w, self.x0, self.saved, self.dx2, self.dx0, self.grads, self.ws)

    def run(self):
        self.forward()
        self.backward()
        torch.cuda.synchronize()
        return self

    def slot(self, name, width=None, rows=None, dtype=torch.bfloat16):
        """A tensor of the saved buffer as a [rows][width] view."""
        off, ld = cola.block_saved_slot(self.desc, name)
        rows = self.T if rows is None else rows
        width = ld if width is None else width
        esz = 2 if dtype == torch.bfloat16 else 4
        raw = self.saved[off: off + rows * ld * esz].view(dtype).view(rows, ld)
        return raw[:, :width]

    def results(self) -> dict:
        f = lambda t: t.detach().float().cpu().numpy().astype(np.float64)
        out = {"x2": f(self.x2), "dx0": f(self.dx0)}
        for k, v in self.grads.items():
            out["d" + k] = f(v)
        return out

    def raw(self) -> dict:
        out = {"x2": self.x2.view(torch.int16).cpu().numpy(), "dx0": self.dx0.view(torch.int16).cpu().numpy()}
        for k, v in self.grads.items():
            out["d" + k] = v.view(torch.int32).cpu().numpy()
        return out
