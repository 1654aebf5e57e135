"""Thin ctypes binding of libcola.so (include/cola.h).

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  Tensors are passed as device pointers (``tensor.data_ptr()``), the
stream is torch's current stream unless one is given.  There is no fallback:
if ``libcola.so`` is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libcola.so")

F32, BF16 = 0, 1
ACT_IDENTITY, ACT_SILU, ACT_GELU = 0, 1, 2
DTYPES = {"f32": F32, "bf16": BF16}
ACTS = {"identity": ACT_IDENTITY, "silu": ACT_SILU, "gelu": ACT_GELU}

OK, ERR_INVALID_ARG, ERR_BAD_SHAPE, ERR_WORKSPACE, ERR_HIP, ERR_UNSUPPORTED, ERR_SCRATCH = range(7)
SCRATCH_BYTES = 64 << 20      # COLA_SCRATCH_BYTES

KERNEL_CLASSES = ("fwd_z_sigma", "fwd_y", "bwd_dz", "bwd_dx", "bwd_da", "bwd_db",
                  "reduce_splits", "dense_fwd", "dense_dx", "dense_dw", "fill_zero", "infer_h",
                  "outer_grad", "bwd_da_db", "attn_fwd", "attn_bwd", "norm", "norm_bwd", "pointwise")


class ColaError(RuntimeError):
    def __init__(self, status: int, text: str):
        super().__init__(f"libcola status {status}: {text}")
        self.status = status


class ColaDesc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("d_in", ctypes.c_int64), ("d_out", ctypes.c_int64),
                ("r", ctypes.c_int64), ("ldx", ctypes.c_int64), ("ldy", ctypes.c_int64),
                ("ldz", ctypes.c_int64), ("dtype", ctypes.c_int32), ("act", ctypes.c_int32),
                ("recompute", ctypes.c_int32)]


class DenseDesc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("d_in", ctypes.c_int64), ("d_out", ctypes.c_int64),
                ("ldx", ctypes.c_int64), ("ldy", ctypes.c_int64), ("dtype", ctypes.c_int32)]


GROUP_MAX = 8


class GroupDesc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("d_in", ctypes.c_int64), ("n", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("act", ctypes.c_int32), ("recompute", ctypes.c_int32),
                ("r", ctypes.c_int64 * GROUP_MAX), ("d_out", ctypes.c_int64 * GROUP_MAX),
                ("ldy", ctypes.c_int64 * GROUP_MAX), ("ldx", ctypes.c_int64), ("ldz", ctypes.c_int64)]


class BlockDesc(ctypes.Structure):
    _fields_ = [("n_seq", ctypes.c_int64), ("seq_len", ctypes.c_int64), ("d", ctypes.c_int64),
                ("ffn", ctypes.c_int64), ("heads", ctypes.c_int64), ("r", ctypes.c_int64),
                ("act", ctypes.c_int32), ("recompute", ctypes.c_int32), ("rope_base", ctypes.c_float),
                ("eps", ctypes.c_float)]


BLOCK_PARAMS = ("g1", "g2", "A_qkv", "B_q", "B_k", "B_v", "A_o", "B_o", "A_gu", "B_g", "B_u", "A_d", "B_d")


class BlockWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in BLOCK_PARAMS]


class BlockGrads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in BLOCK_PARAMS]


# cola_block_slot: tensors of the block's saved buffer
BLOCK_SLOTS = ("x1", "Z_qkv", "Z_o", "Z_gu", "Z_down", "a", "H_qkv", "q", "k", "v", "att", "lse", "H_o", "b",
               "H_gu", "gate", "up", "m", "H_down")

_lib = None

_P = ctypes.c_void_p
_SZ = ctypes.c_size_t

EXPORTS = {
    "cola_abi_version": ([], ctypes.c_int),
    "cola_strerror": ([ctypes.c_int], ctypes.c_char_p),
    "cola_workspace_bytes": ([ctypes.POINTER(ColaDesc), ctypes.c_int], _SZ),
    "cola_fwd": ([ctypes.POINTER(ColaDesc), _P, _P, _P, _P, _P, _P, _P, _SZ, _P], ctypes.c_int),
    "cola_bwd": ([ctypes.POINTER(ColaDesc), _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P],
                 ctypes.c_int),
    "dense_workspace_bytes": ([ctypes.POINTER(DenseDesc), ctypes.c_int], _SZ),
    "dense_fwd": ([ctypes.POINTER(DenseDesc), _P, _P, _P, _P, _SZ, _P], ctypes.c_int),
    "dense_bwd": ([ctypes.POINTER(DenseDesc), _P, _P, _P, _P, _P, _P, _SZ, _P], ctypes.c_int),
    "cola_group_workspace_bytes": ([ctypes.POINTER(GroupDesc), ctypes.c_int], _SZ),
    "cola_group_fwd": ([ctypes.POINTER(GroupDesc), _P, _P, _P, _P, _P, _P, _P, _SZ, _P], ctypes.c_int),
    "cola_group_bwd": ([ctypes.POINTER(GroupDesc), _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P],
                       ctypes.c_int),
    "cola_infer": ([ctypes.POINTER(ColaDesc), _P, _P, _P, _P, _P, _SZ, _P], ctypes.c_int),
    "cola_fwd_outer": ([ctypes.POINTER(ColaDesc), ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P],
                       ctypes.c_int),
    "cola_bwd_outer": ([ctypes.POINTER(ColaDesc), ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ,
                        _P], ctypes.c_int),
    "cola_group_infer": ([ctypes.POINTER(GroupDesc), _P, _P, _P, _P, _P, _SZ, _P], ctypes.c_int),
    "cola_timing_enable": ([ctypes.c_int], ctypes.c_int),
    "cola_timing_reset": ([], ctypes.c_int),
    "cola_timing_read": ([ctypes.c_int, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double),
                          ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)], ctypes.c_int),
    "cola_kernel_name": ([ctypes.c_int], ctypes.c_char_p),
    "cola_bwd_scratch": ([ctypes.POINTER(ColaDesc), _P, _P, _P, _P, _P, _P, _P, _P, _P, _P], ctypes.c_int),
    "cola_block_saved_bytes": ([ctypes.POINTER(BlockDesc)], _SZ),
    "cola_block_saved_slot": ([ctypes.POINTER(BlockDesc), ctypes.c_int, ctypes.POINTER(ctypes.c_size_t),
                               ctypes.POINTER(ctypes.c_int64)], ctypes.c_int),
    "cola_block_workspace_bytes": ([ctypes.POINTER(BlockDesc), ctypes.c_int], _SZ),
    "cola_block_fwd": ([ctypes.POINTER(BlockDesc), ctypes.POINTER(BlockWeights), _P, _P, _P, _SZ, _P, _SZ, _P],
                       ctypes.c_int),
    "cola_block_bwd": ([ctypes.POINTER(BlockDesc), ctypes.POINTER(BlockWeights), _P, _P, _SZ, _P, _P,
                        ctypes.POINTER(BlockGrads), _P, _SZ, _P], ctypes.c_int),
    "cola_set_option": ([ctypes.c_int, ctypes.c_int], ctypes.c_int),
    "cola_get_option": ([ctypes.c_int], ctypes.c_int),
}

OPT_STREAM_ONLY, OPT_WGRAD_PAIR, OPT_FUSE_GATE = 0, 1, 2


def lib():
    """Load libcola.so (built by ``paper_2502_10940_amd.build``); raises if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2502_10940_amd.build` (no fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in EXPORTS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def _check(status: int):
    if status != OK:
        raise ColaError(status, lib().cola_strerror(status).decode())


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


# ---------------------------------------------------------------------------
# Host-side checks of tensors against a descriptor.  The C ABI sees only
# pointers, so a tensor of the wrong dtype (dA allocated as bf16: the kernels
# write fp32, twice the bytes), a non-contiguous view, or rows shorter than
# the pitch would send the kernels outside their buffers; these checks refuse
# such calls with ValueError before anything is enqueued.  Raw integer
# pointers are passed through unchecked (the caller vouches for them).
# ---------------------------------------------------------------------------

def _torch_dtype(code):
    import torch
    return torch.bfloat16 if code == BF16 else torch.float32


def _need(name, t, rows, width, ld, dtype):
    """t must be a 2-D tensor of `dtype` holding `rows` rows of `width` used
    elements with row pitch `ld` elements, its storage covering rows x ld
    elements from its first element, on a GPU."""
    if t is None or isinstance(t, int) or rows == 0:
        return
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor or an integer device pointer")
    if t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, the descriptor needs {dtype}")
    if t.dim() != 2:
        raise ValueError(f"{name}: expected a 2-D tensor, got shape {tuple(t.shape)}")
    if t.shape[0] < rows or t.shape[1] < width:
        raise ValueError(f"{name}: shape {tuple(t.shape)} is smaller than [{rows}][{width}]")
    if t.stride(1) != 1 or (rows > 1 and t.stride(0) != ld):
        raise ValueError(f"{name}: strides {t.stride()} do not match a row pitch of {ld} elements "
                         "with contiguous rows")
    avail = t.untyped_storage().nbytes() - t.storage_offset() * t.element_size()
    if avail < rows * ld * t.element_size():
        raise ValueError(f"{name}: storage holds {avail} bytes from the first element, "
                         f"{rows} rows of pitch {ld} need {rows * ld * t.element_size()}")


def _on_gpu(named):
    """Every tensor of (name, tensor) pairs in GPU memory (checked after the
    shapes, so that a CPU test sees the shape refusals first)."""
    for name, t in named:
        if t is None or isinstance(t, int):
            continue
        if t.device.type != "cuda":
            raise ValueError(f"{name}: tensor is on {t.device}, the library needs GPU memory")


def _need_ws(ws, ws_bytes):
    if ws is None or isinstance(ws, int):
        return
    import torch
    if not isinstance(ws, torch.Tensor):
        raise TypeError("ws: expected a torch.Tensor or an integer device pointer")
    if not ws.is_contiguous():
        raise ValueError("ws: the workspace must be contiguous")
    if ws_bytes > ws.numel() * ws.element_size():
        raise ValueError(f"ws: ws_bytes {ws_bytes} exceeds the tensor's {ws.numel() * ws.element_size()} bytes")
    _on_gpu([("ws", ws)])


def _ws_bytes(ws, ws_bytes):
    if ws_bytes is None:
        ws_bytes = ws.numel() * ws.element_size() if ws is not None and not isinstance(ws, int) else 0
    _need_ws(ws, ws_bytes)
    return ws_bytes


def _layer_dims(d):
    ldx = d.ldx or d.d_in
    ldy = d.ldy or d.d_out
    ldz = d.ldz or d.r
    return d.T, d.d_in, d.d_out, d.r, ldx, ldy, ldz, _torch_dtype(d.dtype)


def _check_layer(d, **ts):
    """Tensors of one layer call, by their names in include/cola.h."""
    import torch
    T, d_in, d_out, r, ldx, ldy, ldz, dt = _layer_dims(d)
    shapes = {"X": (T, d_in, ldx, dt), "dX": (T, d_in, ldx, dt), "Y": (T, d_out, ldy, dt),
              "dY": (T, d_out, ldy, dt), "P": (T, d_out, ldy, dt), "Z": (T, r, ldz, dt),
              "H": (T, r, ldz, dt), "A": (r, d_in, d_in, dt), "B": (d_out, r, r, dt),
              "dA": (r, d_in, d_in, torch.float32), "dB": (d_out, r, r, torch.float32)}
    if d.dtype not in (F32, BF16) or min(T, d_in, d_out, r, ldx, ldy, ldz) < 0:
        return                      # the library refuses the descriptor itself
    for name, t in ts.items():
        rows, width, ld, dtype = shapes[name]
        _need(name, t, rows, width, ld, dtype)
    if T > 0:
        _on_gpu(ts.items())


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def desc(T, d_in, d_out, r, dtype="bf16", act="silu", recompute=False, ldx=0, ldy=0, ldz=0):
    return ColaDesc(T, d_in, d_out, r, ldx, ldy, ldz,
                    DTYPES[dtype] if isinstance(dtype, str) else int(dtype),
                    ACTS[act] if isinstance(act, str) else int(act), int(bool(recompute)))


def group_desc(T, d_in, r, d_out, dtype="bf16", act="silu", recompute=False, ldx=0, ldz=0, ldy=None):
    """Descriptor of n projections reading the same input (r, d_out, ldy: per projection)."""
    n = len(r)
    if len(d_out) != n or not 1 <= n <= GROUP_MAX:
        raise ValueError("r and d_out need the same length, 1 .. %d" % GROUP_MAX)
    ldy = list(ldy) if ldy is not None else [0] * n
    pad = lambda v: (ctypes.c_int64 * GROUP_MAX)(*(list(v) + [0] * (GROUP_MAX - n)))
    return GroupDesc(T, d_in, n, DTYPES[dtype] if isinstance(dtype, str) else int(dtype),
                     ACTS[act] if isinstance(act, str) else int(act), int(bool(recompute)),
                     pad(r), pad(d_out), pad(ldy), ldx, ldz)


def _ptr_array(xs):
    if xs is None:
        return None, None
    arr = (ctypes.c_void_p * len(xs))(*[_ptr(x) for x in xs])
    return ctypes.cast(arr, ctypes.c_void_p), arr      # keep arr alive with the cast


def _check_group(d, X=None, A_all=None, Z_all=None, H_all=None, dX=None, dA_all=None, B=None, Y=None, dY=None,
                 dB=None):
    import torch
    n = d.n
    if not 1 <= n <= GROUP_MAX or d.dtype not in (F32, BF16) or d.T < 0:
        return                      # the library refuses the descriptor itself
    T, d_in = d.T, d.d_in
    R = sum(d.r[p] for p in range(n))
    ldx = d.ldx or d_in
    ldz = d.ldz or R
    dt = _torch_dtype(d.dtype)
    _need("X", X, T, d_in, ldx, dt)
    _need("dX", dX, T, d_in, ldx, dt)
    _need("A_all", A_all, R, d_in, d_in, dt)
    _need("dA_all", dA_all, R, d_in, d_in, torch.float32)
    _need("Z_all", Z_all, T, R, ldz, dt)
    _need("H_all", H_all, T, R, ldz, dt)
    for key, lst in (("B", B), ("Y", Y), ("dY", dY), ("dB", dB)):
        if lst is None:
            continue
        if len(lst) != n:
            raise ValueError(f"{key}: {len(lst)} entries for {n} projections")
        for p, t in enumerate(lst):
            r, d_out = d.r[p], d.d_out[p]
            ldy = d.ldy[p] or d_out
            if key == "B":
                _need(f"B[{p}]", t, d_out, r, r, dt)
            elif key == "dB":
                _need(f"dB[{p}]", t, d_out, r, r, torch.float32)
            else:
                _need(f"{key}[{p}]", t, T, d_out, ldy, dt)
    if T > 0:
        named = [("X", X), ("dX", dX), ("A_all", A_all), ("dA_all", dA_all), ("Z_all", Z_all), ("H_all", H_all)]
        for key, lst in (("B", B), ("Y", Y), ("dY", dY), ("dB", dB)):
            named += [(f"{key}[{p}]", t) for p, t in enumerate(lst or [])]
        _on_gpu(named)


def _check_dense(d, X=None, W=None, Y=None, dY=None, dX=None, dW=None):
    import torch
    T, d_in, d_out = d.T, d.d_in, d.d_out
    if d.dtype not in (F32, BF16) or min(T, d_in, d_out, d.ldx, d.ldy) < 0:
        return                      # the library refuses the descriptor itself
    ldx = d.ldx or d_in
    ldy = d.ldy or d_out
    dt = _torch_dtype(d.dtype)
    _need("X", X, T, d_in, ldx, dt)
    _need("dX", dX, T, d_in, ldx, dt)
    _need("Y", Y, T, d_out, ldy, dt)
    _need("dY", dY, T, d_out, ldy, dt)
    _need("W", W, d_out, d_in, d_in, dt)
    _need("dW", dW, d_out, d_in, d_in, torch.float32)
    if T > 0:
        _on_gpu([("X", X), ("W", W), ("Y", Y), ("dY", dY), ("dX", dX), ("dW", dW)])


def group_workspace_bytes(d: GroupDesc, phase: int) -> int:
    return int(lib().cola_group_workspace_bytes(ctypes.byref(d), phase))


def group_fwd(d: GroupDesc, X, A_all, B, Y, Z_all, H_all, ws=None, ws_bytes=None, stream=None):
    """Z_all = X A_all^T, H_all = sigma(Z_all), Y_p = H_p B_p^T (B, Y: lists)."""
    ws_bytes = _ws_bytes(ws, ws_bytes)
    _check_group(d, X=X, A_all=A_all, Z_all=Z_all, H_all=H_all, B=B, Y=Y)
    pb, _kb = _ptr_array(B)
    py, _ky = _ptr_array(Y)
    _check(lib().cola_group_fwd(ctypes.byref(d), _ptr(X), _ptr(A_all), pb, py, _ptr(Z_all), _ptr(H_all),
                                _ptr(ws), ws_bytes, _stream(stream)))


def group_infer(d: GroupDesc, X, A_all, B, Y, ws=None, ws_bytes=None, stream=None):
    """Inference forward: Y_p = sigma(X A_p^T) B_p^T, nothing kept for a backward pass."""
    ws_bytes = _ws_bytes(ws, ws_bytes)
    _check_group(d, X=X, A_all=A_all, B=B, Y=Y)
    pb, _kb = _ptr_array(B)
    py, _ky = _ptr_array(Y)
    _check(lib().cola_group_infer(ctypes.byref(d), _ptr(X), _ptr(A_all), pb, py, _ptr(ws), ws_bytes,
                                  _stream(stream)))


def group_bwd(d: GroupDesc, dY, X, Z_all, H_all, A_all, B, dX, dA_all, dB, ws=None, ws_bytes=None, stream=None):
    """dZ_p = (dY_p B_p) * sigma'(Z_p), dX = sum_p dZ_p A_p, dA_all = dZ_all^T X, dB_p = dY_p^T H_p."""
    ws_bytes = _ws_bytes(ws, ws_bytes)
    _check_group(d, X=X, A_all=A_all, Z_all=Z_all, H_all=H_all, dX=dX, dA_all=dA_all, B=B, dY=dY, dB=dB)
    pdy, _k1 = _ptr_array(dY)
    pb, _k2 = _ptr_array(B)
    pdb, _k3 = _ptr_array(dB)
    _check(lib().cola_group_bwd(ctypes.byref(d), pdy, _ptr(X), _ptr(Z_all), _ptr(H_all), _ptr(A_all), pb,
                                _ptr(dX), _ptr(dA_all), pdb, _ptr(ws), ws_bytes, _stream(stream)))


def dense_desc(T, d_in, d_out, dtype="bf16", ldx=0, ldy=0):
    return DenseDesc(T, d_in, d_out, ldx, ldy, DTYPES[dtype] if isinstance(dtype, str) else int(dtype))


def workspace_bytes(d: ColaDesc, phase: int) -> int:
    return int(lib().cola_workspace_bytes(ctypes.byref(d), phase))


def dense_workspace_bytes(d: DenseDesc, phase: int) -> int:
    return int(lib().dense_workspace_bytes(ctypes.byref(d), phase))


def fwd(d: ColaDesc, X, A, B, Y, Z, H, ws=None, ws_bytes=None, stream=None):
    """Z = X A^T, H = sigma(Z), Y = H B^T (H is None in CoLA-M mode)."""
    ws_bytes = _ws_bytes(ws, ws_bytes)
    _check_layer(d, X=X, A=A, B=B, Y=Y, Z=Z, H=H)
    _check(lib().cola_fwd(ctypes.byref(d), _ptr(X), _ptr(A), _ptr(B), _ptr(Y), _ptr(Z), _ptr(H),
                          _ptr(ws), ws_bytes, _stream(stream)))


def fwd_outer(d: ColaDesc, outer, X, A, B, Y, P, Z, H, ws=None, ws_bytes=None, stream=None):
    """Both-sigma variant: P = H B^T, Y = sigma_out(P) (outer: a sigma name or code)."""
    ws_bytes = _ws_bytes(ws, ws_bytes)
    _check_layer(d, X=X, A=A, B=B, Y=Y, P=P, Z=Z, H=H)
    _check(lib().cola_fwd_outer(ctypes.byref(d), ACTS[outer] if isinstance(outer, str) else int(outer), _ptr(X),
                                _ptr(A), _ptr(B), _ptr(Y), _ptr(P), _ptr(Z), _ptr(H), _ptr(ws), ws_bytes,
                                _stream(stream)))


def bwd_outer(d: ColaDesc, outer, dY, P, X, Z, H, A, B, dX, dA, dB, ws=None, ws_bytes=None, stream=None):
    """Both-sigma backward: dP = dY * sigma_out'(P), then the layer backward on dP."""
    ws_bytes = _ws_bytes(ws, ws_bytes)
    _check_layer(d, dY=dY, P=P, X=X, Z=Z, H=H, A=A, B=B, dX=dX, dA=dA, dB=dB)
    _check(lib().cola_bwd_outer(ctypes.byref(d), ACTS[outer] if isinstance(outer, str) else int(outer), _ptr(dY),
                                _ptr(P), _ptr(X), _ptr(Z), _ptr(H), _ptr(A), _ptr(B), _ptr(dX), _ptr(dA), _ptr(dB),
                                _ptr(ws), ws_bytes, _stream(stream)))


def infer(d: ColaDesc, X, A, B, Y, ws=None, ws_bytes=None, stream=None):
    """Inference forward: Y = sigma(X A^T) B^T, nothing kept for a backward pass."""
    ws_bytes = _ws_bytes(ws, ws_bytes)
    _check_layer(d, X=X, A=A, B=B, Y=Y)
    _check(lib().cola_infer(ctypes.byref(d), _ptr(X), _ptr(A), _ptr(B), _ptr(Y), _ptr(ws), ws_bytes,
                            _stream(stream)))


def bwd(d: ColaDesc, dY, X, Z, H, A, B, dX, dA, dB, ws=None, ws_bytes=None, stream=None):
    """dZ = (dY B) * sigma'(Z), dX = dZ A, dA = dZ^T X, dB = dY^T H (H None in CoLA-M)."""
    ws_bytes = _ws_bytes(ws, ws_bytes)
    _check_layer(d, dY=dY, X=X, Z=Z, H=H, A=A, B=B, dX=dX, dA=dA, dB=dB)
    _check(lib().cola_bwd(ctypes.byref(d), _ptr(dY), _ptr(X), _ptr(Z), _ptr(H), _ptr(A), _ptr(B),
                          _ptr(dX), _ptr(dA), _ptr(dB), _ptr(ws), ws_bytes, _stream(stream)))


def bwd_scratch(d: ColaDesc, dY, X, Z, H, A, B, dX, dA, dB, stream=None):
    """cola_bwd with the library's static device scratch as its workspace
    (for callers that cannot allocate; overlapping calls on one GPU race)."""
    _check_layer(d, dY=dY, X=X, Z=Z, H=H, A=A, B=B, dX=dX, dA=dA, dB=dB)
    _check(lib().cola_bwd_scratch(ctypes.byref(d), _ptr(dY), _ptr(X), _ptr(Z), _ptr(H), _ptr(A), _ptr(B),
                                  _ptr(dX), _ptr(dA), _ptr(dB), _stream(stream)))


def dense_fwd(d: DenseDesc, X, W, Y, ws=None, ws_bytes=None, stream=None):
    ws_bytes = _ws_bytes(ws, ws_bytes)
    _check_dense(d, X=X, W=W, Y=Y)
    _check(lib().dense_fwd(ctypes.byref(d), _ptr(X), _ptr(W), _ptr(Y), _ptr(ws), ws_bytes,
                           _stream(stream)))


def dense_bwd(d: DenseDesc, dY, X, W, dX, dW, ws=None, ws_bytes=None, stream=None):
    ws_bytes = _ws_bytes(ws, ws_bytes)
    _check_dense(d, dY=dY, X=X, W=W, dX=dX, dW=dW)
    _check(lib().dense_bwd(ctypes.byref(d), _ptr(dY), _ptr(X), _ptr(W), _ptr(dX), _ptr(dW),
                           _ptr(ws), ws_bytes, _stream(stream)))


def timing_enable(on: bool = True):
    _check(lib().cola_timing_enable(int(on)))


def timing_reset():
    _check(lib().cola_timing_reset())


def timing_read(kernel_class: int):
    """(launches, ms, flops, bytes) summed since the last reset."""
    n = ctypes.c_int64()
    ms = ctypes.c_double()
    fl = ctypes.c_double()
    by = ctypes.c_double()
    _check(lib().cola_timing_read(kernel_class, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(fl),
                                  ctypes.byref(by)))
    return n.value, ms.value, fl.value, by.value


def kernel_name(kernel_class: int) -> str:
    return lib().cola_kernel_name(kernel_class).decode()


def set_option(option: int, value: int):
    """Process-wide tuning option (OPT_STREAM_ONLY, OPT_WGRAD_PAIR, OPT_FUSE_GATE) to 0 or 1."""
    _check(lib().cola_set_option(int(option), int(value)))


def get_option(option: int) -> int:
    return int(lib().cola_get_option(int(option)))



# ---------------------------------------------------------------------------
# decoder block (cola_block_*)
# ---------------------------------------------------------------------------

def block_desc(n_seq, seq_len, d, ffn, heads, r, act="silu", recompute=False, rope_base=10000.0, eps=1e-6):
    return BlockDesc(n_seq, seq_len, d, ffn, heads, r, ACTS[act] if isinstance(act, str) else int(act),
                     int(bool(recompute)), rope_base, eps)


def block_shapes(d: BlockDesc) -> dict:
    r, dm, f = d.r, d.d, d.ffn
    return {"g1": (dm,), "g2": (dm,), "A_qkv": (3 * r, dm), "B_q": (dm, r), "B_k": (dm, r), "B_v": (dm, r),
            "A_o": (r, dm), "B_o": (dm, r), "A_gu": (2 * r, dm), "B_g": (f, r), "B_u": (f, r), "A_d": (r, f),
            "B_d": (dm, r)}


def block_saved_bytes(d: BlockDesc) -> int:
    return int(lib().cola_block_saved_bytes(ctypes.byref(d)))


def block_workspace_bytes(d: BlockDesc, phase: int) -> int:
    return int(lib().cola_block_workspace_bytes(ctypes.byref(d), phase))


def block_saved_slot(d: BlockDesc, slot) -> tuple:
    """(byte offset, row pitch in elements) of a tensor in the saved buffer."""
    idx = BLOCK_SLOTS.index(slot) if isinstance(slot, str) else int(slot)
    off = ctypes.c_size_t()
    ld = ctypes.c_int64()
    _check(lib().cola_block_saved_slot(ctypes.byref(d), idx, ctypes.byref(off), ctypes.byref(ld)))
    return int(off.value), int(ld.value)


def _check_block(d: BlockDesc, params: dict, dtype, **acts):
    import torch
    if d.n_seq < 0 or d.seq_len < 1 or d.d < 1 or d.ffn < 1 or d.r < 1:
        return                      # the library refuses the descriptor itself
    for name, shape in block_shapes(d).items():
        t = params.get(name)
        if t is None:
            raise ValueError(f"{name}: missing")
        if isinstance(t, int):
            continue
        if t.dtype != dtype or tuple(t.shape) != shape or not t.is_contiguous():
            raise ValueError(f"{name}: expected a contiguous {dtype} tensor of shape {shape}, got "
                             f"{t.dtype} {tuple(t.shape)}")
    T = d.n_seq * d.seq_len
    for name, t in acts.items():
        _need(name, t, T, d.d, d.d, torch.bfloat16)
    if T > 0:
        _on_gpu(list(acts.items()) + [(k, params[k]) for k in BLOCK_PARAMS])


def _bytes_of(t, n):
    if n is None:
        n = t.numel() * t.element_size() if t is not None and not isinstance(t, int) else 0
    _need_ws(t, n)
    return n


def block_fwd(d: BlockDesc, w: dict, x0, x2, saved, ws, saved_bytes=None, ws_bytes=None, stream=None):
    """x2 = the block applied to x0 (w: bf16 tensors by BLOCK_PARAMS); `saved`
    receives what the backward needs."""
    import torch
    _check_block(d, w, torch.bfloat16, x0=x0, x2=x2)
    saved_bytes = _bytes_of(saved, saved_bytes)
    ws_bytes = _bytes_of(ws, ws_bytes)
    W = BlockWeights(*[_ptr(w[n]) for n in BLOCK_PARAMS])
    _check(lib().cola_block_fwd(ctypes.byref(d), ctypes.byref(W), _ptr(x0), _ptr(x2), _ptr(saved), saved_bytes,
                                _ptr(ws), ws_bytes, _stream(stream)))


def block_bwd(d: BlockDesc, w: dict, x0, saved, dx2, dx0, grads: dict, ws, saved_bytes=None, ws_bytes=None,
              stream=None):
    """dx0 and the fp32 parameter gradients (grads: tensors by BLOCK_PARAMS)."""
    import torch
    _check_block(d, w, torch.bfloat16, x0=x0, dx2=dx2, dx0=dx0)
    _check_block(d, grads, torch.float32)
    saved_bytes = _bytes_of(saved, saved_bytes)
    ws_bytes = _bytes_of(ws, ws_bytes)
    W = BlockWeights(*[_ptr(w[n]) for n in BLOCK_PARAMS])
    G = BlockGrads(*[_ptr(grads[n]) for n in BLOCK_PARAMS])
    _check(lib().cola_block_bwd(ctypes.byref(d), ctypes.byref(W), _ptr(x0), _ptr(saved), saved_bytes, _ptr(dx2),
                                _ptr(dx0), ctypes.byref(G), _ptr(ws), ws_bytes, _stream(stream)))
