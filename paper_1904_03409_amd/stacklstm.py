"""Thin ctypes binding of ``libstacklstm.so`` (include/stacklstm.h).

Argument marshalling only: every step of the forward and backward pass runs in the
HIP library. Tensors must be contiguous device tensors of the documented dtypes;
PyTorch supplies device memory and the current stream. If the library has not been
built this module raises on import of the library -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libstacklstm.so")

SLSTM_FP32 = 0
SLSTM_BF16_GEMM = 1
STATUS = {0: "SLSTM_OK", 1: "SLSTM_EINVAL", 2: "SLSTM_EOPS", 3: "SLSTM_EUNDERFLOW", 4: "SLSTM_EWORKSPACE",
          5: "SLSTM_ENORESIDENT", 6: "SLSTM_EDEVICE", 7: "SLSTM_ETIMEOUT", 8: "SLSTM_EINDEX"}
EXPORTS = ("stacklstm_workspace_bytes", "stacklstm_fwd", "stacklstm_fwd_static", "stacklstm_bwd",
           "stacklstm_sync_status", "stacklstm_status_string", "stacklstm_plan")
SLSTM_FWD_STATIC_MAX_BYTES = 128 << 20


class StackLSTMError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {STATUS.get(code, code)} ({_status_string(code)})")
        self.code = code


class slstm_dims(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("B", ctypes.c_int32), ("I", ctypes.c_int32), ("H", ctypes.c_int32),
                ("precision", ctypes.c_int32), ("spin_limit", ctypes.c_int32), ("phase_events", ctypes.c_void_p),
                ("step_clock", ctypes.c_void_p), ("defer_status", ctypes.c_int32)]

SLSTM_PHASE_EVENTS = 10


class slstm_plan(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "groups", "wg_per_group", "rows_per_group", "k_chunks", "fwd_kernel", "fwd_tiles", "k_chunk_cap",
        "occupancy", "bwd_groups", "bwd_tiles", "bwd_direct", "fused_x", "bwd_split")]


_lib = None


def load_library():
    """Loads the built library (raises FileNotFoundError when it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FileNotFoundError(f"{LIB_PATH} is missing: run __graft_entry__.build() first")
        lib = ctypes.CDLL(LIB_PATH)
        P, I32, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        D = ctypes.POINTER(slstm_dims)
        lib.stacklstm_workspace_bytes.restype = SZ
        lib.stacklstm_workspace_bytes.argtypes = [D]
        lib.stacklstm_fwd.restype = I32
        lib.stacklstm_fwd.argtypes = [D] + [P] * 14 + [SZ, P]
        lib.stacklstm_fwd_static.restype = I32
        lib.stacklstm_fwd_static.argtypes = [D] + [P] * 13 + [P]
        lib.stacklstm_bwd.restype = I32
        lib.stacklstm_bwd.argtypes = [D] + [P] * 10 + [SZ] + [P] * 8 + [P]
        lib.stacklstm_sync_status.restype = I32
        lib.stacklstm_sync_status.argtypes = [P, SZ, P]
        lib.stacklstm_status_string.restype = ctypes.c_char_p
        lib.stacklstm_status_string.argtypes = [I32]
        lib.stacklstm_plan.restype = I32
        lib.stacklstm_plan.argtypes = [D, ctypes.POINTER(slstm_plan)]
        _lib = lib
    return _lib


def _status_string(code: int) -> str:
    try:
        return load_library().stacklstm_status_string(int(code)).decode()
    except Exception:  # library missing: the numeric code is still reported
        return "?"


def make_dims(T: int, B: int, I: int, H: int, precision: int = SLSTM_FP32, spin_limit: int = 0,
              defer_status: int = 0) -> slstm_dims:
    return slstm_dims(int(T), int(B), int(I), int(H), int(precision), int(spin_limit), None, None, int(defer_status))


def _ptr(t: Optional[torch.Tensor], dtype=None, what="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{what} must be {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check(code: int, what: str):
    if code != 0:
        raise StackLSTMError(code, what)


def stacklstm_workspace_bytes(dims: slstm_dims) -> int:
    return int(load_library().stacklstm_workspace_bytes(ctypes.byref(dims)))


def stacklstm_plan(dims: slstm_dims) -> dict:
    out = slstm_plan()
    _check(load_library().stacklstm_plan(ctypes.byref(dims), ctypes.byref(out)), "stacklstm_plan")
    return {n: getattr(out, n) for n, _ in slstm_plan._fields_}


def stacklstm_fwd(dims, x, ops, W, U, b, h0, c0, h_cell, c_cell, h_top, c_top, ptr, top, workspace, stream=None,
                  check=True) -> int:
    f32, i32 = torch.float32, torch.int32
    rc = load_library().stacklstm_fwd(
        ctypes.byref(dims), _ptr(x, f32, "x"), _ptr(ops, torch.int8, "ops"), _ptr(W, f32, "W"), _ptr(U, f32, "U"),
        _ptr(b, f32, "b"), _ptr(h0, f32, "h0"), _ptr(c0, f32, "c0"), _ptr(h_cell, f32, "h_cell"),
        _ptr(c_cell, f32, "c_cell"), _ptr(h_top, f32, "h_top"), _ptr(c_top, f32, "c_top"), _ptr(ptr, i32, "ptr"),
        _ptr(top, i32, "top"), _ptr(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream))
    if check:
        _check(rc, "stacklstm_fwd")
    return rc


def stacklstm_fwd_static(dims, x, ops, W, U, b, h0, c0, h_cell, c_cell, h_top, c_top, ptr, top, stream=None,
                         check=True) -> int:
    """stacklstm_fwd on the library's static per-GPU work space (no work-space argument)."""
    f32, i32 = torch.float32, torch.int32
    rc = load_library().stacklstm_fwd_static(
        ctypes.byref(dims), _ptr(x, f32, "x"), _ptr(ops, torch.int8, "ops"), _ptr(W, f32, "W"), _ptr(U, f32, "U"),
        _ptr(b, f32, "b"), _ptr(h0, f32, "h0"), _ptr(c0, f32, "c0"), _ptr(h_cell, f32, "h_cell"),
        _ptr(c_cell, f32, "c_cell"), _ptr(h_top, f32, "h_top"), _ptr(c_top, f32, "c_top"), _ptr(ptr, i32, "ptr"),
        _ptr(top, i32, "top"), _stream(stream))
    if check:
        _check(rc, "stacklstm_fwd_static")
    return rc


def stacklstm_bwd(dims, x, ops, W, U, h0, c0, h_cell, c_cell, top, workspace, dh_top, dc_top, dx, dW, dU, db, dh0,
                  dc0, stream=None, check=True) -> int:
    f32 = torch.float32
    rc = load_library().stacklstm_bwd(
        ctypes.byref(dims), _ptr(x, f32, "x"), _ptr(ops, torch.int8, "ops"), _ptr(W, f32, "W"), _ptr(U, f32, "U"),
        _ptr(h0, f32, "h0"), _ptr(c0, f32, "c0"), _ptr(h_cell, f32, "h_cell"), _ptr(c_cell, f32, "c_cell"),
        _ptr(top, torch.int32, "top"), _ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
        _ptr(dh_top, f32, "dh_top"), _ptr(dc_top, f32, "dc_top"), _ptr(dx, f32, "dx"), _ptr(dW, f32, "dW"),
        _ptr(dU, f32, "dU"), _ptr(db, f32, "db"), _ptr(dh0, f32, "dh0"), _ptr(dc0, f32, "dc0"), _stream(stream))
    if check:
        _check(rc, "stacklstm_bwd")
    return rc


def stacklstm_sync_status(workspace: torch.Tensor, stream=None) -> int:
    return int(load_library().stacklstm_sync_status(_ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
                                                    _stream(stream)))


# ----------------------------------------------------------------------------- device buffers for one workload

@dataclass
class DeviceRun:
    """Device copies of a workload's inputs plus every output buffer of one fwd + bwd."""
    dims: slstm_dims
    x: torch.Tensor
    ops: torch.Tensor
    W: torch.Tensor
    U: torch.Tensor
    b: torch.Tensor
    h0: torch.Tensor
    c0: torch.Tensor
    dh_top: torch.Tensor
    dc_top: Optional[torch.Tensor]
    h_cell: torch.Tensor
    c_cell: torch.Tensor
    h_top: Optional[torch.Tensor]
    c_top: Optional[torch.Tensor]
    ptr: torch.Tensor
    top: torch.Tensor
    workspace: torch.Tensor
    dx: torch.Tensor
    dW: torch.Tensor
    dU: torch.Tensor
    db: torch.Tensor
    dh0: torch.Tensor
    dc0: torch.Tensor

    @classmethod
    def from_workload(cls, wl, device="cuda", precision: Optional[int] = None, want_top: bool = True,
                      spin_limit: int = 0) -> "DeviceRun":
        prec = wl.precision if precision is None else precision
        dims = make_dims(wl.T, wl.B, wl.I, wl.H, prec, spin_limit)
        ws = stacklstm_workspace_bytes(dims)
        if ws == 0:
            raise StackLSTMError(1, "stacklstm_workspace_bytes")
        dev = torch.device(device)

        def up(a):
            return None if a is None else torch.from_numpy(a).to(dev)

        T, B, I, H = wl.T, wl.B, wl.I, wl.H
        e = lambda *s: torch.empty(*s, dtype=torch.float32, device=dev)
        return cls(dims=dims, x=up(wl.x), ops=up(wl.ops), W=up(wl.W), U=up(wl.U), b=up(wl.b), h0=up(wl.h0),
                   c0=up(wl.c0), dh_top=up(wl.dh_top), dc_top=up(wl.dc_top), h_cell=e(T, B, H), c_cell=e(T, B, H),
                   h_top=e(T, B, H) if want_top else None, c_top=e(T, B, H) if want_top else None,
                   ptr=torch.empty(T + 1, B, dtype=torch.int32, device=dev),
                   top=torch.empty(T, B, dtype=torch.int32, device=dev),
                   workspace=torch.empty(ws, dtype=torch.uint8, device=dev), dx=e(T, B, I), dW=e(I, 4 * H),
                   dU=e(H, 4 * H), db=e(4 * H), dh0=e(B, H), dc0=e(B, H))

    def forward(self, stream=None, check=True) -> int:
        return stacklstm_fwd(self.dims, self.x, self.ops, self.W, self.U, self.b, self.h0, self.c0, self.h_cell,
                             self.c_cell, self.h_top, self.c_top, self.ptr, self.top, self.workspace, stream, check)

    def backward(self, stream=None, check=True) -> int:
        return stacklstm_bwd(self.dims, self.x, self.ops, self.W, self.U, self.h0, self.c0, self.h_cell,
                             self.c_cell, self.top, self.workspace, self.dh_top, self.dc_top, self.dx, self.dW,
                             self.dU, self.db, self.dh0, self.dc0, stream, check)

    def results(self) -> dict:
        out = {}
        for k in ("h_cell", "c_cell", "h_top", "c_top", "ptr", "top", "dx", "dW", "dU", "db", "dh0", "dc0"):
            v = getattr(self, k)
            if v is not None:
                out[k] = v.cpu().numpy()
        return out


def multilayer_runs(ops, x, layers, h0, c0, dh_top, dc_top=None, device="cuda", precision: int = 0,
                    want_top: bool = True) -> list:
    """Device buffers for L stacked StackLSTM layers driven by one op stream: the stack
    element holds every layer's state, so layer l (l > 0) reads as its input at step t
    the state at the top of layer l-1 after that step (on push steps the state layer l-1
    just produced; on pop and hold steps the written state is discarded and its
    gradient is exactly zero). Layer l's input buffer is layer l-1's h_top buffer, and
    in the backward layer l-1's dh_top buffer is layer l's dx buffer, so running
    [r.forward() for r in runs] and then [r.backward() for r in reversed(runs)] is the
    multi-layer forward and backward (every step on the GPU; this only wires buffers).

    ops [T, B] int8, x [T, B, I], layers = [(W_l, U_l, b_l)] with W_1 [I, 4H] and W_l
    [H, 4H] after, h0/c0 = per layer [B, H], dh_top/dc_top [T, B, H] on the last layer.
    """
    T, B = ops.shape
    H = layers[0][1].shape[0]
    dev = torch.device(device)
    up = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    e = lambda *sh: torch.empty(*sh, dtype=torch.float32, device=dev)
    ops_d = up(np.asarray(ops, dtype=np.int8))
    runs = []
    prev_top = up(np.asarray(x, dtype=np.float32))
    for l, (W, U, bias) in enumerate(layers):
        I = W.shape[0]
        dims = make_dims(T, B, I, H, precision, 0)
        ws = stacklstm_workspace_bytes(dims)
        if ws == 0:
            raise StackLSTMError(1, "stacklstm_workspace_bytes")
        last = l == len(layers) - 1
        r = DeviceRun(dims=dims, x=prev_top, ops=ops_d, W=up(W), U=up(U), b=up(bias), h0=up(h0[l]), c0=up(c0[l]),
                      dh_top=up(dh_top) if last else None, dc_top=up(dc_top) if last else None,
                      h_cell=e(T, B, H), c_cell=e(T, B, H), h_top=e(T, B, H),
                      c_top=e(T, B, H) if (want_top or not last) else None,
                      ptr=torch.empty(T + 1, B, dtype=torch.int32, device=dev),
                      top=torch.empty(T, B, dtype=torch.int32, device=dev),
                      workspace=torch.empty(ws, dtype=torch.uint8, device=dev), dx=e(T, B, I), dW=e(I, 4 * H),
                      dU=e(H, 4 * H), db=e(4 * H), dh0=e(B, H), dc0=e(B, H))
        if l > 0:
            runs[-1].dh_top = r.dx
        runs.append(r)
        prev_top = r.h_top
    return runs
