"""ctypes binding of libvitattn.so (argument marshalling only).

Raw entry points (`library().vitattn_fwd(...)` etc.) take integer device
pointers exactly like the C ABI. The tensor helpers below allocate outputs
with PyTorch, pass `data_ptr()`s and the current HIP stream, and raise
VitattnError on a non-zero status.
"""
from __future__ import annotations

import ctypes
import math
import os
import threading

from ._build import LIB_PATH

_lock = threading.Lock()
_lib = None

c_int, c_float, c_size_t, c_void_p = ctypes.c_int, ctypes.c_float, ctypes.c_size_t, ctypes.c_void_p


class Strides(ctypes.Structure):
    """vitattn_strides: element strides of an operand viewed as [B, H, N, d]."""
    _fields_ = [("batch", ctypes.c_longlong), ("head", ctypes.c_longlong), ("row", ctypes.c_longlong)]


_S = Strides

_SIGNATURES = {
    "vitattn_fwd": (c_int, [c_void_p] * 5 + [c_int] * 4 + [c_float, c_void_p]),
    "vitattn_bwd_workspace_bytes": (c_size_t, [c_int] * 4),
    "vitattn_bwd": (c_int, [c_void_p] * 9 + [c_int] * 4 + [c_float, c_void_p, c_size_t, c_void_p]),
    "vitattn_bwd_rowdot": (c_int, [c_void_p] * 3 + [c_int] * 4 + [c_void_p, c_size_t, c_void_p]),
    "vitattn_bwd_dkdv": (c_int, [c_void_p] * 7 + [c_int] * 4 + [c_float, c_void_p, c_size_t, c_void_p]),
    "vitattn_bwd_dq": (c_int, [c_void_p] * 6 + [c_int] * 4 + [c_float, c_void_p, c_size_t, c_void_p]),
    "vitattn_fwd_kv": (c_int, [c_void_p] * 5 + [c_int] * 5 + [c_float, c_void_p]),
    "vitattn_bwd_kv": (c_int, [c_void_p] * 9 + [c_int] * 5 + [c_float, c_int, c_void_p, c_size_t, c_void_p]),
    "vitattn_bwd_workspace_bytes_kv": (c_size_t, [c_int] * 6),
    "vitattn_bwd_dkdv_ds": (c_int, [c_void_p] * 7 + [c_int] * 4 + [c_float, c_void_p, c_size_t, c_void_p]),
    "vitattn_bwd_dq_from_ds": (c_int, [c_void_p] * 2 + [c_int] * 4 + [c_float, c_void_p, c_size_t, c_void_p]),
    "vitattn_fwd_strided": (c_int, [c_void_p, _S] * 4 + [c_void_p] + [c_int] * 5 + [c_float, c_void_p]),
    "vitattn_bwd_strided": (c_int, [c_void_p, _S] * 5 + [c_void_p] + [c_void_p, _S] * 3 + [c_int] * 5
                            + [c_float, c_int, c_void_p, c_size_t, c_void_p]),
    "vitattn_merge": (c_int, [c_void_p] * 2 + [c_int] + [c_void_p] * 2 + [c_int] * 4 + [c_void_p]),
    "vitattn_agg_fwd": (c_int, [c_void_p] * 5 + [c_int] * 4 + [c_float, c_void_p]),
    "vitattn_agg_bwd_workspace_bytes": (c_size_t, [c_int] * 4),
    "vitattn_agg_bwd": (c_int, [c_void_p] * 9 + [c_int] * 4 + [c_float, c_void_p, c_size_t, c_void_p]),
    "vitattn_ulysses_pack": (c_int, [c_void_p] * 2 + [c_int] * 5 + [c_void_p]),
    "vitattn_ulysses_unpack": (c_int, [c_void_p] * 2 + [c_int] * 5 + [c_void_p]),
    "vitattn_ulysses_pack_out": (c_int, [c_void_p] * 2 + [c_int] * 5 + [c_void_p]),
    "vitattn_ulysses_unpack_out": (c_int, [c_void_p] * 2 + [c_int] * 5 + [c_void_p]),
    "vitattn_bwd_noalloc": (c_int, [c_void_p] * 9 + [c_int] * 4 + [c_float, c_void_p]),
    "vitattn_status_str": (ctypes.c_char_p, [c_int]),
    "vitattn_version": (ctypes.c_char_p, []),
}


class VitattnError(RuntimeError):
    def __init__(self, status: int):
        self.status = status
        super().__init__(status_str(status))


def open_library(path):
    """ctypes handle of a built library at `path` with every entry point's
    signature set (library() uses it for the package's own build)."""
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


def library():
    """Load libvitattn.so once. Raises if it has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise ImportError(f"{LIB_PATH} is missing: build it with paper_2405_15780_amd._build.build()")
            _lib = open_library(LIB_PATH)
    return _lib


def status_str(status: int) -> str:
    return library().vitattn_status_str(status).decode()


def version() -> str:
    return library().vitattn_version().decode()


def workspace_bytes(B: int, H: int, N: int, d: int) -> int:
    return int(library().vitattn_bwd_workspace_bytes(B, H, N, d))


def _check(status: int):
    if status != 0:
        raise VitattnError(status)


def _torch():
    import torch

    return torch


def _stream_ptr(t) -> int:
    torch = _torch()
    return torch.cuda.current_stream(t.device).cuda_stream


def _as_input(t, name, device=None):
    torch = _torch()
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == torch.bfloat16 and t.dim() == 4
            and (t.shape[3] == 1 or t.stride(3) == 1) and (device is None or t.device == device)):
        raise TypeError(f"{name} must be a 4-D bfloat16 CUDA tensor [B, H, N, d] with unit stride along d, on the "
                        "device of q (other strides are free, e.g. a [B, N, H, d] tensor passed as .transpose(1, 2))")
    return t


def _expect(t, name, dtype, shape, device, dense=False):
    """Raise TypeError unless t is a CUDA tensor of this dtype and exact shape
    on `device`, with unit stride along its last dim (contiguous if dense).
    A mismatch would otherwise become an out-of-bounds access on the GPU."""
    torch = _torch()
    shape = tuple(int(n) for n in shape)
    ok = (isinstance(t, torch.Tensor) and t.is_cuda and t.device == device and t.dtype == dtype
          and tuple(t.shape) == shape)
    if ok:
        ok = t.is_contiguous() if dense else (shape[-1] == 1 or t.stride(-1) == 1)
    if not ok:
        layout = "contiguous" if dense else "unit stride along the last dim"
        raise TypeError(f"{name} must be a {dtype} CUDA tensor of shape {shape} on {device} ({layout})")
    return t


def _expect_workspace(ws, device):
    torch = _torch()
    if not (isinstance(ws, torch.Tensor) and ws.is_cuda and ws.device == device and ws.is_contiguous()):
        raise TypeError(f"workspace must be a contiguous CUDA tensor on {device}")
    return ws


def strides_of(t):
    """vitattn_strides of a [B, H, N, d] view (d contiguous)."""
    return Strides(t.stride(0), t.stride(1), t.stride(2))


def _dense(*ts):
    return all(t.is_contiguous() for t in ts)


def _default_scale(d, scale):
    return 1.0 / math.sqrt(d) if scale is None else float(scale)


VITATTN_BWD_ACCUMULATE_DQ = 1
VITATTN_BWD_STORE_DS = 2


def workspace_bytes_kv(B: int, H: int, Nq: int, Nk: int, d: int, flags: int = 0) -> int:
    """Workspace bytes of the backward pass for these sizes and flags (0 if invalid)."""
    return int(library().vitattn_bwd_workspace_bytes_kv(B, H, Nq, Nk, d, flags))


def _kv_shapes(q, k, v):
    B, H, Nq, d = q.shape
    if k.shape != v.shape or k.shape[:2] != q.shape[:2] or k.shape[3] != d:
        raise ValueError("k and v must be [B, H, Nk, d] with the B, H and d of q")
    return B, H, Nq, k.shape[2], d


def fwd(q, k, v, scale=None, out=None):
    """O (fp32 [B,H,Nq,d]) and LSE (fp32 [B,H,Nq]) of softmax(scale Q K^T) V;
    k and v may hold a different number of rows Nk (one key segment)."""
    torch = _torch()
    _as_input(q, "q")
    for t, n in ((k, "k"), (v, "v")):
        _as_input(t, n, q.device)
    B, H, Nq, Nk, d = _kv_shapes(q, k, v)
    if out is None:
        o = torch.empty((B, H, Nq, d), dtype=torch.float32, device=q.device)
        lse = torch.empty((B, H, Nq), dtype=torch.float32, device=q.device)
    else:
        o, lse = out
        _expect(o, "o", torch.float32, (B, H, Nq, d), q.device)
        _expect(lse, "lse", torch.float32, (B, H, Nq), q.device, dense=True)
    lib = library()
    if not _dense(q, k, v, o):
        st = lib.vitattn_fwd_strided(q.data_ptr(), strides_of(q), k.data_ptr(), strides_of(k), v.data_ptr(),
                                     strides_of(v), o.data_ptr(), strides_of(o), lse.data_ptr(), B, H, Nq, Nk, d,
                                     _default_scale(d, scale), _stream_ptr(q))
    elif Nq == Nk:
        st = lib.vitattn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), B, H, Nq, d,
                             _default_scale(d, scale), _stream_ptr(q))
    else:
        st = lib.vitattn_fwd_kv(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), B, H, Nq, Nk,
                                d, _default_scale(d, scale), _stream_ptr(q))
    _check(st)
    return o, lse


def _workspace(q, k, workspace, flags=0):
    torch = _torch()
    B, H, N, d = q.shape
    need = workspace_bytes_kv(B, H, N, k.shape[2], d, flags)
    if workspace is None:
        workspace = torch.empty(max(need, 4) // 4, dtype=torch.float32, device=q.device)
    _expect_workspace(workspace, q.device)
    return workspace, workspace.numel() * workspace.element_size()


def bwd(q, k, v, o, lse, dout, scale=None, workspace=None, out=None, accumulate_dq=False, store_ds=False):
    """dQ (fp32 [B,H,Nq,d]), dK, dV (fp32 [B,H,Nk,d]) for the upstream gradient
    dout (bf16). For one key segment pass the merged o and lse of all keys;
    accumulate_dq adds this segment's share to out[0] instead of overwriting.
    store_ds selects the dS mode (dQ from stored dS; a workspace of about
    B*H*Nq*Nk*2 bytes, see workspace_bytes_kv)."""
    torch = _torch()
    _as_input(q, "q")
    for t, n in ((k, "k"), (v, "v"), (dout, "dout")):
        _as_input(t, n, q.device)
    B, H, Nq, Nk, d = _kv_shapes(q, k, v)
    _expect(dout, "dout", torch.bfloat16, (B, H, Nq, d), q.device)
    _expect(o, "o", torch.float32, (B, H, Nq, d), q.device)
    _expect(lse, "lse", torch.float32, (B, H, Nq), q.device, dense=True)
    flags = (VITATTN_BWD_ACCUMULATE_DQ if accumulate_dq else 0) | (VITATTN_BWD_STORE_DS if store_ds else 0)
    ws, ws_bytes = _workspace(q, k, workspace, flags)
    if out is None:
        if accumulate_dq:
            raise ValueError("accumulate_dq needs out=(dq, dk, dv) holding the running dq")
        dq = torch.empty((B, H, Nq, d), dtype=torch.float32, device=q.device)
        dk, dv = (torch.empty((B, H, Nk, d), dtype=torch.float32, device=q.device) for _ in range(2))
    else:
        dq, dk, dv = out
        _expect(dq, "dq", torch.float32, (B, H, Nq, d), q.device)
        _expect(dk, "dk", torch.float32, (B, H, Nk, d), q.device)
        _expect(dv, "dv", torch.float32, (B, H, Nk, d), q.device)
    lib = library()
    if not _dense(q, k, v, o, dout, dq, dk, dv):
        st = lib.vitattn_bwd_strided(q.data_ptr(), strides_of(q), k.data_ptr(), strides_of(k), v.data_ptr(),
                                     strides_of(v), o.data_ptr(), strides_of(o), dout.data_ptr(), strides_of(dout),
                                     lse.data_ptr(), dq.data_ptr(), strides_of(dq), dk.data_ptr(), strides_of(dk),
                                     dv.data_ptr(), strides_of(dv), B, H, Nq, Nk, d, _default_scale(d, scale),
                                     flags, ws.data_ptr(), ws_bytes, _stream_ptr(q))
    elif Nq == Nk and flags == 0:
        st = lib.vitattn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), dout.data_ptr(), lse.data_ptr(),
                             dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), B, H, Nq, d, _default_scale(d, scale),
                             ws.data_ptr(), ws_bytes, _stream_ptr(q))
    else:
        st = lib.vitattn_bwd_kv(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), dout.data_ptr(),
                                lse.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), B, H, Nq, Nk, d,
                                _default_scale(d, scale), flags, ws.data_ptr(), ws_bytes, _stream_ptr(q))
    _check(st)
    return dq, dk, dv


VITATTN_NOALLOC_MAX_ROWS = 4194304


def bwd_noalloc(q, k, v, o, lse, dout, scale=None, out=None):
    """The backward pass through vitattn_bwd_noalloc (no workspace: the
    library's static scratch; B*H*N at most VITATTN_NOALLOC_MAX_ROWS; calls on
    one device must not overlap). Dense [B,H,N,d] operands; out=(dq, dk, dv)
    to write into existing tensors."""
    torch = _torch()
    B, H, N, d = _shape4(q, "q")
    dev = q.device
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (dout, "dout")):
        _expect(t, n, torch.bfloat16, (B, H, N, d), dev, dense=True)
    _expect(o, "o", torch.float32, (B, H, N, d), dev, dense=True)
    _expect(lse, "lse", torch.float32, (B, H, N), dev, dense=True)
    if out is None:
        dq, dk, dv = (torch.empty((B, H, N, d), dtype=torch.float32, device=dev) for _ in range(3))
    else:
        dq, dk, dv = out
        for t, n in ((dq, "dq"), (dk, "dk"), (dv, "dv")):
            _expect(t, n, torch.float32, (B, H, N, d), dev, dense=True)
    _check(library().vitattn_bwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), dout.data_ptr(),
                                         lse.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), B, H, N, d,
                                         _default_scale(d, scale), _stream_ptr(q)))
    return dq, dk, dv


def merge(o_parts, lse_parts, out=None):
    """Merge partial results over disjoint key segments: o_parts fp32
    [P,B,H,N,d], lse_parts fp32 [P,B,H,N] -> (o [B,H,N,d], lse [B,H,N])."""
    torch = _torch()
    if not (o_parts.is_cuda and o_parts.dtype == torch.float32 and o_parts.dim() == 5 and o_parts.is_contiguous()):
        raise TypeError("o_parts must be a contiguous 5-D float32 CUDA tensor [P, B, H, N, d]")
    P, B, H, N, d = o_parts.shape
    _expect(lse_parts, "lse_parts", torch.float32, (P, B, H, N), o_parts.device, dense=True)
    if out is None:
        o = torch.empty((B, H, N, d), dtype=torch.float32, device=o_parts.device)
        lse = torch.empty((B, H, N), dtype=torch.float32, device=o_parts.device)
    else:
        o, lse = out
        _expect(o, "o", torch.float32, (B, H, N, d), o_parts.device, dense=True)
        _expect(lse, "lse", torch.float32, (B, H, N), o_parts.device, dense=True)
    _check(library().vitattn_merge(o_parts.data_ptr(), lse_parts.data_ptr(), P, o.data_ptr(), lse.data_ptr(), B, H,
                                   N, d, _stream_ptr(o_parts)))
    return o, lse


def _stage_args(q, names_bf16, names_f32_rows, names_f32_out, lse, workspace, B, H, N, d):
    """Checks for the dense stage entry points: bf16 operands and fp32 outputs
    of shape [B, H, N, d], lse [B, H, N], all contiguous on q's device."""
    torch = _torch()
    dev = q.device
    for t, n in names_bf16:
        _expect(t, n, torch.bfloat16, (B, H, N, d), dev, dense=True)
    for t, n in names_f32_rows + names_f32_out:
        _expect(t, n, torch.float32, (B, H, N, d), dev, dense=True)
    if lse is not None:
        _expect(lse, "lse", torch.float32, (B, H, N), dev, dense=True)
    _expect_workspace(workspace, dev)


def _shape4(t, name):
    torch = _torch()
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dim() == 4):
        raise TypeError(f"{name} must be a 4-D CUDA tensor [B, H, N, d]")
    return tuple(int(n) for n in t.shape)


def bwd_rowdot(o, dout, lse, workspace):
    B, H, N, d = _shape4(dout, "dout")
    _stage_args(dout, [(dout, "dout")], [(o, "o")], [], lse, workspace, B, H, N, d)
    _check(library().vitattn_bwd_rowdot(o.data_ptr(), dout.data_ptr(), lse.data_ptr(), B, H, N, d, workspace.data_ptr(),
                                        workspace.numel() * workspace.element_size(), _stream_ptr(dout)))


def bwd_dkdv(q, k, v, dout, lse, dk, dv, workspace, scale=None):
    B, H, N, d = _shape4(q, "q")
    _stage_args(q, [(q, "q"), (k, "k"), (v, "v"), (dout, "dout")], [], [(dk, "dk"), (dv, "dv")], lse, workspace,
                B, H, N, d)
    _check(library().vitattn_bwd_dkdv(q.data_ptr(), k.data_ptr(), v.data_ptr(), dout.data_ptr(), lse.data_ptr(),
                                      dk.data_ptr(), dv.data_ptr(), B, H, N, d, _default_scale(d, scale),
                                      workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                      _stream_ptr(q)))


def bwd_dkdv_ds(q, k, v, dout, lse, dk, dv, workspace, scale=None):
    """The dK/dV stage of the dS mode (also writes the dS blocks into workspace)."""
    B, H, N, d = _shape4(q, "q")
    _stage_args(q, [(q, "q"), (k, "k"), (v, "v"), (dout, "dout")], [], [(dk, "dk"), (dv, "dv")], lse, workspace,
                B, H, N, d)
    _check(library().vitattn_bwd_dkdv_ds(q.data_ptr(), k.data_ptr(), v.data_ptr(), dout.data_ptr(), lse.data_ptr(),
                                         dk.data_ptr(), dv.data_ptr(), B, H, N, d, _default_scale(d, scale),
                                         workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                         _stream_ptr(q)))


def bwd_dq_from_ds(k, dq, workspace, scale=None):
    """The dQ stage of the dS mode, from the dS blocks bwd_dkdv_ds stored."""
    B, H, N, d = _shape4(k, "k")
    _stage_args(k, [(k, "k")], [], [(dq, "dq")], None, workspace, B, H, N, d)
    _check(library().vitattn_bwd_dq_from_ds(k.data_ptr(), dq.data_ptr(), B, H, N, d, _default_scale(d, scale),
                                            workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                            _stream_ptr(k)))


def bwd_dq(q, k, v, dout, lse, dq, workspace, scale=None):
    B, H, N, d = _shape4(q, "q")
    _stage_args(q, [(q, "q"), (k, "k"), (v, "v"), (dout, "dout")], [], [(dq, "dq")], lse, workspace, B, H, N, d)
    _check(library().vitattn_bwd_dq(q.data_ptr(), k.data_ptr(), v.data_ptr(), dout.data_ptr(), lse.data_ptr(),
                                    dq.data_ptr(), B, H, N, d, _default_scale(d, scale), workspace.data_ptr(),
                                    workspace.numel() * workspace.element_size(), _stream_ptr(q)))


def _rows(t, lead, name):
    """(leading dims, row shape, row_bytes) of a contiguous CUDA tensor whose
    first `lead` dims index rows."""
    if not (t.is_cuda and t.is_contiguous() and t.dim() > lead):
        raise TypeError(f"{name} must be a contiguous CUDA tensor with more than {lead} dims")
    row_shape = tuple(t.shape[lead:])
    row_bytes = t.element_size()
    for n in row_shape:
        row_bytes *= n
    return tuple(t.shape[:lead]), row_shape, row_bytes


def _ulysses(status, dst):
    _check(status)
    return dst


def _dst(out, shape, like):
    """`out` if given (checked), else a new tensor of `shape` like `like`."""
    torch = _torch()
    if out is None:
        return torch.empty(shape, dtype=like.dtype, device=like.device)
    if not (isinstance(out, torch.Tensor) and out.is_cuda and out.device == like.device and out.dtype == like.dtype
            and out.is_contiguous() and tuple(out.shape) == tuple(shape)):
        raise TypeError(f"out must be a contiguous {like.dtype} CUDA tensor of shape {tuple(shape)} on {like.device}")
    return out


def ulysses_pack(x, P, out=None):
    """x [B, Nl, H, *row] -> send [P, B, H/P, Nl, *row] (head group p in chunk p)."""
    (B, Nl, H), row, rb = _rows(x, 3, "x")
    if P < 1 or H % P != 0:
        raise ValueError("H must be a multiple of P")
    send = _dst(out, (P, B, H // P, Nl) + row, x)
    return _ulysses(library().vitattn_ulysses_pack(x.data_ptr(), send.data_ptr(), B, Nl, H, P, rb, _stream_ptr(x)),
                    send)


def ulysses_unpack(recv, out=None):
    """recv [P, B, Hl, Nl, *row] (chunk r from rank r) -> y [B, Hl, P*Nl, *row]."""
    (P, B, Hl, Nl), row, rb = _rows(recv, 4, "recv")
    y = _dst(out, (B, Hl, P * Nl) + row, recv)
    return _ulysses(library().vitattn_ulysses_unpack(recv.data_ptr(), y.data_ptr(), B, Nl, Hl * P, P, rb,
                                                     _stream_ptr(recv)), y)


def ulysses_pack_out(y, P, out=None):
    """y [B, Hl, P*Nl, *row] -> send [P, B, Hl, Nl, *row] (the inverse of unpack)."""
    (B, Hl, N), row, rb = _rows(y, 3, "y")
    if P < 1 or N % P != 0:
        raise ValueError("the sequence length must be divisible by P")
    send = _dst(out, (P, B, Hl, N // P) + row, y)
    return _ulysses(library().vitattn_ulysses_pack_out(y.data_ptr(), send.data_ptr(), B, N // P, Hl * P, P, rb,
                                                       _stream_ptr(y)), send)


def ulysses_unpack_out(recv, out=None):
    """recv [P, B, Hl, Nl, *row] -> x [B, Nl, P*Hl, *row] (the inverse of pack)."""
    (P, B, Hl, Nl), row, rb = _rows(recv, 4, "recv")
    x = _dst(out, (B, Nl, P * Hl) + row, recv)
    return _ulysses(library().vitattn_ulysses_unpack_out(recv.data_ptr(), x.data_ptr(), B, Nl, Hl * P, P, rb,
                                                         _stream_ptr(recv)), x)


def _agg_shapes(q, k, v):
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        if not (isinstance(t, _torch().Tensor) and t.is_cuda and t.dtype == _torch().bfloat16 and t.is_contiguous()
                and t.device == k.device):
            raise TypeError(f"{n} must be a contiguous bfloat16 CUDA tensor on the device of k")
    if q.dim() != 2 or k.dim() != 4 or k.shape != v.shape or k.shape[1] != q.shape[0] or k.shape[3] != q.shape[1]:
        raise ValueError("q must be [H, d] and k, v [M, H, C, d]")
    M, H, C, d = k.shape
    return M, H, C, d


def agg_fwd(q, k, v, scale=None):
    """Channel aggregation: o (fp32 [M,H,d]) and lse (fp32 [M,H]) of one shared
    query per head (q [H,d]) over each patch's C channel keys (k, v [M,H,C,d])."""
    torch = _torch()
    M, H, C, d = _agg_shapes(q, k, v)
    o = torch.empty((M, H, d), dtype=torch.float32, device=k.device)
    lse = torch.empty((M, H), dtype=torch.float32, device=k.device)
    _check(library().vitattn_agg_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), M, H, C,
                                     d, _default_scale(d, scale), _stream_ptr(k)))
    return o, lse


def agg_bwd(q, k, v, o, lse, dout, scale=None):
    """Gradients of the channel aggregation: dq (fp32 [H,d], summed over all
    patches), dk and dv (fp32 [M,H,C,d])."""
    torch = _torch()
    M, H, C, d = _agg_shapes(q, k, v)
    _expect(dout, "dout", torch.bfloat16, (M, H, d), k.device, dense=True)
    _expect(o, "o", torch.float32, (M, H, d), k.device, dense=True)
    _expect(lse, "lse", torch.float32, (M, H), k.device, dense=True)
    lib = library()
    wsb = int(lib.vitattn_agg_bwd_workspace_bytes(M, H, C, d))
    ws = torch.empty(max(wsb, 4) // 4, dtype=torch.float32, device=k.device)
    dq = torch.empty((H, d), dtype=torch.float32, device=k.device)
    dk = torch.empty((M, H, C, d), dtype=torch.float32, device=k.device)
    dv = torch.empty_like(dk)
    _check(lib.vitattn_agg_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), dout.data_ptr(),
                               lse.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), M, H, C, d,
                               _default_scale(d, scale), ws.data_ptr(), ws.numel() * 4, _stream_ptr(k)))
    return dq, dk, dv
