"""ctypes binding of libmas (include/mas.h); argument marshalling only.

Every step of the alignment runs in the HIP kernels of ``libmas.so``; this
module checks tensor dtypes, devices and shapes, passes raw device pointers
and the current HIP stream, and turns non-zero status codes into exceptions.
PyTorch is used only for device memory and streams.  When the library is not
built the binding raises instead of computing anything another way.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmas.so")

MAS_OK = 0
STATUS_NAMES = {0: "MAS_OK", 1: "MAS_ERR_NULL_POINTER", 2: "MAS_ERR_BAD_SHAPE", 3: "MAS_ERR_WORKSPACE", 4: "MAS_ERR_HIP",
                5: "MAS_ERR_SCRATCH", 6: "MAS_ERR_BAD_VALUE"}
STATIC_SCRATCH_BYTES = 80 << 20  # MAS_STATIC_SCRATCH_BYTES
ITEM_OK, ITEM_EMPTY, ITEM_INFEASIBLE, ITEM_OUT_OF_RANGE, ITEM_SYNC_TIMEOUT, ITEM_BAD_WORKSPACE = 0, 1, 2, 3, 4, 5

# Every function declared in include/mas.h, with its ctypes signature.
_P, _I32, _SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
SIGNATURES = {
    "mas_workspace_bytes": ([_I32, _I32, _I32], _SZ),
    "mas_workspace_init": ([_P, _SZ, _P], ctypes.c_int),
    "mas_search": ([_P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _P, _P, _SZ, _P], ctypes.c_int),
    "mas_expand_path": ([_P, _I32, _I32, _I32, _P, _P], ctypes.c_int),
    "mas_expand_text": ([_P, _P, _I32, _I32, _I32, _I32, _I32, _P, _P], ctypes.c_int),
    "mas_loglik": ([_P, _P, _P, _P, _P, _I32, _I32, _I32, _I32, _P, _P], ctypes.c_int),
    "mas_forward_ex": ([_P, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _SZ, _P], ctypes.c_int),
    "mas_forward_sentinel": ([_P, _P, _P, _P, _I32, _I32, _I32, ctypes.c_float, _P, _P, _P, _SZ, _P], ctypes.c_int),
    "mas_forward": ([_P, _P, _P, _P, _I32, _I32, _I32, _P], ctypes.c_int),
    "mas_forward_static": ([_P, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P], ctypes.c_int),
    "mas_status_string": ([ctypes.c_int], ctypes.c_char_p),
    "mas_version": ([], ctypes.c_int),
}


class MasError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn} failed: {STATUS_NAMES.get(code, code)}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libmas.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -c \"import __graft_entry__ as g; g.build()\"` "
                "or `python paper_2409_07704_amd/build.py`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def _check(fn: str, code: int) -> None:
    if code != MAS_OK:
        raise MasError(fn, code)


def _dev_ptr(t: torch.Tensor | None, name: str, dtype: torch.dtype, shape=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a device (cuda/hip) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t.data_ptr()


def _stream(stream, device) -> int:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def mas_workspace_bytes(B: int, T: int, S: int) -> int:
    return int(lib().mas_workspace_bytes(B, T, S))


def mas_status_string(code: int) -> str:
    return lib().mas_status_string(code).decode()


def mas_version() -> int:
    return int(lib().mas_version())


class Workspace:
    """Device workspace for mas_search / mas_forward_ex, initialised once."""

    def __init__(self, B: int, T: int, S: int, device=None, stream=None):
        n = mas_workspace_bytes(B, T, S)
        if n == 0:
            raise ValueError(f"invalid shape B={B} T={T} S={S}")
        self.shape = (B, T, S)
        self.nbytes = n
        self._buf = torch.empty(n + 256, dtype=torch.uint8, device=device or "cuda")
        off = (-self._buf.data_ptr()) % 256
        self.ptr = self._buf.data_ptr() + off
        self.device = self._buf.device
        mas_workspace_init(self.ptr, self.nbytes, stream=stream, device=self.device)

    def fits(self, B: int, T: int, S: int) -> bool:
        return mas_workspace_bytes(B, T, S) <= self.nbytes


def mas_workspace_init(ptr: int, nbytes: int, stream=None, device=None) -> None:
    _check("mas_workspace_init", lib().mas_workspace_init(ptr, nbytes, _stream(stream, device)))


def _batch(value, t_x, t_y):
    if value.dim() != 3:
        raise ValueError("value must be [B, T, S]")
    B, T, S = value.shape
    pv = _dev_ptr(value, "value", torch.float32)
    px = _dev_ptr(t_x, "t_x", torch.int32, (B,))
    py = _dev_ptr(t_y, "t_y", torch.int32, (B,))
    return B, T, S, pv, px, py


def _workspace(ws, B, T, S, device, stream):
    if ws is None:
        ws = Workspace(B, T, S, device=device, stream=stream)
    if not ws.fits(B, T, S):
        raise ValueError("workspace too small for this batch")
    return ws


def mas_search(value, t_x, t_y, row_start_out=None, score_out=None, item_status_out=None, workspace=None, stream=None,
               durations_out=None):
    """Forward pass + backtrack without the dense path; returns row_start
    [B, T+1] int32 (see mas.h).  durations_out [B, T] int32 is optional."""
    B, T, S, pv, px, py = _batch(value, t_x, t_y)
    if row_start_out is None:
        row_start_out = torch.empty((B, T + 1), dtype=torch.int32, device=value.device)
    prs = _dev_ptr(row_start_out, "row_start_out", torch.int32, (B, T + 1))
    pdu = _dev_ptr(durations_out, "durations_out", torch.int32, (B, T))
    psc = _dev_ptr(score_out, "score_out", torch.float32, (B,))
    pst = _dev_ptr(item_status_out, "item_status_out", torch.int32, (B,))
    s = _stream(stream, value.device)
    ws = _workspace(workspace, B, T, S, value.device, s)
    _check("mas_search", lib().mas_search(pv, px, py, B, T, S, prs, pdu, psc, pst, ws.ptr, ws.nbytes, s))
    return row_start_out


def mas_expand_path(row_start, S: int, path_out=None, stream=None):
    """Dense [B, T, S] uint8 path from row_start [B, T+1]."""
    if row_start.dim() != 2:
        raise ValueError("row_start must be [B, T+1]")
    B, T1 = row_start.shape
    T = T1 - 1
    prs = _dev_ptr(row_start, "row_start", torch.int32)
    if path_out is None:
        path_out = torch.empty((B, T, S), dtype=torch.uint8, device=row_start.device)
    pp = _dev_ptr(path_out, "path_out", torch.uint8, (B, T, S))
    _check("mas_expand_path", lib().mas_expand_path(prs, B, T, S, pp, _stream(stream, row_start.device)))
    return path_out


def mas_expand_text(text, row_start, S: int, out=None, stream=None):
    """Aligned text grid [B, S, C] from text [B, T, C] (any 1, 2, 4 or 8-byte
    dtype) and row_start [B, T+1]: frame j copies the text row whose segment
    holds it, zeros where none does."""
    if text.dim() != 3 or row_start.dim() != 2:
        raise ValueError("text must be [B, T, C] and row_start [B, T+1]")
    B, T, C = text.shape
    prs = _dev_ptr(row_start, "row_start", torch.int32, (B, T + 1))
    pt = _dev_ptr(text, "text", text.dtype)
    if out is None:
        out = torch.empty((B, S, C), dtype=text.dtype, device=text.device)
    po = _dev_ptr(out, "out", text.dtype, (B, S, C))
    _check("mas_expand_text", lib().mas_expand_text(pt, prs, B, T, S, C, text.element_size(), po,
                                                    _stream(stream, text.device)))
    return out


def mas_loglik(mu, log_sigma, z, t_x, t_y, value_out=None, stream=None):
    """Gaussian log-likelihood value [B, T, S] fp32 of frames z [B, S, D]
    under text-token Gaussians mu, log_sigma [B, T, D] (log_sigma None: unit
    variance), written for the cells of each item's feasible band only (the
    cells MAS reads); other cells of value_out are left as they are."""
    if mu.dim() != 3 or z.dim() != 3:
        raise ValueError("mu must be [B, T, D] and z [B, S, D]")
    B, T, D = mu.shape
    S = z.shape[1]
    pm = _dev_ptr(mu, "mu", torch.float32)
    pl = _dev_ptr(log_sigma, "log_sigma", torch.float32, (B, T, D))
    pz = _dev_ptr(z, "z", torch.float32, (B, S, D))
    px = _dev_ptr(t_x, "t_x", torch.int32, (B,))
    py = _dev_ptr(t_y, "t_y", torch.int32, (B,))
    if value_out is None:
        value_out = torch.empty((B, T, S), dtype=torch.float32, device=mu.device)
    pv = _dev_ptr(value_out, "value_out", torch.float32, (B, T, S))
    _check("mas_loglik", lib().mas_loglik(pm, pl, pz, px, py, B, T, S, D, pv, _stream(stream, mu.device)))
    return value_out


def mas_forward_ex(value, t_x, t_y, path_out=None, score_out=None, item_status_out=None, workspace=None, stream=None):
    """Full alignment into path_out [B, T, S] uint8 with a caller workspace."""
    B, T, S, pv, px, py = _batch(value, t_x, t_y)
    if path_out is None:
        path_out = torch.empty((B, T, S), dtype=torch.uint8, device=value.device)
    pp = _dev_ptr(path_out, "path_out", torch.uint8, (B, T, S))
    psc = _dev_ptr(score_out, "score_out", torch.float32, (B,))
    pst = _dev_ptr(item_status_out, "item_status_out", torch.int32, (B,))
    s = _stream(stream, value.device)
    ws = _workspace(workspace, B, T, S, value.device, s)
    _check("mas_forward_ex", lib().mas_forward_ex(pv, px, py, pp, B, T, S, psc, pst, ws.ptr, ws.nbytes, s))
    return path_out


def mas_forward_sentinel(value, t_x, t_y, sentinel, path_out=None, score_out=None, item_status_out=None,
                         workspace=None, stream=None):
    """Full alignment in the legacy-sentinel mode: the cells Algorithm 1
    masks hold the finite negative `sentinel` (e.g. -1e9) instead of -inf."""
    B, T, S, pv, px, py = _batch(value, t_x, t_y)
    if path_out is None:
        path_out = torch.empty((B, T, S), dtype=torch.uint8, device=value.device)
    pp = _dev_ptr(path_out, "path_out", torch.uint8, (B, T, S))
    psc = _dev_ptr(score_out, "score_out", torch.float32, (B,))
    pst = _dev_ptr(item_status_out, "item_status_out", torch.int32, (B,))
    s = _stream(stream, value.device)
    ws = _workspace(workspace, B, T, S, value.device, s)
    _check("mas_forward_sentinel",
           lib().mas_forward_sentinel(pv, px, py, pp, B, T, S, float(sentinel), psc, pst, ws.ptr, ws.nbytes, s))
    return path_out


def mas_forward_static(value, t_x, t_y, path_out=None, score_out=None, item_status_out=None, stream=None):
    """Full alignment with the library's static per-device scratch as the
    workspace: allocates no device memory (see mas.h for the limit)."""
    B, T, S, pv, px, py = _batch(value, t_x, t_y)
    if path_out is None:
        path_out = torch.empty((B, T, S), dtype=torch.uint8, device=value.device)
    pp = _dev_ptr(path_out, "path_out", torch.uint8, (B, T, S))
    psc = _dev_ptr(score_out, "score_out", torch.float32, (B,))
    pst = _dev_ptr(item_status_out, "item_status_out", torch.int32, (B,))
    _check("mas_forward_static", lib().mas_forward_static(pv, px, py, pp, B, T, S, psc, pst, _stream(stream, value.device)))
    return path_out


def mas_forward(value, t_x, t_y, path_out=None, stream=None):
    """Full alignment; the library allocates its workspace stream-ordered."""
    B, T, S, pv, px, py = _batch(value, t_x, t_y)
    if path_out is None:
        path_out = torch.empty((B, T, S), dtype=torch.uint8, device=value.device)
    pp = _dev_ptr(path_out, "path_out", torch.uint8, (B, T, S))
    _check("mas_forward", lib().mas_forward(pv, px, py, pp, B, T, S, _stream(stream, value.device)))
    return path_out
