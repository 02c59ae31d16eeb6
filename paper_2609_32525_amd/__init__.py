"""Python binding of libflashslice (the fused slice -> token mix -> deslice path, HIP/gfx950).

Argument marshalling only: every step of the path runs in the library's kernels. Tensors
(torch device tensors) are passed as raw device pointers with ``data_ptr()``; PyTorch only
provides memory and the current stream. There is no fallback: if the library is not built,
every call raises.

Function names and argument order follow include/flashslice.h.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

__all__ = [
    "F32", "BF16", "MIX_IDENTITY", "MIX_LINEAR_G", "MIX_LINEAR_C", "MIX_ATTN",
    "FsError", "Problem", "MixDesc", "lib", "lib_path", "workspace_bytes", "slice_fwd",
    "slice_fwd_noalloc", "mix",
    "mix_bwd", "deslice_fwd", "deslice_stats_fwd", "slice_deslice_bwd", "untied_bwd",
    "linearno_slice_fwd", "linearno_bwd", "status_string", "last_hip_error",
    "set_pass_events", "EXPORTED", "PASS_SLICE", "PASS_DESLICE", "PASS_BWD_A", "PASS_BWD_B",
]

F32, BF16 = 0, 1
MIX_IDENTITY, MIX_LINEAR_G, MIX_LINEAR_C, MIX_ATTN = 0, 1, 2, 3

EXPORTED = ("fs_workspace_bytes", "fs_slice_fwd", "fs_slice_fwd_noalloc", "fs_mix", "fs_mix_bwd", "fs_deslice_fwd",
            "fs_deslice_stats_fwd", "fs_slice_deslice_bwd", "fs_untied_bwd",
            "fs_linearno_slice_fwd", "fs_linearno_bwd", "fs_set_pass_events", "fs_status_string",
            "fs_last_hip_error")

PASS_SLICE, PASS_DESLICE, PASS_BWD_A, PASS_BWD_B = 0, 1, 2, 3

_HERE = os.path.dirname(os.path.abspath(__file__))


def lib_path() -> str:
    return os.path.join(_HERE, "libflashslice.so")


class Problem(ctypes.Structure):
    """fs_problem: B, N, H, D, V, G, dtype (F32/BF16), eps, ws_per_head."""
    _fields_ = [("B", ctypes.c_int64), ("N", ctypes.c_int64), ("H", ctypes.c_int32),
                ("D", ctypes.c_int32), ("V", ctypes.c_int32), ("G", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("eps", ctypes.c_float),
                ("ws_per_head", ctypes.c_int32)]

    @classmethod
    def make(cls, B, N, H, D, V, G, dtype=F32, eps=1e-5, ws_per_head=0) -> "Problem":
        return cls(B, N, H, D, V, G, dtype, eps, ws_per_head)


class MixDesc(ctypes.Structure):
    """fs_mix_desc: kind, a_per_head, A, Wc, Wq, Wk, Wv (device pointers), scale."""
    _fields_ = [("kind", ctypes.c_int32), ("a_per_head", ctypes.c_int32),
                ("A", ctypes.c_void_p), ("Wc", ctypes.c_void_p), ("Wq", ctypes.c_void_p),
                ("Wk", ctypes.c_void_p), ("Wv", ctypes.c_void_p), ("scale", ctypes.c_float)]

    @classmethod
    def make(cls, kind, A=None, Wc=None, Wq=None, Wk=None, Wv=None, scale=1.0,
             a_per_head=0) -> "MixDesc":
        return cls(kind, a_per_head, _ptr(A), _ptr(Wc), _ptr(Wq), _ptr(Wk), _ptr(Wv), scale)


class FsError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = status_string(status)
        if status == -9:
            msg += f" (hipError_t {last_hip_error()})"
        super().__init__(f"{where}: {msg} [{status}]")


_LIB = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built (no fallback exists)."""
    global _LIB
    if _LIB is None:
        path = lib_path()
        if not os.path.exists(path):
            raise RuntimeError(f"libflashslice.so is not built ({path}); run "
                               "`python -c 'import __graft_entry__ as g; g.build()'`")
        L = ctypes.CDLL(path)
        P, S = ctypes.c_void_p, ctypes.c_size_t
        prob = ctypes.POINTER(Problem)
        mixp = ctypes.POINTER(MixDesc)
        L.fs_workspace_bytes.argtypes = [prob, ctypes.c_int, ctypes.POINTER(S)]
        L.fs_slice_fwd.argtypes = [prob, P, P, P, P, P, P, P, P, P, S, P]
        L.fs_slice_fwd_noalloc.argtypes = [prob, P, P, P, P, P, P, P, P, P]
        L.fs_mix.argtypes = [prob, mixp, P, P, P, P]
        L.fs_mix_bwd.argtypes = [prob, mixp, P, P, P, P, P, P, S, P]
        L.fs_deslice_fwd.argtypes = [prob, P, P, P, P, P, P, P, P]
        L.fs_deslice_stats_fwd.argtypes = [prob, P, P, P, P, P, P, P, P]
        L.fs_slice_deslice_bwd.argtypes = [prob, mixp] + [P] * 19 + [S, P]
        L.fs_untied_bwd.argtypes = [prob, mixp] + [P] * 26 + [S, P]
        L.fs_linearno_slice_fwd.argtypes = [prob] + [P] * 8 + [S, P]
        L.fs_linearno_bwd.argtypes = [prob, mixp] + [P] * 25 + [S, P]
        L.fs_status_string.argtypes = [ctypes.c_int]
        L.fs_status_string.restype = ctypes.c_char_p
        L.fs_last_hip_error.argtypes = []
        L.fs_set_pass_events.argtypes = [ctypes.c_int, P, P]
        for name in EXPORTED:
            if name not in ("fs_status_string",):
                getattr(L, name).restype = ctypes.c_int
        _LIB = L
    return _LIB


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _nbytes(t) -> int:
    if t is None:
        return 0
    return t.numel() * t.element_size()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int, where: str) -> None:
    if status != 0:
        raise FsError(status, where)


def status_string(status: int) -> str:
    return lib().fs_status_string(status).decode()


def last_hip_error() -> int:
    return lib().fs_last_hip_error()


def set_pass_events(pass_id: int, before=None, after=None) -> None:
    """Record torch.cuda.Event objects (or raw hipEvent_t ints) around one streaming pass of
    later calls on this thread; pass_id = -1 clears."""
    def ev(e):
        if e is None or isinstance(e, int):
            return e
        return e.cuda_event
    _check(lib().fs_set_pass_events(pass_id, ev(before), ev(after)), "fs_set_pass_events")


def workspace_bytes(prob: Problem, for_backward) -> int:
    """for_backward: 0 / False forward, 1 / True backward, 2 untied backward, 3 LinearNO
    slice, 4 LinearNO backward."""
    out = ctypes.c_size_t(0)
    _check(lib().fs_workspace_bytes(ctypes.byref(prob), int(for_backward),
                                    ctypes.byref(out)), "fs_workspace_bytes")
    return out.value


def slice_fwd(prob, x, fx, Ws, b, tau, z, s, lse, ws, ws_bytes=None, stream=None) -> None:
    _check(lib().fs_slice_fwd(ctypes.byref(prob), _ptr(x), _ptr(fx), _ptr(Ws), _ptr(b),
                              _ptr(tau), _ptr(z), _ptr(s), _ptr(lse), _ptr(ws),
                              _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream)),
           "fs_slice_fwd")


def slice_fwd_noalloc(prob, x, fx, Ws, b, tau, z, s, lse, stream=None) -> None:
    _check(lib().fs_slice_fwd_noalloc(ctypes.byref(prob), _ptr(x), _ptr(fx), _ptr(Ws), _ptr(b),
                                      _ptr(tau), _ptr(z), _ptr(s), _ptr(lse), _stream(stream)),
           "fs_slice_fwd_noalloc")


def mix(prob, mixdesc, z, zmix, attn=None, stream=None) -> None:
    _check(lib().fs_mix(ctypes.byref(prob), ctypes.byref(mixdesc), _ptr(z), _ptr(zmix),
                        _ptr(attn), _stream(stream)), "fs_mix")


def mix_bwd(prob, mixdesc, z, attn, dzmix, dz, dmix, ws, ws_bytes=None, stream=None) -> None:
    _check(lib().fs_mix_bwd(ctypes.byref(prob), ctypes.byref(mixdesc), _ptr(z), _ptr(attn),
                            _ptr(dzmix), _ptr(dz), _ptr(dmix), _ptr(ws),
                            _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream)),
           "fs_mix_bwd")


def deslice_fwd(prob, x, Ws, b, tau, zmix, lse, out, stream=None) -> None:
    _check(lib().fs_deslice_fwd(ctypes.byref(prob), _ptr(x), _ptr(Ws), _ptr(b), _ptr(tau),
                                _ptr(zmix), _ptr(lse), _ptr(out), _stream(stream)),
           "fs_deslice_fwd")


def deslice_stats_fwd(prob, x, Ws, b, tau, zmix, lse_out, out, stream=None) -> None:
    _check(lib().fs_deslice_stats_fwd(ctypes.byref(prob), _ptr(x), _ptr(Ws), _ptr(b),
                                      _ptr(tau), _ptr(zmix), _ptr(lse_out), _ptr(out),
                                      _stream(stream)),
           "fs_deslice_stats_fwd")


def slice_deslice_bwd(prob, mixdesc, x, fx, Ws, b, tau, z, s, zmix, attn, lse, dout, dx, dfx,
                      dWs, db, dtau, dmix, dzmix_out, ws, ws_bytes=None, stream=None) -> None:
    _check(lib().fs_slice_deslice_bwd(
        ctypes.byref(prob), ctypes.byref(mixdesc), _ptr(x), _ptr(fx), _ptr(Ws), _ptr(b),
        _ptr(tau), _ptr(z), _ptr(s), _ptr(zmix), _ptr(attn), _ptr(lse), _ptr(dout), _ptr(dx),
        _ptr(dfx), _ptr(dWs), _ptr(db), _ptr(dtau), _ptr(dmix), _ptr(dzmix_out), _ptr(ws),
        _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream)),
        "fs_slice_deslice_bwd")


def untied_bwd(prob, mixdesc, x, fx, Ws, b, tau, Wd, bd, taud, z, s, zmix, attn, lse, lse_d,
               dout, dx, dfx, dWs, db, dtau, dWd, dbd, dtaud, dmix, dzmix_out, ws,
               ws_bytes=None, stream=None) -> None:
    _check(lib().fs_untied_bwd(
        ctypes.byref(prob), ctypes.byref(mixdesc), _ptr(x), _ptr(fx), _ptr(Ws), _ptr(b),
        _ptr(tau), _ptr(Wd), _ptr(bd), _ptr(taud), _ptr(z), _ptr(s), _ptr(zmix), _ptr(attn),
        _ptr(lse), _ptr(lse_d), _ptr(dout), _ptr(dx), _ptr(dfx), _ptr(dWs), _ptr(db),
        _ptr(dtau), _ptr(dWd), _ptr(dbd), _ptr(dtaud), _ptr(dmix), _ptr(dzmix_out), _ptr(ws),
        _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream)),
        "fs_untied_bwd")


def linearno_slice_fwd(prob, x, fx, Ws, b, tau, z, clse, ws, ws_bytes=None, stream=None) -> None:
    _check(lib().fs_linearno_slice_fwd(ctypes.byref(prob), _ptr(x), _ptr(fx), _ptr(Ws), _ptr(b),
                                       _ptr(tau), _ptr(z), _ptr(clse), _ptr(ws),
                                       _nbytes(ws) if ws_bytes is None else ws_bytes,
                                       _stream(stream)),
           "fs_linearno_slice_fwd")


def linearno_bwd(prob, mixdesc, x, fx, Ws, b, tau, Wd, bd, taud, z, clse, zmix, attn, lse_d,
                 dout, dx, dfx, dWs, db, dtau, dWd, dbd, dtaud, dmix, dzmix_out, ws,
                 ws_bytes=None, stream=None) -> None:
    _check(lib().fs_linearno_bwd(
        ctypes.byref(prob), ctypes.byref(mixdesc), _ptr(x), _ptr(fx), _ptr(Ws), _ptr(b),
        _ptr(tau), _ptr(Wd), _ptr(bd), _ptr(taud), _ptr(z), _ptr(clse), _ptr(zmix), _ptr(attn),
        _ptr(lse_d), _ptr(dout), _ptr(dx), _ptr(dfx), _ptr(dWs), _ptr(db), _ptr(dtau), _ptr(dWd),
        _ptr(dbd), _ptr(dtaud), _ptr(dmix), _ptr(dzmix_out), _ptr(ws),
        _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream)),
        "fs_linearno_bwd")
