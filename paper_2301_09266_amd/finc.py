"""Python binding of libfinc (include/finc.h): argument marshalling only.

Every function takes and returns torch tensors on the current HIP device and
enqueues on torch's current stream; all arithmetic runs in the HIP kernels of
csrc/finc.hip.  There is no fallback: if the library is missing or a call
fails, FincError is raised.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "libfinc.so")

TL, TR, BL, BR = 0, 1, 2, 3
OK, EINVAL, ESINGULAR, EUNSUPPORTED, EHIP = 0, -1, -2, -3, -4
PLAN_LAYER, PLAN_UNIT, PLAN_SPLIT, PLAN_STACK = 0, 1, 2, 3

_vp = ctypes.c_void_p
_i = ctypes.c_int
_sz = ctypes.c_size_t

# name -> (restype, argtypes); mirrors include/finc.h
SIGNATURES = {
    "finc_version": (_i, []),
    "finc_strerror": (ctypes.c_char_p, [_i]),
    "finc_inverse_plan": (_i, [_i, _i, _i, _i, _i, _i, _i, ctypes.POINTER(_i), _i]),
    "finc_forward_plan": (_i, [_i, _i, _i, _i, _i, _i, _i, ctypes.POINTER(_i)]),
    "finc_inverse_steps": (_i, [_i, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _i, _vp]),
    "finc_inverse_timeline": (_i, [_i, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _i, _vp]),
    "finc_banded_plan": (_i, [_i, _i, _i, _i, ctypes.POINTER(_i)]),
    "finc_banded_workspace_bytes": (_sz, [_i, _i, _i, _i, _i, _i]),
    "finc_inverse_banded": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _vp]),
    "finc_unit_inverse_banded": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _vp, _vp]),
    "finc_workspace_bytes": (_sz, [_i, _i, _i]),
    "finc_prepare": (_i, [_vp, _i, ctypes.POINTER(_i), _i, _i, _vp, _vp]),
    "finc_forward": (_i, [_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp]),
    "finc_logdet": (_i, [_vp, _i, _i, _i, _i, _i, _vp, _vp]),
    "finc_inverse": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _vp]),
    "finc_inverse_prepared": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp]),
    "finc_inverse_noalloc": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp]),
    "finc_backward_workspace_bytes": (_sz, [_i, _i, _i, _i, _i]),
    "finc_backward": (_i, [_vp, _vp, _vp, _vp, _vp, ctypes.c_double, _i, _i, _i, _i, _i, _i,
                           _vp, _vp]),
    "finc_unit_backward_workspace_bytes": (_sz, [_i, _i, _i, _i, _i]),
    "finc_unit_backward": (_i, [_vp, _vp, _vp, _vp, _vp, ctypes.c_double, _i, _i, _i, _i, _i,
                                _vp, _vp]),
    "finc_split_backward_workspace_bytes": (_sz, [_i, _i, _i, _i, _i]),
    "finc_split_backward": (_i, [_vp, _vp, _vp, _vp, _vp, ctypes.c_double, _i, _i, _i, _i, _i,
                                 _vp, _vp]),
    "finc_actnorm_backward_workspace_bytes": (_sz, [_i, _i, _i, _i]),
    "finc_actnorm_backward": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_double, _i, _i, _i,
                                   _i, _vp, _vp]),
    "finc_gauss_nll": (_i, [ctypes.POINTER(_vp), ctypes.POINTER(ctypes.c_longlong), _i, _i, _vp,
                            _vp, _vp, _vp]),
    "finc_stack_train_workspace_bytes": (_sz, [_i, _i, _i, _i, _i, _i, _i]),
    "finc_stack_forward": (_i, [_vp, ctypes.POINTER(_vp), _vp, _vp, _vp, _vp, _i, _i, _i, _i,
                                _i, _i, _i, _vp, _vp]),
    "finc_stack_backward": (_i, [_vp, ctypes.POINTER(_vp), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                 ctypes.c_double, _i, _i, _i, _i, _i, _i, _i, _vp, _vp]),
    "finc_unit_forward": (_i, [_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _vp]),
    "finc_unit_logdet": (_i, [_vp, _i, _i, _i, _i, _vp, _vp]),
    "finc_unit_inverse": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _vp, _vp]),
    "finc_unit_inverse_prepared": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _vp]),
    "finc_split_forward": (_i, [_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _vp]),
    "finc_split_logdet": (_i, [_vp, _i, _i, _i, _i, _vp, _vp]),
    "finc_split_inverse": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _vp, _vp]),
    "finc_split_inverse_prepared": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _vp]),
    "finc_stack_workspace_bytes": (_sz, [_i, _i, _i, _i]),
    "finc_stack_inverse": (_i, [ctypes.POINTER(_vp), _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i,
                                _i, _i, _vp, _vp]),
    "finc_stack_prepare": (_i, [_vp, _i, _i, _i, _i, _vp, _vp]),
    "finc_stack_inverse_prepared": (_i, [ctypes.POINTER(_vp), _vp, _vp, _vp, _vp, _i, _i,
                                         _i, _i, _i, _i, _i, _vp]),
    "finc_step_param_count": (_sz, [_i, _i, _i]),
    "finc_step_prepared_bytes": (_sz, [_i, _i]),
    "finc_step_workspace_bytes": (_sz, [_i, _i, _i, _i, _i]),
    "finc_step_prepare": (_i, [_vp, _i, _i, _i, _vp, _vp]),
    "finc_step_forward": (_i, [_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _vp]),
    "finc_step_inverse": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _vp]),
    "finc_flow_param_count": (_sz, [_i, _i, _i, _i, _i]),
    "finc_flow_prepared_bytes": (_sz, [_i, _i, _i, _i]),
    "finc_flow_workspace_bytes": (_sz, [_i, _i, _i, _i, _i, _i]),
    "finc_flow_prepare": (_i, [_vp, _i, _i, _i, _i, _i, _vp, _vp]),
    "finc_flow_forward": (_i, [_vp, ctypes.POINTER(_vp), _vp, _vp, _vp, _i, _i, _i, _i, _i, _i,
                               _i, _i, _vp, _vp]),
    "finc_flow_sample": (_i, [ctypes.POINTER(_vp), _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i,
                              _i, _vp, _vp]),
    "finc_conv1x1_workspace_bytes": (_sz, [_i]),
    "finc_conv1x1_forward": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _vp, _vp]),
    "finc_conv1x1_inverse": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _vp, _vp]),
}


class FincError(RuntimeError):
    def __init__(self, code: int, what: str):
        msg = _lib.finc_strerror(code).decode() if _lib is not None else str(code)
        super().__init__(f"{what}: {msg} ({code})")
        self.code = code


_lib = None


def lib(path: str = LIB_PATH):
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"libfinc is not built ({path}); run __graft_entry__.build() first")
    handle = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(handle, name)
        fn.restype = res
        fn.argtypes = args
    _lib = handle
    return _lib


def _require_lib():
    return lib()


def _check(code: int, what: str):
    if code != OK:
        raise FincError(code, what)


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t: torch.Tensor, name: str, shape=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != torch.float32:
        raise ValueError(f"{name} must be float32")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def _logdet_out(t: torch.Tensor | None):
    if t is None:
        return None
    if not t.is_cuda or t.dtype != torch.float64 or t.numel() < 1:
        raise ValueError("logdet must be a device float64 tensor with at least one element")
    return t


def _bytes_buf(t: torch.Tensor, nbytes: int, name: str):
    """A device buffer of at least nbytes (prepared weights, workspaces)."""
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() * t.element_size() < nbytes:
        raise ValueError(f"{name} holds {t.numel() * t.element_size()} bytes, needs {nbytes}")
    return t


def _workspace(nbytes: int, device, ws):
    if ws is None:
        return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
    return _bytes_buf(ws, nbytes, "workspace")


# ---------------------------------------------------------------------------

def version() -> int:
    return _require_lib().finc_version()


def inverse_plan(kind: int, C: int, H: int, W: int, k: int, L: int = 1, U: int = 1):
    """The inverse kernel launches a call would make (finc_inverse_plan): a
    list of dicts (threads, mode, groups, streamed, lds, compact), one per
    distinct launch, or the negative status (EUNSUPPORTED, EINVAL)."""
    info = (ctypes.c_int * (6 * 8))()
    n = _require_lib().finc_inverse_plan(kind, L, U, C, H, W, k, info, 8)
    if n < 0:
        return n
    keys = ("threads", "mode", "groups", "streamed", "lds", "compact")
    return [dict(zip(keys, info[6 * i:6 * i + 6])) for i in range(n)]


def forward_plan(kind: int, B: int, C: int, H: int, W: int, k: int, in_place: bool = False):
    """The forward's row blocks (finc_forward_plan): dict(blocks, rows, lds),
    or the negative status (EUNSUPPORTED when a block does not fit)."""
    info = (ctypes.c_int * 3)()
    rc = _require_lib().finc_forward_plan(kind, B, C, H, W, k, int(in_place), info)
    if rc < 0:
        return rc
    return dict(blocks=info[0], rows=info[1], lds=info[2])


def workspace_bytes(C: int, k: int, n_layers: int = 1) -> int:
    return int(_require_lib().finc_workspace_bytes(C, k, n_layers))


def stack_workspace_bytes(L: int, U: int, C1: int, k: int) -> int:
    return int(_require_lib().finc_stack_workspace_bytes(L, U, C1, k))


def prepare(K: torch.Tensor, corners, out: torch.Tensor | None = None) -> torch.Tensor:
    """K: (n, C, C, k, k) or (C, C, k, k); corners: one id per layer."""
    L = _require_lib()
    _dev(K, "K")
    if K.dim() not in (4, 5) or K.shape[-4] != K.shape[-3] or K.shape[-2] != K.shape[-1]:
        raise ValueError(f"K has shape {tuple(K.shape)}, expected ([n,] C, C, k, k)")
    n = 1 if K.dim() == 4 else K.shape[0]
    C, k = K.shape[-3], K.shape[-1]
    corners = [int(c) for c in (corners if hasattr(corners, "__len__") else [corners])]
    if len(corners) != n:
        raise ValueError("one corner per layer")
    out = _workspace(workspace_bytes(C, k, n), K.device, out)
    arr = (ctypes.c_int * n)(*corners)
    _check(L.finc_prepare(_ptr(K), n, arr, C, k, _ptr(out), _stream()), "finc_prepare")
    return out


def forward(x: torch.Tensor, K: torch.Tensor, corner: int, out: torch.Tensor | None = None,
            logdet: torch.Tensor | None = None, prepared: torch.Tensor | None = None):
    """y = layer(x); with `logdet` (a device float64 tensor of one element) the
    same launch also writes the layer's log|det|; with `prepared` (a uint8
    device tensor of workspace_bytes(C, k, 1)) it also writes the weights
    prepared for inverse_prepared."""
    L = _require_lib()
    _dev(x, "x")
    B, C, H, W = x.shape
    k = K.shape[-1]
    _dev(K, "K", (C, C, k, k))
    y = torch.empty_like(x) if out is None else _dev(out, "out", x.shape)
    pp = None if prepared is None else _workspace(workspace_bytes(C, k, 1), x.device, prepared)
    _check(L.finc_forward(_ptr(x), _ptr(y), _ptr(K), _ptr(_logdet_out(logdet)), _ptr(pp), B, C,
                          H, W, k, corner, _stream()), "finc_forward")
    return y


def logdet(K: torch.Tensor, corner: int, H: int, W: int, out: torch.Tensor | None = None):
    L = _require_lib()
    _dev(K, "K")
    out = torch.empty(1, dtype=torch.float64, device=K.device) if out is None else out
    _check(L.finc_logdet(_ptr(K), K.shape[0], K.shape[-1], corner, H, W, _ptr(out),
                         _stream()), "finc_logdet")
    return out


def inverse(y: torch.Tensor, K: torch.Tensor, corner: int, out: torch.Tensor | None = None,
            workspace: torch.Tensor | None = None):
    L = _require_lib()
    _dev(y, "y")
    B, C, H, W = y.shape
    k = K.shape[-1]
    _dev(K, "K", (C, C, k, k))
    x = torch.empty_like(y) if out is None else _dev(out, "out", y.shape)
    ws = _workspace(workspace_bytes(C, k, 1), y.device, workspace)
    _check(L.finc_inverse(_ptr(y), _ptr(x), _ptr(K), B, C, H, W, k, corner, _ptr(ws),
                          _stream()), "finc_inverse")
    return x


def inverse_noalloc(y: torch.Tensor, K: torch.Tensor, corner: int,
                    out: torch.Tensor | None = None):
    """finc_inverse with the library's own device array for the prepared
    weights (no workspace); calls on one device must not overlap."""
    L = _require_lib()
    _dev(y, "y")
    B, C, H, W = y.shape
    k = K.shape[-1]
    _dev(K, "K", (C, C, k, k))
    x = torch.empty_like(y) if out is None else _dev(out, "out", y.shape)
    _check(L.finc_inverse_noalloc(_ptr(y), _ptr(x), _ptr(K), B, C, H, W, k, corner, _stream()),
           "finc_inverse_noalloc")
    return x


def inverse_prepared(y: torch.Tensor, prepared: torch.Tensor, k: int, corner: int,
                     out: torch.Tensor | None = None):
    L = _require_lib()
    _dev(y, "y")
    B, C, H, W = y.shape
    _bytes_buf(prepared, workspace_bytes(C, k, 1), "prepared")
    x = torch.empty_like(y) if out is None else _dev(out, "out", y.shape)
    _check(L.finc_inverse_prepared(_ptr(y), _ptr(x), _ptr(prepared), B, C, H, W, k, corner,
                                   _stream()), "finc_inverse_prepared")
    return x


def inverse_steps(y: torch.Tensor, prepared: torch.Tensor, k: int, corner: int = TL,
                  split: bool = False):
    """(x, steps): the inverse of a prepared layer (or, split=True, of a
    prepared channel-split unit) and the number of diagonal steps every wave
    of every workgroup ran, as (workgroups, waves) int32 (see
    finc_inverse_steps)."""
    L = _require_lib()
    _dev(y, "y")
    B, C, H, W = y.shape
    kind = PLAN_SPLIT if split else PLAN_LAYER
    _bytes_buf(prepared, workspace_bytes(C // 4 if split else C, k, 4 if split else 1),
               "prepared")
    info = inverse_plan(kind, C, H, W, k)
    if isinstance(info, int):
        _check(info, "finc_inverse_steps")
    waves = info[0]["threads"] // 64
    nwg = (4 * B if split else B)
    steps = torch.full((nwg, waves), -1, dtype=torch.int32, device=y.device)
    x = torch.empty_like(y)
    n = L.finc_inverse_steps(kind, _ptr(y), _ptr(x), _ptr(prepared), B, C, H, W, k, corner,
                             _ptr(steps), steps.numel(), _stream())
    if n < 0:
        _check(n, "finc_inverse_steps")
    return x, steps


def inverse_timeline(y: torch.Tensor, prepared: torch.Tensor, k: int, corner: int = TL,
                     split: bool = False):
    """(x, stamps): the inverse of a prepared layer (or, split=True, of a
    prepared channel-split unit) and, for every wave of every workgroup, the
    GPU's 100 MHz clock when its arguments arrived, its set-up was done, its
    last step was done and its store was issued, as (workgroups, waves, 4)
    int64 (see finc_inverse_timeline)."""
    L = _require_lib()
    _dev(y, "y")
    B, C, H, W = y.shape
    kind = PLAN_SPLIT if split else PLAN_LAYER
    _bytes_buf(prepared, workspace_bytes(C // 4 if split else C, k, 4 if split else 1),
               "prepared")
    info = inverse_plan(kind, C, H, W, k)
    if isinstance(info, int):
        _check(info, "finc_inverse_timeline")
    waves = info[0]["threads"] // 64
    nwg = (4 * B if split else B)
    stamps = torch.full((nwg, waves, 4), -1, dtype=torch.int64, device=y.device)
    x = torch.empty_like(y)
    n = L.finc_inverse_timeline(kind, _ptr(y), _ptr(x), _ptr(prepared), B, C, H, W, k, corner,
                                _ptr(stamps), stamps.numel(), _stream())
    if n < 0:
        _check(n, "finc_inverse_timeline")
    return x, stamps


def banded_plan(C: int, H: int, W: int, k: int):
    """dict(threads, rows, bands, lds) of the banded stream form
    (finc_banded_plan), or the negative status."""
    info = (ctypes.c_int * 4)()
    rc = _require_lib().finc_banded_plan(C, H, W, k, info)
    if rc < 0:
        return rc
    return dict(threads=info[0], rows=info[1], bands=info[2], lds=info[3])


def _banded(fn, y, K, n_layers, corner, out, workspace):
    L = _require_lib()
    _dev(y, "y")
    B, C, H, W = y.shape
    k = K.shape[-1]
    _dev(K, "K", (C, C, k, k) if n_layers == 1 else (4, C, C, k, k))
    nbytes = int(L.finc_banded_workspace_bytes(B, C, H, W, k, n_layers))
    if nbytes == 0:
        raise FincError(EUNSUPPORTED if isinstance(banded_plan(C, H, W, k), int) else EINVAL, fn)
    ws = _workspace(nbytes, y.device, workspace)
    x = torch.empty_like(y) if out is None else _dev(out, "out", y.shape)
    args = (_ptr(y), _ptr(x), _ptr(K), B, C, H, W, k) + ((corner,) if n_layers == 1 else ())
    _check(getattr(L, fn)(*args, _ptr(ws), _stream()), fn)
    return x, ws


def inverse_banded(y, K, corner: int, out=None, workspace=None):
    """(x, workspace) of finc_inverse_banded; the workspace's int at byte
    offset workspace_bytes(C, k, 1) is the timeout flag."""
    return _banded("finc_inverse_banded", y, K, 1, corner, out, workspace)


def unit_inverse_banded(y, K4, out=None, workspace=None):
    """(x, workspace) of finc_unit_inverse_banded (timeout flag at byte
    offset workspace_bytes(C, k, 4))."""
    return _banded("finc_unit_inverse_banded", y, K4, 4, TL, out, workspace)


def backward(x: torch.Tensor, dy: torch.Tensor, K: torch.Tensor, corner: int,
             gld: float = 0.0, want_dx: bool = True, want_dK: bool = True,
             dx: torch.Tensor | None = None, dK: torch.Tensor | None = None,
             workspace: torch.Tensor | None = None):
    """(dx, dK) of one layer for the loss gradient dy (see finc_backward);
    either is None when not wanted."""
    L = _require_lib()
    _dev(x, "x")
    B, C, H, W = x.shape
    _dev(dy, "dy", x.shape)
    k = K.shape[-1]
    _dev(K, "K", (C, C, k, k))
    if want_dx:
        dx = torch.empty_like(x) if dx is None else _dev(dx, "dx", x.shape)
    else:
        dx = None
    if want_dK:
        dK = torch.empty_like(K) if dK is None else _dev(dK, "dK", K.shape)
    else:
        dK = None
    ws = _workspace(int(L.finc_backward_workspace_bytes(B, C, H, W, k)), x.device, workspace)
    _check(L.finc_backward(_ptr(x), _ptr(dy), _ptr(K), _ptr(dx), _ptr(dK), float(gld), B, C, H,
                           W, k, corner, _ptr(ws), _stream()), "finc_backward")
    return dx, dK


def _unit_grads(fn, wsfn, x, dy, Kw, wshape, gld, want_dx, want_dK, dx, dKw, workspace):
    L = _require_lib()
    _dev(x, "x")
    B, C, H, W = x.shape
    _dev(dy, "dy", x.shape)
    k = Kw.shape[-1]
    _dev(Kw, "K", wshape(C, k))
    dx = (torch.empty_like(x) if dx is None else _dev(dx, "dx", x.shape)) if want_dx else None
    dKw = ((torch.empty_like(Kw) if dKw is None else _dev(dKw, "dK", Kw.shape))
           if want_dK else None)
    nbytes = int(getattr(L, wsfn)(B, C, H, W, k))
    if nbytes == 0:
        raise FincError(EINVAL, fn)
    ws = _workspace(nbytes, x.device, workspace)
    _check(getattr(L, fn)(_ptr(x), _ptr(dy), _ptr(Kw), _ptr(dx), _ptr(dKw), float(gld), B, C, H,
                          W, k, _ptr(ws), _stream()), fn)
    return dx, dKw


def unit_backward(x, dy, K4, gld: float = 0.0, want_dx: bool = True, want_dK: bool = True,
                  dx=None, dK4=None, workspace=None):
    """(dx, dK4) of the sequential unit (see finc_unit_backward); K4 is
    (4, C, C, k, k)."""
    return _unit_grads("finc_unit_backward", "finc_unit_backward_workspace_bytes", x, dy, K4,
                       lambda C, k: (4, C, C, k, k), gld, want_dx, want_dK, dx, dK4, workspace)


def split_backward(x, dy, Kq4, gld: float = 0.0, want_dx: bool = True, want_dK: bool = True,
                   dx=None, dKq4=None, workspace=None):
    """(dx, dKq4) of the channel-split unit (see finc_split_backward); Kq4 is
    (4, C/4, C/4, k, k)."""
    return _unit_grads("finc_split_backward", "finc_split_backward_workspace_bytes", x, dy,
                       Kq4, lambda C, k: (4, C // 4, C // 4, k, k), gld, want_dx, want_dK, dx,
                       dKq4, workspace)


def actnorm_backward(x, dy, s, gld: float = 0.0, workspace=None):
    """(dx, ds, db) of actnorm y = s x + b (see finc_actnorm_backward)."""
    L = _require_lib()
    _dev(x, "x")
    B, C, H, W = x.shape
    _dev(dy, "dy", x.shape)
    _dev(s, "s", (C,))
    dx, ds, db = torch.empty_like(x), torch.empty_like(s), torch.empty_like(s)
    nbytes = int(L.finc_actnorm_backward_workspace_bytes(B, C, H, W))
    if nbytes == 0:
        raise FincError(EINVAL, "finc_actnorm_backward")
    ws = _workspace(nbytes, x.device, workspace)
    _check(L.finc_actnorm_backward(_ptr(x), _ptr(dy), _ptr(s), _ptr(dx), _ptr(ds), _ptr(db),
                                   float(gld), B, C, H, W, _ptr(ws), _stream()),
           "finc_actnorm_backward")
    return dx, ds, db


def _stack_latents(B, L_levels, C1, H1, W1, device):
    return [torch.empty((B, (C1 << l) if l == L_levels - 1 else (C1 << l) // 2, H1 >> l, W1 >> l),
                        device=device) for l in range(L_levels)]


def stack_forward(x, K, scale, bias, L_levels: int, U: int, k: int, workspace=None):
    """(latents, logdet) of the stack's forward direction (finc_stack_forward);
    K, scale, bias flat in the stack's layout."""
    L = _require_lib()
    _dev(x, "x")
    B, C1, H1, W1 = x.shape
    _stack_params(L_levels, U, C1, k, scale, bias, K)
    z = _stack_latents(B, L_levels, C1, H1, W1, x.device)
    zp = (ctypes.c_void_p * L_levels)(*[t.data_ptr() for t in z])
    ld = torch.empty(B, dtype=torch.float64, device=x.device)
    nbytes = int(L.finc_stack_train_workspace_bytes(B, L_levels, U, C1, H1, W1, k))
    if nbytes == 0:
        raise FincError(EINVAL, "finc_stack_forward")
    ws = _workspace(nbytes, x.device, workspace)
    _check(L.finc_stack_forward(_ptr(x), zp, _ptr(ld), _ptr(K), _ptr(scale), _ptr(bias), B,
                                L_levels, U, C1, H1, W1, k, _ptr(ws), _stream()),
           "finc_stack_forward")
    return z, ld


def stack_backward(x, dz, K, scale, bias, L_levels: int, U: int, k: int, gld: float = 0.0,
                   want_dx: bool = True, workspace=None):
    """(dx, dK, dscale, dbias) of the stack's forward direction for latent
    gradients dz (finc_stack_backward); dx is None when not wanted."""
    L = _require_lib()
    _dev(x, "x")
    B, C1, H1, W1 = x.shape
    _stack_params(L_levels, U, C1, k, scale, bias, K)
    zp = _stack_args(dz, L_levels, C1, H1, W1)
    dx = torch.empty_like(x) if want_dx else None
    dK, ds, db = torch.empty_like(K), torch.empty_like(scale), torch.empty_like(bias)
    nbytes = int(L.finc_stack_train_workspace_bytes(B, L_levels, U, C1, H1, W1, k))
    if nbytes == 0:
        raise FincError(EINVAL, "finc_stack_backward")
    ws = _workspace(nbytes, x.device, workspace)
    _check(L.finc_stack_backward(_ptr(x), zp, _ptr(K), _ptr(scale), _ptr(bias), _ptr(dx),
                                 _ptr(dK), _ptr(ds), _ptr(db), float(gld), B, L_levels, U, C1,
                                 H1, W1, k, _ptr(ws), _stream()), "finc_stack_backward")
    return dx, dK, ds, db


def gauss_nll(zs, logdet):
    """(nll, bpd) per image (device float64, B each) for latents zs (float32
    tensors with the batch first) and per-image log|det| (float64, B); see
    finc_gauss_nll."""
    L = _require_lib()
    if not logdet.is_cuda or logdet.dtype != torch.float64 or logdet.dim() != 1:
        raise ValueError("logdet must be a 1-d float64 device tensor")
    B = logdet.shape[0]
    for z in zs:
        _dev(z, "z")
        if z.shape[0] != B:
            raise ValueError(f"latent has batch {z.shape[0]}, expected {B}")
    n = (ctypes.c_longlong * len(zs))(*[math.prod(z.shape[1:]) for z in zs])
    ptrs = (_vp * len(zs))(*[z.data_ptr() for z in zs])
    nll = torch.empty(B, dtype=torch.float64, device=logdet.device)
    bpd = torch.empty_like(nll)
    _check(L.finc_gauss_nll(ptrs, n, len(zs), B, _ptr(logdet), _ptr(nll), _ptr(bpd), _stream()),
           "finc_gauss_nll")
    return nll, bpd


def unit_forward(x: torch.Tensor, K4: torch.Tensor, out: torch.Tensor | None = None,
                 logdet: torch.Tensor | None = None, prepared: torch.Tensor | None = None):
    """The unit (TL, TR, BL, BR); optional side outputs as for forward, with
    `prepared` of workspace_bytes(C, k, 4) for unit_inverse_prepared."""
    L = _require_lib()
    _dev(x, "x")
    B, C, H, W = x.shape
    k = K4.shape[-1]
    _dev(K4, "K4", (4, C, C, k, k))
    y = torch.empty_like(x) if out is None else _dev(out, "out", x.shape)
    pp = None if prepared is None else _workspace(workspace_bytes(C, k, 4), x.device, prepared)
    _check(L.finc_unit_forward(_ptr(x), _ptr(y), _ptr(K4), _ptr(_logdet_out(logdet)), _ptr(pp),
                               B, C, H, W, k, _stream()), "finc_unit_forward")
    return y


def unit_logdet(K4: torch.Tensor, H: int, W: int, out: torch.Tensor | None = None):
    L = _require_lib()
    _dev(K4, "K4")
    out = torch.empty(1, dtype=torch.float64, device=K4.device) if out is None else out
    _check(L.finc_unit_logdet(_ptr(K4), K4.shape[1], K4.shape[-1], H, W, _ptr(out),
                              _stream()), "finc_unit_logdet")
    return out


def unit_inverse(y: torch.Tensor, K4: torch.Tensor, out: torch.Tensor | None = None,
                 workspace: torch.Tensor | None = None):
    L = _require_lib()
    _dev(y, "y")
    B, C, H, W = y.shape
    k = K4.shape[-1]
    _dev(K4, "K4", (4, C, C, k, k))
    x = torch.empty_like(y) if out is None else _dev(out, "out", y.shape)
    ws = _workspace(workspace_bytes(C, k, 4), y.device, workspace)
    _check(L.finc_unit_inverse(_ptr(y), _ptr(x), _ptr(K4), B, C, H, W, k, _ptr(ws),
                               _stream()), "finc_unit_inverse")
    return x


def unit_inverse_prepared(y: torch.Tensor, prepared4: torch.Tensor, k: int,
                          out: torch.Tensor | None = None):
    L = _require_lib()
    _dev(y, "y")
    B, C, H, W = y.shape
    _bytes_buf(prepared4, workspace_bytes(C, k, 4), "prepared4")
    x = torch.empty_like(y) if out is None else _dev(out, "out", y.shape)
    _check(L.finc_unit_inverse_prepared(_ptr(y), _ptr(x), _ptr(prepared4), B, C, H, W, k,
                                        _stream()), "finc_unit_inverse_prepared")
    return x


# channel-split unit (four quarter-channel PCBs side by side; quarter g has
# corner g): Kq4 of shape (4, C/4, C/4, k, k)

def split_forward(x: torch.Tensor, Kq4: torch.Tensor, out: torch.Tensor | None = None,
                  logdet: torch.Tensor | None = None, prepared: torch.Tensor | None = None):
    """Optional side outputs as for forward, with `prepared` of
    workspace_bytes(C/4, k, 4) for split_inverse_prepared."""
    L = _require_lib()
    _dev(x, "x")
    B, C, H, W = x.shape
    k = Kq4.shape[-1]
    _dev(Kq4, "Kq4", (4, C // 4, C // 4, k, k))
    y = torch.empty_like(x) if out is None else _dev(out, "out", x.shape)
    pp = None if prepared is None else _workspace(workspace_bytes(C // 4, k, 4), x.device,
                                                  prepared)
    _check(L.finc_split_forward(_ptr(x), _ptr(y), _ptr(Kq4), _ptr(_logdet_out(logdet)), _ptr(pp),
                                B, C, H, W, k, _stream()), "finc_split_forward")
    return y


def split_logdet(Kq4: torch.Tensor, H: int, W: int, out: torch.Tensor | None = None):
    L = _require_lib()
    _dev(Kq4, "Kq4")
    out = torch.empty(1, dtype=torch.float64, device=Kq4.device) if out is None else out
    _check(L.finc_split_logdet(_ptr(Kq4), 4 * Kq4.shape[1], Kq4.shape[-1], H, W, _ptr(out),
                               _stream()), "finc_split_logdet")
    return out


def split_inverse(y: torch.Tensor, Kq4: torch.Tensor, out: torch.Tensor | None = None,
                  workspace: torch.Tensor | None = None):
    L = _require_lib()
    _dev(y, "y")
    B, C, H, W = y.shape
    k = Kq4.shape[-1]
    _dev(Kq4, "Kq4", (4, C // 4, C // 4, k, k))
    x = torch.empty_like(y) if out is None else _dev(out, "out", y.shape)
    ws = _workspace(workspace_bytes(C // 4, k, 4), y.device, workspace)
    _check(L.finc_split_inverse(_ptr(y), _ptr(x), _ptr(Kq4), B, C, H, W, k, _ptr(ws),
                                _stream()), "finc_split_inverse")
    return x


def split_inverse_prepared(y: torch.Tensor, prepared4: torch.Tensor, k: int,
                           out: torch.Tensor | None = None):
    L = _require_lib()
    _dev(y, "y")
    B, C, H, W = y.shape
    _bytes_buf(prepared4, workspace_bytes(C // 4, k, 4), "prepared4")
    x = torch.empty_like(y) if out is None else _dev(out, "out", y.shape)
    _check(L.finc_split_inverse_prepared(_ptr(y), _ptr(x), _ptr(prepared4), B, C, H, W, k,
                                         _stream()), "finc_split_inverse_prepared")
    return x


def _stack_args(z, L_levels, C1, H1, W1):
    """Latents z[l]: (B, C_l / 2, H_l, W_l) below the top, (B, C_top, H_top,
    W_top) at the top, C_l = C1 2^l, H_l = H1 / 2^l."""
    if len(z) != L_levels:
        raise ValueError("one latent per level")
    B = z[0].shape[0] if z[0].dim() == 4 else -1
    for l, t in enumerate(z):
        C = C1 << l
        _dev(t, f"z[{l}]", (B, C if l == L_levels - 1 else C // 2, H1 >> l, W1 >> l))
    return (ctypes.c_void_p * L_levels)(*[t.data_ptr() for t in z])


def _stack_params(L_levels, U, C1, k, scale, bias, K=None):
    """scale, bias: U * sum_l C_l floats; K: U * 4 * sum_l C_l^2 k^2 floats."""
    chans = sum(C1 << l for l in range(L_levels))
    for name, t in (("scale", scale), ("bias", bias)):
        _dev(t, name)
        if t.numel() != U * chans:
            raise ValueError(f"{name} has {t.numel()} elements, expected {U * chans}")
    if K is not None:
        _dev(K, "K")
        n = U * 4 * sum((C1 << l) ** 2 for l in range(L_levels)) * k * k
        if K.numel() != n:
            raise ValueError(f"K has {K.numel()} elements, expected {n}")


def stack_prepare(K: torch.Tensor, L: int, U: int, C1: int, k: int,
                  out: torch.Tensor | None = None):
    lb = _require_lib()
    _dev(K, "K")
    n = U * 4 * sum((C1 << l) ** 2 for l in range(L)) * k * k
    if K.numel() != n:
        raise ValueError(f"K has {K.numel()} elements, expected {n}")
    out = _workspace(stack_workspace_bytes(L, U, C1, k), K.device, out)
    _check(lb.finc_stack_prepare(_ptr(K), L, U, C1, k, _ptr(out), _stream()),
           "finc_stack_prepare")
    return out


def stack_inverse(z, K: torch.Tensor, scale: torch.Tensor, bias: torch.Tensor, L: int,
                  U: int, C1: int, H1: int, W1: int, k: int, out: torch.Tensor | None = None,
                  workspace: torch.Tensor | None = None):
    """z: list of L latents (see finc.h); K, scale, bias: flat device tensors."""
    lb = _require_lib()
    zp = _stack_args(z, L, C1, H1, W1)
    _stack_params(L, U, C1, k, scale, bias, K)
    B = z[0].shape[0]
    x = (torch.empty((B, C1, H1, W1), dtype=torch.float32, device=z[0].device)
         if out is None else _dev(out, "out", (B, C1, H1, W1)))
    ws = _workspace(stack_workspace_bytes(L, U, C1, k), z[0].device, workspace)
    _check(lb.finc_stack_inverse(zp, _ptr(x), _ptr(K), _ptr(scale), _ptr(bias), B, L, U, C1,
                                 H1, W1, k, _ptr(ws), _stream()), "finc_stack_inverse")
    return x


def stack_inverse_prepared(z, prepared: torch.Tensor, scale: torch.Tensor,
                           bias: torch.Tensor, L: int, U: int, C1: int, H1: int, W1: int,
                           k: int, out: torch.Tensor | None = None):
    lb = _require_lib()
    zp = _stack_args(z, L, C1, H1, W1)
    _stack_params(L, U, C1, k, scale, bias)
    _bytes_buf(prepared, stack_workspace_bytes(L, U, C1, k), "prepared")
    B = z[0].shape[0]
    x = (torch.empty((B, C1, H1, W1), dtype=torch.float32, device=z[0].device)
         if out is None else _dev(out, "out", (B, C1, H1, W1)))
    _check(lb.finc_stack_inverse_prepared(zp, _ptr(x), _ptr(prepared), _ptr(scale),
                                          _ptr(bias), B, L, U, C1, H1, W1, k, _stream()),
           "finc_stack_inverse_prepared")
    return x


# ---------------------------------------------------------------------------
# The full FInC Flow (Step and multi-scale flow; parameter layout in finc.h)

def conv1x1_forward(x: torch.Tensor, Wm: torch.Tensor, out: torch.Tensor | None = None,
                    logdet: torch.Tensor | None = None, workspace: torch.Tensor | None = None):
    lb = _require_lib()
    _dev(x, "x")
    B, C, H, W = x.shape
    _dev(Wm, "Wm", (C, C))
    y = torch.empty_like(x) if out is None else _dev(out, "out", x.shape)
    ws = _workspace(int(lb.finc_conv1x1_workspace_bytes(C)), x.device, workspace)
    _check(lb.finc_conv1x1_forward(_ptr(x), _ptr(y), _ptr(Wm), _ptr(_logdet_out(logdet)), B, C,
                                   H, W, _ptr(ws), _stream()), "finc_conv1x1_forward")
    return y


def conv1x1_inverse(y: torch.Tensor, Wm: torch.Tensor, out: torch.Tensor | None = None,
                    workspace: torch.Tensor | None = None):
    lb = _require_lib()
    _dev(y, "y")
    B, C, H, W = y.shape
    _dev(Wm, "Wm", (C, C))
    x = torch.empty_like(y) if out is None else _dev(out, "out", y.shape)
    ws = _workspace(int(lb.finc_conv1x1_workspace_bytes(C)), y.device, workspace)
    _check(lb.finc_conv1x1_inverse(_ptr(y), _ptr(x), _ptr(Wm), B, C, H, W, _ptr(ws), _stream()),
           "finc_conv1x1_inverse")
    return x


def step_param_count(C: int, k: int, hid: int) -> int:
    return int(_require_lib().finc_step_param_count(C, k, hid))


def step_prepare(sp: torch.Tensor, C: int, k: int, hid: int, out: torch.Tensor | None = None):
    lb = _require_lib()
    _dev(sp, "sp")
    if sp.numel() != step_param_count(C, k, hid):
        raise ValueError(f"sp has {sp.numel()} elements, expected {step_param_count(C, k, hid)}")
    pp = _workspace(int(lb.finc_step_prepared_bytes(C, k)), sp.device, out)
    _check(lb.finc_step_prepare(_ptr(sp), C, k, hid, _ptr(pp), _stream()), "finc_step_prepare")
    return pp


def _step_call(name, a, sp, prepared, k, hid, out, workspace, logdet=None):
    lb = _require_lib()
    _dev(a, "input")
    B, C, H, W = a.shape
    _dev(sp, "sp")
    if sp.numel() != step_param_count(C, k, hid):
        raise ValueError("sp does not match (C, k, hid)")
    _bytes_buf(prepared, int(lb.finc_step_prepared_bytes(C, k)), "prepared")
    b = torch.empty_like(a) if out is None else _dev(out, "out", a.shape)
    ws = _workspace(int(lb.finc_step_workspace_bytes(B, C, H, W, hid)), a.device, workspace)
    if name == "finc_step_forward":
        if logdet is not None and (not logdet.is_cuda or logdet.dtype != torch.float64 or
                                   logdet.numel() < B):
            raise ValueError("logdet must be a device float64 tensor of B elements")
        rc = lb.finc_step_forward(_ptr(a), _ptr(b), _ptr(logdet), _ptr(sp), _ptr(prepared), B, C,
                                  H, W, k, hid, _ptr(ws), _stream())
    else:
        rc = lb.finc_step_inverse(_ptr(a), _ptr(b), _ptr(sp), _ptr(prepared), B, C, H, W, k, hid,
                                  _ptr(ws), _stream())
    _check(rc, name)
    return b


def step_forward(x, sp, prepared, k: int, hid: int, out=None, logdet=None, workspace=None):
    """y = Step(x); logdet (B float64, device) is incremented if given."""
    return _step_call("finc_step_forward", x, sp, prepared, k, hid, out, workspace, logdet)


def step_inverse(y, sp, prepared, k: int, hid: int, out=None, workspace=None):
    return _step_call("finc_step_inverse", y, sp, prepared, k, hid, out, workspace)


def flow_param_count(L: int, K: int, C0: int, k: int, hid: int) -> int:
    return int(_require_lib().finc_flow_param_count(L, K, C0, k, hid))


def flow_latent_shapes(B: int, L: int, C0: int, H0: int, W0: int):
    return [(B, ((4 * C0) << l) // (1 if l == L - 1 else 2), H0 >> (l + 1), W0 >> (l + 1))
            for l in range(L)]


def flow_prepare(params: torch.Tensor, L: int, K: int, C0: int, k: int, hid: int,
                 out: torch.Tensor | None = None):
    lb = _require_lib()
    _dev(params, "params")
    if params.numel() != flow_param_count(L, K, C0, k, hid):
        raise ValueError("params does not match (L, K, C0, k, hid)")
    pp = _workspace(int(lb.finc_flow_prepared_bytes(L, K, C0, k)), params.device, out)
    _check(lb.finc_flow_prepare(_ptr(params), L, K, C0, k, hid, _ptr(pp), _stream()),
           "finc_flow_prepare")
    return pp


def _flow_common(params, prepared, L, K, C0, k, hid):
    lb = _require_lib()
    _dev(params, "params")
    if params.numel() != flow_param_count(L, K, C0, k, hid):
        raise ValueError("params does not match (L, K, C0, k, hid)")
    _bytes_buf(prepared, int(lb.finc_flow_prepared_bytes(L, K, C0, k)), "prepared")
    return lb


def flow_forward(x: torch.Tensor, params: torch.Tensor, prepared: torch.Tensor, L: int, K: int,
                 k: int, hid: int, workspace: torch.Tensor | None = None):
    """(latents z[0..L-1], logdet per image) of images x."""
    _dev(x, "x")
    B, C0, H0, W0 = x.shape
    lb = _flow_common(params, prepared, L, K, C0, k, hid)
    z = [torch.empty(s, dtype=torch.float32, device=x.device)
         for s in flow_latent_shapes(B, L, C0, H0, W0)]
    ld = torch.empty(B, dtype=torch.float64, device=x.device)
    ws = _workspace(int(lb.finc_flow_workspace_bytes(B, L, C0, H0, W0, hid)), x.device, workspace)
    zp = (ctypes.c_void_p * L)(*[t.data_ptr() for t in z])
    _check(lb.finc_flow_forward(_ptr(x), zp, _ptr(ld), _ptr(params), _ptr(prepared), B, L, K, C0,
                                H0, W0, k, hid, _ptr(ws), _stream()), "finc_flow_forward")
    return z, ld


def flow_sample(z, params: torch.Tensor, prepared: torch.Tensor, L: int, K: int, C0: int,
                H0: int, W0: int, k: int, hid: int, out: torch.Tensor | None = None,
                workspace: torch.Tensor | None = None):
    """Images from latents z[0..L-1] (shapes as flow_latent_shapes)."""
    if len(z) != L:
        raise ValueError("one latent per level")
    B = z[0].shape[0]
    for l, (t, shp) in enumerate(zip(z, flow_latent_shapes(B, L, C0, H0, W0))):
        _dev(t, f"z[{l}]", shp)
    lb = _flow_common(params, prepared, L, K, C0, k, hid)
    x = (torch.empty((B, C0, H0, W0), dtype=torch.float32, device=z[0].device)
         if out is None else _dev(out, "out", (B, C0, H0, W0)))
    ws = _workspace(int(lb.finc_flow_workspace_bytes(B, L, C0, H0, W0, hid)), z[0].device,
                    workspace)
    zp = (ctypes.c_void_p * L)(*[t.data_ptr() for t in z])
    _check(lb.finc_flow_sample(zp, _ptr(x), _ptr(params), _ptr(prepared), B, L, K, C0, H0, W0, k,
                               hid, _ptr(ws), _stream()), "finc_flow_sample")
    return x
