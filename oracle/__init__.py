"""CPU oracle for the FInC masked convolution: ctypes wrapper over finc_oracle.c.

TEST INFRASTRUCTURE ONLY.  The product path (the HIP library and its binding)
never imports this package; only the tests, the smoke check and the
benchmark's CPU-baseline leg do.  Every array crossing this wrapper is float64
and C-contiguous; the wrapper only marshals, all arithmetic is in the C file.

Parity status of each function (see the pins in tests/test_oracle_pins.py):
forward, logdet, inverse, unit_*, squeeze/unsqueeze, actnorm_*, stack_* are
all pinned; nothing here is "parity unpinned".
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "finc_oracle.c")
LIB = os.path.join(HERE, "libfinc_oracle.so")

_dp = ctypes.POINTER(ctypes.c_double)
_lib = None


def build(src: str = SRC, out: str = LIB) -> str:
    """Compile the oracle with gcc (plain -O2, no fast-math, no FMA contraction)."""
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c99",
           "-shared", "-fPIC", "-o", out, src, "-lm"]
    subprocess.run(cmd, check=True)
    return out


def load(path: str = LIB):
    """Load (building first if absent) and declare the C signatures."""
    global _lib
    if path == LIB and _lib is not None:
        return _lib
    if not os.path.exists(path):
        build(out=path)
    lib = ctypes.CDLL(path)
    L, I = ctypes.c_long, ctypes.c_int
    sig = {
        "orc_forward": [_dp, _dp, _dp, L, I, I, I, I, I],
        "orc_inverse": [_dp, _dp, _dp, L, I, I, I, I, I],
        "orc_logdet": [_dp, I, I, I, I, I, _dp],
        "orc_backward": [_dp, _dp, _dp, _dp, _dp, ctypes.c_double, L, I, I, I, I, I],
        "orc_unit_backward": [_dp, _dp, _dp, _dp, _dp, ctypes.c_double, L, I, I, I, I],
        "orc_split_backward": [_dp, _dp, _dp, _dp, _dp, ctypes.c_double, L, I, I, I, I],
        "orc_actnorm_backward": [_dp, _dp, _dp, _dp, _dp, _dp, ctypes.c_double, L, I, I, I],
        "orc_gauss_nll": [ctypes.POINTER(_dp), ctypes.POINTER(L), I, L, _dp, _dp, _dp],
        "orc_stack_logdet": [_dp, _dp, I, I, I, I, I, I, _dp],
        "orc_stack_backward": [_dp, ctypes.POINTER(_dp), _dp, _dp, _dp, _dp, _dp, _dp, _dp,
                               ctypes.c_double, L, I, I, I, I, I, I],
        "orc_unit_forward": [_dp, _dp, _dp, L, I, I, I, I],
        "orc_unit_inverse": [_dp, _dp, _dp, L, I, I, I, I],
        "orc_unit_logdet": [_dp, I, I, I, I, _dp],
        "orc_split_forward": [_dp, _dp, _dp, L, I, I, I, I],
        "orc_split_inverse": [_dp, _dp, _dp, L, I, I, I, I],
        "orc_split_logdet": [_dp, I, I, I, I, _dp],
        "orc_actnorm_forward": [_dp, _dp, _dp, _dp, L, I, I, I],
        "orc_actnorm_inverse": [_dp, _dp, _dp, _dp, L, I, I, I],
        "orc_squeeze": [_dp, _dp, L, I, I, I],
        "orc_unsqueeze": [_dp, _dp, L, I, I, I],
        "orc_stack_forward": [_dp, ctypes.POINTER(_dp), _dp, _dp, _dp, L, I, I, I, I, I, I],
        "orc_stack_inverse": [ctypes.POINTER(_dp), _dp, _dp, _dp, _dp, L, I, I, I, I, I, I],
        "orc_conv1x1_forward": [_dp, _dp, _dp, L, I, I, I],
        "orc_conv1x1_inverse": [_dp, _dp, _dp, L, I, I, I],
        "orc_conv1x1_logdet": [_dp, I, I, I, _dp],
        "orc_coupling_net": [_dp, _dp, _dp, L, I, I, I, I],
        "orc_coupling_forward": [_dp, _dp, _dp, L, I, I, I, I, _dp],
        "orc_coupling_inverse": [_dp, _dp, _dp, L, I, I, I, I],
        "orc_step_forward": [_dp, _dp, _dp, L, I, I, I, I, I, _dp],
        "orc_step_inverse": [_dp, _dp, _dp, L, I, I, I, I, I],
        "orc_flow_params": [I, I, I, I, I],
        "orc_flow_forward": [_dp, ctypes.POINTER(_dp), _dp, L, I, I, I, I, I, I, I, _dp],
        "orc_flow_sample": [ctypes.POINTER(_dp), _dp, _dp, L, I, I, I, I, I, I, I],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = None if name.startswith(("orc_actnorm_f", "orc_actnorm_i", "orc_squeeze",
                                              "orc_unsqueeze")) else I
    lib.orc_flow_params.restype = L
    if path == LIB:
        _lib = lib
    return lib


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"oracle returned {code}")
        self.code = code


def _c(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a: np.ndarray):
    return a.ctypes.data_as(_dp)


def _check(rc: int, allow_singular: bool = False):
    if rc != 0 and not (allow_singular and rc == -2):
        raise OracleError(rc)


class Oracle:
    """Bound oracle; `Oracle(path)` loads another build (used by mutation tests)."""

    def __init__(self, path: str = LIB):
        self.lib = load(path)

    def forward(self, x, K, corner: int) -> np.ndarray:
        x, K = _c(x), _c(K)
        B, C, H, W = x.shape
        y = np.empty_like(x)
        _check(self.lib.orc_forward(_p(x), _p(y), _p(K), B, C, H, W, K.shape[-1], corner))
        return y

    def inverse(self, y, K, corner: int) -> np.ndarray:
        y, K = _c(y), _c(K)
        B, C, H, W = y.shape
        x = np.empty_like(y)
        _check(self.lib.orc_inverse(_p(y), _p(x), _p(K), B, C, H, W, K.shape[-1], corner))
        return x

    def logdet(self, K, corner: int, H: int, W: int, allow_singular=False) -> float:
        K = _c(K)
        out = np.zeros(1)
        _check(self.lib.orc_logdet(_p(K), K.shape[0], K.shape[-1], corner, H, W, _p(out)),
               allow_singular)
        return float(out[0])

    def backward(self, x, dy, K, corner: int, gld: float = 0.0):
        """(dx, dK) of one layer for the loss gradient dy (see orc_backward)."""
        x, dy, K = _c(x), _c(dy), _c(K)
        B, C, H, W = x.shape
        dx, dK = np.empty_like(x), np.empty_like(K)
        _check(self.lib.orc_backward(_p(x), _p(dy), _p(K), _p(dx), _p(dK), float(gld), B, C,
                                     H, W, K.shape[-1], corner))
        return dx, dK

    def unit_backward(self, x, dy, K4, gld: float = 0.0):
        """(dx, dK4) of the sequential unit (see orc_unit_backward)."""
        x, dy, K4 = _c(x), _c(dy), _c(K4)
        B, C, H, W = x.shape
        dx, dK4 = np.empty_like(x), np.empty_like(K4)
        _check(self.lib.orc_unit_backward(_p(x), _p(dy), _p(K4), _p(dx), _p(dK4), float(gld),
                                          B, C, H, W, K4.shape[-1]))
        return dx, dK4

    def split_backward(self, x, dy, Kq4, gld: float = 0.0):
        """(dx, dKq4) of the channel-split unit (see orc_split_backward)."""
        x, dy, Kq4 = _c(x), _c(dy), _c(Kq4)
        B, C, H, W = x.shape
        dx, dKq4 = np.empty_like(x), np.empty_like(Kq4)
        _check(self.lib.orc_split_backward(_p(x), _p(dy), _p(Kq4), _p(dx), _p(dKq4),
                                           float(gld), B, C, H, W, Kq4.shape[-1]))
        return dx, dKq4

    def actnorm_backward(self, x, dy, s, gld: float = 0.0):
        """(dx, ds, db) of actnorm (see orc_actnorm_backward)."""
        x, dy, s = _c(x), _c(dy), _c(s)
        B, C, H, W = x.shape
        dx, ds, db = np.empty_like(x), np.empty(C), np.empty(C)
        _check(self.lib.orc_actnorm_backward(_p(x), _p(dy), _p(s), _p(dx), _p(ds), _p(db),
                                             float(gld), B, C, H, W))
        return dx, ds, db

    def gauss_nll(self, zs, logdet):
        """(nll, bpd) per image for latents zs (arrays with the batch first)
        and per-image log|det| (see orc_gauss_nll)."""
        zs = [_c(z) for z in zs]
        logdet = _c(logdet)
        B = logdet.shape[0]
        n = (ctypes.c_long * len(zs))(*[int(np.prod(z.shape[1:])) for z in zs])
        ptrs = (_dp * len(zs))(*[_p(z) for z in zs])
        nll, bpd = np.empty(B), np.empty(B)
        _check(self.lib.orc_gauss_nll(ptrs, n, len(zs), B, _p(logdet), _p(nll), _p(bpd)))
        return nll, bpd

    def unit_forward(self, x, K4) -> np.ndarray:
        x, K4 = _c(x), _c(K4)
        B, C, H, W = x.shape
        y = np.empty_like(x)
        _check(self.lib.orc_unit_forward(_p(x), _p(y), _p(K4), B, C, H, W, K4.shape[-1]))
        return y

    def unit_inverse(self, y, K4) -> np.ndarray:
        y, K4 = _c(y), _c(K4)
        B, C, H, W = y.shape
        x = np.empty_like(y)
        _check(self.lib.orc_unit_inverse(_p(y), _p(x), _p(K4), B, C, H, W, K4.shape[-1]))
        return x

    def unit_logdet(self, K4, H: int, W: int) -> float:
        K4 = _c(K4)
        out = np.zeros(1)
        _check(self.lib.orc_unit_logdet(_p(K4), K4.shape[1], K4.shape[-1], H, W, _p(out)))
        return float(out[0])

    # channel-split unit: Kq4 = (4, C/4, C/4, k, k); quarter g has corner g
    def split_forward(self, x, Kq4) -> np.ndarray:
        x, Kq4 = _c(x), _c(Kq4)
        B, C, H, W = x.shape
        y = np.empty_like(x)
        _check(self.lib.orc_split_forward(_p(x), _p(y), _p(Kq4), B, C, H, W, Kq4.shape[-1]))
        return y

    def split_inverse(self, y, Kq4) -> np.ndarray:
        y, Kq4 = _c(y), _c(Kq4)
        B, C, H, W = y.shape
        x = np.empty_like(y)
        _check(self.lib.orc_split_inverse(_p(y), _p(x), _p(Kq4), B, C, H, W, Kq4.shape[-1]))
        return x

    def split_logdet(self, Kq4, H: int, W: int) -> float:
        Kq4 = _c(Kq4)
        out = np.zeros(1)
        _check(self.lib.orc_split_logdet(_p(Kq4), 4 * Kq4.shape[1], Kq4.shape[-1], H, W,
                                         _p(out)))
        return float(out[0])

    def actnorm_forward(self, x, s, b) -> np.ndarray:
        x, s, b = _c(x), _c(s), _c(b)
        y = np.empty_like(x)
        self.lib.orc_actnorm_forward(_p(x), _p(y), _p(s), _p(b), *x.shape)
        return y

    def actnorm_inverse(self, y, s, b) -> np.ndarray:
        y, s, b = _c(y), _c(s), _c(b)
        x = np.empty_like(y)
        self.lib.orc_actnorm_inverse(_p(y), _p(x), _p(s), _p(b), *y.shape)
        return x

    def squeeze(self, x) -> np.ndarray:
        x = _c(x)
        B, C, H, W = x.shape
        out = np.empty((B, 4 * C, H // 2, W // 2))
        self.lib.orc_squeeze(_p(x), _p(out), B, C, H, W)
        return out

    def unsqueeze(self, x) -> np.ndarray:
        x = _c(x)
        B, C4, H2, W2 = x.shape
        out = np.empty((B, C4 // 4, 2 * H2, 2 * W2))
        self.lib.orc_unsqueeze(_p(x), _p(out), B, C4, H2, W2)
        return out

    @staticmethod
    def _stack_params(K, scale, bias):
        Kf = _c(np.concatenate([np.ravel(a) for a in K]))
        sf = _c(np.concatenate([np.ravel(a) for a in scale]))
        bf = _c(np.concatenate([np.ravel(a) for a in bias]))
        return Kf, sf, bf

    def stack_forward(self, x, K, scale, bias, levels: int, units: int, k: int):
        x = _c(x)
        B, C1, H1, W1 = x.shape
        Kf, sf, bf = self._stack_params(K, scale, bias)
        z = []
        for l in range(levels):
            C, H, W = C1 << l, H1 >> l, W1 >> l
            z.append(np.empty((B, C if l == levels - 1 else C // 2, H, W)))
        zp = (_dp * levels)(*[_p(a) for a in z])
        _check(self.lib.orc_stack_forward(_p(x), zp, _p(Kf), _p(sf), _p(bf), B, levels,
                                          units, C1, H1, W1, k))
        return z

    def stack_logdet(self, K, scale, levels: int, units: int, C1: int, H1: int, W1: int,
                     k: int) -> float:
        """log|det| of the stack's forward direction, one image."""
        Kf, sf, _ = self._stack_params(K, scale, scale)
        out = np.zeros(1)
        _check(self.lib.orc_stack_logdet(_p(Kf), _p(sf), levels, units, C1, H1, W1, k, _p(out)))
        return float(out[0])

    def stack_backward(self, x, dz, K, scale, bias, levels: int, units: int, k: int,
                       gld: float = 0.0):
        """(dx, dK, dscale, dbias) of the stack's forward direction, flat
        parameter layouts as K, scale, bias (see orc_stack_backward)."""
        x = _c(x)
        B, C1, H1, W1 = x.shape
        Kf, sf, bf = self._stack_params(K, scale, bias)
        dzs = [_c(a) for a in dz]
        zp = (_dp * levels)(*[_p(a) for a in dzs])
        dx, dK, ds, db = np.empty_like(x), np.empty_like(Kf), np.empty_like(sf), np.empty_like(bf)
        _check(self.lib.orc_stack_backward(_p(x), zp, _p(Kf), _p(sf), _p(bf), _p(dx), _p(dK),
                                           _p(ds), _p(db), float(gld), B, levels, units, C1, H1,
                                           W1, k))
        return dx, dK, ds, db

    def stack_inverse(self, z, K, scale, bias, levels: int, units: int, k: int,
                      C1: int, H1: int, W1: int) -> np.ndarray:
        z = [_c(a) for a in z]
        B = z[0].shape[0]
        Kf, sf, bf = self._stack_params(K, scale, bias)
        x = np.empty((B, C1, H1, W1))
        zp = (_dp * levels)(*[_p(a) for a in z])
        _check(self.lib.orc_stack_inverse(zp, _p(x), _p(Kf), _p(sf), _p(bf), B, levels,
                                          units, C1, H1, W1, k))
        return x


    # ---- the full FInC Flow: 1x1 convolution, coupling, Step, multi-scale
    # flow (parameter layout: see finc_oracle.c)
    def conv1x1_forward(self, x, Wm) -> np.ndarray:
        x, Wm = _c(x), _c(Wm)
        y = np.empty_like(x)
        _check(self.lib.orc_conv1x1_forward(_p(x), _p(y), _p(Wm), *x.shape))
        return y

    def conv1x1_inverse(self, y, Wm) -> np.ndarray:
        y, Wm = _c(y), _c(Wm)
        x = np.empty_like(y)
        _check(self.lib.orc_conv1x1_inverse(_p(y), _p(x), _p(Wm), *y.shape))
        return x

    def conv1x1_logdet(self, Wm, H: int, W: int) -> float:
        Wm = _c(Wm)
        out = np.zeros(1)
        _check(self.lib.orc_conv1x1_logdet(_p(Wm), Wm.shape[0], H, W, _p(out)))
        return float(out[0])

    def coupling_net(self, xa, cp, hid: int) -> np.ndarray:
        xa, cp = _c(xa), _c(cp)
        B, Ch, H, W = xa.shape
        h = np.empty((B, 2 * Ch, H, W))
        _check(self.lib.orc_coupling_net(_p(xa), _p(h), _p(cp), B, 2 * Ch, H, W, hid))
        return h

    def coupling_forward(self, x, cp, hid: int):
        """(y, logdet per image)."""
        x, cp = _c(x), _c(cp)
        y, ld = np.empty_like(x), np.zeros(x.shape[0])
        _check(self.lib.orc_coupling_forward(_p(x), _p(y), _p(cp), *x.shape, hid, _p(ld)))
        return y, ld

    def coupling_inverse(self, y, cp, hid: int) -> np.ndarray:
        y, cp = _c(y), _c(cp)
        x = np.empty_like(y)
        _check(self.lib.orc_coupling_inverse(_p(y), _p(x), _p(cp), *y.shape, hid))
        return x

    def step_forward(self, x, sp, k: int, hid: int):
        """(y, logdet per image) of one FInC Flow Step."""
        x, sp = _c(x), _c(sp)
        y, ld = np.empty_like(x), np.zeros(x.shape[0])
        _check(self.lib.orc_step_forward(_p(x), _p(y), _p(sp), *x.shape, k, hid, _p(ld)))
        return y, ld

    def step_inverse(self, y, sp, k: int, hid: int) -> np.ndarray:
        y, sp = _c(y), _c(sp)
        x = np.empty_like(y)
        _check(self.lib.orc_step_inverse(_p(y), _p(x), _p(sp), *y.shape, k, hid))
        return x

    def flow_params(self, L: int, K: int, C0: int, k: int, hid: int) -> int:
        return int(self.lib.orc_flow_params(L, K, C0, k, hid))

    @staticmethod
    def flow_latent_shapes(B, L, C0, H0, W0):
        out = []
        for l in range(L):
            C, H, W = (4 * C0) << l, H0 >> (l + 1), W0 >> (l + 1)
            out.append((B, C if l == L - 1 else C // 2, H, W))
        return out

    def flow_forward(self, x, params, L: int, K: int, k: int, hid: int):
        """(latents z[0..L-1], logdet per image)."""
        x, params = _c(x), _c(params)
        B, C0, H0, W0 = x.shape
        z = [np.empty(s) for s in self.flow_latent_shapes(B, L, C0, H0, W0)]
        ld = np.zeros(B)
        zp = (_dp * L)(*[_p(a) for a in z])
        _check(self.lib.orc_flow_forward(_p(x), zp, _p(params), B, L, K, C0, H0, W0, k, hid,
                                         _p(ld)))
        return z, ld

    def flow_sample(self, z, params, L: int, K: int, C0: int, H0: int, W0: int, k: int,
                    hid: int) -> np.ndarray:
        z = [_c(a) for a in z]
        params = _c(params)
        B = z[0].shape[0]
        x = np.empty((B, C0, H0, W0))
        zp = (_dp * L)(*[_p(a) for a in z])
        _check(self.lib.orc_flow_sample(zp, _p(x), _p(params), B, L, K, C0, H0, W0, k, hid))
        return x


_default = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default
