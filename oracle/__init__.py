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
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = None if name.startswith(("orc_actnorm", "orc_squeeze", "orc_unsqueeze")) else I
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


_default = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default
