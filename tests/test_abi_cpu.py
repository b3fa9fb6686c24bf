"""The C ABI without a GPU: the library loads, exports every function that
include/finc.h declares, and rejects bad arguments before any HIP call."""
import ctypes
import os
import re

import pytest

from paper_2301_09266_amd import finc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "finc.h")

FAKE = ctypes.c_void_p(0x100000)     # never dereferenced on the host
FAKE2 = ctypes.c_void_p(0x900000)
NULL = None


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(finc_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for want in ("finc_forward", "finc_logdet", "finc_inverse", "finc_unit_forward",
                 "finc_unit_inverse", "finc_unit_logdet", "finc_stack_inverse",
                 "finc_split_forward", "finc_split_inverse", "finc_split_logdet",
                 "finc_prepare", "finc_strerror"):
        assert want in names


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(finc.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    # and the binding knows every one of them
    assert set(declared_functions()) == set(finc.SIGNATURES)


def test_version_and_strerror():
    lib = finc.lib()
    assert lib.finc_version() >= 100
    for code in (0, -1, -2, -3, -4, 12345):
        assert lib.finc_strerror(code)


def test_workspace_bytes():
    lib = finc.lib()
    for C, k in [(3, 3), (12, 3), (12, 5), (48, 3), (64, 7), (1, 1)]:
        cp = (C + 3) // 4 * 4
        floats = -(-(k * k * cp * cp) // 64) * 64 + 64
        assert lib.finc_workspace_bytes(C, k, 1) == floats * 4
        assert lib.finc_workspace_bytes(C, k, 4) == 4 * floats * 4
    for bad in [(0, 3, 1), (65, 3, 1), (12, 0, 1), (12, 8, 1), (12, 3, -1)]:
        assert lib.finc_workspace_bytes(*bad) == 0
    assert lib.finc_stack_workspace_bytes(3, 8, 12, 3) == sum(
        8 * 4 * lib.finc_workspace_bytes(12 << l, 3, 1) for l in range(3))
    assert lib.finc_stack_workspace_bytes(3, 8, 24, 3) == 0   # 96 channels at the top


SHAPE = (2, 12, 16, 16, 3)


@pytest.mark.parametrize("args", [
    (NULL, FAKE2, FAKE, NULL, NULL, *SHAPE, 0),
    (FAKE, NULL, FAKE2, NULL, NULL, *SHAPE, 0),
    (FAKE, FAKE2, NULL, NULL, NULL, *SHAPE, 0),
    (FAKE, FAKE2, FAKE, NULL, NULL, -1, 12, 16, 16, 3, 0),
    (FAKE, FAKE2, FAKE, NULL, NULL, 2, 0, 16, 16, 3, 0),
    (FAKE, FAKE2, FAKE, NULL, NULL, 2, 65, 16, 16, 3, 0),
    (FAKE, FAKE2, FAKE, NULL, NULL, 2, 12, 0, 16, 3, 0),
    (FAKE, FAKE2, FAKE, NULL, NULL, 2, 12, 16, 16, 0, 0),
    (FAKE, FAKE2, FAKE, NULL, NULL, 2, 12, 16, 16, 8, 0),
    (FAKE, FAKE2, FAKE, NULL, NULL, *SHAPE, 4),
    (FAKE, FAKE2, FAKE, NULL, NULL, *SHAPE, -1),
    (FAKE, ctypes.c_void_p(0x100000 + 64), FAKE2, NULL, NULL, *SHAPE, 0),   # overlapping x / y
    (FAKE, FAKE2, FAKE, NULL, NULL, 1 << 20, 64, 64, 64, 3, 0),            # > 2^31 elements
    (FAKE, FAKE2, FAKE, NULL, ctypes.c_void_p(0x4000000 + 16), *SHAPE, 0),  # unaligned prepared
    (FAKE, FAKE2, FAKE, NULL, ctypes.c_void_p(0x100000), *SHAPE, 0),        # prepared over x
])
def test_forward_rejects(args):
    assert finc.lib().finc_forward(*args, None) == finc.EINVAL


FAKE3 = ctypes.c_void_p(0x1100000)
FAKE4 = ctypes.c_void_p(0x1900000)


@pytest.mark.parametrize("args", [
    (NULL, FAKE2, FAKE3, FAKE4, NULL, 0.0, *SHAPE, 0),                       # no x
    (FAKE, NULL, FAKE3, FAKE4, NULL, 0.0, *SHAPE, 0),                        # no dy
    (FAKE, FAKE2, NULL, FAKE4, NULL, 0.0, *SHAPE, 0),                        # no K
    (FAKE, FAKE2, FAKE3, FAKE4, NULL, 0.0, 2, 0, 16, 16, 3, 0),              # C = 0
    (FAKE, FAKE2, FAKE3, FAKE4, NULL, 0.0, *SHAPE, 4),                       # bad corner
    (FAKE, FAKE2, FAKE3, ctypes.c_void_p(0x100000 + 64), NULL, 0.0, *SHAPE, 0),   # dx over x
    (FAKE, FAKE2, FAKE3, ctypes.c_void_p(0x900000 + 64), NULL, 0.0, *SHAPE, 0),   # dx over dy
    (FAKE, FAKE2, FAKE3, NULL, ctypes.c_void_p(0x100000 + 64), 0.0, *SHAPE, 0),   # dK over x
    (FAKE, FAKE2, FAKE3, NULL, FAKE3, 0.0, *SHAPE, 0),                        # dK over K
    (FAKE, FAKE2, FAKE3, FAKE4, ctypes.c_void_p(0x1900000 + 64), 0.0, *SHAPE, 0),  # dK over dx
])
def test_backward_rejects(args):
    ws = ctypes.c_void_p(0x40000000)
    assert finc.lib().finc_backward(*args, ws, None) == finc.EINVAL


def test_backward_workspace_rules():
    lib = finc.lib()
    args = (FAKE, FAKE2, FAKE3, FAKE4, NULL, 0.0, *SHAPE, 0)
    assert lib.finc_backward(*args, NULL, None) == finc.EINVAL                         # none
    assert lib.finc_backward(*args, ctypes.c_void_p(0x40000010), None) == finc.EINVAL  # misaligned
    assert lib.finc_backward(*args, ctypes.c_void_p(0x1900000), None) == finc.EINVAL   # over dx
    assert lib.finc_backward(*args, ctypes.c_void_p(0x1100000), None) == finc.EINVAL   # over K
    B, C, H, W, k = SHAPE
    n = lib.finc_backward_workspace_bytes(B, C, H, W, k)
    assert n >= C * C * k * k * 4 and n % 256 == 0
    assert lib.finc_backward_workspace_bytes(B, 65, H, W, k) == 0


def test_unit_split_backward_rejects():
    lib = finc.lib()
    ws = ctypes.c_void_p(0x40000000)
    B, C, H, W, k = SHAPE
    args = (FAKE, FAKE2, FAKE3, FAKE4, NULL, 0.0)
    assert lib.finc_unit_backward(*args, B, C, H, W, k, NULL, None) == finc.EINVAL    # no ws
    assert lib.finc_unit_backward(*args, B, C, H, W, k, ctypes.c_void_p(0x40000010),
                                  None) == finc.EINVAL                                # misaligned
    assert lib.finc_unit_backward(FAKE, FAKE2, FAKE3, ctypes.c_void_p(0x100000 + 64), NULL, 0.0,
                                  B, C, H, W, k, ws, None) == finc.EINVAL            # dx over x
    assert lib.finc_unit_backward(*args, B, 65, H, W, k, ws, None) == finc.EINVAL
    assert lib.finc_unit_backward(NULL, FAKE2, FAKE3, FAKE4, NULL, 0.0, B, C, H, W, k, ws,
                                  None) == finc.EINVAL                                # no x
    assert lib.finc_split_backward(*args, B, 6, H, W, k, ws, None) == finc.EINVAL     # C % 4
    assert lib.finc_split_backward(*args, B, 8, H, W, 8, ws, None) == finc.EINVAL     # k > 7
    assert lib.finc_split_backward_workspace_bytes(B, 6, H, W, k) == 0
    assert lib.finc_split_backward_workspace_bytes(B, 8, H, W, k) >= 4 * 4 * k * k
    n = lib.finc_unit_backward_workspace_bytes(B, C, H, W, k)
    assert n >= 4 * B * C * H * W * 4 and n % 256 == 0


def test_actnorm_backward_and_nll_reject():
    lib = finc.lib()
    ws = ctypes.c_void_p(0x40000000)
    B, C, H, W = 2, 3, 4, 5
    S = ctypes.c_void_p(0x2000000)
    assert lib.finc_actnorm_backward(FAKE, FAKE2, S, FAKE4, NULL, NULL, 0.0, B, C, H, W, NULL,
                                     None) == finc.EINVAL                            # no ws
    assert lib.finc_actnorm_backward(FAKE, FAKE2, S, ctypes.c_void_p(0x100000 + 8), NULL, NULL,
                                     0.0, B, C, H, W, ws, None) == finc.EINVAL       # dx over x
    assert lib.finc_actnorm_backward(FAKE, FAKE2, S, NULL, S, NULL, 0.0, B, C, H, W, ws,
                                     None) == finc.EINVAL                            # ds over s
    assert lib.finc_actnorm_backward(FAKE, FAKE2, S, NULL, FAKE4, FAKE4, 0.0, B, C, H, W, ws,
                                     None) == finc.EINVAL                            # ds over db
    assert lib.finc_actnorm_backward_workspace_bytes(B, 0, H, W) == 0
    z = (ctypes.c_void_p * 2)(0x100000, 0x900000)
    n = (ctypes.c_longlong * 2)(16, 8)
    LD, OUT = ctypes.c_void_p(0x3000000), ctypes.c_void_p(0x3100000)
    assert lib.finc_gauss_nll(z, n, 0, B, LD, OUT, NULL, None) == finc.EINVAL        # L = 0
    assert lib.finc_gauss_nll(z, n, 17, B, LD, OUT, NULL, None) == finc.EINVAL       # L > 16
    assert lib.finc_gauss_nll(z, n, 2, B, LD, LD, NULL, None) == finc.EINVAL         # nll over logdet
    assert lib.finc_gauss_nll(z, n, 2, B, LD, OUT, OUT, None) == finc.EINVAL         # bpd over nll
    assert lib.finc_gauss_nll(z, n, 2, B, LD, ctypes.c_void_p(0x100000), NULL,
                              None) == finc.EINVAL                                   # nll over z
    n0 = (ctypes.c_longlong * 2)(16, 0)
    assert lib.finc_gauss_nll(z, n0, 2, B, LD, OUT, NULL, None) == finc.EINVAL       # empty latent


def test_inverse_rejects():
    lib = finc.lib()
    ws = ctypes.c_void_p(0x4000000)
    assert lib.finc_inverse(FAKE, FAKE2, FAKE, *SHAPE, 0, NULL, None) == finc.EINVAL
    assert lib.finc_inverse(FAKE, FAKE2, FAKE, *SHAPE, 0, ctypes.c_void_p(0x4000010),
                            None) == finc.EINVAL                         # misaligned
    assert lib.finc_inverse(FAKE, FAKE2, FAKE, *SHAPE, 7, ws, None) == finc.EINVAL
    # partial overlap of y and x is rejected, identical pointers (in place) are not
    assert lib.finc_inverse(FAKE, ctypes.c_void_p(0x100000 + 64), FAKE2, *SHAPE, 0, ws,
                            None) == finc.EINVAL
    # workspace overlapping the output
    assert lib.finc_inverse(FAKE2, FAKE, ctypes.c_void_p(0x8000000), *SHAPE, 0,
                            ctypes.c_void_p(0x100000), None) == finc.EINVAL
    assert lib.finc_inverse_prepared(FAKE, FAKE2, NULL, *SHAPE, 0, None) == finc.EINVAL
    assert lib.finc_unit_inverse(FAKE, FAKE2, FAKE, *SHAPE, NULL, None) == finc.EINVAL
    assert lib.finc_unit_inverse_prepared(FAKE, FAKE2, NULL, *SHAPE, None) == finc.EINVAL


def test_logdet_and_prepare_reject():
    lib = finc.lib()
    out = ctypes.c_void_p(0x200000)
    assert lib.finc_logdet(NULL, 12, 3, 0, 16, 16, out, None) == finc.EINVAL
    assert lib.finc_logdet(FAKE, 12, 3, 5, 16, 16, out, None) == finc.EINVAL
    assert lib.finc_logdet(FAKE, 12, 3, 0, 16, 16, NULL, None) == finc.EINVAL
    assert lib.finc_unit_logdet(FAKE, 0, 3, 16, 16, out, None) == finc.EINVAL
    corners = (ctypes.c_int * 2)(0, 9)
    ws = ctypes.c_void_p(0x4000000)
    assert lib.finc_prepare(FAKE, 2, corners, 12, 3, ws, None) == finc.EINVAL
    corners = (ctypes.c_int * 2)(0, 1)
    assert lib.finc_prepare(FAKE, 2, corners, 12, 3, ctypes.c_void_p(0x4000004),
                            None) == finc.EINVAL
    assert lib.finc_prepare(FAKE, -1, corners, 12, 3, ws, None) == finc.EINVAL
    assert lib.finc_prepare(FAKE, 0, corners, 12, 3, ws, None) == finc.OK   # nothing to do


def test_split_rejects():
    lib = finc.lib()
    ws = ctypes.c_void_p(0x4000000)
    for C in (0, 2, 13, 260):   # not a multiple of 4, or quarters above FINC_MAX_C
        assert lib.finc_split_forward(FAKE, FAKE2, FAKE, NULL, NULL, 2, C, 8, 8, 3,
                                      None) == finc.EINVAL
        assert lib.finc_split_inverse(FAKE, FAKE2, FAKE, 2, C, 8, 8, 3, ws, None) == finc.EINVAL
        assert lib.finc_split_logdet(FAKE, C, 3, 8, 8, ctypes.c_void_p(0x200000),
                                     None) == finc.EINVAL
    assert lib.finc_split_forward(NULL, FAKE2, FAKE, NULL, NULL, 2, 12, 8, 8, 3, None) == finc.EINVAL
    assert lib.finc_split_forward(FAKE, ctypes.c_void_p(0x100000 + 64), FAKE2, NULL, NULL, 2,
                                  12, 8, 8, 3, None) == finc.EINVAL   # x / y overlap
    assert lib.finc_split_inverse(FAKE, FAKE2, FAKE, 2, 12, 8, 8, 3, NULL, None) == finc.EINVAL
    assert lib.finc_split_inverse_prepared(FAKE, FAKE2, ctypes.c_void_p(0x4000010), 2, 12, 8,
                                           8, 3, None) == finc.EINVAL   # misaligned
    assert lib.finc_split_inverse_prepared(FAKE, FAKE2, ws, 0, 12, 8, 8, 3, None) == finc.OK
    assert lib.finc_split_inverse(FAKE, FAKE2, FAKE, 0, 12, 8, 8, 3, ws, None) == finc.OK


def test_stack_rejects():
    lib = finc.lib()
    z = (ctypes.c_void_p * 3)(0x1000000, 0x2000000, 0x3000000)
    ws = ctypes.c_void_p(0x40000000)
    x = ctypes.c_void_p(0x50000000)
    ok = dict(B=64, L=3, U=8, C1=12, H1=32, W1=32, k=3)

    def call(**kw):
        a = dict(ok, **kw)
        return lib.finc_stack_inverse(z, x, FAKE, FAKE, FAKE, a["B"], a["L"], a["U"], a["C1"],
                                      a["H1"], a["W1"], a["k"], ws, None)

    assert call(C1=13) == finc.EINVAL          # odd channels cannot be split
    assert call(H1=30) == finc.EINVAL          # not divisible by 4
    assert call(L=9) == finc.EINVAL
    assert call(C1=24) == finc.EINVAL          # 96 channels at the top
    assert call(k=0) == finc.EINVAL
    assert call(B=0) == finc.OK                # nothing to enqueue
    assert lib.finc_stack_inverse(None, x, FAKE, FAKE, FAKE, 64, 3, 8, 12, 32, 32, 3, ws,
                                  None) == finc.EINVAL


def test_stack_overlaps_rejected():
    """The output x is written, so every buffer the stack reads (latents,
    scale, bias, K or the prepared weights) must be clear of it; the
    workspace is written too and must be clear of all of them."""
    lib = finc.lib()
    x, ws = 0x50000000, 0x40000000     # x: 3 MB, workspace: 3.4 MB
    zs = [0x1000000, 0x2000000, 0x3000000]
    K, S, Bi = 0x60000000, 0x61000000, 0x62000000
    shape = (64, 3, 8, 12, 32, 32, 3)

    def full(z=zs, K=K, S=S, Bi=Bi, x=x, ws=ws):
        zz = (ctypes.c_void_p * 3)(*z)
        return lib.finc_stack_inverse(zz, ctypes.c_void_p(x), ctypes.c_void_p(K),
                                      ctypes.c_void_p(S), ctypes.c_void_p(Bi), *shape,
                                      ctypes.c_void_p(ws), None)

    def prepared(z=zs, S=S, Bi=Bi, x=x, p=ws, B=64):
        # (B = 64 only where the checks reject the call before any HIP call)
        zz = (ctypes.c_void_p * 3)(*z)
        return lib.finc_stack_inverse_prepared(zz, ctypes.c_void_p(x), ctypes.c_void_p(p),
                                               ctypes.c_void_p(S), ctypes.c_void_p(Bi), B,
                                               *shape[1:], None)

    assert prepared(B=0) == finc.OK                           # (B = 0: checks only)
    assert full(S=x + 64) == finc.EINVAL                      # scale inside x
    assert full(Bi=x + 4096) == finc.EINVAL                   # bias inside x
    assert full(K=x + 1024) == finc.EINVAL                    # K inside x
    assert full(K=ws + 1024) == finc.EINVAL                   # K inside the workspace
    assert full(S=ws + 64) == finc.EINVAL                     # scale inside the workspace
    assert full(z=[zs[0], ws + 512, zs[2]]) == finc.EINVAL    # a latent inside the workspace
    assert full(z=[x + 4, zs[1], zs[2]]) == finc.EINVAL       # a latent inside x
    assert prepared(p=x) == finc.EINVAL                       # prepared weights inside x
    assert prepared(S=x + 64) == finc.EINVAL
    assert prepared(Bi=x + 64) == finc.EINVAL
    assert prepared(S=ws, Bi=ws + 8, B=0) == finc.OK          # read-only buffers may share


def test_noalloc_rejects_before_any_hip_call():
    lib = finc.lib()
    assert lib.finc_inverse_noalloc(NULL, FAKE2, FAKE, 2, 12, 16, 16, 3, 0, None) == finc.EINVAL
    assert lib.finc_inverse_noalloc(FAKE, FAKE2, NULL, 2, 12, 16, 16, 3, 0, None) == finc.EINVAL
    assert lib.finc_inverse_noalloc(FAKE, FAKE2, FAKE, 2, 65, 16, 16, 3, 0, None) == finc.EINVAL
    assert lib.finc_inverse_noalloc(FAKE, FAKE2, FAKE, 2, 12, 16, 16, 3, 4, None) == finc.EINVAL
    # x overlapping y other than exactly (in place) is rejected
    assert lib.finc_inverse_noalloc(FAKE, ctypes.c_void_p(0x100000 + 64), FAKE, 2, 12, 16, 16, 3,
                                    0, None) == finc.EINVAL
    # an empty batch checks the shape and enqueues nothing
    assert lib.finc_inverse_noalloc(FAKE, FAKE2, FAKE, 0, 12, 16, 16, 3, 0, None) == finc.OK
    assert lib.finc_inverse_noalloc(FAKE, FAKE2, FAKE, 0, 64, 16, 16, 7, 0,
                                    None) == finc.EUNSUPPORTED


def test_empty_batch_enqueues_nothing():
    lib = finc.lib()
    ws = ctypes.c_void_p(0x4000000)
    assert lib.finc_forward(FAKE, FAKE2, FAKE, NULL, NULL, 0, 12, 16, 16, 3, 0, None) == finc.OK
    assert lib.finc_unit_forward(FAKE, FAKE2, FAKE, NULL, NULL, 0, 12, 16, 16, 3, None) == finc.OK
    assert lib.finc_inverse(FAKE, FAKE2, FAKE, 0, 12, 16, 16, 3, 0, ws, None) == finc.OK
    assert lib.finc_inverse_prepared(FAKE, FAKE2, ws, 0, 12, 16, 16, 3, 0, None) == finc.OK
    assert lib.finc_unit_inverse(FAKE, FAKE2, FAKE, 0, 12, 16, 16, 3, ws, None) == finc.OK


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(finc, "_lib", None)
    with pytest.raises(RuntimeError, match="not built"):
        finc.lib(str(tmp_path / "missing.so"))


def test_inverse_steps_rejects():
    lib = finc.lib()
    S = ctypes.c_void_p(0x2000000)
    P = ctypes.c_void_p(0x40000000)
    B, C, H, W, k = SHAPE
    # unit kind, too small a buffer, steps over y, misaligned prepared, bad corner
    assert lib.finc_inverse_steps(finc.PLAN_UNIT, FAKE, FAKE2, P, B, C, H, W, k, 0, S, 100,
                                  None) == finc.EINVAL
    assert lib.finc_inverse_steps(finc.PLAN_LAYER, FAKE, FAKE2, P, B, C, H, W, k, 0, S, 1,
                                  None) == finc.EINVAL
    assert lib.finc_inverse_steps(finc.PLAN_LAYER, FAKE, FAKE2, P, B, C, H, W, k, 0, FAKE, 100,
                                  None) == finc.EINVAL
    assert lib.finc_inverse_steps(finc.PLAN_LAYER, FAKE, FAKE2, ctypes.c_void_p(0x40000010), B,
                                  C, H, W, k, 0, S, 100, None) == finc.EINVAL
    assert lib.finc_inverse_steps(finc.PLAN_LAYER, FAKE, FAKE2, P, B, C, H, W, k, 4, S, 100,
                                  None) == finc.EINVAL
    assert lib.finc_inverse_steps(finc.PLAN_SPLIT, FAKE, FAKE2, P, B, 6, H, W, k, 0, S, 100,
                                  None) == finc.EINVAL


def test_inverse_timeline_rejects():
    lib = finc.lib()
    S = ctypes.c_void_p(0x2000000)
    P = ctypes.c_void_p(0x40000000)
    B, C, H, W, k = SHAPE
    waves = finc.inverse_plan(finc.PLAN_LAYER, C, H, W, k)[0]["threads"] // 64
    need = B * waves * 4
    # unit kind, no buffer, one stamp short, stamps over y, misaligned
    # prepared, bad corner, channels the split unit cannot take
    assert lib.finc_inverse_timeline(finc.PLAN_UNIT, FAKE, FAKE2, P, B, C, H, W, k, 0, S, need,
                                     None) == finc.EINVAL
    assert lib.finc_inverse_timeline(finc.PLAN_LAYER, FAKE, FAKE2, P, B, C, H, W, k, 0, None,
                                     need, None) == finc.EINVAL
    assert lib.finc_inverse_timeline(finc.PLAN_LAYER, FAKE, FAKE2, P, B, C, H, W, k, 0, S,
                                     need - 1, None) == finc.EINVAL
    assert lib.finc_inverse_timeline(finc.PLAN_LAYER, FAKE, FAKE2, P, B, C, H, W, k, 0, FAKE,
                                     need, None) == finc.EINVAL
    assert lib.finc_inverse_timeline(finc.PLAN_LAYER, FAKE, FAKE2, ctypes.c_void_p(0x40000010),
                                     B, C, H, W, k, 0, S, need, None) == finc.EINVAL
    assert lib.finc_inverse_timeline(finc.PLAN_LAYER, FAKE, FAKE2, P, B, C, H, W, k, 4, S, need,
                                     None) == finc.EINVAL
    assert lib.finc_inverse_timeline(finc.PLAN_SPLIT, FAKE, FAKE2, P, B, 6, H, W, k, 0, S, need,
                                     None) == finc.EINVAL


def test_banded_rejects():
    lib = finc.lib()
    ws = ctypes.c_void_p(0x40000000)
    info = (ctypes.c_int * 4)()
    assert lib.finc_banded_plan(17, 256, 256, 3, info) == finc.EUNSUPPORTED   # C > 16
    assert lib.finc_banded_plan(2, 256, 256, 1, info) == finc.EUNSUPPORTED    # k = 1
    assert lib.finc_banded_plan(2, 256, 256, 3, None) == finc.EINVAL
    assert lib.finc_banded_plan(2, 256, 256, 3, info) == finc.OK
    assert info[1] == 128 and info[2] == 2 and info[0] % 64 == 0
    assert lib.finc_banded_workspace_bytes(1, 17, 256, 256, 3, 1) == 0
    assert lib.finc_banded_workspace_bytes(1, 2, 256, 256, 3, 2) == 0        # 1 or 4 layers
    n1 = lib.finc_banded_workspace_bytes(3, 2, 256, 256, 3, 1)
    assert n1 >= lib.finc_workspace_bytes(2, 3, 1) + 4 * (2 + 3 * 2)
    args = (FAKE, FAKE2, FAKE3, 1, 2, 256, 256, 3)
    assert lib.finc_inverse_banded(*args, 0, NULL, None) == finc.EINVAL              # no ws
    assert lib.finc_inverse_banded(*args, 4, ws, None) == finc.EINVAL                # corner
    assert lib.finc_inverse_banded(*args, 0, ctypes.c_void_p(0x40000010), None) == finc.EINVAL
    assert lib.finc_inverse_banded(FAKE, ctypes.c_void_p(0x100000 + 64), FAKE3, 1, 2, 256, 256, 3,
                                   0, ws, None) == finc.EINVAL                       # x over y
    assert lib.finc_unit_inverse_banded(FAKE, FAKE2, FAKE3, 1, 17, 64, 64, 3, ws,
                                        None) == finc.EUNSUPPORTED
    assert lib.finc_unit_inverse_banded(FAKE, FAKE2, FAKE3, 1, 2, 64, 64, 3,
                                        ctypes.c_void_p(0x1100000 - 256), None) == finc.EINVAL


def test_stack_train_rejects():
    lib = finc.lib()
    ws = ctypes.c_void_p(0x40000000)
    z = (ctypes.c_void_p * 2)(0x2000000, 0x3000000)
    K, S, Bb = ctypes.c_void_p(0x5000000), ctypes.c_void_p(0x6000000), ctypes.c_void_p(0x6100000)
    args = (FAKE, z, NULL, K, S, Bb)
    assert lib.finc_stack_train_workspace_bytes(2, 2, 2, 3, 16, 16, 3) == 0        # odd C1
    assert lib.finc_stack_train_workspace_bytes(2, 2, 2, 4, 15, 16, 3) == 0        # odd H1
    assert lib.finc_stack_train_workspace_bytes(2, 2, 2, 48, 16, 16, 3) == 0       # 96 > 64
    assert lib.finc_stack_train_workspace_bytes(2, 2, 2, 4, 16, 16, 3) > 0
    assert lib.finc_stack_forward(*args, 2, 2, 2, 4, 16, 16, 3, NULL, None) == finc.EINVAL
    assert lib.finc_stack_forward(*args, 2, 2, 2, 4, 16, 16, 3, ctypes.c_void_p(0x40000010),
                                  None) == finc.EINVAL
    zbad = (ctypes.c_void_p * 2)(0x100000 + 64, 0x3000000)                        # z over x
    assert lib.finc_stack_forward(FAKE, zbad, NULL, K, S, Bb, 2, 2, 2, 4, 16, 16, 3, ws,
                                  None) == finc.EINVAL
    assert lib.finc_stack_backward(FAKE, z, K, S, Bb, NULL, S, NULL, NULL, 0.0, 2, 2, 2, 4, 16,
                                   16, 3, ws, None) == finc.EINVAL                 # dK over scale
    assert lib.finc_stack_backward(FAKE, z, K, S, Bb, NULL, NULL, NULL, NULL, 0.0, 2, 2, 2, 4, 16,
                                   16, 3, ctypes.c_void_p(0x2000000 - 256), None) == finc.EINVAL
