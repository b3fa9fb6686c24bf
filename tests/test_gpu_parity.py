"""HIP path vs the CPU oracle, element by element, through the C ABI.

Bar: |gpu - oracle| <= 1e-4 * max(1, |oracle|) elementwise for single
layers and units; the round trip inverse(forward(x)) within 1e-4 of x.  Both
sides see the same fp32 inputs (the oracle computes on them in fp64).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2301_09266_amd import finc, synth

pytestmark = pytest.mark.gpu

from gpu_util import (DEV, TOL, assert_close, assert_round_trip, dev, f64, host,  # noqa: E402
                      poisoned)


@pytest.fixture(scope="module")
def orc():
    return oracle.default()


SHAPES = [
    # (B, C, H, W, k)
    (2, 1, 1, 1, 3), (2, 3, 1, 7, 3), (2, 3, 7, 1, 3), (3, 5, 5, 9, 2), (2, 12, 13, 17, 3),
    (2, 4, 6, 6, 1), (1, 7, 9, 6, 5), (2, 12, 24, 24, 3), (1, 16, 11, 8, 4), (1, 33, 7, 9, 3),
]


@pytest.mark.parametrize("corner", [0, 1, 2, 3])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_layer_forward_inverse(orc, shape, corner):
    B, C, H, W, k = shape
    print(f"layer B={B} C={C} H={H} W={W} k={k} corner={corner}", flush=True)
    rng = np.random.default_rng(hash((shape, corner)) % 2**32)
    x = rng.normal(size=(B, C, H, W))
    K = synth.garbage_in_mask(synth.masked_kernel(C, k, corner, 1000 + corner), corner)
    xd, Kd = dev(x), dev(K)
    y = finc.forward(xd, Kd, corner, out=poisoned(x.shape))
    assert_close(host(y), orc.forward(f64(x), f64(K), corner), "forward")
    # inverse of the GPU forward output, against the oracle on the same input
    yh = host(y)
    xr = finc.inverse(y, Kd, corner, out=poisoned(x.shape))
    assert_close(host(xr), orc.inverse(yh, f64(K), corner), "inverse")
    assert_round_trip(host(xr), f64(x), "layer")
    # inverse of an arbitrary input
    z = rng.normal(size=(B, C, H, W))
    xz = finc.inverse(dev(z), Kd, corner)
    assert_close(host(xz), orc.inverse(f64(z), f64(K), corner), "inverse of z")
    ld = finc.logdet(Kd, corner, H, W)
    r = orc.logdet(f64(K), corner, H, W)
    assert abs(float(ld.cpu()[0]) - r) <= TOL * max(1.0, abs(r))
    # the forward's own log|det| output, and its y unchanged by asking for it
    ldf = torch.full((1,), float("nan"), dtype=torch.float64, device=DEV)
    y2 = finc.forward(xd, Kd, corner, logdet=ldf)
    assert abs(float(ldf.cpu()[0]) - r) <= TOL * max(1.0, abs(r))
    assert torch.equal(y2, y)


# Single layers whose rows are stored as they complete (one channel tile,
# rows of at most 512 values) next to ones just past that bound, which store
# the image after the last diagonal: every corner (the frame's rows run
# bottom-up for the lower corners), one and several 16-row tiles, one row.
DRAIN_SHAPES = [
    # (B, C, H, W, k)
    (2, 16, 16, 32, 3), (2, 16, 16, 33, 3), (1, 12, 20, 40, 3), (1, 12, 20, 43, 3),
    (3, 12, 16, 16, 3), (1, 1, 1, 512, 3), (1, 1, 3, 513, 3), (2, 4, 9, 20, 7),
]


@pytest.mark.parametrize("corner", [0, 1, 2, 3])
@pytest.mark.parametrize("shape", DRAIN_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_layer_inverse_row_drain(orc, shape, corner):
    B, C, H, W, k = shape
    print(f"drain B={B} C={C} H={H} W={W} k={k} corner={corner}", flush=True)
    rng = np.random.default_rng(hash(("drain", shape, corner)) % 2**32)
    K = synth.masked_kernel(C, k, corner, 2000 + corner)
    z = rng.normal(size=(B, C, H, W))
    xz = finc.inverse(dev(z), dev(K), corner, out=poisoned(z.shape))
    assert_close(host(xz), orc.inverse(f64(z), f64(K), corner), "inverse")
    # in place: the whole image is in LDS before the first row goes out
    zi = dev(z)
    finc.inverse(zi, dev(K), corner, out=zi)
    assert torch.equal(zi, xz)


# Layers at the largest C the forward supports at k = 3, where the padding
# quad groups' weight fragments do not fit in LDS beside the rows (those
# groups read one shared zero fragment): every C from 57 at 8 x 8 and from 49
# at 32 x 32 takes that form.
@pytest.mark.parametrize("corner", [0, 3])
@pytest.mark.parametrize("shape", [(2, 57, 8, 8, 3), (2, 60, 8, 8, 3), (1, 52, 32, 32, 3)],
                         ids=lambda s: "x".join(map(str, s)))
def test_forward_zero_fragment(orc, shape, corner):
    B, C, H, W, k = shape
    print(f"forward B={B} C={C} H={H} W={W} k={k} corner={corner}", flush=True)
    rng = np.random.default_rng(hash(("zf", shape, corner)) % 2**32)
    x = rng.normal(size=(B, C, H, W))
    K = synth.garbage_in_mask(synth.masked_kernel(C, k, corner, 3000 + corner), corner)
    y = finc.forward(dev(x), dev(K), corner, out=poisoned(x.shape))
    assert_close(host(y), orc.forward(f64(x), f64(K), corner), "forward")


def test_inverse_in_place(orc):
    c = synth.make("layer_c12_16x16_b64_k3", B=5)
    y = dev(orc.forward(c["x"], c["K"], 0))
    want = orc.inverse(host(y), f64(c["K"]), 0)
    finc.inverse(y, dev(c["K"]), 0, out=y)
    assert_close(host(y), want, "in-place inverse")


def offset_copy(t, floats=1):
    """A copy of t whose data starts `floats` floats past a 256-byte boundary."""
    buf = torch.empty(t.numel() + floats, dtype=t.dtype, device=t.device)
    u = buf[floats:].view(t.shape)
    u.copy_(t)
    return u


@pytest.mark.parametrize("shape", [(3, 12, 16, 16, 3), (2, 5, 8, 12, 3), (2, 3, 6, 10, 2)],
                         ids=lambda s: "x".join(map(str, s)))
def test_unaligned_buffers(orc, shape):
    """Input and output 4 bytes off 16-byte alignment: the inverse's staging
    takes its scalar route and gives the aligned call's result bit for bit."""
    B, C, H, W, k = shape
    print(f"unaligned B={B} C={C} H={H} W={W} k={k}", flush=True)
    rng = np.random.default_rng(7 + C)
    K = dev(synth.masked_kernel(C, k, 1, 21))
    y = dev(rng.normal(size=(B, C, H, W)))
    want = finc.inverse(y, K, 1)
    assert_close(host(want), orc.inverse(host(y), host(K), 1), "aligned inverse")
    for fi, fo in [(1, 0), (0, 1), (1, 3), (2, 2)]:
        yu = offset_copy(y, fi) if fi else y
        out = offset_copy(poisoned(y.shape), fo) if fo else poisoned(y.shape)
        got = finc.inverse(yu, K, 1, out=out)
        assert torch.equal(got, want), (fi, fo)
    # the forward and the unit (four layers in one launch) likewise
    assert torch.equal(finc.forward(offset_copy(y, 3), K, 1, out=offset_copy(y, 1)),
                       finc.forward(y, K, 1))
    K4 = dev(synth.unit_kernels(C, k))
    wantu = finc.unit_inverse(y, K4)
    gotu = finc.unit_inverse(offset_copy(y, 1), K4, out=offset_copy(poisoned(y.shape), 3))
    assert torch.equal(gotu, wantu)


def test_logdet_singular():
    K = synth.masked_kernel(4, 3, 2, 5)
    K[2, 2, 0, 2] = 0.0
    assert float(finc.logdet(dev(K), 2, 5, 5).cpu()[0]) == -np.inf


def test_prepared_matches_unprepared(orc):
    c = synth.make("layer_c12_16x16_b64_k3", B=4)
    Kd = dev(c["K"])
    y = dev(orc.forward(c["x"], c["K"], 0))
    prep = finc.prepare(Kd, [0])
    a = finc.inverse_prepared(y, prep, 3, 0)
    b = finc.inverse(y, Kd, 0)
    assert torch.equal(a, b)


@pytest.mark.parametrize("C,k,unit", [(12, 3, False), (3, 2, False), (33, 3, False),
                                      (12, 3, True), (20, 5, True)])
def test_forward_prepares_weights(C, k, unit):
    """The forward's prepared-weights side output equals finc_prepare's, bit for
    bit (its own workgroups for C <= 16, a second launch above), and the
    forward's y is unchanged by asking for it."""
    print(f"forward+prepare C={C} k={k} unit={unit}", flush=True)
    rng = np.random.default_rng(C * 10 + k)
    x = dev(rng.normal(size=(3, C, 9, 7)))
    if unit:
        Kd = dev(synth.unit_kernels(C, k, 0))
        ref = torch.full((finc.workspace_bytes(C, k, 4),), 0xAB, dtype=torch.uint8, device=DEV)
        finc.prepare(Kd, [0, 1, 2, 3], out=ref)   # (the same filler in unwritten gaps)
        pp = torch.full_like(ref, 0xAB)
        y = finc.unit_forward(x, Kd, prepared=pp)
        assert torch.equal(y, finc.unit_forward(x, Kd))
    else:
        Kd = dev(synth.masked_kernel(C, k, 1, 77))
        ref = torch.full((finc.workspace_bytes(C, k, 1),), 0xAB, dtype=torch.uint8, device=DEV)
        finc.prepare(Kd, [1], out=ref)
        pp = torch.full_like(ref, 0xAB)
        y = finc.forward(x, Kd, 1, prepared=pp)
        assert torch.equal(y, finc.forward(x, Kd, 1))
    assert torch.equal(pp, ref)


# --- the workloads at full size ------------------------------------------------

def _layer_workload(orc, name):
    c = synth.make(name)
    x, K, corner = c["x"], c["K"], c["corner"]
    xd, Kd = dev(x), dev(K)
    y = finc.forward(xd, Kd, corner, out=poisoned(x.shape))
    yh = host(y)
    assert_close(yh, orc.forward(f64(x), f64(K), corner), f"{name} forward")
    xr = finc.inverse(y, Kd, corner, out=poisoned(x.shape))
    assert_close(host(xr), orc.inverse(yh, f64(K), corner), f"{name} inverse")
    assert_round_trip(host(xr), f64(x), name)
    xz = finc.inverse(dev(c["z"]), Kd, corner)
    assert_close(host(xz), orc.inverse(f64(c["z"]), f64(K), corner), f"{name} inverse(z)")
    ld = float(finc.logdet(Kd, corner, c["H"], c["W"]).cpu()[0])
    r = orc.logdet(f64(K), corner, c["H"], c["W"])
    assert abs(ld - r) <= TOL * max(1.0, abs(r))
    # bitwise determinism and batch invariance
    xr2 = finc.inverse(y, Kd, corner)
    assert torch.equal(xr, xr2)
    one = finc.inverse(y[-1:].contiguous(), Kd, corner)
    assert torch.equal(one[0], xr[-1])
    y2 = finc.forward(xd, Kd, corner)
    assert torch.equal(y, y2)
    assert torch.equal(finc.forward(xd[-1:].contiguous(), Kd, corner)[0], y[-1])


@pytest.mark.parametrize("name", ["layer_c3_8x8_b1_k3", "layer_c12_16x16_b64_k3",
                                  "layer_c12_32x32_b64_k3", "layer_c12_32x32_b64_k5"])
def test_layer_workload(orc, name):
    print(f"workload {name}", flush=True)
    _layer_workload(orc, name)


def test_dense_jacobian_slogdet_8x8():
    """8x8x3 workload: the GPU forward applied to all 192 basis images gives
    the dense Jacobian; its slogdet equals the GPU log|det|."""
    c = synth.make("layer_c3_8x8_b1_k3")
    n = 3 * 8 * 8
    basis = torch.eye(n, device=DEV).reshape(n, 3, 8, 8).contiguous()
    J = host(finc.forward(basis, dev(c["K"]), 0)).reshape(n, n).T
    sign, ld = np.linalg.slogdet(J)
    assert sign == 1.0
    g = float(finc.logdet(dev(c["K"]), 0, 8, 8).cpu()[0])
    assert abs(g - ld) <= TOL * max(1.0, abs(ld))


@pytest.mark.parametrize("name", ["unit_c12_16x16_b256_k3", "unit_c48_8x8_b256_k3",
                                  "unit_c12_32x32_b64_k3", "unit_c12_32x32_b64_k5"])
def test_unit_workload(orc, name):
    print(f"workload {name}", flush=True)
    c = synth.make(name)
    x, K4 = c["x"], c["K4"]
    xd, K4d = dev(x), dev(K4)
    y = finc.unit_forward(xd, K4d, out=poisoned(x.shape))
    yh = host(y)
    assert_close(yh, orc.unit_forward(f64(x), f64(K4)), f"{name} unit forward")
    xr = finc.unit_inverse(y, K4d, out=poisoned(x.shape))
    assert_close(host(xr), orc.unit_inverse(yh, f64(K4)), f"{name} unit inverse")
    assert_round_trip(host(xr), f64(x), f"{name} unit")
    ld = float(finc.unit_logdet(K4d, c["H"], c["W"]).cpu()[0])
    r = orc.unit_logdet(f64(K4), c["H"], c["W"])
    assert abs(ld - r) <= TOL * max(1.0, abs(r))
    ldf = torch.full((1,), float("nan"), dtype=torch.float64, device=DEV)
    assert torch.equal(finc.unit_forward(xd, K4d, logdet=ldf), y)
    assert abs(float(ldf.cpu()[0]) - r) <= TOL * max(1.0, abs(r))
    xr2 = finc.unit_inverse(y, K4d)
    assert torch.equal(xr, xr2)
    inplace = xd.clone()
    finc.unit_forward(inplace, K4d, out=inplace)
    assert torch.equal(inplace, y)
    assert torch.equal(finc.unit_inverse(y[3:4].contiguous(), K4d)[0], xr[3])


@pytest.mark.parametrize("shape", [(2, 2, 64, 64, 3), (1, 3, 48, 64, 3), (1, 2, 64, 40, 2)],
                         ids=lambda s: "x".join(map(str, s)))
def test_large_images(orc, shape):
    """Images whose padded partial-tile layout does not fit in LDS (the
    compact one is used): layer and unit, against the oracle."""
    B, C, H, W, k = shape
    print(f"large B={B} C={C} H={H} W={W} k={k}", flush=True)
    rng = np.random.default_rng(C * 1000 + H + W)
    x = rng.normal(size=(B, C, H, W))
    K = synth.masked_kernel(C, k, 3, 55)
    xd, Kd = dev(x), dev(K)
    y = finc.forward(xd, Kd, 3)
    yh = host(y)
    assert_close(yh, orc.forward(f64(x), f64(K), 3), "forward")
    xr = finc.inverse(y, Kd, 3, out=poisoned(x.shape))
    assert_close(host(xr), orc.inverse(yh, f64(K), 3), "inverse")
    assert_round_trip(host(xr), f64(x), "layer")
    K4 = synth.unit_kernels(C, k, 4)
    K4d = dev(K4)
    yu = finc.unit_forward(xd, K4d)
    yuh = host(yu)
    assert_close(yuh, orc.unit_forward(f64(x), f64(K4)), "unit forward")
    xu = finc.unit_inverse(yu, K4d, out=poisoned(x.shape))
    assert_close(host(xu), orc.unit_inverse(yuh, f64(K4)), "unit inverse")
    assert_round_trip(host(xu), f64(x), "unit")


@pytest.mark.parametrize("shape,corner", [((2, 2, 128, 128, 3), 0), ((1, 3, 16, 600, 3), 3),
                                          ((2, 4, 40, 300, 2), 1), ((1, 2, 100, 130, 5), 2)],
                         ids=lambda s: "x".join(map(str, s)) if isinstance(s, tuple) else str(s))
def test_stream_images(orc, shape, corner):
    """Images too large for LDS: the inverse streams them through column
    rings (layer, in place, and the unit as four launches) -- against the
    oracle."""
    B, C, H, W, k = shape
    print(f"stream B={B} C={C} H={H} W={W} k={k} corner={corner}", flush=True)
    rng = np.random.default_rng(H * W + C)
    x = rng.normal(size=(B, C, H, W))
    K = synth.garbage_in_mask(synth.masked_kernel(C, k, corner, 31), corner)
    Kd = dev(K)
    y = finc.forward(dev(x), Kd, corner)
    yh = host(y)
    assert_close(yh, orc.forward(f64(x), f64(K), corner), "forward")
    xr = finc.inverse(y, Kd, corner, out=poisoned(x.shape))
    assert_close(host(xr), orc.inverse(yh, f64(K), corner), "inverse")
    assert_round_trip(host(xr), f64(x), "layer")
    z = rng.normal(size=x.shape)
    zd = dev(z)
    finc.inverse(zd, Kd, corner, out=zd)   # in place
    assert_close(host(zd), orc.inverse(f64(z), f64(K), corner), "in-place inverse of z")
    assert torch.equal(finc.inverse(y[-1:].contiguous(), Kd, corner)[0], xr[-1])
    K4 = synth.unit_kernels(C, k, 8)
    yu = orc.unit_forward(f64(x), f64(K4)).astype(np.float32)
    xu = finc.unit_inverse(dev(yu), dev(K4), out=poisoned(x.shape))
    assert_close(host(xu), orc.unit_inverse(f64(yu), f64(K4)), "unit inverse")
    assert_round_trip(host(xu), f64(x), "unit")


SPLIT_SHAPES = [
    # (B, C, H, W, k): quarters of 1 .. 16 channels, ragged sizes, k = 1 .. 5
    (2, 4, 5, 7, 3), (3, 8, 6, 4, 2), (2, 12, 13, 17, 3), (1, 16, 9, 6, 5), (2, 4, 3, 3, 1),
    (1, 64, 8, 8, 3), (2, 20, 1, 9, 3),
]


@pytest.mark.parametrize("shape", [(3, 5, 37, 9, 3), (2, 12, 24, 20, 5), (1, 3, 9, 40, 2)],
                         ids=lambda s: "x".join(map(str, s)))
def test_unit_forward_bands(orc, shape):
    """Unit forward of a batch smaller than the compute units: images split
    into bands of rows, each recomputing the rows its neighbours' later
    layers read, the last band ragged.  Against the oracle elementwise, and
    in place (then whole images) bit for bit the same."""
    B, C, H, W, k = shape
    c = synth.unit_case(B, C, H, W, k)
    x, K4 = c["x"], c["K4"]
    y = finc.unit_forward(dev(x), dev(K4), out=poisoned(x.shape))
    assert_close(host(y), orc.unit_forward(f64(x), f64(K4)), f"unit forward {shape}")
    inplace = dev(x)
    finc.unit_forward(inplace, dev(K4), out=inplace)
    assert torch.equal(inplace, y)


@pytest.mark.parametrize("shape", [(2, 3, 5, 7, 3), (3, 12, 16, 16, 3), (1, 7, 9, 6, 5),
                                   (2, 4, 6, 6, 1), (2, 5, 8, 11, 2), (1, 20, 9, 10, 7),
                                   (2, 64, 5, 6, 3), (1, 33, 7, 5, 4), (3, 2, 11, 4, 6)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("corner", [0, 1, 2, 3])
def test_backward(orc, shape, corner):
    """Backward of one layer (dx = J^T dy; dK with the masked entries reset
    and the log|det| term) against the oracle; junk in the masked weight
    slots is ignored; the same bits on a second run."""
    B, C, H, W, k = shape
    rng = np.random.default_rng(100 + corner)
    x = rng.normal(size=(B, C, H, W))
    dy = rng.normal(size=(B, C, H, W))
    K = synth.garbage_in_mask(synth.masked_kernel(C, k, corner, 1000 + corner), corner)
    gld = -0.75
    dx, dK = finc.backward(dev(x), dev(dy), dev(K), corner, gld, dx=poisoned(x.shape),
                           dK=poisoned(K.shape))
    want_dx, want_dK = orc.backward(f64(x), f64(dy), f64(K), corner, gld)
    assert_close(host(dx), want_dx, f"backward dx {shape} corner {corner}")
    assert_close(host(dK), want_dK, f"backward dK {shape} corner {corner}")
    dx2, dK2 = finc.backward(dev(x), dev(dy), dev(K), corner, gld)
    assert torch.equal(dx, dx2) and torch.equal(dK, dK2)


@pytest.mark.parametrize("name", ["layer_c12_16x16_b64_k3", "layer_c12_32x32_b64_k3",
                                  "layer_c12_32x32_b64_k5"])
def test_backward_workload(orc, name):
    """Backward at the single-layer workloads' shapes (64 images of 12
    channels, 16 x 16 or 32 x 32, k = 3 or 5): dK sums 16,384 or 65,536
    pixels per tap, each entry held to the size of its terms (the root sum
    of squares of the products it adds, from the oracle's dK of x^2 and
    dy^2); dx checked on three sampled images; dx alone and dK alone give
    the same bits as both together."""
    c = synth.make(name)
    x, K, corner = c["x"], c["K"], c["corner"]
    dy = np.random.default_rng(5).normal(size=x.shape)
    dx, dK = finc.backward(dev(x), dev(dy), dev(K), corner, -1.0)
    want_dx, want_dK = orc.backward(f64(x), f64(dy), f64(K), corner, -1.0)
    _, sq = orc.backward(f64(x) ** 2, f64(dy) ** 2, f64(K), corner, 0.0)
    assert_close(host(dK), want_dK, f"backward dK, {name}", scale=np.sqrt(sq))
    pick = [0, 21, 63]
    assert_close(host(dx)[pick], want_dx[pick], f"backward dx, {name}")
    only_dk = finc.backward(dev(x), dev(dy), dev(K), corner, -1.0, want_dx=False)
    assert only_dk[0] is None and torch.equal(only_dk[1], dK)
    only_dx = finc.backward(dev(x), dev(dy), dev(K), corner, -1.0, want_dK=False)
    assert only_dx[1] is None and torch.equal(only_dx[0], dx)


def test_backward_empty_batch(orc):
    """No images: dx is empty and dK holds only the log|det| term (masked
    entries 0), as the oracle gives it."""
    C, H, W, k, corner = 5, 6, 7, 3, 2
    K = synth.masked_kernel(C, k, corner, 77)
    x = np.zeros((0, C, H, W))
    dx, dK = finc.backward(dev(x), dev(x), dev(K), corner, -1.0, dK=poisoned(K.shape))
    want_dx, want_dK = orc.backward(f64(x), f64(x), f64(K), corner, -1.0)
    assert dx.shape == (0, C, H, W)
    assert_close(host(dK), want_dK, "backward dK, no images")


def test_unsupported_shapes_rejected():
    """Shapes beyond what a workgroup can hold are rejected before any launch
    with FINC_EUNSUPPORTED, the output untouched: 8 channels at 128 x 128
    (the stream form's phase input exceeds its prefetch registers) and 129
    rows (more row tiles than a workgroup has waves)."""
    for C, H, W in [(8, 128, 128), (2, 129, 16)]:
        K = dev(synth.masked_kernel(C, 3, 0, 1000))
        prep = finc.prepare(K, [0])
        y = torch.zeros((1, C, H, W), dtype=torch.float32, device=DEV)
        out = poisoned((1, C, H, W))
        with pytest.raises(finc.FincError) as err:
            finc.inverse_prepared(y, prep, 3, 0, out=out)
        assert err.value.code == finc.EUNSUPPORTED, (C, H, W)
        torch.cuda.synchronize()
        assert torch.isnan(out).all(), (C, H, W)


@pytest.mark.parametrize("shape", SPLIT_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_split_unit(orc, shape):
    """Channel-split unit (Sec. 4.3, Alg. 2): forward, log|det|, inverse and the
    prepared side output, elementwise against the oracle; junk in the masked
    slots is ignored."""
    B, C, H, W, k = shape
    print(f"split B={B} C={C} H={H} W={W} k={k}", flush=True)
    rng = np.random.default_rng(hash(shape) % 2**32)
    x = rng.normal(size=(B, C, H, W))
    Kq4 = np.stack([synth.garbage_in_mask(synth.masked_kernel(C // 4, k, g, 1200 + g), g)
                    for g in range(4)])
    xd, Kd = dev(x), dev(Kq4)
    ldf = torch.full((1,), float("nan"), dtype=torch.float64, device=DEV)
    y = finc.split_forward(xd, Kd, out=poisoned(x.shape), logdet=ldf)
    yh = host(y)
    assert_close(yh, orc.split_forward(f64(x), f64(Kq4)), "split forward")
    r = orc.split_logdet(f64(Kq4), H, W)
    assert abs(float(ldf.cpu()[0]) - r) <= TOL * max(1.0, abs(r))
    ld = float(finc.split_logdet(Kd, H, W).cpu()[0])
    assert abs(ld - r) <= TOL * max(1.0, abs(r))
    xr = finc.split_inverse(y, Kd, out=poisoned(x.shape))
    assert_close(host(xr), orc.split_inverse(yh, f64(Kq4)), "split inverse")
    assert_round_trip(host(xr), f64(x), "split")
    z = rng.normal(size=(B, C, H, W))
    assert_close(host(finc.split_inverse(dev(z), Kd)), orc.split_inverse(f64(z), f64(Kq4)),
                 "split inverse of arbitrary input")
    # the forward's prepared side output is what prepare writes, and drives
    # the prepared inverse to the same bits
    nb = finc.workspace_bytes(C // 4, k, 4)
    pp = torch.full((nb,), 0xAB, dtype=torch.uint8, device=DEV)
    ref = torch.full((nb,), 0xAB, dtype=torch.uint8, device=DEV)
    assert torch.equal(finc.split_forward(xd, Kd, prepared=pp), y)
    finc.prepare(Kd, [0, 1, 2, 3], out=ref)
    assert torch.equal(pp, ref)
    assert torch.equal(finc.split_inverse_prepared(y, pp, k, out=poisoned(x.shape)), xr)
    # in place, and batch-invariant bits
    inplace = y.clone()
    finc.split_inverse(inplace, Kd, out=inplace)
    assert torch.equal(inplace, xr)
    assert torch.equal(finc.split_inverse(y[B - 1:B].contiguous(), Kd)[0], xr[B - 1])


@pytest.mark.parametrize("name", [n for n, s in synth.WORKLOADS.items() if s["kind"] == "split"])
def test_split_workload(orc, name):
    """Full-size channel-split workloads; the oracle runs on four sampled images
    (results do not depend on the batch)."""
    print(f"workload {name}", flush=True)
    c = synth.make(name)
    x, Kq4 = c["x"], c["Kq4"]
    xd, Kd = dev(x), dev(Kq4)
    y = finc.split_forward(xd, Kd, out=poisoned(x.shape))
    xr = finc.split_inverse(y, Kd, out=poisoned(x.shape))
    idx = [0, 1, c["B"] // 2, c["B"] - 1]
    yh, xh = host(y)[idx], host(xr)[idx]
    assert_close(yh, orc.split_forward(f64(x[idx]), f64(Kq4)), f"{name} forward")
    assert_close(xh, orc.split_inverse(yh, f64(Kq4)), f"{name} inverse")
    assert_round_trip(host(xr), f64(x), f"{name} round trip")


def _stack_flat(c):
    Kf = np.concatenate([a.ravel() for a in c["K"]])
    sf = np.concatenate([a.ravel() for a in c["scale"]])
    bf = np.concatenate([a.ravel() for a in c["bias"]])
    return Kf, sf, bf


def test_stack_small(orc):
    """Small stack (2 images, 3 levels of 2 units): elementwise vs oracle."""
    c = synth.stack_case(B=2, C1=4, H1=8, W1=8, levels=3, units=2, k=3)
    Kf, sf, bf = _stack_flat(c)
    x = finc.stack_inverse([dev(z) for z in c["z"]], dev(Kf), dev(sf), dev(bf), 3, 2, 4, 8,
                           8, 3)
    want = orc.stack_inverse([f64(z) for z in c["z"]], [f64(a) for a in c["K"]],
                             [f64(a) for a in c["scale"]], [f64(a) for a in c["bias"]],
                             3, 2, 3, 4, 8, 8)
    assert_close(host(x), want, "small stack")


def test_stack_levels_in_own_launches(orc):
    """Small stack whose levels need different kernel instances (12, 24 and
    48 channels: one, two and three channel tiles), so each level runs in a
    launch of its own and hands its solution to the next through the output
    tensor: per image max|gpu - oracle| / max(1, max|oracle|) <= 1e-4 (the
    stack workload's criterion), and each image independent of the batch."""
    c = synth.stack_case(B=3, C1=12, H1=16, W1=16, levels=3, units=2, k=3)
    Kf, sf, bf = _stack_flat(c)
    zd = [dev(z) for z in c["z"]]
    args = (dev(Kf), dev(sf), dev(bf), 3, 2, 12, 16, 16, 3)
    x = finc.stack_inverse(zd, *args, out=poisoned((3, 12, 16, 16)))
    want = orc.stack_inverse([f64(z) for z in c["z"]], [f64(a) for a in c["K"]],
                             [f64(a) for a in c["scale"]], [f64(a) for a in c["bias"]],
                             3, 2, 3, 12, 16, 16)
    xh = host(x)
    assert np.isfinite(xh).all()
    for b in range(3):
        err = np.max(np.abs(xh[b] - want[b])) / max(1.0, np.max(np.abs(want[b])))
        assert err <= TOL, f"image {b}: inf-norm relative error {err:.3e}"
    one = finc.stack_inverse([z[2:3].contiguous() for z in zd], *args)
    assert torch.equal(one[0], x[2])


def test_stack_workload(orc):
    """Three levels of eight units (12x32x32 -> 24x16x16 -> 48x8x8), batch 64:
    the oracle runs on four sampled images (results do not depend on the
    batch); criterion is max|gpu - oracle| / max(1, max|oracle|) <= 1e-4,
    because the random stack's inverse reaches magnitudes where elementwise
    fp32 error is dominated by cancellation."""
    print("workload stack_3x8_c12_32x32_b64_k3", flush=True)
    c = synth.make("stack_3x8_c12_32x32_b64_k3")
    Kf, sf, bf = _stack_flat(c)
    zd = [dev(z) for z in c["z"]]
    args = (dev(Kf), dev(sf), dev(bf), 3, 8, 12, 32, 32, 3)
    x = finc.stack_inverse(zd, *args, out=poisoned((64, 12, 32, 32)))
    xh = host(x)
    assert np.isfinite(xh).all()
    pick = [0, 17, 42, 63]
    want = orc.stack_inverse([f64(z[pick]) for z in c["z"]], [f64(a) for a in c["K"]],
                             [f64(a) for a in c["scale"]], [f64(a) for a in c["bias"]],
                             3, 8, 3, 12, 32, 32)
    for n, b in enumerate(pick):
        err = np.max(np.abs(xh[b] - want[n])) / max(1.0, np.max(np.abs(want[n])))
        assert err <= TOL, f"image {b}: inf-norm relative error {err:.3e}"
    x2 = finc.stack_inverse(zd, *args)
    assert torch.equal(x, x2)
    one = finc.stack_inverse([z[5:6].contiguous() for z in zd], *args)
    assert torch.equal(one[0], x[5])
