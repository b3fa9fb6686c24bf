"""Images whose level does not fit one workgroup, on the GPU, against the
oracle: the banded stream form (finc_inverse_banded,
finc_unit_inverse_banded) -- bands of rows in workgroups of their own,
pipelined through drained-diagonal counts.  Shapes: 256 x 256 at C = 2 and
128 x 128 at C = 12 (beyond one workgroup), ragged last bands, every corner,
k = 2 .. 7, a unit, and a seeded sweep of random shapes.

Bar: 1e-4 * max(1, |oracle|) elementwise against the oracle's raster-order
inverse of the oracle's forward of x, and the round trip to x within 1e-4;
the workspace's timeout flag stays 0; the same bits on a second call and
for the last image alone."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import TOL, assert_close, assert_round_trip, dev, f64, host
from paper_2301_09266_amd import finc, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def orc():
    return oracle.default()


def timeout_flag(ws, C, k, n_layers):
    off = finc.workspace_bytes(C, k, n_layers)
    return int(ws[off:off + 4].view(torch.int32).item())


LAYER_CASES = [
    # (B, C, H, W, k, corner)
    (2, 2, 200, 40, 3, 0), (2, 12, 64, 24, 3, 1), (1, 16, 100, 30, 5, 2), (1, 4, 300, 17, 7, 3),
    (3, 12, 40, 19, 5, 0), (1, 3, 129, 16, 2, 1), (2, 2, 48, 40, 3, 2),
    (1, 2, 256, 256, 3, 0), (2, 12, 128, 128, 3, 3),
]


@pytest.mark.parametrize("case", LAYER_CASES, ids=lambda c: "x".join(map(str, c)))
def test_banded_layer(orc, case):
    B, C, H, W, k, corner = case
    plan = finc.banded_plan(C, H, W, k)
    print(f"banded layer {case} {plan}", flush=True)
    assert not isinstance(plan, int)
    K = synth.garbage_in_mask(synth.masked_kernel(C, k, corner, 1000 + C + k), corner)
    x = np.random.default_rng(C * 7 + H).normal(size=(B, C, H, W))
    y = orc.forward(f64(x), f64(K), corner)
    xr, ws = finc.inverse_banded(dev(y), dev(K), corner)
    assert timeout_flag(ws, C, k, 1) == 0
    assert_close(host(xr), orc.inverse(f64(y), f64(K), corner), f"banded inverse {case}")
    assert_round_trip(host(xr), f64(x), f"banded round trip {case}")
    again, ws2 = finc.inverse_banded(dev(y), dev(K), corner, workspace=ws)
    assert torch.equal(again, xr) and timeout_flag(ws2, C, k, 1) == 0
    one, _ = finc.inverse_banded(dev(y[-1:]), dev(K), corner)
    assert torch.equal(one[0], xr[-1])


def draw_banded(seed):
    """A seeded banded layer shape (B, C, H, W, k, corner) that the banded
    form takes: C 1..16, k 2..7, H 17..159, W 2..47."""
    rng = np.random.default_rng(seed)
    while True:
        C, k = int(rng.integers(1, 17)), int(rng.integers(2, 8))
        H, W = int(rng.integers(17, 160)), int(rng.integers(2, 48))
        corner, B = int(rng.integers(0, 4)), int(rng.integers(1, 3))
        if C * H * W * C * k * k <= 6_000_000 and not isinstance(finc.banded_plan(C, H, W, k), int):
            return B, C, H, W, k, corner


@pytest.mark.parametrize("seed", range(24))
def test_banded_layer_sweep(orc, seed):
    """Random shapes cover band heights, thread counts and register budgets
    that the listed cases miss."""
    B, C, H, W, k, corner = case = draw_banded(500 + seed)
    print(f"banded sweep {seed} {case} {finc.banded_plan(C, H, W, k)}", flush=True)
    K = synth.garbage_in_mask(synth.masked_kernel(C, k, corner, 3000 + seed), corner)
    x = np.random.default_rng(seed).normal(size=(B, C, H, W))
    y = orc.forward(f64(x), f64(K), corner)
    xr, ws = finc.inverse_banded(dev(y), dev(K), corner)
    assert timeout_flag(ws, C, k, 1) == 0
    assert_close(host(xr), orc.inverse(f64(y), f64(K), corner), f"banded sweep {case}")


def test_banded_in_place(orc):
    B, C, H, W, k, corner = 2, 12, 70, 21, 3, 0
    K = synth.masked_kernel(C, k, corner, 77)
    x = np.random.default_rng(3).normal(size=(B, C, H, W))
    y = orc.forward(f64(x), f64(K), corner)
    t = dev(y)
    finc.inverse_banded(t, dev(K), corner, out=t)
    assert_close(host(t), orc.inverse(f64(y), f64(K), corner), "banded inverse in place")


@pytest.mark.parametrize("case", [(2, 2, 160, 33, 3), (1, 12, 96, 40, 3), (1, 2, 256, 256, 3)],
                         ids=lambda c: "x".join(map(str, c)))
def test_banded_unit(orc, case):
    B, C, H, W, k = case
    print(f"banded unit {case} {finc.banded_plan(C, H, W, k)}", flush=True)
    K4 = np.stack([synth.garbage_in_mask(synth.masked_kernel(C, k, q, 2000 + q), q)
                   for q in range(4)])
    x = np.random.default_rng(H + W).normal(size=(B, C, H, W))
    y = orc.unit_forward(f64(x), f64(K4))
    xr, ws = finc.unit_inverse_banded(dev(y), dev(K4))
    assert timeout_flag(ws, C, k, 4) == 0
    assert_close(host(xr), orc.unit_inverse(f64(y), f64(K4)), f"banded unit {case}")
    assert_round_trip(host(xr), f64(x), f"banded unit round trip {case}")


def test_banded_unsupported():
    """No band fits a workgroup beyond 16 channels or at k = 1."""
    y = torch.zeros((1, 17, 256, 16), device="cuda:0")
    with pytest.raises(finc.FincError) as e:
        finc.inverse_banded(y, torch.zeros((17, 17, 3, 3), device="cuda:0"), 0)
    assert e.value.code == finc.EUNSUPPORTED
