"""The inverse over the whole supported domain, on the GPU, against the
oracle: every kernel instance the host can select (one or two shapes each,
tests/domain.py) and a seeded sweep of random shapes -- k = 1 .. 7, up to 64
channels, up to 128 rows, single layers, units and channel-split units, all
four corners.

Per shape: the forward elementwise against the oracle (or, for rows too
wide for its LDS blocks, its FINC_EUNSUPPORTED); the inverse of the
GPU forward's output elementwise against the oracle's inverse of the same
bits; the round trip within 1e-4 of x; the inverse of an arbitrary input;
log|det|; the last image alone giving the same bits as in its batch.  The
masked weight slots hold junk, and outputs start NaN-poisoned.
"""
import numpy as np
import pytest
import torch

import domain
import oracle
from gpu_util import TOL, assert_close, assert_round_trip, dev, f64, host, poisoned
from paper_2301_09266_amd import finc, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def orc():
    return oracle.default()


def _check_logdet(got, want):
    assert abs(float(got.cpu()[0]) - want) <= TOL * max(1.0, abs(want))


def run_case(orc, kind, B, C, H, W, k, corner, seed):
    print(f"domain {kind} B={B} C={C} H={H} W={W} k={k} corner={corner} seed={seed} "
          f"instance={domain.instance(kind, C, H, W, k)}", flush=True)
    rng = np.random.default_rng(seed)
    x = rng.normal(size=(B, C, H, W))
    z = rng.normal(size=(B, C, H, W))
    shape = x.shape
    if kind == "layer":
        K = synth.garbage_in_mask(synth.masked_kernel(C, k, corner, 1000 + seed % 997), corner)
        Kd = dev(K)
        fwd = lambda t, out=None: finc.forward(t, Kd, corner, out=out)
        inv = lambda t, out=None: finc.inverse(t, Kd, corner, out=out)
        ofwd = lambda a: orc.forward(a, f64(K), corner)
        oinv = lambda a: orc.inverse(a, f64(K), corner)
        ld, ld_ref = finc.logdet(Kd, corner, H, W), orc.logdet(f64(K), corner, H, W)
    elif kind == "unit":
        K4 = synth.unit_kernels(C, k, seed % 997)
        K4 = np.stack([synth.garbage_in_mask(K4[q], q) for q in range(4)])
        Kd = dev(K4)
        fwd = lambda t, out=None: finc.unit_forward(t, Kd, out=out)
        inv = lambda t, out=None: finc.unit_inverse(t, Kd, out=out)
        ofwd = lambda a: orc.unit_forward(a, f64(K4))
        oinv = lambda a: orc.unit_inverse(a, f64(K4))
        ld, ld_ref = finc.unit_logdet(Kd, H, W), orc.unit_logdet(f64(K4), H, W)
    else:
        Kq4 = synth.split_kernels(C, k, seed % 997)
        Kq4 = np.stack([synth.garbage_in_mask(Kq4[g], g) for g in range(4)])
        Kd = dev(Kq4)
        fwd = lambda t, out=None: finc.split_forward(t, Kd, out=out)
        inv = lambda t, out=None: finc.split_inverse(t, Kd, out=out)
        ofwd = lambda a: orc.split_forward(a, f64(Kq4))
        oinv = lambda a: orc.split_inverse(a, f64(Kq4))
        ld, ld_ref = finc.split_logdet(Kd, H, W), orc.split_logdet(f64(Kq4), H, W)
    what = f"{kind} {shape} k={k} corner={corner}"
    if isinstance(finc.forward_plan(domain.KINDS[kind], B, C, H, W, k), int):
        # rows too wide for the forward's LDS blocks: it must say so, and the
        # inverse is checked on the oracle's forward
        with pytest.raises(finc.FincError) as err:
            fwd(dev(x), out=poisoned(shape))
        assert err.value.code == finc.EUNSUPPORTED
        y = dev(ofwd(f64(x)))
    else:
        y = fwd(dev(x), out=poisoned(shape))
        assert_close(host(y), ofwd(f64(x)), f"{what} forward")
    yh = host(y)
    xr = inv(y, out=poisoned(shape))
    assert_close(host(xr), oinv(yh), f"{what} inverse")
    assert_round_trip(host(xr), f64(x), what)
    xz = inv(dev(z), out=poisoned(shape))
    assert_close(host(xz), oinv(f64(z)), f"{what} inverse of z")
    _check_logdet(ld, ld_ref)
    if B > 1:
        assert torch.equal(inv(y[-1:].contiguous())[0], xr[-1]), f"{what}: batch invariance"


@pytest.mark.parametrize("case", domain.COVER, ids=lambda c: "-".join(map(str, c)))
def test_every_instance(orc, case):
    kind, C, H, W, k = case
    corner = (C + H + W + k) % 4
    run_case(orc, kind, 2, C, H, W, k, corner, seed=C * 131 + H * 17 + W * 3 + k)


@pytest.mark.parametrize("seed", domain.RANDOM_SEEDS)
def test_random_shapes(orc, seed):
    for n, (kind, B, C, H, W, k, corner) in enumerate(domain.random_cases(seed)):
        run_case(orc, kind, B, C, H, W, k, corner, seed=seed * 100 + n)


def test_stack_single_launch(orc):
    """A stack whose levels share one plan (2 levels of 2 units, 2 -> 4
    channels, 16x16 -> 8x8) runs as one launch, handing over between levels
    in LDS: elementwise against the oracle, and each image independent of
    its batch."""
    assert len(finc.inverse_plan(finc.PLAN_STACK, 2, 16, 16, 3, L=2, U=2)) == 1
    c = synth.stack_case(B=3, C1=2, H1=16, W1=16, levels=2, units=2, k=3)
    Kf = np.concatenate([a.ravel() for a in c["K"]])
    sf = np.concatenate([a.ravel() for a in c["scale"]])
    bf = np.concatenate([a.ravel() for a in c["bias"]])
    zd = [dev(z) for z in c["z"]]
    args = (dev(Kf), dev(sf), dev(bf), 2, 2, 2, 16, 16, 3)
    x = finc.stack_inverse(zd, *args, out=poisoned((3, 2, 16, 16)))
    want = orc.stack_inverse([f64(z) for z in c["z"]], [f64(a) for a in c["K"]],
                             [f64(a) for a in c["scale"]], [f64(a) for a in c["bias"]],
                             2, 2, 3, 2, 16, 16)
    assert_close(host(x), want, "single-launch stack")
    one = finc.stack_inverse([z[1:2].contiguous() for z in zd], *args)
    assert torch.equal(one[0], x[1])
