"""Theorem 2's step count, on the GPU: the inverse of a layer runs H + W - 1
dependent diagonal steps.  finc_inverse_steps has every wave of every
workgroup count the steps it ran (each ended by the workgroup's step
barrier); for one shape per kernel instance of the single layer and of the
channel-split unit (tests/domain.py) and the benchmark shape, every count
is H + W - 1, and the inverse it returns is bit for bit that of the
uncounted call."""
import numpy as np
import pytest
import torch

import domain
from gpu_util import dev
from paper_2301_09266_amd import finc, synth

pytestmark = pytest.mark.gpu

CASES = [c for c in domain.COVER if c[0] in ("layer", "split")] + [("layer", 12, 16, 16, 3)]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c)))
def test_step_count(case):
    kind, C, H, W, k = case
    split = kind == "split"
    corner = (C + H + W + k) % 4
    print(f"steps {case}", flush=True)
    if split:
        K = synth.split_kernels(C, k)
        prep = finc.prepare(dev(K), [0, 1, 2, 3])
    else:
        K = synth.masked_kernel(C, k, corner, 1000 + C)
        prep = finc.prepare(dev(K), [corner])
    y = dev(np.random.default_rng(C + H).normal(size=(2, C, H, W)))
    x, steps = finc.inverse_steps(y, prep, k, corner, split=split)
    want = H + W - 1
    assert steps.min().item() == want and steps.max().item() == want, \
        (case, steps.min().item(), steps.max().item())
    ref = (finc.split_inverse_prepared(y, prep, k) if split
           else finc.inverse_prepared(y, prep, k, corner))
    assert torch.equal(x, ref)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c)))
def test_timeline(case):
    """finc_inverse_timeline: four stamps a wave, in order (start, set-up done,
    last step done, store issued), and the inverse bit for bit that of the
    call without stamps."""
    kind, C, H, W, k = case
    split = kind == "split"
    corner = (C + H + W + k) % 4
    print(f"timeline {case}", flush=True)
    if split:
        K = synth.split_kernels(C, k)
        prep = finc.prepare(dev(K), [0, 1, 2, 3])
    else:
        K = synth.masked_kernel(C, k, corner, 1000 + C)
        prep = finc.prepare(dev(K), [corner])
    y = dev(np.random.default_rng(C + W).normal(size=(2, C, H, W)))
    x, st = finc.inverse_timeline(y, prep, k, corner, split=split)
    t = st.cpu().numpy()
    assert (t > 0).all(), case
    assert (np.diff(t, axis=2) >= 0).all(), case
    ref = (finc.split_inverse_prepared(y, prep, k) if split
           else finc.inverse_prepared(y, prep, k, corner))
    assert torch.equal(x, ref)
