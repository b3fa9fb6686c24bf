"""Seeded synthetic inputs for the masked k x k convolution, the FInC unit and
the multi-scale sampling stack.

This module only draws random numbers and lays them out; it holds none of the
layer's arithmetic (no convolution, no solve, no determinant).  Both the HIP
path and the CPU oracle are fed from here, so that every comparison runs on the
same bits.

Recipe (the paper trains on MNIST / CIFAR-10 / ImageNet / CelebA, Sec. 5 and
the appendix "Datasets"; those images and any trained weights are replaced by
tensors of the same shapes drawn here):

* weights of one padded convolution block (Sec. 4.1, Alg. 1 input K of shape
  (C, C, k, k)): every entry ~ N(0, 0.05^2), drawn for the full OIHW tensor in
  C order; at the self tap (the kernel position that multiplies the output
  pixel itself) the entries with c_in > c_out are set to zero (the channel mask)
  and the diagonal K[c, c, self] is then set to 1 + U(-0.1, 0.1), c ascending.
  Layer number l of a configuration (forward order) uses default_rng(1000 + l).
* activations and latents ~ N(0, 1) from default_rng(0), in the order the
  configuration lists them.
* actnorm (Sec. 4.4) of level L, unit u: default_rng(2000 + 8 L + u);
  scale = exp(N(0, 0.1^2)) per channel, then bias ~ N(0, 0.1^2) per channel.
"""
from __future__ import annotations

import numpy as np

CORNERS = ("TL", "TR", "BL", "BR")
CORNER_ID = {name: i for i, name in enumerate(CORNERS)}

# The FInC unit applies its four padded blocks in this corner order
# (Sec. 4.3; the order of the four corners is listed in Fig. 2a).
UNIT_CORNERS = (0, 1, 2, 3)


def self_tap(corner: int, k: int) -> tuple[int, int]:
    """Kernel position (a, b) that multiplies the output pixel itself.

    With k-1 zero rows/cols padded on the two named sides (Sec. 4.1,
    corner paddings), the input pixel aligned with the output sits at the
    kernel corner opposite to the padding: TL -> (k-1, k-1), TR -> (k-1, 0),
    BL -> (0, k-1), BR -> (0, 0).
    """
    top = corner in (0, 1)
    left = corner in (0, 2)
    return (k - 1 if top else 0, k - 1 if left else 0)


def masked_kernel(C: int, k: int, corner: int, seed: int) -> np.ndarray:
    """One block's weights (C_out, C_in, k, k) as float64, recipe above."""
    rng = np.random.default_rng(seed)
    K = rng.normal(0.0, 0.05, size=(C, C, k, k))
    sh, sw = self_tap(corner, k)
    for co in range(C):
        K[co, co + 1:, sh, sw] = 0.0
    diag = 1.0 + rng.uniform(-0.1, 0.1, size=C)
    for c in range(C):
        K[c, c, sh, sw] = diag[c]
    return K


def unit_kernels(C: int, k: int, first_layer: int = 0) -> np.ndarray:
    """Four blocks of one unit, stacked (4, C, C, k, k), corners TL, TR, BL, BR."""
    return np.stack([masked_kernel(C, k, q, 1000 + first_layer + i)
                     for i, q in enumerate(UNIT_CORNERS)])


def actnorm_params(C: int, level: int, unit: int) -> tuple[np.ndarray, np.ndarray]:
    rng = np.random.default_rng(2000 + 8 * level + unit)
    scale = np.exp(rng.normal(0.0, 0.1, size=C))
    bias = rng.normal(0.0, 0.1, size=C)
    return scale, bias


def gaussian(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.normal(0.0, 1.0, size=shape)


def garbage_in_mask(K: np.ndarray, corner: int, seed: int = 7) -> np.ndarray:
    """Copy of K whose masked entries (self tap, c_in > c_out) hold large junk.

    The layer is defined for any buffer: those entries must be ignored.
    """
    K = np.array(K, copy=True)
    C, k = K.shape[0], K.shape[-1]
    sh, sw = self_tap(corner, k)
    rng = np.random.default_rng(seed)
    for co in range(C):
        n = C - co - 1
        if n:
            K[co, co + 1:, sh, sw] = rng.uniform(-50.0, 50.0, size=n)
    return K


# ---------------------------------------------------------------------------
# Workloads.  Shapes follow the paper's datasets after one 2x2 squeeze
# (CIFAR-10 32x32x3 -> 16x16x12, ImageNet-64 64x64x3 -> 32x32x12, Sec. 4.4),
# plus the small 8x8 case.  Each builder returns plain float64 arrays.
# ---------------------------------------------------------------------------

def layer_case(B: int, C: int, H: int, W: int, k: int, corner: int = 0,
               seed: int = 0, layer: int = 0) -> dict:
    rng = np.random.default_rng(seed)
    x = gaussian(rng, (B, C, H, W))
    z = gaussian(rng, (B, C, H, W))
    K = masked_kernel(C, k, corner, 1000 + layer)
    return dict(x=x, z=z, K=K, B=B, C=C, H=H, W=W, k=k, corner=corner)


def unit_case(B: int, C: int, H: int, W: int, k: int, seed: int = 0) -> dict:
    rng = np.random.default_rng(seed)
    x = gaussian(rng, (B, C, H, W))
    z = gaussian(rng, (B, C, H, W))
    K4 = unit_kernels(C, k, 0)
    return dict(x=x, z=z, K4=K4, B=B, C=C, H=H, W=W, k=k)


def split_kernels(C: int, k: int, first_layer: int = 0) -> np.ndarray:
    """The four quarter-channel blocks of one channel-split unit, stacked
    (4, C/4, C/4, k, k); quarter g has corner g (TL, TR, BL, BR)."""
    return np.stack([masked_kernel(C // 4, k, g, 1000 + first_layer + g) for g in range(4)])


def split_case(B: int, C: int, H: int, W: int, k: int, seed: int = 0) -> dict:
    rng = np.random.default_rng(seed)
    x = gaussian(rng, (B, C, H, W))
    z = gaussian(rng, (B, C, H, W))
    Kq4 = split_kernels(C, k, 0)
    return dict(x=x, z=z, Kq4=Kq4, B=B, C=C, H=H, W=W, k=k)


def stack_case(B: int = 64, C1: int = 12, H1: int = 32, W1: int = 32,
               levels: int = 3, units: int = 8, k: int = 3, seed: int = 0) -> dict:
    """Multi-scale sampling stack: `levels` levels of `units` FInC units, each
    unit followed by an actnorm; between levels the channels are split in
    half and the rest squeezed (Sec. 4.4, Fig. 2c).

    Latents: z[l] for l < levels-1 is the half split off at level l,
    shape (B, C_l/2, H_l, W_l); z[levels-1] is the top, (B, C_top, H_top, W_top),
    with C_l = C1 * 2**l and H_l = H1 / 2**l.  Draw order: top latent first,
    then downwards (z[levels-1], ..., z[0]).
    """
    rng = np.random.default_rng(seed)
    dims = [(C1 * 2 ** l, H1 >> l, W1 >> l) for l in range(levels)]
    z = [None] * levels
    for l in reversed(range(levels)):
        C, H, W = dims[l]
        cz = C if l == levels - 1 else C // 2
        z[l] = gaussian(rng, (B, cz, H, W))
    K = []      # K[l]: (units, 4, C, C, k, k)
    scale = []  # scale[l]: (units, C)
    bias = []
    for l, (C, H, W) in enumerate(dims):
        K.append(np.stack([unit_kernels(C, k, 32 * l + 4 * u) for u in range(units)]))
        sb = [actnorm_params(C, l, u) for u in range(units)]
        scale.append(np.stack([s for s, _ in sb]))
        bias.append(np.stack([b for _, b in sb]))
    x = gaussian(np.random.default_rng(seed + 1), (B, C1, H1, W1))
    return dict(z=z, K=K, scale=scale, bias=bias, x=x, B=B, C1=C1, H1=H1, W1=W1,
                levels=levels, units=units, k=k, dims=dims)


# The workloads, by what they are.
WORKLOADS = {
    "layer_c3_8x8_b1_k3": dict(kind="layer", B=1, C=3, H=8, W=8, k=3),
    "layer_c12_16x16_b64_k3": dict(kind="layer", B=64, C=12, H=16, W=16, k=3),
    "unit_c12_16x16_b256_k3": dict(kind="unit", B=256, C=12, H=16, W=16, k=3),
    "unit_c48_8x8_b256_k3": dict(kind="unit", B=256, C=48, H=8, W=8, k=3),
    "layer_c12_32x32_b64_k3": dict(kind="layer", B=64, C=12, H=32, W=32, k=3),
    "layer_c12_32x32_b64_k5": dict(kind="layer", B=64, C=12, H=32, W=32, k=5),
    "unit_c12_32x32_b64_k3": dict(kind="unit", B=64, C=12, H=32, W=32, k=3),
    "unit_c12_32x32_b64_k5": dict(kind="unit", B=64, C=12, H=32, W=32, k=5),
    "stack_3x8_c12_32x32_b64_k3": dict(kind="stack", B=64, C1=12, H1=32, W1=32,
                                       levels=3, units=8, k=3),
    # the paper's channel-split unit (Sec. 4.3, Alg. 2): quarters of 3 and 12
    # channels
    "split_c12_16x16_b64_k3": dict(kind="split", B=64, C=12, H=16, W=16, k=3),
    "split_c48_16x16_b64_k3": dict(kind="split", B=64, C=48, H=16, W=16, k=3),
}


# Scaling sweep after the paper's sampling-time study (Sec. 5, Fig. 3): one
# FInC unit at C = 2, k = 3, square images of 16 .. 128 pixels a side,
# batches of 1 .. 128 (the larger images exceed LDS and stream).
SWEEP_SIZES = (16, 32, 64, 128)
SWEEP_BATCHES = (1, 8, 32, 128)
# sizes beyond one workgroup (the banded stream form)
SWEEP_BANDED_SIZES = (256,)


def sweep_case(n: int, B: int, C: int = 2, k: int = 3, seed: int = 0) -> dict:
    return unit_case(B, C, n, n, k, seed)


def make(name: str, **override) -> dict:
    spec = dict(WORKLOADS[name])
    spec.update(override)
    kind = spec.pop("kind")
    if kind == "layer":
        return layer_case(**spec)
    if kind == "unit":
        return unit_case(**spec)
    if kind == "split":
        return split_case(**spec)
    return stack_case(**spec)


# ---------------------------------------------------------------------------
# The full FInC Flow (Sec. 4.4, Fig. 2b/2c): Steps of [channel-split unit,
# actnorm, invertible 1x1 convolution, affine coupling] in a multi-scale
# architecture with split priors.  The paper times untrained models; these
# are random untrained weights, drawn in the parameter layout below, all from
# one default_rng(seed) stream in layout order:
#   step:  Kq4 (4, C/4, C/4, k, k) masked as above but std 0.02 (diagonal
#          1 + U(-0.1, 0.1)) | actnorm scale exp(N(0, 0.1^2)) (C) | bias
#          N(0, 0.1^2) (C) | Wm (C, C): a random rotation (Q of the QR of a
#          N(0, 1) matrix, columns' signs fixed by R's diagonal, as Glow
#          initialises it) | coupling network: W1 (hid, C/2, 3, 3) He-normal
#          (std sqrt(2 / fan_in)), b1 (hid) N(0, 0.01^2), W2 (hid, hid, 1, 1)
#          He-normal, b2 (hid) N(0, 0.01^2), W3 (C, hid, 3, 3) N(0, (0.02 /
#          sqrt(fan_in))^2) (Glow starts it at zero; small and nonzero here so
#          that the coupling does something), b3 (C) N(0, 0.01^2) with 2 added
#          to its scale half (scale = sigmoid(r + 2) near 0.98), ls3 (C)
#          N(0, 0.01^2)
#   prior (levels below the top): Wp (C, C/2, 3, 3) N(0, (0.02 /
#          sqrt(fan_in))^2), bp (C) N(0, 0.01^2), lsp (C) N(0, 0.01^2)
# With the single layer's std 0.05, Glow's fixed coupling scale
# sigmoid(2) = 0.88 and larger output weights, the inverse of 84 random Steps
# grows by about 1.17 a Step and the split prior's exp(logsd) overflows; the
# scales above keep the sampled images finite (rms about 7 from N(0, 1)
# latents at the CIFAR-10 setting).
#   flow:  for level l: K steps, then (l < L-1) the prior; level l has
#          C_l = 4 C0 2^l channels at H0 / 2^(l+1) x W0 / 2^(l+1).
# ---------------------------------------------------------------------------

def _flow_step(rng, C, k, hid, unit_std=0.02, out_std=0.02, rbias=2.0):
    q = C // 4
    Kq4 = np.empty((4, q, q, k, k))
    for g in range(4):
        K = rng.normal(0.0, unit_std, size=(q, q, k, k))
        sh, sw = self_tap(g, k)
        for co in range(q):
            K[co, co + 1:, sh, sw] = 0.0
        K[np.arange(q), np.arange(q), sh, sw] = 1.0 + rng.uniform(-0.1, 0.1, size=q)
        Kq4[g] = K
    an_s = np.exp(rng.normal(0.0, 0.1, size=C))
    an_b = rng.normal(0.0, 0.1, size=C)
    Q, R = np.linalg.qr(rng.normal(size=(C, C)))
    Wm = Q * np.sign(np.diag(R))[None, :]
    Ch = C // 2
    W1 = rng.normal(0.0, np.sqrt(2.0 / (Ch * 9)), size=(hid, Ch, 3, 3))
    b1 = rng.normal(0.0, 0.01, size=hid)
    W2 = rng.normal(0.0, np.sqrt(2.0 / hid), size=(hid, hid, 1, 1))
    b2 = rng.normal(0.0, 0.01, size=hid)
    W3 = rng.normal(0.0, out_std / np.sqrt(hid * 9), size=(C, hid, 3, 3))
    b3 = rng.normal(0.0, 0.01, size=C)
    b3[C // 2:] += rbias
    ls3 = rng.normal(0.0, 0.01, size=C)
    return [Kq4, an_s, an_b, Wm, W1, b1, W2, b2, W3, b3, ls3]


def _flow_prior(rng, C, prior_std=0.02):
    Wp = rng.normal(0.0, prior_std / np.sqrt(C // 2 * 9), size=(C, C // 2, 3, 3))
    bp = rng.normal(0.0, 0.01, size=C)
    lsp = rng.normal(0.0, 0.01, size=C)
    return [Wp, bp, lsp]


def step_params(C: int, k: int, hid: int, seed: int = 3000) -> np.ndarray:
    """One Step's parameters, flat, in the layout above."""
    rng = np.random.default_rng(seed)
    return np.concatenate([a.ravel() for a in _flow_step(rng, C, k, hid)])


def flow_params(L: int, K: int, C0: int, k: int, hid: int, seed: int = 3000,
                unit_std: float = 0.02, out_std: float = 0.02, rbias: float = 2.0,
                prior_std: float = 0.02) -> np.ndarray:
    """All parameters of an L-level flow of K Steps per level, flat."""
    rng = np.random.default_rng(seed)
    parts = []
    for l in range(L):
        C = (4 * C0) << l
        for _ in range(K):
            parts += _flow_step(rng, C, k, hid, unit_std, out_std, rbias)
        if l < L - 1:
            parts += _flow_prior(rng, C, prior_std)
    return np.concatenate([a.ravel() for a in parts])


def flow_latent_shapes(B: int, L: int, C0: int, H0: int, W0: int):
    out = []
    for l in range(L):
        C, H, W = (4 * C0) << l, H0 >> (l + 1), W0 >> (l + 1)
        out.append((B, C if l == L - 1 else C // 2, H, W))
    return out


def flow_case(B: int, L: int, K: int, C0: int, H0: int, W0: int, k: int = 3, hid: int = 512,
              seed: int = 0) -> dict:
    """Images x ~ N(0, 1) (seed) and latents z[l] ~ N(0, 1) (seed + 1, level 0
    first) for a flow, with its parameters."""
    x = gaussian(np.random.default_rng(seed), (B, C0, H0, W0))
    rz = np.random.default_rng(seed + 1)
    z = [gaussian(rz, s) for s in flow_latent_shapes(B, L, C0, H0, W0)]
    return dict(x=x, z=z, params=flow_params(L, K, C0, k, hid), B=B, L=L, K=K, C0=C0, H0=H0,
                W0=W0, k=k, hid=hid)


# The paper's CIFAR-10 model (Table 3: setting [28, 28, 28], i.e. three
# levels of 28 Steps on 3 x 32 x 32 images; its sampling time is for n = 100
# images), and a small one the oracle runs in a blink.
FLOWS = {
    "flow_cifar10_L3_K28_b100": dict(B=100, L=3, K=28, C0=3, H0=32, W0=32, k=3, hid=512),
    "flow_small_L2_K2_b4": dict(B=4, L=2, K=2, C0=1, H0=8, W0=8, k=3, hid=16),
}
