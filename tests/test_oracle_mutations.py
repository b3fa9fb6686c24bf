"""Plant plausible mistakes in copies of the oracle (on the CPU) and check
that the pins catch every one of them."""
import os

import pytest

import oracle
import pins

# (label, text in finc_oracle.c, replacement, which occurrence (0-based))
MUTANTS = [
    ("forward reads the mirrored tap",
     "int ii = i + a - oh, jj = j + b - ow;", "int ii = i - a + oh, jj = j + b - ow;", 0),
    ("forward drops the self diagonal", "if (a == oh && b == ow && ci > co)",
     "if (a == oh && b == ow && ci >= co)", 0),
    ("forward keeps the masked entries", "if (a == oh && b == ow && ci > co)",
     "if (a == oh && b == ow && ci > co + C)", 0),
    ("forward transposes channels", "s += kmasked(K, C, k, oh, ow, co, ci, a, b)",
     "s += kmasked(K, C, k, oh, ow, ci, co, a, b)", 0),
    ("inverse reads the mirrored column",
     "int ii = i + a - oh, jj = j + b - ow;", "int ii = i + a - oh, jj = j - b + ow;", 1),
    ("inverse counts the diagonal twice", "int cmax = self ? c : C;",
     "int cmax = self ? c + 1 : C;", 0),
    ("inverse drops the self block", "int cmax = self ? c : C;",
     "int cmax = self ? 0 : C;", 0),
    ("inverse adds instead of subtracting", "r -= kw(K, C, k, c, ci, a, b)",
     "r += kw(K, C, k, c, ci, a, b)", 0),
    ("inverse transposes channels", "r -= kw(K, C, k, c, ci, a, b)",
     "r -= kw(K, C, k, ci, c, a, b)", 0),
    ("inverse skips the divide", "= r / kw(K, C, k, c, c, oh, ow);", "= r;", 0),
    ("inverse walks rows the wrong way", "int rows_down = (corner == 0 || corner == 1);",
     "int rows_down = (corner == 0 || corner == 2);", 0),
    ("logdet forgets W", "*out = (double)H * (double)W * s;", "*out = (double)H * s;", 0),
    ("logdet reads the wrong tap", "double d = kw(K, C, k, c, c, oh, ow);",
     "double d = kw(K, C, k, c, c, ow, oh);", 0),
    ("corner offsets swapped", "*ow = (corner == 0 || corner == 2) ? k - 1 : 0;",
     "*ow = (corner == 0 || corner == 1) ? k - 1 : 0;", 0),
    ("unit inverse runs the blocks forwards",
     "for (int q = 3; q >= 0 && rc == ORC_OK; --q)",
     "for (int q = 0; q < 4 && rc == ORC_OK; ++q)", 0),
    ("squeeze swaps dy and dx", "int co = 4 * c + 2 * dy + dx;",
     "int co = 4 * c + dy + 2 * dx;", 0),
    ("actnorm inverse subtracts after scaling", "x[o] = (y[o] - b[c]) / s[c];",
     "x[o] = y[o] / s[c] - b[c];", 0),
    ("stack inverse runs units forwards",
     "for (int u = U - 1; u >= 0 && rc == ORC_OK; --u)",
     "for (int u = 0; u < U && rc == ORC_OK; ++u)", 0),
    ("stack inverse concatenates latent first",
     "memcpy(h + b * 2 * Cq * hw, t + b * Cq * hw, sizeof(double) * Cq * hw);",
     "memcpy(h + (b * 2 * Cq + Cq) * hw, t + b * Cq * hw, sizeof(double) * Cq * hw);", 0),
    ("backward input gradient transposes channels",
     "kmasked(K, C, k, oh, ow, co, ci, a, b) * g;", "kmasked(K, C, k, oh, ow, ci, co, a, b) * g;",
     0),
    ("backward keeps the masked weight gradients", "if (!(a == oh && b == ow && ci > co))",
     "if (1)", 0),
    ("backward forgets the log|det| term",
     "s += gld * (double)H * (double)W / kw(K, C, k, co, co, a, b);", "s += 0.0;", 0),
    ("unit backward feeds each block its own output",
     "rc = orc_backward(h[q], g, K4 + q * ksz, gn,",
     "rc = orc_backward(h[q < 3 ? q + 1 : 3], g, K4 + q * ksz, gn,", 0),
    ("unit backward gives the log|det| term to the last block only",
     "dK4 ? dK4 + q * ksz : NULL, gld, B, C, H,", "dK4 ? dK4 + q * ksz : NULL, q == 3 ? gld : 0.0, B, C, H,", 0),
    ("split backward gives every quarter the first corner",
     "H, W, k, g);\n        for (long b = 0; dx", "H, W, k, 0);\n        for (long b = 0; dx", 0),
    ("actnorm backward forgets the log|det| term", "ds[c] = sx + gld * (double)plane / s[c];",
     "ds[c] = sx;", 0),
    ("actnorm backward scales dx by 1/s", "dx[o] = s[c] * dy[o];", "dx[o] = dy[o] / s[c];", 0),
    ("nll drops the normalising constant", "q += 0.5 * (v * v + log2pi);", "q += 0.5 * v * v;", 0),
    ("nll adds the log|det|", "nll[b] = q - logdet[b];", "nll[b] = q + logdet[b];", 0),
    ("bpd in nats", "bpd[b] = nll[b] / ((double)D * log(2.0));", "bpd[b] = nll[b] / (double)D;", 0),
    ("stack forward keeps the latent half",
     "memcpy(t + b * Ch * hw, h + b * C * hw, sizeof(double) * Ch * hw);",
     "memcpy(t + b * Ch * hw, h + (b * C + Ch) * hw, sizeof(double) * Ch * hw);", 0),
    ("stack forward passes the scale as the bias",
     "orc_actnorm_forward(t, h, sl + (long)u * C, bl + (long)u * C, B, C, H, W);",
     "orc_actnorm_forward(t, h, sl + (long)u * C, sl + (long)u * C, B, C, H, W);", 0),
    ("actnorm forward reads the scale of the next channel", "y[o] = s[c] * x[o] + b[c];",
     "y[o] = s[(c + 1) % C] * x[o] + b[c];", 0),
    ("stack logdet forgets the actnorms", "s += (double)H * W * log(fabs(sl[(long)u * C + c]));",
     "s += 0.0;", 0),
    ("stack backward puts the latent gradient first",
     "memcpy(g + (b * C + Ch) * hw, dz[l] + b * Ch * hw, sizeof(double) * Ch * hw);",
     "memcpy(g + b * C * hw, dz[l] + b * Ch * hw, sizeof(double) * Ch * hw);", 0),
    ("stack backward feeds the unit's output to its actnorm's backward as input",
     "rc = orc_actnorm_backward(tu, g, sl + (long)u * C, gt,",
     "rc = orc_actnorm_backward(tu + n, g, sl + (long)u * C, gt,", 0),
    ("backward weight gradient reads the mirrored tap",
     "x[n * img + ci * plane + (long)ii * W + jj];",
     "x[n * img + ci * plane + (long)(H - 1 - ii) * W + jj];", 0),
    ("1x1 forward transposes the matrix", "s += Wm[(long)co * C + ci] * x[(n * C + ci) * plane + p];",
     "s += Wm[(long)ci * C + co] * x[(n * C + ci) * plane + p];", 0),
    ("1x1 inverse forgets the row order", "double s = y[(n * C + perm[r]) * plane + p];",
     "double s = y[(n * C + r) * plane + p];", 0),
    ("1x1 logdet drops a pivot", "ld += log(fabs(d));", "ld += c ? log(fabs(d)) : 0.0;", 0),
    ("coupling network pads on one side only", "int ii = i + a - pad, jj = j + b - pad;",
     "int ii = i + a - 2 * pad, jj = j + b - pad;", 0),
    ("coupling network skips a ReLU", "conv_same(t1, t2, W2, b2, NULL, B, hid, hid, H, W, 1, 1);",
     "conv_same(t1, t2, W2, b2, NULL, B, hid, hid, H, W, 1, 0);", 0),
    ("coupling scale without the +2", "double s = sigmoid(r + 2.0);", "double s = sigmoid(r);", 0),
    ("coupling adds the shift after scaling",
     "y[n * 2 * half + half + e] = (x[n * 2 * half + half + e] + t) * s;",
     "y[n * 2 * half + half + e] = x[n * 2 * half + half + e] * s + t;", 0),
    ("coupling inverse multiplies by the scale",
     "y[n * 2 * half + half + e] / sigmoid(r + 2.0) - t;",
     "y[n * 2 * half + half + e] * sigmoid(r + 2.0) - t;", 0),
    ("step inverse undoes actnorm before the 1x1",
     "rc = orc_conv1x1_inverse(t1, t2, Wm, B, C, H, W);",
     "rc = orc_conv1x1_inverse(t1, t2, Wm, B, C, H, W); orc_actnorm_inverse(t2, t1, s, b, B, C, H, W); orc_conv1x1_inverse(t1, t2, Wm, B, C, H, W);", 0),
    ("step logdet forgets the actnorm", "logdet[n] += lu + la + lw;", "logdet[n] += lu + lw;", 0),
    ("split prior latent uses exp(+logsd)",
     "z[l][n * Ch * plane + e] = (t[n * C * plane + Ch * plane + e] - mean) * exp(-logsd);",
     "z[l][n * Ch * plane + e] = (t[n * C * plane + Ch * plane + e] - mean) * exp(logsd);", 0),
    ("split prior forgets its log|det|", "ld -= logsd;", "ld -= 0.0;", 0),
    ("flow sample runs the steps forwards", "for (int s = K - 1; s >= 0 && rc == ORC_OK; --s) {",
     "for (int s = 0; s < K && rc == ORC_OK; ++s) {", 0),
]


def _mutate(src: str, old: str, new: str, nth: int) -> str:
    pos = -1
    for _ in range(nth + 1):
        pos = src.index(old, pos + 1)
    return src[:pos] + new + src[pos + len(old):]


@pytest.mark.parametrize("label,old,new,nth", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, label, old, new, nth):
    src = open(oracle.SRC).read()
    mutated = _mutate(src, old, new, nth)
    assert mutated != src
    cpath = os.path.join(tmp_path, "mutant.c")
    open(cpath, "w").write(mutated)
    lib = oracle.build(src=cpath, out=os.path.join(tmp_path, "libmutant.so"))
    o = oracle.Oracle(lib)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(o)
        except (AssertionError, oracle.OracleError) as e:
            failed.append((pin.__name__, str(e)[:80]))
            break
    assert failed, f"no pin caught mutant: {label}"
