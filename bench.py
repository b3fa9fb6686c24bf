"""Throughput of the FInC masked-conv hot path on one MI355X.

A step is one pass of the whole path over one batch: the forward masked
convolution, with log|det| and the weight preparation for the inverse (L^-1
and L^-1 K_s) as side outputs of the same launch, then the diagonal-wavefront
inverse of the forward's output.  The default workload is
the single masked 3x3 layer, TL padding, batch 64, 12 channels, 16x16 (a
CIFAR-10 image after one 2x2 squeeze), fp32.

Prints one JSON line.  `value` is sampled images per second through the
step; `roofline` is for the inverse kernel (the dominant one): algorithmic
bytes (read y + write x + the layer's weights) per launch over its mean
duration, timed with HIP events on the stream it runs on; `cpu_baseline`
times the CPU oracle on a bounded sample of the same step.

    python bench.py [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0         # MI355X HBM3E
FP32_VALU_PEAK_TFLOPS = 157.3
METRIC = "masked-conv inverse: images/sec & achieved HBM GB/s (fp32, k=3, batch 64)"
KERNEL_SRC = os.path.join(ROOT, "paper_2301_09266_amd", "csrc", "finc.hip")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=400)
    p.add_argument("--warmup", type=int, default=40)
    p.add_argument("--workload", default="layer_c12_16x16_b64_k3")
    p.add_argument("--cpu-seconds", type=float, default=10.0,
                   help="bound on the CPU-oracle sample (0 disables it)")
    p.add_argument("--graph-steps", type=int, default=20,
                   help="steps captured in one HIP graph (the timed region replays it)")
    p.add_argument("--no-graph", action="store_true",
                   help="launch every step eagerly instead of replaying a HIP graph")
    p.add_argument("--no-configs", action="store_true",
                   help="skip the per-configuration table (forward / inverse of every workload) and the scaling sweep")
    p.add_argument("--no-flow", action="store_true",
                   help="skip the full-flow sampling at the CIFAR-10 setting")
    p.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                   help="only run a plain device copy of MIB MiB ten times (the known-size "
                        "reference for rocprofv3 FETCH_SIZE / WRITE_SIZE) and exit")
    return p.parse_args()


def calibrate_copy(mib: int):
    """Ten plain device-to-device copies of `mib` MiB: each dispatch reads and
    writes exactly mib MiB, the scale for the HBM byte counters."""
    import torch

    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_dispatch": n * 4, "dispatches": 10}))


def kernel_hash() -> str:
    return hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]


def traffic_for(workload: str):
    """HBM bytes per inverse launch from committed rocprofv3 counter runs,
    only if they were taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_sha") != kernel_hash():
        return None
    return rec.get("bytes_per_launch")


class LayerStep:
    """forward (with log|det| and the prepared weights) + inverse of one padded
    masked conv block."""

    def __init__(self, case, dev):
        import numpy as np
        import torch

        from paper_2301_09266_amd import finc

        self.finc = finc
        self.B, self.C, self.H, self.W, self.k = (case[n] for n in "BCHWk")
        self.corner = case["corner"]
        self.x = torch.from_numpy(case["x"].astype(np.float32)).to(dev)
        self.K = torch.from_numpy(case["K"].astype(np.float32)).to(dev)
        self.y = torch.empty_like(self.x)
        self.xr = torch.empty_like(self.x)
        self.ld = torch.empty(1, dtype=torch.float64, device=dev)
        self.prep = torch.empty(finc.workspace_bytes(self.C, self.k, 1), dtype=torch.uint8,
                                device=dev)
        self.case = case

    def forward(self):
        # y, log|det| and the weights prepared for the inverse, from one launch
        self.finc.forward(self.x, self.K, self.corner, out=self.y, logdet=self.ld,
                          prepared=self.prep)

    def inverse(self):
        self.finc.inverse_prepared(self.y, self.prep, self.k, self.corner, out=self.xr)

    def step(self):
        self.forward()
        self.inverse()

    def inverse_bytes(self):
        return 2 * self.B * self.C * self.H * self.W * 4 + self.C * self.C * self.k ** 2 * 4

    def inverse_flops(self):
        C, k = self.C, self.k
        return 2 * self.B * self.H * self.W * (C * C * k * k - C * (C - 1) // 2)

    def steps_per_inverse(self):
        return self.H + self.W - 1

    def pixels(self):
        return self.B * self.H * self.W

    def cpu_step(self, orc, imgs):
        import numpy as np

        x = self.case["x"][imgs].astype(np.float32).astype(np.float64)
        K = self.case["K"].astype(np.float32).astype(np.float64)
        y = orc.forward(x, K, self.corner)
        orc.logdet(K, self.corner, self.H, self.W)
        orc.inverse(y, K, self.corner)


def time_back_to_back(fn, stream, n: int, use_graph: bool) -> float:
    """Mean milliseconds per call of `fn` over about `n` back-to-back calls on
    `stream`, bracketed by HIP events."""
    import torch

    per = 20
    reps = max(1, n // per)
    g = None
    if use_graph:
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(per):
                fn()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(reps):
        if g is not None:
            g.replay()
        else:
            for _ in range(per):
                fn()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (reps * per)


def graph_time_us(fn, reps: int, per: int) -> float:
    """Mean microseconds per call of `fn`: a HIP graph of `per` back-to-back
    calls replayed `reps` times between two events on the current stream."""
    import torch

    return time_back_to_back(fn, torch.cuda.current_stream(), reps * per, True) * 1e3


def per_config(dev) -> list:
    """Forward and inverse of every workload (inputs resident, weights
    prepared once outside the timed region), with the inverse's algorithmic
    HBM bytes over its time against the HBM peak."""
    import numpy as np
    import torch

    from paper_2301_09266_amd import finc, synth

    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
    rows = []
    for name, spec in synth.WORKLOADS.items():
        c = synth.make(name)
        kind = spec["kind"]
        bwd = None
        if kind == "layer":
            B, C, H, W, k = (c[n] for n in "BCHWk")
            x, K = d(c["x"]), d(c["K"])
            y = finc.forward(x, K, c["corner"])
            prep = finc.prepare(K, [c["corner"]])
            out = torch.empty_like(x)
            fwd = graph_time_us(lambda: finc.forward(x, K, c["corner"], out=out), 5, 20)
            inv = graph_time_us(lambda: finc.inverse_prepared(y, prep, k, c["corner"], out=out), 5, 20)
            act, wts, layers = 2 * C * H * W * 4, C * C * k * k * 4, 1
            # training direction: dx and dK of the layer for a loss gradient dy
            dyt = torch.randn_like(x)
            dxo, dKo = torch.empty_like(x), torch.empty_like(K)
            bws = torch.empty(finc.lib().finc_backward_workspace_bytes(B, C, H, W, k),
                              dtype=torch.uint8, device=dev)
            bwd = graph_time_us(lambda: finc.backward(x, dyt, K, c["corner"], -1.0, dx=dxo, dK=dKo,
                                                      workspace=bws), 5, 20)
        elif kind == "unit":
            B, C, H, W, k = (c[n] for n in "BCHWk")
            x, K4 = d(c["x"]), d(c["K4"])
            y = finc.unit_forward(x, K4)
            prep = finc.prepare(K4, [0, 1, 2, 3])
            out = torch.empty_like(x)
            fwd = graph_time_us(lambda: finc.unit_forward(x, K4, out=out), 5, 10)
            inv = graph_time_us(lambda: finc.unit_inverse_prepared(y, prep, k, out=out), 5, 10)
            act, wts, layers = 2 * C * H * W * 4, 4 * C * C * k * k * 4, 4
            # training direction: recompute of the blocks' inputs, four layer backwards
            dyt, dxo, dKo = torch.randn_like(x), torch.empty_like(x), torch.empty_like(K4)
            bws = torch.empty(finc.lib().finc_unit_backward_workspace_bytes(B, C, H, W, k),
                              dtype=torch.uint8, device=dev)
            bwd = graph_time_us(lambda: finc.unit_backward(x, dyt, K4, -1.0, dx=dxo, dK4=dKo,
                                                           workspace=bws), 5, 10)
        elif kind == "split":
            B, C, H, W, k = (c[n] for n in "BCHWk")
            x, Kq4 = d(c["x"]), d(c["Kq4"])
            y = finc.split_forward(x, Kq4)
            prep = finc.prepare(Kq4, [0, 1, 2, 3])
            out = torch.empty_like(x)
            fwd = graph_time_us(lambda: finc.split_forward(x, Kq4, out=out), 5, 20)
            inv = graph_time_us(lambda: finc.split_inverse_prepared(y, prep, k, out=out), 5, 20)
            act, wts, layers = 2 * C * H * W * 4, 4 * (C // 4) ** 2 * k * k * 4, 1
            dyt, dxo, dKo = torch.randn_like(x), torch.empty_like(x), torch.empty_like(Kq4)
            bws = torch.empty(finc.lib().finc_split_backward_workspace_bytes(B, C, H, W, k),
                              dtype=torch.uint8, device=dev)
            bwd = graph_time_us(lambda: finc.split_backward(x, dyt, Kq4, -1.0, dx=dxo, dKq4=dKo,
                                                            workspace=bws), 5, 20)
        else:
            B, C1, H1, W1, k, L, U = (c[n] for n in ("B", "C1", "H1", "W1", "k", "levels", "units"))
            Kf = d(np.concatenate([a.ravel() for a in c["K"]]))
            sf = d(np.concatenate([a.ravel() for a in c["scale"]]))
            bf = d(np.concatenate([a.ravel() for a in c["bias"]]))
            zd = [d(z) for z in c["z"]]
            prep = finc.stack_prepare(Kf, L, U, C1, k)
            out = torch.empty((B, C1, H1, W1), device=dev)
            fwd = None
            inv = graph_time_us(lambda: finc.stack_inverse_prepared(zd, prep, sf, bf, L, U, C1, H1,
                                                                    W1, k, out=out), 2, 3)
            C, H, W = C1, H1, W1
            act = (sum(z[0].size for z in c["z"]) + C1 * H1 * W1) * 4
            wts = sum(a.size for a in c["K"]) * 4
            layers = 4 * U * L
        alg = B * act + wts
        gbs = alg / (inv * 1e-6) / 1e9
        steps = (H + W - 1) * layers if kind != "stack" else None
        row = {"workload": name, "B": B, "C": C, "H": H, "W": W, "k": k, "layers": layers,
               "forward_us": fwd, "inverse_us": inv, "backward_us": bwd,
               "inverse_images_per_s": B / (inv * 1e-6),
               "inverse_pixels_per_s": B * H * W / (inv * 1e-6),
               "inverse_alg_bytes": alg, "inverse_hbm_gbs": gbs,
               "inverse_hbm_frac": gbs / HBM_PEAK_GBS,
               "us_per_diagonal_step": inv / steps if steps else None}
        if kind == "layer":   # set-up, loop and store of one launch (finc_inverse_timeline)
            row["inverse_timeline"] = inverse_timeline(dev, name, reps=5)
        row.update(oracle_row(c, kind, zd if kind == "stack" else y, out))
        rows.append(row)
    return rows


def oracle_row(c, kind, gpu_in, gpu_out):
    """The oracle's inverse on image 0 of a workload: its images/s on the
    host cores (at most 16 threads, each inverting image 0, about two
    seconds), and max |gpu - oracle| / max(1, max |oracle|) for that image
    (gpu_out: the last timed inverse; gpu_in: its input, or the latents of
    the stack)."""
    import numpy as np

    import oracle

    orc = oracle.default()
    f64 = lambda a: np.asarray(a, dtype=np.float32).astype(np.float64)
    h = lambda t: t.detach().cpu().numpy().astype(np.float64)
    if kind == "stack":
        zs = [h(z[:1]) for z in gpu_in]
        Ks, ss, bs = ([f64(a) for a in c[n]] for n in ("K", "scale", "bias"))
        inv = lambda: orc.stack_inverse(zs, Ks, ss, bs, c["levels"], c["units"], c["k"], c["C1"],
                                        c["H1"], c["W1"])
    else:
        y = h(gpu_in[:1])
        if kind == "layer":
            inv = lambda: orc.inverse(y, f64(c["K"]), c["corner"])
        elif kind == "unit":
            inv = lambda: orc.unit_inverse(y, f64(c["K4"]))
        else:
            inv = lambda: orc.split_inverse(y, f64(c["Kq4"]))
    n = oracle_threads()
    rate, _, _ = cpu_rate(lambda i: inv(), 2.0, n)
    want = inv()[0]
    g = h(gpu_out[0])
    return {"oracle_images_per_s": rate, "oracle_cores": n,
            "parity_image0_inf_rel": float(np.abs(g - want).max() / max(1.0, np.abs(want).max())),
            "parity_image0_max_abs": float(np.abs(g - want).max())}


def scaling_sweep(dev) -> dict:
    """Unit inverse (four layers, prepared weights) at C = 2, k = 3 over image
    sizes and batches, after the paper's sampling-time sweep (Sec. 5, Fig. 3)."""
    import numpy as np
    import torch

    from paper_2301_09266_amd import finc, synth

    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
    rows = []
    for n in synth.SWEEP_SIZES:
        for B in synth.SWEEP_BATCHES:
            c = synth.sweep_case(n, B)
            x, K4 = d(c["x"]), d(c["K4"])
            y = x
            for q in range(4):   # the unit's layers one by one (any image size)
                y = finc.forward(y, K4[q].contiguous(), q)
            prep = finc.prepare(K4, [0, 1, 2, 3])
            out = torch.empty_like(x)
            finc.unit_inverse_prepared(y, prep, c["k"], out=out)
            err = float((out - x).abs().max())
            per = 20 if n <= 32 else 5
            us = graph_time_us(lambda: finc.unit_inverse_prepared(y, prep, c["k"], out=out), 3, per)
            rows.append({"n": n, "B": B, "unit_inverse_us": us, "images_per_s": B / (us * 1e-6),
                         "us_per_diagonal_step": us / (4 * (2 * n - 1)),
                         "round_trip_max_abs": err, "form": "one workgroup per image"})
    # beyond one workgroup: the banded stream form (bands of rows in
    # workgroups of their own, pipelined)
    for n in synth.SWEEP_BANDED_SIZES:
        for B in synth.SWEEP_BATCHES:
            c = synth.sweep_case(n, B)
            x, K4 = d(c["x"]), d(c["K4"])
            y = x
            for q in range(4):
                y = finc.forward(y, K4[q].contiguous(), q)
            out, ws = finc.unit_inverse_banded(y, K4)
            err = float((out - x).abs().max())
            us = graph_time_us(lambda: finc.unit_inverse_banded(y, K4, out=out, workspace=ws), 2, 3)
            plan = finc.banded_plan(2, n, n, c["k"])
            rows.append({"n": n, "B": B, "unit_inverse_us": us, "images_per_s": B / (us * 1e-6),
                         "us_per_diagonal_step": us / (4 * (2 * n - 1)),
                         "round_trip_max_abs": err,
                         "form": f"banded: {plan['bands']} bands of {plan['rows']} rows"})
    return {"what": "FInC unit inverse (TL, TR, BL, BR), C = 2, k = 3, n x n images "
                    "(the banded unit call includes its weight preparation)",
            "rows": rows}


def stack_training(dev) -> dict:
    """One training step of the sampling stack's model (3 levels x 8 units
    with actnorm, 12 x 32 x 32, batch 64): the forward to latents and
    log|det|, the batch's negative log-likelihood, and the backward of the
    summed NLL to every weight, scale and bias (the forward is run again
    inside it); by the paper's protocol (11 runs, the first dropped)."""
    import numpy as np
    import torch

    from paper_2301_09266_amd import finc, synth

    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
    spec = synth.WORKLOADS["stack_3x8_c12_32x32_b64_k3"]
    B, C1, H1, W1, L, U, k = (spec[n] for n in ("B", "C1", "H1", "W1", "levels", "units", "k"))
    c = synth.stack_case(B=B, C1=C1, H1=H1, W1=W1, levels=L, units=U, k=k)
    x = d(c["x"][:, :C1, :H1, :W1])
    Kf = d(np.concatenate([np.ravel(a) for a in c["K"]]))
    sf = d(np.concatenate([np.ravel(a) for a in c["scale"]]))
    bf = d(np.concatenate([np.ravel(a) for a in c["bias"]]))
    ws = torch.empty(finc.lib().finc_stack_train_workspace_bytes(B, L, U, C1, H1, W1, k),
                     dtype=torch.uint8, device=dev)
    state = {}

    def fwd():
        state["z"], state["ld"] = finc.stack_forward(x, Kf, sf, bf, L, U, k, workspace=ws)

    def nll():
        state["nll"], state["bpd"] = finc.gauss_nll(state["z"], state["ld"])

    def bwd():
        finc.stack_backward(x, state["z"], Kf, sf, bf, L, U, k, gld=-float(B), workspace=ws)

    fwd(), nll(), bwd()
    torch.cuda.synchronize()
    out = {"workload": "stack_3x8_c12_32x32_b64_k3", "B": B}
    for name, fn in (("forward", fwd), ("nll", nll), ("backward", bwd)):
        out[name] = protocol_runs(lambda: event_ms(fn))
    step = sum(out[n]["mean_ms"] for n in ("forward", "nll", "backward"))
    out["step_ms"] = step
    out["images_per_s"] = B / (step * 1e-3)
    out["note"] = ("untrained random weights (the latents grow to ~1e9 through 24 units): the "
                   "NLL value is not a model quality figure")
    return out


def banded_layers(dev) -> list:
    """Single layers beyond one workgroup (banded stream form): 12 x 128 x 128
    and 16 x 256 x 64 at k = 3, batch 8, weights prepared inside the call."""
    import numpy as np
    import torch

    from paper_2301_09266_amd import finc, synth

    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
    rows = []
    for (B, C, H, W, k) in ((8, 12, 128, 128, 3), (8, 16, 256, 64, 3)):
        c = synth.layer_case(B, C, H, W, k)
        x, K = d(c["x"]), d(c["K"])
        y = finc.forward(x, K, 0)
        out, ws = finc.inverse_banded(y, K, 0)
        err = float((out - x).abs().max())
        us = graph_time_us(lambda: finc.inverse_banded(y, K, 0, out=out, workspace=ws), 3, 5)
        plan = finc.banded_plan(C, H, W, k)
        rows.append({"B": B, "C": C, "H": H, "W": W, "k": k, "inverse_us": us,
                     "images_per_s": B / (us * 1e-6), "us_per_diagonal_step": us / (H + W - 1),
                     "bands": plan["bands"], "band_rows": plan["rows"],
                     "threads": plan["threads"], "round_trip_max_abs": err})
    return rows


def protocol_runs(fn, runs: int = 11) -> dict:
    """The paper's timing protocol (appendix, run-time and confidence
    intervals): `runs` runs, the first dropped, mean, standard deviation and
    the 95% confidence interval of the mean (Student t, runs - 2 degrees of
    freedom).  fn() returns one run's time in milliseconds."""
    import statistics

    t = [fn() for _ in range(runs)][1:]
    m = statistics.mean(t)
    sd = statistics.stdev(t) if len(t) > 1 else 0.0
    tq = {9: 2.262, 4: 2.776, 19: 2.093}.get(len(t) - 1, 1.96)
    half = tq * sd / (len(t) ** 0.5)
    return {"runs": runs, "dropped": 1, "mean_ms": m, "std_ms": sd,
            "ci95_ms": [m - half, m + half]}


def event_ms(fn) -> float:
    import torch

    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b)


def step_cost(dev) -> dict:
    """Where an inverse launch's time goes, from shipped kernels only.
    t_step: the inverse of the same batch and channels at two image widths
    (e.g. H + W - 1 = 31 and 55 diagonal steps for 16 x 16 and 16 x 40), the
    time difference over the extra steps (it also carries those columns' share
    of the load and store); fixed: the 16 x 16 time less 31 t_step (launch,
    argument and weight loads, staging, the store).  t_barrier: a kernel
    doing nothing but the steps' synchronisation (each thread writes an LDS
    value, a barrier, each reads another wave's), 64 workgroups of 256
    threads, per step from 31 and 1031 steps."""
    import ctypes

    import numpy as np
    import torch

    from paper_2301_09266_amd import build, finc, synth

    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
    rows = []
    # (second widths: the widest that keeps the first's kernel instance and
    # partial-tile layout, per finc_inverse_plan)
    for C, H, W1, W2, k in ((12, 16, 16, 40, 3), (12, 32, 24, 40, 3), (48, 8, 8, 32, 3),
                            (24, 16, 16, 32, 3)):
        inst = lambda W: [{key: v for key, v in p.items() if key != "lds"}
                          for p in finc.inverse_plan(finc.PLAN_LAYER, C, H, W, k)]
        assert inst(W1) == inst(W2), (C, H, W1, W2)
        t = []
        for W in (W1, W2):
            c = synth.layer_case(64, C, H, W, k)
            y, K = d(c["x"]), d(c["K"])
            prep = finc.prepare(K, [0])
            out = torch.empty_like(y)
            t.append(graph_time_us(lambda: finc.inverse_prepared(y, prep, k, 0, out=out), 5, 20))
        ts = (t[1] - t[0]) / (W2 - W1)
        rows.append({"C": C, "H": H, "W": [W1, W2], "k": k, "B": 64, "inverse_us": t,
                     "t_step_us": ts, "fixed_us": t[0] - (H + W1 - 1) * ts})
    lib = ctypes.CDLL(build.CALIB_LIB)
    lib.finc_calib_barrier_chain.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                             ctypes.c_void_p]
    buf = torch.empty(64 * 256, dtype=torch.float32, device=dev)
    tb = []
    for steps in (31, 1031):
        # (the stream is taken at each call: graph capture runs on its own)
        run = lambda: lib.finc_calib_barrier_chain(
            ctypes.c_void_p(buf.data_ptr()), 64, steps,
            ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        tb.append(graph_time_us(run, 5, 20))
    return {"rows": rows, "t_barrier_us": (tb[1] - tb[0]) / 1000,
            "barrier_kernel_us": {"31": tb[0], "1031": tb[1]}}


def inverse_timeline(dev, name: str = "layer_c12_16x16_b64_k3", reps: int = 20) -> dict:
    """Where one inverse launch's time goes, from the shipped diagnostic
    finc_inverse_timeline (the GPU's 100 MHz clock read by every wave when
    its arguments arrived, its set-up was done, its last diagonal step was done
    and its store was issued): per workgroup, set-up = the last wave's set-up
    done less the first wave's arguments (weights, the image into LDS, roles
    and addresses), loop = the last wave's
    last step less that, store = the last store issued less the loop's end;
    medians over the workgroups of `reps` launches, in microseconds, and the
    spread of the workgroups' starts within a launch."""
    import numpy as np
    import torch

    from paper_2301_09266_amd import finc, synth

    c = synth.make(name)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
    y, K = d(c["x"]), d(c["K"])
    prep = finc.prepare(K, [c["corner"]])
    rows = []
    for r in range(reps + 3):
        _, st = finc.inverse_timeline(y, prep, c["k"], c["corner"])
        if r < 3:
            continue   # (warm-up)
        t = st.cpu().numpy().astype(np.int64)
        start, setup = t[:, :, 0].min(axis=1), t[:, :, 1].max(axis=1)
        loop_end, store = t[:, :, 2].max(axis=1), t[:, :, 3].max(axis=1)
        rows.append(np.stack([setup - start, loop_end - setup, store - loop_end,
                              start - start.min()], axis=1))
    a = np.concatenate(rows) * 0.01   # 100 MHz ticks -> microseconds
    med = np.median(a, axis=0)
    steps = c["H"] + c["W"] - 1
    return {"workload": name, "launches": reps, "clock_mhz": 100,
            "setup_us": float(med[0]), "loop_us": float(med[1]), "store_us": float(med[2]),
            "loop_us_per_step": float(med[1] / steps),
            "workgroup_start_spread_us": float(np.max(a[:, 3]))}


def flow_sampling(dev, name: str = "flow_cifar10_L3_K28_b100") -> dict:
    """The whole FInC Flow at the paper's CIFAR-10 setting (Table 3: three
    levels of 28 Steps, 3 x 32 x 32, 512-wide coupling networks, n = 100
    images): sampling (latents to images) and the forward (images to latents
    and log|det|), each timed by the paper's protocol; weights prepared once
    outside the timed region."""
    import numpy as np
    import torch

    from paper_2301_09266_amd import finc, synth

    c = synth.flow_case(**synth.FLOWS[name])
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
    a = dict(L=c["L"], K=c["K"], k=c["k"], hid=c["hid"])
    geo = dict(C0=c["C0"], H0=c["H0"], W0=c["W0"])
    params = d(c["params"])
    prep = finc.flow_prepare(params, c["L"], c["K"], c["C0"], c["k"], c["hid"])
    zs = [d(t) for t in c["z"]]
    x = torch.empty((c["B"], c["C0"], c["H0"], c["W0"]), device=dev)
    ws = torch.empty(finc.lib().finc_flow_workspace_bytes(c["B"], c["L"], c["C0"], c["H0"],
                                                          c["W0"], c["hid"]),
                     dtype=torch.uint8, device=dev)
    sample = lambda: finc.flow_sample(zs, params, prep, out=x, workspace=ws, **geo, **a)
    forward = lambda: finc.flow_forward(x, params, prep, workspace=ws, **a)
    sample()
    torch.cuda.synchronize()
    st = protocol_runs(lambda: event_ms(sample))
    ft = protocol_runs(lambda: event_ms(forward))
    # conv flops of the coupling and prior networks (2 per multiply-add), per image
    fl = 0
    for l in range(c["L"]):
        C, hw = (4 * c["C0"]) << l, (c["H0"] >> (l + 1)) * (c["W0"] >> (l + 1))
        hid = c["hid"]
        fl += c["K"] * 2 * hw * (hid * C // 2 * 9 + hid * hid + C * hid * 9)
        if l < c["L"] - 1:
            fl += 2 * hw * C * C // 2 * 9
    B = c["B"]
    return {"workload": name, "B": B, "params": int(params.numel()),
            "sample": st, "sample_images_per_s": B / (st["mean_ms"] * 1e-3),
            "forward": ft, "forward_images_per_s": B / (ft["mean_ms"] * 1e-3),
            "network_gflop_per_image": fl / 1e9,
            "sample_network_tflops": fl * B / (st["mean_ms"] * 1e-3) / 1e12,
            "paper_context": "FInC Flow, CIFAR-10 [28,28,28], 39.46M parameters: ST 0.41 s, "
                             "FT 0.37 s for 100 images on a GTX 1080Ti (Table 3); untrained "
                             "models in both"}


def batch_scaling(dev) -> dict:
    """The benchmark layer (12 x 16 x 16, k = 3, TL) at batches 1, 8 and 64:
    one GPU's share of a batch of 64 sharded over 64, 8 and 1 GPUs."""
    import numpy as np
    import torch

    from paper_2301_09266_amd import finc, synth

    d = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
    rows = []
    for B in (1, 8, 64):
        c = synth.layer_case(B, 12, 16, 16, 3)
        x, K = d(c["x"]), d(c["K"])
        y = finc.forward(x, K, 0)
        prep = finc.prepare(K, [0])
        out = torch.empty_like(x)
        fwd = graph_time_us(lambda: finc.forward(x, K, 0, out=out), 5, 20)
        inv = graph_time_us(lambda: finc.inverse_prepared(y, prep, 3, 0, out=out), 5, 20)
        rows.append({"B": B, "forward_us": fwd, "inverse_us": inv,
                     "inverse_images_per_s": B / (inv * 1e-6)})
    return {"what": "layer 12 x 16 x 16, k = 3, TL, by batch", "rows": rows}


def host_info() -> dict:
    """CPU model and the cores this process may use."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"cpu_model": model, "nproc": len(os.sched_getaffinity(0)),
            "os_cpu_count": os.cpu_count()}


def oracle_threads() -> int:
    # at most 16: a one-GPU machine's share of the host, whatever nproc shows
    return max(1, min(16, len(os.sched_getaffinity(0))))


def cpu_rate(work, seconds: float, threads: int):
    """Images per second of `work(i)` (one image each, i counting up) run on
    `threads` threads until `seconds` have passed (at least one round).  The
    oracle's C calls release the interpreter lock, so threads run in parallel."""
    import concurrent.futures

    done = 0
    t0 = time.perf_counter()
    with concurrent.futures.ThreadPoolExecutor(threads) as pool:
        while True:
            list(pool.map(work, range(done, done + threads)))
            done += threads
            el = time.perf_counter() - t0
            if el >= seconds:
                break
    return done / el, done, el


def cpu_baseline(step, seconds: float):
    """The oracle on the same step (forward, log|det|, raster-order inverse,
    fp64), image by image: on all the host cores this process may use (at
    most 16), and on one thread, each for about `seconds`."""
    import oracle

    orc = oracle.default()
    work = lambda i: step.cpu_step(orc, [i % step.B])
    n = oracle_threads()
    rate, done, el = cpu_rate(work, seconds, n)
    rate1, done1, el1 = cpu_rate(work, seconds / 2, 1)
    return dict(value=rate, unit="images/s", cores=n, kind="oracle",
                sample=f"{done} images of the same step (forward, logdet, raster-order inverse) "
                       f"in fp64 on {n} threads, {el:.1f} s",
                single_thread={"value": rate1, "unit": "images/s", "cores": 1,
                               "sample": f"{done1} images, {el1:.1f} s"},
                host=host_info())


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the path shards by "
              "batch with no communication, so one GPU's throughput is the figure.",
              file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    import numpy as np
    import torch

    from paper_2301_09266_amd import finc, synth

    finc.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    case = synth.make(args.workload)
    if "K" not in case:
        print("bench.py times single-layer workloads", file=sys.stderr)
        sys.exit(2)
    st = LayerStep(case, dev)

    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        st.step()
    torch.cuda.synchronize()

    # HIP graphs of P steps each (and one of the remainder), so that exactly
    # `steps` steps run in the timed region with one submission per P steps
    graphs = []
    if not args.no_graph:
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            st.step()
        torch.cuda.synchronize()
        per = max(1, min(args.graph_steps, args.steps))

        def capture(n):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for _ in range(n):
                    st.step()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            return g

        full = capture(per) if args.steps >= per else None
        graphs = [full] * (args.steps // per) if full is not None else []
        if args.steps % per:
            graphs.append(capture(args.steps % per))
    graph = graphs[0] if graphs else None

    # timed region: exactly `steps` steps
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    if graphs:
        for g in graphs:
            g.replay()
    else:
        for _ in range(args.steps):
            st.step()
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_total = t_start.elapsed_time(t_end)
    ms_per_step = ms_total / args.steps

    # the dominant kernel alone, on the stream it is launched on: HIP events
    # around `steps` back-to-back launches (replays of a graph of 20 launches
    # when graphs are on), and around every single launch for comparison
    inv_ms = time_back_to_back(st.inverse, stream, args.steps, graph is not None)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for a, b in ev:
        a.record(stream)
        st.inverse()
        b.record(stream)
    torch.cuda.synchronize()
    inv_single_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))

    # correctness guard on what was timed
    err = float((st.xr - st.x).abs().max())
    if not err <= 1e-4:
        print(f"round-trip error {err:.3e} exceeds 1e-4", file=sys.stderr)
        sys.exit(1)

    achieved = st.inverse_bytes() / (inv_ms * 1e-3) / 1e9
    traffic = traffic_for(args.workload)
    out = {
        "metric": METRIC,
        "value": st.B / (ms_per_step * 1e-3),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "B": st.B, "C": st.C, "H": st.H, "W": st.W,
                   "k": st.k, "corner": "TL",
                   "graph_steps": (min(args.graph_steps, args.steps) if graphs else 0),
                   "step": "forward + logdet + weight preparation (one launch), inverse"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": "inverse_chain_kernel",
                     "alg_bytes_per_launch": st.inverse_bytes(),
                     "mean_launch_us": inv_ms * 1e3,
                     "timing": "HIP events around back-to-back launches on the kernel's stream",
                     "single_launch_event_us": inv_single_ms * 1e3},
        "inverse": {
            "images_per_s": st.B / (inv_ms * 1e-3),
            "pixels_per_s": st.pixels() / (inv_ms * 1e-3),
            "us_per_diagonal_step": inv_ms * 1e3 / st.steps_per_inverse(),
            "fp32_tflops": st.inverse_flops() / (inv_ms * 1e-3) / 1e12,
            "fp32_frac": st.inverse_flops() / (inv_ms * 1e-3) / 1e12 / FP32_VALU_PEAK_TFLOPS,
        },
        "wall_s_timed": wall,
        "round_trip_max_abs": err,
    }
    # the paper's protocol on the dominant kernel: 11 runs of a graph of 20
    # inverse launches, the first dropped
    if graph is not None:
        g20 = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g20):
            for _ in range(20):
                st.inverse()
        torch.cuda.synchronize()
        pr = protocol_runs(lambda: event_ms(g20.replay))
        out["inverse"]["protocol"] = {k: (v / 20 * 1e3 if k == "mean_ms" or k == "std_ms" else
                                          ([w / 20 * 1e3 for w in v] if k == "ci95_ms" else v))
                                      for k, v in pr.items()}
        out["inverse"]["protocol"]["unit"] = "us per launch (graph of 20)"
    if not args.no_configs:
        out["per_config"] = per_config(dev)
        out["scaling_sweep"] = scaling_sweep(dev)
        out["banded_layers"] = banded_layers(dev)
        out["stack_training"] = stack_training(dev)
        out["batch_scaling"] = batch_scaling(dev)
    if not args.no_configs:
        out["step_cost"] = step_cost(dev)
        out["inverse_timeline"] = inverse_timeline(dev)
    if not args.no_flow:
        out["flow_sampling"] = flow_sampling(dev)
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline(st, args.cpu_seconds)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
