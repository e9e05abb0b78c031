#!/usr/bin/env python3
"""Benchmark of the SS-Conv hot path on one MI355X.

A step is one pass of the whole path over one seeded synthetic input already
resident in HBM: rule book (hash build, output sites, neighbour probes, pair
compaction), kernel synthesis, forward gather-MFMA, and backward (feature and
coefficient gradients; for the five-layer stack also the gates).  The rule
book is rebuilt every step, as it would be for every new input.

Prints ONE JSON line: throughput in M active output sites/s, the roofline of
the dominant kernel (timed with events on the stream it runs on) and the CPU
oracle timed on a bounded sample on this host.

    python bench.py [--steps K] [--warmup W] [--config {1..9}] [--no-cpu-baseline]
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "SS-Conv layer throughput: M active output sites/s + % of MFMA/HBM roofline"
PEAK = {"f32": 157.3, "bf16": 2516.6}     # dense MFMA TFLOP/s, MI355X
HBM_PEAK_GBS = 8000.0


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------
# HBM traffic of the gather-GEMM kernel from rocprofv3 counter runs
# ---------------------------------------------------------------------------
CSRC = os.path.join(ROOT, "paper_2111_07383_amd", "csrc")
# kernel symbol and the source files that decide its device code, per compute dtype
GATHER_KERNEL = {"bf16": ("gather_bf16_kernel", ["gather_bf16.hip", "lds_dma.hpp", "gather_mfma.hpp", "common.hpp"]),
                 "f32": ("gather_mfma_kernel", ["gather_mfma.hip", "lds_dma.hpp", "gather_mfma.hpp", "common.hpp"])}
COPY_KERNEL = "__amd_rocclr_copyBuffer"


def kernel_name(dtype):
    return GATHER_KERNEL[dtype][0]


def kernel_source_hash(dtype):
    import hashlib
    h = hashlib.sha256()
    for f in GATHER_KERNEL[dtype][1]:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def traffic_path(spec):
    return os.path.join(ROOT, "profiles", f"traffic_{kernel_name(spec.dtype)}_{spec.name}.txt")


def traffic_from_summary(spec):
    """HBM bytes per gather-GEMM launch from the committed counter summary, or None when
    there is none or the kernel's sources changed since the counters were taken."""
    path = traffic_path(spec)
    if not os.path.exists(path):
        return None, "no counter summary"
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith(" "):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != kernel_source_hash(spec.dtype):
        return None, f"{os.path.relpath(path, ROOT)} predates the current kernel source"
    return float(kv["traffic_bytes_per_launch"]), os.path.relpath(path, ROOT)


def _counter_rows(d):
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    rows = []
    for f in files:
        rows += list(csv.DictReader(open(f)))
    return rows


def _per_dispatch(rows, name_part, counter):
    vals = {}
    for r in rows:
        if name_part in r["Kernel_Name"] and r["Counter_Name"] == counter:
            vals[r["Dispatch_Id"]] = vals.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    return list(vals.values())


def write_traffic_summary(args):
    """Turns four rocprofv3 --pmc runs into the summary that traffic_from_summary reads:
    fetch/ and write/ under args.traffic_summary (the workload), copy_fetch/ and
    copy_write/ under args.copy_pmc (a plain device copy of args.copy_mb MiB)."""
    from workloads import CONFIGS
    spec = CONFIGS[args.config]
    d = args.traffic_summary
    dc = args.copy_pmc or d
    kname = kernel_name(spec.dtype)
    mb = args.copy_mb or 256
    fetch = _per_dispatch(_counter_rows(os.path.join(d, "fetch")), kname, "FETCH_SIZE")
    write = _per_dispatch(_counter_rows(os.path.join(d, "write")), kname, "WRITE_SIZE")
    cf = _per_dispatch(_counter_rows(os.path.join(dc, "copy_fetch")), COPY_KERNEL, "FETCH_SIZE")
    cw = _per_dispatch(_counter_rows(os.path.join(dc, "copy_write")), COPY_KERNEL, "WRITE_SIZE")
    if not (fetch and write and cf and cw):
        raise SystemExit("missing dispatches of the kernel or of the copy in the counter runs")
    kib = mb * 1024.0
    ff, fw = kib / float(np.mean(cf)), kib / float(np.mean(cw))
    fk, wk = float(np.mean(fetch)), float(np.mean(write))
    traffic = (fk * ff + wk * fw) * 1024.0
    run = (f"python3 bench.py --config {spec.index} --steps 3 --warmup 1 --no-cpu-baseline --secondary 0")
    cmds = [f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d {d}/fetch -o p -- {run}",
            f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d {d}/write -o p -- {run}",
            f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d {dc}/copy_fetch -o p -- "
            f"python3 bench.py --copy-mb {mb} --steps 2",
            f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d {dc}/copy_write -o p -- "
            f"python3 bench.py --copy-mb {mb} --steps 2",
            f"python3 bench.py --config {spec.index} --copy-mb {mb} --traffic-summary {d}"
            + (f" --copy-pmc {dc}" if dc != d else "")]
    lines = [f"# HBM traffic of {kname} on {spec.name} (rocprofv3 counters, KiB per dispatch)",
             "commands (from the repository root, TMPDIR=/tmp, each rocprofv3 run under timeout -s KILL 120):"]
    lines += [f"  {c}" for c in cmds]
    lines += [f"kernel: {kname}",
              f"source_sha256: {kernel_source_hash(spec.dtype)}",
              f"dispatches: {len(fetch)} (FETCH_SIZE run), {len(write)} (WRITE_SIZE run)",
              f"fetch_kib_per_dispatch: {fk:.1f}",
              f"write_kib_per_dispatch: {wk:.1f}",
              f"copy_calibration: {COPY_KERNEL} of {mb} MiB reads FETCH_SIZE {np.mean(cf):.1f} KiB, "
              f"WRITE_SIZE {np.mean(cw):.1f} KiB",
              f"fetch_factor: {ff:.4f}",
              f"write_factor: {fw:.4f}",
              f"traffic_bytes_per_launch: {traffic:.0f}"]
    path = traffic_path(spec)
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    log(f"wrote {os.path.relpath(path, ROOT)}: {traffic / 1e6:.1f} MB per launch")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=4, help="workload index 1..9 (default: the 128^3 3x3x3 208-channel "
                    "bf16 layer; 2: the 64^3 5x5x5 104-channel fp32 layer; 5: the five-layer stack; 6: the "
                    "downsampling block conv + norm + gate + pooling; 7: input voxelisation; "
                    "8: Feature-Steering; 9: Tensor-to-Point)")
    ap.add_argument("--secondary", type=int, default=-1,
                    help="a second workload measured after the first and reported in the same line under "
                         "'secondary' (default: 2 after the bf16 layer 4, none otherwise; 0: none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle work to aim for")
    ap.add_argument("--only", choices=["step", "forward"], default="step",
                    help="'forward' times the forward gather-GEMM alone over one prebuilt rule book")
    ap.add_argument("--variant", type=int, default=0, help="gather-GEMM tile-configuration override (tuning)")
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="instead of the benchmark, run plain device copies of this many MiB (counter calibration)")
    ap.add_argument("--traffic-summary", default="",
                    help="write the HBM-traffic summary under profiles/ from the rocprofv3 counter runs in this "
                         "directory (runs on the CPU; --copy-mb gives the calibration copy size)")
    ap.add_argument("--stats-summary", default="",
                    help="write profiles/kernels_<workload>.txt from the rocprofv3 --kernel-trace --stats run in this "
                         "directory (runs on the CPU)")
    ap.add_argument("--stats-log", default="", help="stdout of that profiled run (holds the benchmark's JSON line)")
    ap.add_argument("--counter-summary", default="",
                    help="write profiles/counters_<workload>.txt from the rocprofv3 --pmc runs (fetch/, write/, mfma/) "
                         "in this directory (runs on the CPU)")
    ap.add_argument("--copy-pmc", default="",
                    help="directory of the copy-calibration counter runs (default: the --traffic-summary one)")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# GPU side
# ---------------------------------------------------------------------------

class StreamOrder:
    """Orders a stream after the work queued so far on another one, through a reused HIP event
    created without timing and without the system-scope fence: device-side ordering needs
    neither, and a fenced record writes back the caches between two kernels of the stream.
    Calls the HIP runtime the library itself links (same process-wide instance as torch's)."""

    def __init__(self):
        import ctypes
        self.ct = ctypes
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.events = {}

    def _check(self, rc, what):
        if rc != 0:
            raise RuntimeError(f"{what} failed with HIP error {rc}")

    def wait(self, waiter, signaller):
        ct, hip = self.ct, self.hip
        key = (waiter.cuda_stream, signaller.cuda_stream)
        ev = self.events.get(key)
        if ev is None:
            ev = ct.c_void_p()
            self._check(hip.hipEventCreateWithFlags(ct.byref(ev), ct.c_uint(0x2 | 0x20000000)),
                        "hipEventCreateWithFlags")  # hipEventDisableTiming | hipEventDisableSystemFence
            self.events[key] = ev
        self._check(hip.hipEventRecord(ev, ct.c_void_p(signaller.cuda_stream)), "hipEventRecord")
        self._check(hip.hipStreamWaitEvent(ct.c_void_p(waiter.cuda_stream), ev, ct.c_uint(0)), "hipStreamWaitEvent")


class SingleLayer:
    def __init__(self, i, dev):
        import torch
        import paper_2111_07383_amd as P
        from workloads import CONFIGS
        from workloads.gen import make_coeffs, make_coords, make_features, make_grad
        self.P, self.torch = P, torch
        spec = CONFIGS[i]
        self.spec, self.L = spec, spec.layers[0]
        self.dt = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
        self.desc = P.layer_desc(self.L)
        self.basis = torch.from_numpy(P.basis_build(self.desc)).to(dev)
        self.n_coeff = P.basis_info(self.desc)[1]
        coords = make_coords(spec)
        self.coords = torch.from_numpy(coords).to(dev)
        self.feats = torch.from_numpy(make_features(spec, len(coords), self.L.cin)).to(dev).to(self.dt)
        self.coeffs = torch.from_numpy(make_coeffs(spec, [self.n_coeff])[0]).to(dev)
        rb = P.Rulebook(self.coords, spec.grid, self.L.ksize, self.L.stride, self.L.submanifold)
        self.n_out, self.n_pairs = rb.n_out, rb.n_pairs
        rb.close()
        self.grad = torch.from_numpy(make_grad(spec, self.n_out, self.L.cout)).to(dev).to(self.dt)
        rb = P.Rulebook(self.coords, spec.grid, self.L.ksize, self.L.stride, self.L.submanifold)
        ws = P.backward_workspace_size(rb, self.dt, self.L.cin, self.L.cout)
        self.hash_cap = int(rb.hash_slots(0).shape[0])
        rb.close()
        self.ws = torch.empty((ws,), dtype=torch.uint8, device=dev)
        K = self.L.ksize ** 3
        self.W = torch.empty((K, self.L.cout, self.L.cin), dtype=self.dt, device=dev)
        self.side = torch.cuda.Stream(device=dev)  # default priority, like every stream here
        self.pending = None     # rule book of the next step, queued on the side stream
        self.done = None        # rule book of the previous step, closed once its backward is ordered
        self.order = StreamOrder()
        self.events = None      # per-step [synth, rulebook, forward, backward] boundaries when set

    def forward_only(self):
        P, torch = self.P, self.torch
        if not hasattr(self, "_rb"):
            L = self.L
            self._rb = P.Rulebook(self.coords, self.spec.grid, L.ksize, L.stride, L.submanifold)
            self._W = P.synth_kernel(self.desc, self.basis, self.coeffs, self.dt)
            self._out = torch.empty((self.n_out, L.cout), dtype=self.dt, device=self.feats.device)
        P.forward(self.feats, self._rb, self._W, out=self._out)

    def _build_next(self):
        """The rule-book build of a next step, queued on the side stream."""
        L = self.L
        return self.P.Rulebook(self.coords, self.spec.grid, L.ksize, L.stride, L.submanifold, stream=self.side,
                               asynchronous=True)

    def step(self):
        """One training step of the layer: synthesis, rule book, forward, backward.

        Timed steps prefetch the rule book: it needs only the coordinates (the next batch's are
        known to a training loop), so each step's build is queued on the side stream behind the
        previous step's forward and runs beside that step's backward (its kernel gradient, not a
        gather); the main stream waits for it before its forward.  The synthesis stays at the
        head of the step on the main stream, after the previous backward in stream order: it
        needs the coefficients as updated from that backward's gradient.  Every step still
        synthesises one kernel, builds one rule book and runs one forward and one backward.  A
        step's rule book is closed (its blocks freed, stream-ordered on the side stream) in the
        next step, after the side stream's wait for that step's forward, which follows the
        backward that last read it."""
        if self.events is not None:
            return self.step_in_sequence()
        P, torch = self.P, self.torch
        main = torch.cuda.current_stream()
        if self.pending is None:
            self.order.wait(self.side, main)
            self.pending = self._build_next()
        rb = self.pending
        self.order.wait(main, self.side)   # next to the step boundary's records, not between kernels
        W = P.synth_kernel(self.desc, self.basis, self.coeffs, self.dt, out=self.W)
        out = P.forward(self.feats, rb, W)
        self.order.wait(self.side, main)
        if self.done is not None:
            self.done.close()
        self.pending = self._build_next()
        P.backward(self.feats, self.grad, rb, W, self.desc, self.basis, n_coeff=self.n_coeff, workspace=self.ws)
        self.done = rb
        return out

    def drain(self):
        """Closes the rule books still held by the pipelined steps (after the device is idle)."""
        if self.pending is not None or self.done is not None:
            self.torch.cuda.synchronize()
        for rb in (self.pending, self.done):
            if rb is not None:
                rb.close()
        self.pending = self.done = None

    def step_in_sequence(self):
        """The same step with every phase in sequence on one stream, bracketed by events (the
        per-phase report)."""
        P, L, torch = self.P, self.L, self.torch
        self.drain()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
        self.events.append(ev)
        ev[0].record()
        W = P.synth_kernel(self.desc, self.basis, self.coeffs, self.dt, out=self.W)
        ev[1].record()
        # asynchronous build: the forward is queued behind it without a host round trip (a bf16
        # forward needs only the neighbour map; the backward settles the build)
        rb = P.Rulebook(self.coords, self.spec.grid, L.ksize, L.stride, L.submanifold, asynchronous=True)
        ev[2].record()
        out = P.forward(self.feats, rb, W)
        ev[3].record()
        P.backward(self.feats, self.grad, rb, W, self.desc, self.basis, n_coeff=self.n_coeff, workspace=self.ws)
        ev[4].record()
        rb.close()
        return out

    def phase_report(self):
        """Per-phase medians of the timed steps against each phase's roofline time, as defined for
        the layer: rule book and synthesis bound by HBM bytes, each GEMM phase by the larger of
        useful FLOPs / MFMA peak and algorithmic bytes / HBM peak."""
        if not self.events:
            return None
        L, K = self.L, self.L.ksize ** 3
        t = np.array([[a.elapsed_time(b) for a, b in zip(ev, ev[1:])] for ev in self.events])  # ms
        med = np.median(t, 0)
        b = 2 if self.spec.dtype == "bf16" else 4
        n_in, n_out, P_ = int(self.coords.shape[0]), int(self.n_out), int(self.n_pairs)
        peak = PEAK[self.spec.dtype] * 1e12
        hbm = HBM_PEAK_GBS * 1e9
        flops = 2.0 * P_ * L.cin * L.cout
        w_bytes = K * L.cin * L.cout * b
        rb_bytes = 16 * n_in + 8 * self.hash_cap + 8 * n_in + 12 * n_out * K + 8 * P_
        synth_bytes = w_bytes + 4 * int(self.basis.numel()) + 4 * int(self.n_coeff)
        gemm_bytes = n_in * L.cin * b + n_out * L.cout * b + w_bytes + 4 * P_
        dw_bytes = n_in * L.cin * b + n_out * L.cout * b + 8 * P_ + K * L.cin * L.cout * 4
        roof = [synth_bytes / hbm, rb_bytes / hbm, max(flops / peak, gemm_bytes / hbm),
                max(flops / peak, gemm_bytes / hbm) + max(flops / peak, dw_bytes / hbm)]
        names = ["synth", "rulebook", "forward", "backward"]  # launch order of the step
        out = {n: {"ms": float(m), "roofline_ms": float(r) * 1e3, "frac": float(r * 1e3 / m)}
               for n, m, r in zip(names, med, roof)}
        layer_ms = float(med[:3].sum())
        layer_roof = float(sum(roof[:3])) * 1e3
        out["layer"] = {"what": "synth+rulebook+forward", "ms": layer_ms, "roofline_ms": layer_roof,
                        "frac": layer_roof / layer_ms, "M_sites_per_s": n_out / layer_ms / 1e3}
        out["forward"]["M_sites_per_s"] = n_out / float(med[2]) / 1e3
        out["backward"]["M_sites_per_s"] = n_out / float(med[3]) / 1e3
        step = t.sum(1)
        out["step_ms"] = {"p10": float(np.percentile(step, 10)), "median": float(np.median(step)),
                          "p90": float(np.percentile(step, 90))}
        return out

    def sites(self):
        return self.n_out

    def gather_flops(self, forward_only):
        """Algorithmic flops of the gather-GEMM launches of one step: the forward and, in a
        full step, the input-feature gradient, each 2 * pairs * cin * cout."""
        f = 2.0 * self.n_pairs * self.L.cin * self.L.cout
        return (f, 1) if forward_only else (2 * f, 2)

    def config(self):
        L = self.L
        return {"workload": self.spec.name, "grid": self.spec.grid, "batch": self.spec.batch, "ksize": L.ksize,
                "stride": L.stride, "submanifold": L.submanifold, "cin": L.cin, "cout": L.cout,
                "n_in": int(self.coords.shape[0]), "n_out": int(self.n_out), "pairs": int(self.n_pairs),
                "step": "synth+rulebook+forward+backward(dfeats,dcoeffs)"}


class StackBench:
    def __init__(self, dev):
        import torch
        import paper_2111_07383_amd as P
        from paper_2111_07383_amd.stack import Stack
        from workloads import CONFIGS
        from workloads.gen import make_coeffs, make_coords, make_features, make_grad
        self.P, self.torch = P, torch
        spec = CONFIGS[5]
        self.spec = spec
        counts = [P.basis_info(P.layer_desc(L))[1] for L in spec.layers]
        self.st = Stack.create(spec.layers, make_coeffs(spec, counts), spec.grid, dev)
        coords = make_coords(spec)
        self.coords = torch.from_numpy(coords).to(dev)
        self.feats = torch.from_numpy(make_features(spec, len(coords), spec.layers[0].cin)).to(dev)
        self.st.forward(self.coords, self.feats)
        self.n_outs = [L.rb.n_out for L in self.st.layers]
        self.pairs = [L.rb.n_pairs for L in self.st.layers]
        self.grad = torch.from_numpy(make_grad(spec, self.n_outs[-1], spec.layers[-1].cout)).to(dev)

    def step(self, overlap=True):
        self.st.forward(self.coords, self.feats, overlap=overlap)
        self.st.backward(self.grad, need_input_grad=False)

    def sites(self):
        return sum(self.n_outs)

    def roofline_ms(self):
        """The stack's roofline time: per layer, synthesis and rule book at HBM bandwidth on their
        algorithmic bytes, each GEMM phase (forward, input-feature gradient for layers 2..5,
        kernel gradient) at the fp32 MFMA peak on its useful FLOPs, gates at HBM bandwidth."""
        P = self.P
        hbm, peak = HBM_PEAK_GBS * 1e9, PEAK["f32"] * 1e12
        t = 0.0
        n_in = int(self.coords.shape[0])
        for i, (L, p, n_out, lay) in enumerate(zip(self.spec.layers, self.pairs, self.n_outs, self.st.layers)):
            K = L.ksize ** 3
            cap = 64
            while cap < 2 * n_in:
                cap *= 2
            rb_bytes = 16 * n_in + 8 * cap + 8 * n_in + 12 * n_out * K + 8 * p
            synth_bytes = K * L.cin * L.cout * 4 + 4 * int(lay.basis.numel())
            f = 2.0 * p * L.cin * L.cout
            gemms = f * (3 if i > 0 else 2)
            gate = 0
            if L.gated:
                c = P.n_channels(L.fields_out[:-1])
                gate = 2 * (n_out * L.cout * 4 + n_out * c * 4)      # forward and backward
            t += (rb_bytes + synth_bytes + gate) / hbm + gemms / peak
            n_in = n_out
        return t * 1e3

    def serial_report(self, steps=10):
        """Extra steps with the side stream and the backward fork off, so that no kernel overlaps
        another: the stack's time against its roofline, and the gather-GEMM launches timed alone."""
        torch, P = self.torch, self.P
        P.debug_set(3, 11)
        try:
            self.step(overlap=False)
            torch.cuda.synchronize()
            P.debug_set(4, 1)
            t0 = time.perf_counter()
            for _ in range(steps):
                self.step(overlap=False)
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) / steps * 1e3
            n_timed, kern_ms = P.debug_kernel_ms()
            P.debug_set(4, 0)
        finally:
            P.debug_set(3, 0)
        flops, launches = self.gather_flops(False)
        achieved = flops * steps / (kern_ms / 1e3) / 1e12
        roof = self.roofline_ms()
        return {"what": "serialised steps (no side stream, no backward fork): stack forward + backward",
                "stack": {"ms": ms, "roofline_ms": roof, "frac": roof / ms, "M_sites_per_s": self.sites() / ms / 1e3},
                "gather_gemm": {"launches": n_timed, "avg_launch_ms": kern_ms / max(n_timed, 1),
                                "achieved_tflops": achieved, "frac": achieved / PEAK["f32"]}}

    def gather_flops(self, forward_only):
        """Forward gather-GEMM of every layer plus the input-feature gradient of layers 2..5
        (the stack input needs no gradient)."""
        f = [2.0 * p * L.cin * L.cout for p, L in zip(self.pairs, self.spec.layers)]
        return sum(f) + sum(f[1:]), 2 * len(f) - 1

    def config(self):
        return {"workload": self.spec.name, "grid": self.spec.grid, "batch": self.spec.batch,
                "layers": len(self.spec.layers), "n_in": int(self.coords.shape[0]), "n_out_per_layer": self.n_outs,
                "pairs_per_layer": [int(p) for p in self.pairs],
                "step": "5 x (rulebook+synth+forward+gate) + backward"}


class BlockBench:
    """The paper's downsampling block (workload 6): stride-1 submanifold SS-Conv -> Norm -> gate
    -> 2x2x2 average pooling, forward and backward (feature and coefficient gradients).  The
    same calls, in the same order, as ``stack.DownBlock``, with an event between every two."""
    NAMES = ["synth", "rulebook", "conv_norm_forward", "gate_forward", "pool_rulebook",
             "pool_forward", "pool_backward", "gate_backward", "norm_backward", "conv_backward"]

    def __init__(self, i, dev):
        import torch
        import paper_2111_07383_amd as P
        from paper_2111_07383_amd.stack import regular_fields
        from workloads import CONFIGS
        from workloads.gen import make_coeffs, make_coords, make_features, make_grad
        self.P, self.torch = P, torch
        spec = CONFIGS[i]
        self.spec, self.L = spec, spec.layers[0]
        self.regular = regular_fields(self.L)
        self.desc = P.layer_desc(self.L)
        self.basis = torch.from_numpy(P.basis_build(self.desc)).to(dev)
        self.n_coeff = P.basis_info(self.desc)[1]
        coords = make_coords(spec)
        self.coords = torch.from_numpy(coords).to(dev)
        self.feats = torch.from_numpy(make_features(spec, len(coords), self.L.cin)).to(dev)
        self.coeffs = torch.from_numpy(make_coeffs(spec, [self.n_coeff])[0]).to(dev)
        rb = P.Rulebook(self.coords, spec.grid, self.L.ksize, 1, True)
        self.n_pairs = rb.n_pairs
        self.ws = torch.empty((P.backward_workspace_size(rb, torch.float32, self.L.cin, self.L.cout),),
                              dtype=torch.uint8, device=dev)
        rb.close()
        prb = P.Rulebook(self.coords, spec.grid, 2, 2, False)
        self.n_out = prb.n_out
        prb.close()
        self.grad = torch.from_numpy(make_grad(spec, self.n_out, P.n_channels(self.regular))).to(dev)
        self.events = None
        from paper_2111_07383_amd.stack import LayerState
        self.state = LayerState(self.L, self.desc, self.basis, self.coeffs, self.n_coeff, spec.grid)
        self.blk = None

    def step(self):
        """One block forward + backward as DownBlock runs it (pooling rule book on a side
        stream, overlapping the convolution, Norm and gate)."""
        if self.blk is None:
            from paper_2111_07383_amd.stack import DownBlock
            self.blk = DownBlock(self.state, self.torch.float32)
        _, out = self.blk.forward(self.coords, self.feats)
        self.blk.backward(self.grad)
        return out

    def phase_step(self):
        """The same calls one after another on one stream, with an event between every two (for
        the per-phase report)."""
        P, L, torch = self.P, self.L, self.torch
        ev = None
        if self.events is not None:
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(self.NAMES) + 1)]
            self.events.append(ev)
            ev[0].record()
        marks = iter(ev[1:] if ev else [])

        def mark():
            if ev:
                next(marks).record()
        W = P.synth_kernel(self.desc, self.basis, self.coeffs, torch.float32)
        mark()
        rb = P.Rulebook(self.coords, self.spec.grid, L.ksize, 1, True, asynchronous=True)
        mark()
        y, z = P.forward_norm(self.feats, rb, W, L.fields_out)
        mark()
        h = P.gate_forward(self.regular, z)
        mark()
        prb = P.Rulebook(self.coords, self.spec.grid, 2, 2, False)
        mark()
        out = P.pool_forward(h, prb)
        mark()
        g = P.pool_backward(self.grad, prb)
        mark()
        g = P.gate_backward(self.regular, z, g)
        mark()
        g = P.norm_backward(L.fields_out, y, g)
        mark()
        P.backward(self.feats, g, rb, W, self.desc, self.basis, n_coeff=self.n_coeff, workspace=self.ws)
        mark()
        rb.close()
        prb.close()
        return out

    def phase_report(self):
        """Per-phase medians against HBM (norm, gate, pooling: algorithmic bytes = one read of each
        operand and one write of each result) or MFMA (the convolution GEMMs) roofline times."""
        if not self.events:
            return None
        L = self.L
        t = np.array([[a.elapsed_time(b) for a, b in zip(ev, ev[1:])] for ev in self.events])
        med = np.median(t, 0)
        n_in, n_out, P_ = int(self.coords.shape[0]), int(self.n_out), int(self.n_pairs)
        C, Cg, Cin = L.cout, self.P.n_channels(self.regular), L.cin
        hbm, peak = HBM_PEAK_GBS * 1e9, PEAK["f32"] * 1e12
        flops = 2.0 * P_ * Cin * C
        # the convolution with its Norm: the GEMM at the MFMA peak plus the Norm's elementwise pass
        # (one read of y, one write of z) at the HBM peak
        roof = {"conv_norm_forward": flops / peak + 2 * n_in * C * 4 / hbm,
                "gate_forward": (n_in * C + n_in * Cg) * 4 / hbm,
                "pool_forward": ((n_in + n_out) * Cg * 4 + 32 * n_out) / hbm,
                "pool_backward": ((n_in + n_out) * Cg * 4 + 32 * n_out) / hbm,
                "gate_backward": (2 * n_in * C + n_in * Cg) * 4 / hbm, "norm_backward": 3 * n_in * C * 4 / hbm,
                "conv_backward": 2 * flops / peak}
        out = {}
        for n, m in zip(self.NAMES, med):
            out[n] = {"ms": float(m)}
            if n in roof:
                out[n]["roofline_ms"] = roof[n] * 1e3
                out[n]["frac"] = roof[n] * 1e3 / float(m)
        step = t.sum(1)
        out["step_ms"] = {"p10": float(np.percentile(step, 10)), "median": float(np.median(step)),
                          "p90": float(np.percentile(step, 90))}
        return out

    def sites(self):
        return self.n_out

    def gather_flops(self, forward_only):
        f = 2.0 * self.n_pairs * self.L.cin * self.L.cout
        return 2 * f, 2

    def config(self):
        L = self.L
        return {"workload": self.spec.name, "grid": self.spec.grid, "batch": self.spec.batch, "ksize": L.ksize,
                "cin": L.cin, "cout": L.cout, "n_in": int(self.coords.shape[0]), "n_out": int(self.n_out),
                "pairs": int(self.n_pairs),
                "step": "synth+rulebook+conv+norm+gate+pool rulebook+pool, then pool+gate+norm+conv backward"}


class VoxelBench:
    """Input voxelisation (workload 7, Sec. 4.1): one step = ssconv_voxelize over the object
    point clouds (cells, site order, per-cell averages of (R, G, B, 1)); bandwidth-bound."""

    def __init__(self, i, dev):
        import torch
        import paper_2111_07383_amd as P
        from workloads import CONFIGS
        from workloads.gen import make_point_cloud
        self.P, self.torch = P, torch
        self.spec = CONFIGS[i]
        pts, bat, feats = make_point_cloud(self.spec)
        self.points = torch.from_numpy(pts).to(dev)
        self.batch = torch.from_numpy(bat).to(dev)
        self.feats = torch.from_numpy(feats).to(dev)
        self.events = None
        c, _, _ = self.step()
        self.n_sites = int(c.shape[0])

    def step(self):
        P, torch = self.P, self.torch
        if self.events is not None:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
        out = P.voxelize(self.points, self.feats, self.batch, self.spec.batch, (0.0, 0.0, 0.0), 1.0, self.spec.grid)
        if self.events is not None:
            e1.record()
            self.events.append((e0, e1))
        return out

    def sites(self):
        return self.n_sites

    def algorithmic_bytes(self):
        """Points (12 B), batch index (4 B) and features (4 C B) read once; site coordinates
        (16 B) and averages (4 C B) written once; the site row of every point (4 B) written."""
        n, C = int(self.points.shape[0]), int(self.feats.shape[1])
        return n * (12 + 4 + 4 * C + 4) + self.n_sites * (16 + 4 * C)

    def config(self):
        return {"workload": self.spec.name, "grid": self.spec.grid, "batch": self.spec.batch,
                "points": int(self.points.shape[0]), "channels": int(self.feats.shape[1]), "n_out": self.n_sites,
                "step": "voxelise (cells, lexicographic sites, per-cell averages); includes its one synchronisation"}


class SteerBench:
    """Feature-Steering (workload 8, Sec. 4.1): one step = ssconv_steer of the 64^3 map with 104
    channels by its seeded rigid motion (Wigner-D rotation of the fields, moved cell centres,
    re-voxelisation averaging merged sites); bandwidth-bound."""

    def __init__(self, i, dev):
        import torch
        import paper_2111_07383_amd as P
        from workloads import CONFIGS
        from workloads.gen import make_coords, make_features, make_motion
        self.P, self.torch = P, torch
        self.spec = CONFIGS[i]
        self.fields = self.spec.layers[0].fields_in
        coords = make_coords(self.spec)
        self.coords = torch.from_numpy(coords).to(dev)
        self.feats = torch.from_numpy(make_features(self.spec, len(coords), self.spec.layers[0].cin)).to(dev)
        self.R, self.t = make_motion(self.spec)
        self.events = None
        c, _, _ = self.step()
        self.n_sites = int(c.shape[0])

    def step(self):
        P, torch = self.P, self.torch
        if self.events is not None:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
        out = P.steer(self.coords, self.feats, self.fields, self.R, self.t, 1, (0.0, 0.0, 0.0), 1.0, self.spec.grid)
        if self.events is not None:
            e1.record()
            self.events.append((e0, e1))
        return out

    def sites(self):
        return self.n_sites

    def algorithmic_bytes(self):
        """Input sites (16 B) and features (4 C B) read once, output sites and averaged
        features written once, the new row of every input site (4 B) written."""
        n, C = int(self.coords.shape[0]), int(self.feats.shape[1])
        return n * (16 + 4 * C + 4) + self.n_sites * (16 + 4 * C)

    def config(self):
        return {"workload": self.spec.name, "grid": self.spec.grid, "n_in": int(self.coords.shape[0]),
                "channels": int(self.feats.shape[1]), "n_out": self.n_sites,
                "step": "steer (Wigner-D rotation, moved cell centres, re-voxelisation with averaging); "
                        "includes its one synchronisation"}


class InterpBench:
    """Tensor-to-Point (workload 9, Sec. 4.1): one step = ssconv_interpolate and
    ssconv_interpolate_backward of the 64^3 104-channel map at 4 points per site, over the map's
    rule-book hash (built once per map, outside the step)."""

    def __init__(self, i, dev):
        import torch
        import paper_2111_07383_amd as P
        from workloads import CONFIGS
        from workloads.gen import make_coords, make_features, make_query_points
        self.P, self.torch = P, torch
        self.spec = CONFIGS[i]
        coords = make_coords(self.spec)
        self.rb = P.Rulebook(torch.from_numpy(coords).to(dev), self.spec.grid, 1, 1, True)
        self.feats = torch.from_numpy(make_features(self.spec, len(coords), self.spec.layers[0].cin)).to(dev)
        pts, b = make_query_points(self.spec, coords)
        self.points = torch.from_numpy(pts).to(dev)
        self.batch = torch.from_numpy(b).to(dev)
        g = torch.Generator(dev).manual_seed(0)
        self.grad = torch.randn((len(pts), self.feats.shape[1]), device=dev, generator=g)
        self.events = None
        self.n_sites = len(pts)

    def step(self):
        P, torch = self.P, self.torch
        if self.events is not None:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
        out = P.interpolate(self.rb, self.feats, self.points, self.batch)
        P.interpolate_backward(self.rb, self.grad, self.points, self.batch)
        if self.events is not None:
            e1.record()
            self.events.append((e0, e1))
        return out

    def sites(self):
        return self.n_sites

    def algorithmic_bytes(self):
        """Forward: points (12 B) and batch (4 B) read, the 8 corner slots of the hash (8 B each),
        site features read once (n C 4 B), point features written (m C 4 B); backward: the same
        lookups, point gradients read once, site gradients written once."""
        m, C, n = int(self.points.shape[0]), int(self.feats.shape[1]), int(self.feats.shape[0])
        return 2 * (m * (16 + 64) + (n + m) * C * 4)

    def config(self):
        return {"workload": self.spec.name, "grid": self.spec.grid, "sites": int(self.feats.shape[0]),
                "points": int(self.points.shape[0]), "channels": int(self.feats.shape[1]), "n_out": self.n_sites,
                "step": "interpolate + interpolate_backward at every point (rule book of the map prebuilt)"}


# ---------------------------------------------------------------------------
# CPU oracle baseline (bounded sample of the same workload)
# ---------------------------------------------------------------------------

def cpu_model():
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    import subprocess
    try:
        txt = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in txt.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(i, budget_s):
    """The fp64 oracle on this host's cores over the first m output rows of the workload (all their
    offsets), m grown until the work fills about half the budget; timed per phase."""
    from threadpoolctl import threadpool_info
    from oracle import conv as oc
    from oracle import rulebook as orb
    from workloads import CONFIGS
    from workloads.gen import make_coeffs, make_coords, make_features, make_grad
    spec = CONFIGS[i]
    L = spec.layers[0]
    coords = make_coords(spec)
    lay = oc.Layer(L)
    w = make_coeffs(spec, [lay.n_coeff])[0]
    f = make_features(spec, len(coords), L.cin)
    t0 = time.perf_counter()
    co = orb.output_sites(coords, spec.grid, L.ksize, L.stride, L.submanifold)
    t_sites = time.perf_counter() - t0
    m = min(len(co), 256)
    while True:
        g = make_grad(spec, len(co), L.cout)[:m]
        t = [time.perf_counter()]
        R = orb.rulebook(coords, co[:m], L.ksize, L.stride)
        t.append(time.perf_counter())
        kap = lay.kappa(w, bf16=spec.dtype == "bf16")
        t.append(time.perf_counter())
        oc.forward(f, R, kap, m)
        t.append(time.perf_counter())
        oc.grad_feats(g, R, kap, len(coords))
        dk = oc.grad_kappa(f, g, R, kap.shape)
        oc.synth_adjoint(L, lay.basis, dk)
        t.append(time.perf_counter())
        ph = np.diff(t)
        ph[0] += t_sites * m / max(len(co), 1)          # the output-site pass, pro rata
        tot = float(ph.sum())
        if m == len(co) or tot >= 0.5 * budget_s:
            break
        m = int(min(len(co), max(2 * m, m * 0.8 * budget_s / max(tot, 1e-3))))
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    names = ("rulebook", "synth", "forward", "backward")
    phases = {n: {"s": float(x), "M_sites_per_s": m / float(x) / 1e6} for n, x in zip(names, ph)}
    phases["rulebook"]["threads"] = 1
    phases["synth"]["what"] = "the whole kernel (independent of the sample size)"
    phases["backward"]["what"] = "feature gradient + kernel gradient + coefficient gradient"
    return {"value": m / tot / 1e6, "unit": "M active output sites/s", "cores": int(threads), "kind": "oracle",
            "cpu_model": cpu_model(), "phases": phases,
            "sample": f"{spec.name}: first {m} of {len(co)} output rows, all offsets; rulebook (dict, 1 thread) + "
                      f"synth + forward + backward (fp64 numpy, BLAS on {threads} threads), {tot:.1f} s"}


def cpu_baseline_block(i):
    """The whole block on the oracle (Norm needs every row's statistics, so no row sample)."""
    from threadpoolctl import threadpool_info
    from oracle import conv as oc
    from oracle import norm_pool as onp
    from oracle import rulebook as orb
    from workloads import CONFIGS
    from workloads.gen import make_coeffs, make_coords, make_features, make_grad
    spec = CONFIGS[i]
    L = spec.layers[0]
    coords = make_coords(spec)
    lay = oc.Layer(L)
    w = make_coeffs(spec, [lay.n_coeff])[0]
    f = make_features(spec, len(coords), L.cin)
    regular = L.fields_out[:-1]
    t0 = time.perf_counter()
    R = orb.rulebook(coords, coords, L.ksize, 1)
    kap = lay.kappa(w)
    y = oc.forward(f, R, kap, len(coords))
    z = onp.norm_forward(y, L.fields_out)
    h = oc.gate_forward(z, regular)
    pc = onp.pool_sites(coords)
    member = onp.pool_members(coords, pc)
    onp.pool_forward(h, member, len(pc))
    g = make_grad(spec, len(pc), h.shape[1])
    g = oc.gate_backward(z, onp.pool_backward(g, member), regular)
    g = onp.norm_backward(y, g, L.fields_out)
    oc.grad_feats(g, R, kap, len(coords))
    oc.synth_adjoint(L, lay.basis, oc.grad_kappa(f, g, R, kap.shape))
    t = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": len(pc) / t / 1e6, "unit": "M active output sites/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{spec.name}: the whole block, {len(pc)} pooled sites; rule books (dict, 1 thread) + synth + "
                      f"conv + norm + gate + pool, forward and backward (fp64 numpy), {t:.1f} s"}


def step_text(spec):
    if spec.index == 9:
        return "Tensor-to-Point interpolation and its adjoint at 4 points per site of the 64^3 104-channel map"
    if spec.index == 8:
        return "Feature-Steering of the 64^3 104-channel map (Wigner-D rotation, moved centres, re-voxelisation)"
    if spec.index == 7:
        return "voxelisation of the object point clouds (cells, sites, per-cell averages)"
    if spec.index == 6:
        return ("synthesis + rule book + conv + norm + gate + pooling rule book + pooling, then pooling, gate, norm "
                "and conv backward")
    if spec.index == 5:
        return "per layer synthesis + rule book + forward (+ gate), then the backward of every layer"
    return "synthesis + rule book + forward + backward"


def cpu_baseline_voxel(i):
    from oracle import voxel as ov
    from workloads import CONFIGS
    from workloads.gen import make_point_cloud
    spec = CONFIGS[i]
    pts, bat, feats = make_point_cloud(spec)
    t0 = time.perf_counter()
    c, _, _ = ov.voxelize(pts, bat, feats, (0.0, 0.0, 0.0), 1.0, spec.grid)
    t = time.perf_counter() - t0
    return {"value": len(c) / t / 1e6, "unit": "M active output sites/s", "cores": 1, "kind": "oracle",
            "sample": f"{spec.name}: all {len(pts)} points, {len(c)} sites (numpy cells + dict averaging, "
                      f"1 thread), {t:.1f} s"}


def cpu_baseline_steer(i):
    from oracle import steer as ost
    from workloads import CONFIGS
    from workloads.gen import make_coords, make_features, make_motion
    spec = CONFIGS[i]
    coords = make_coords(spec)
    feats = make_features(spec, len(coords), spec.layers[0].cin)
    R, t = make_motion(spec)
    t0 = time.perf_counter()
    c, _, _ = ost.steer(coords, feats, spec.layers[0].fields_in, R, t, (0.0, 0.0, 0.0), 1.0, spec.grid)
    dt = time.perf_counter() - t0
    return {"value": len(c) / dt / 1e6, "unit": "M active output sites/s", "cores": 1, "kind": "oracle",
            "sample": f"{spec.name}: all {len(coords)} sites -> {len(c)} (numpy Wigner-D product, fp32 centres, "
                      f"dict averaging, 1 thread), {dt:.2f} s"}


def cpu_baseline_interp(i):
    from oracle import interp as oi
    from workloads import CONFIGS
    from workloads.gen import make_coords, make_features, make_query_points
    spec = CONFIGS[i]
    coords = make_coords(spec)
    feats = make_features(spec, len(coords), spec.layers[0].cin)
    pts, b = make_query_points(spec, coords)
    m = min(len(pts), 20000)
    g = np.random.default_rng(0).standard_normal((m, feats.shape[1]))
    t0 = time.perf_counter()
    oi.interpolate(coords, feats, pts[:m], b[:m], (0.0, 0.0, 0.0), 1.0)
    oi.interpolate_backward(coords, len(coords), pts[:m], b[:m], g, (0.0, 0.0, 0.0), 1.0)
    dt = time.perf_counter() - t0
    return {"value": m / dt / 1e6, "unit": "M active output sites/s", "cores": 1, "kind": "oracle",
            "sample": f"{spec.name}: first {m} of {len(pts)} points, forward + backward (dict corner lookups, "
                      f"1 thread), {dt:.1f} s"}


def write_stats_summary(args):
    """Tabulates a rocprofv3 --kernel-trace --stats run of this benchmark (directory
    args.stats_summary, with the benchmark's own JSON line in args.stats_log) into
    profiles/kernels_<workload>.txt, next to the gather-GEMM launch time the benchmark
    measured with its events in the same run."""
    import csv
    import glob
    import re
    from workloads import CONFIGS
    spec = CONFIGS[args.config]
    d = args.stats_summary
    stats = list(csv.DictReader(open(glob.glob(os.path.join(d, "*_kernel_stats.csv"))[0])))
    trace = list(csv.DictReader(open(glob.glob(os.path.join(d, "*_kernel_trace.csv"))[0])))
    bench = None
    for line in open(args.stats_log):
        if line.startswith("{"):
            bench = json.loads(line)

    def short(n):
        n = n.replace("(anonymous namespace)::", "").replace("void ", "").replace("ssconv::", "")
        return re.sub(r"\(.*", "", n)[:70]

    steps, warmup = (bench["steps"], bench["warmup"]) if bench else (args.steps, args.warmup)
    run = f"python3 bench.py --config {spec.index} --steps {steps} --warmup {warmup} --no-cpu-baseline --secondary 0"
    out = [f"# rocprofv3 kernel statistics: {spec.name} ({spec.dtype}), one step = {step_text(spec)}",
           f"command: rocprofv3 --kernel-trace --stats --output-format csv -d {d} -o p -- {run} > {args.stats_log}",
           f"summary: python3 bench.py --config {spec.index} --stats-summary {d} --stats-log {args.stats_log}", "",
           f"{'kernel':70s} {'calls':>6s} {'avg_us':>9s} {'min_us':>9s} {'max_us':>9s} {'pct':>6s}"]
    for r in stats[:18]:
        out.append(f"{short(r['Name']):70s} {r['Calls']:>6s} {float(r['AverageNs']) / 1e3:9.1f} "
                   f"{float(r['MinNs']) / 1e3:9.1f} {float(r['MaxNs']) / 1e3:9.1f} {float(r['Percentage']):6.1f}")
    kname = kernel_name(spec.dtype)
    g = sorted((int(t["Start_Timestamp"]), int(t["End_Timestamp"])) for t in trace if kname in t["Kernel_Name"])
    if g:
        durs = [(e - b) / 1e3 for b, e in g]
        n_timed = bench["roofline"]["launches_timed"] if bench else 0
        # the timed steps follow the warmup ones (setup launches no gather-GEMM); the phase pass,
        # if any, comes after them
        per_step = n_timed // steps if n_timed else 0
        first = per_step * warmup
        timed = durs[first:first + n_timed] if n_timed and first + n_timed <= len(durs) else durs
        out += ["", f"{kname} dispatches in launch order (us): " + " ".join(f"{x:.0f}" for x in durs),
                f"{kname} average over the {len(timed)} timed dispatches (trace; launches {first + 1}-"
                f"{first + len(timed)}): {np.mean(timed):.1f} us"]
        if bench:
            r = bench["roofline"]
            out.append(f"{kname} average launch time measured by the benchmark's HIP events in the same run: "
                       f"{r['avg_launch_ms'] * 1e3:.1f} us ({r['achieved']:.1f} {r['unit']}, "
                       f"{100 * r['frac']:.1f}% of {r['peak']})")
    if bench:
        out.append(f"step: {bench['ms_per_step']:.3f} ms ({bench['value']:.2f} {bench['unit']}) under the profiler")
    path = os.path.join(ROOT, "profiles", f"kernels_{spec.name}.txt")
    with open(path, "w") as fh:
        fh.write("\n".join(out) + "\n")
    log(f"wrote {os.path.relpath(path, ROOT)}")


def write_counter_summary(args):
    """Per-kernel HBM bandwidth and MFMA utilisation of one workload's step from rocprofv3 --pmc
    runs: fetch/ and write/ (FETCH_SIZE, WRITE_SIZE) and mfma/ (GRBM_GUI_ACTIVE,
    SQ_VALU_MFMA_BUSY_CYCLES) under args.counter_summary, copy calibration under args.copy_pmc;
    writes profiles/counters_<workload>.txt."""
    import collections
    import re
    from workloads import CONFIGS
    spec = CONFIGS[args.config]
    d, dc = args.counter_summary, args.copy_pmc or args.counter_summary
    mb = args.copy_mb or 256

    def name(r):
        n = r["Kernel_Name"].replace("(anonymous namespace)::", "").replace("void ", "").replace("ssconv::", "")
        return re.sub(r"\(.*", "", n)[:44]

    def per_kernel(rows, counter):
        vals, dur = collections.defaultdict(dict), collections.defaultdict(dict)
        for r in rows:
            if r["Counter_Name"] != counter:
                continue
            k = name(r)
            vals[k][r["Dispatch_Id"]] = vals[k].get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
            dur[k][r["Dispatch_Id"]] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        return ({k: float(np.mean(list(v.values()))) for k, v in vals.items()},
                {k: float(np.mean(list(v.values()))) for k, v in dur.items()},
                {k: len(v) for k, v in vals.items()})

    fetch, fdur, calls = per_kernel(_counter_rows(os.path.join(d, "fetch")), "FETCH_SIZE")
    write, _, _ = per_kernel(_counter_rows(os.path.join(d, "write")), "WRITE_SIZE")
    busy, mdur, _ = per_kernel(_counter_rows(os.path.join(d, "mfma")), "SQ_VALU_MFMA_BUSY_CYCLES")
    gui, _, _ = per_kernel(_counter_rows(os.path.join(d, "mfma")), "GRBM_GUI_ACTIVE")
    cf = _per_dispatch(_counter_rows(os.path.join(dc, "copy_fetch")), COPY_KERNEL, "FETCH_SIZE")
    cw = _per_dispatch(_counter_rows(os.path.join(dc, "copy_write")), COPY_KERNEL, "WRITE_SIZE")
    ff, fw = mb * 1024.0 / float(np.mean(cf)), mb * 1024.0 / float(np.mean(cw))
    run = f"python3 bench.py --config {spec.index} --steps 3 --warmup 1 --no-cpu-baseline --secondary 0"
    lines = [f"# rocprofv3 counters per kernel: {spec.name} ({spec.dtype}), one step = {step_text(spec)}",
             "commands (from the repository root, TMPDIR=/tmp, each under timeout -s KILL 120):",
             f"  rocprofv3 --pmc FETCH_SIZE --output-format csv -d {d}/fetch -o p -- {run}",
             f"  rocprofv3 --pmc WRITE_SIZE --output-format csv -d {d}/write -o p -- {run}",
             f"  rocprofv3 --pmc GRBM_GUI_ACTIVE SQ_VALU_MFMA_BUSY_CYCLES --output-format csv -d {d}/mfma -o p -- {run}",
             f"  (copy calibration as in profiles/traffic_*.txt: fetch factor {ff:.4f}, write factor {fw:.4f})",
             f"  python3 bench.py --config {spec.index} --copy-mb {mb} --counter-summary {d}"
             + (f" --copy-pmc {dc}" if dc != d else ""),
             "HBM bytes = FETCH_SIZE and WRITE_SIZE scaled by the copy calibration; GB/s over the dispatch's own",
             "duration in the counter run; MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE / 8",
             "XCDs), i.e. the share of all SIMD cycles with the matrix core busy; clock = GRBM_GUI_ACTIVE / 8 / duration",
             "(shown for launches of 100 us or more; shorter ones are dominated by launch overhead).",
             "",
             f"{'kernel':44s} {'calls':>5s} {'us':>8s} {'MB read':>9s} {'MB write':>9s} {'GB/s':>8s} {'%HBM':>6s} "
             f"{'MFMA%':>6s} {'GHz':>5s}"]
    order = sorted(fetch, key=lambda k: -fdur.get(k, 0.0) * calls.get(k, 0))
    for k in order[:16]:
        rd, wr = fetch[k] * ff * 1024, write.get(k, 0.0) * fw * 1024
        us = fdur[k] / 1e3
        gbs = (rd + wr) / max(fdur[k], 1.0)
        mf = busy.get(k, 0.0) / (1024.0 * gui[k] / 8.0) if gui.get(k) else 0.0
        ghz = gui[k] / 8.0 / mdur[k] if gui.get(k) and mdur.get(k) else 0.0
        clk = f"{ghz:5.2f}" if us >= 100 else "    -"   # GUI_ACTIVE includes launch overhead
        lines.append(f"{k:44s} {calls[k]:5d} {us:8.1f} {rd / 1e6:9.1f} {wr / 1e6:9.1f} {gbs:8.0f} "
                     f"{100 * gbs / HBM_PEAK_GBS:6.1f} {100 * mf:6.1f} {clk}")
    path = os.path.join(ROOT, "profiles", f"counters_{spec.name}.txt")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    log(f"wrote {os.path.relpath(path, ROOT)}")


def run_voxel_bench(args, dev):
    import torch
    b = {7: VoxelBench, 8: SteerBench, 9: InterpBench}[args.config](args.config, dev)
    for _ in range(args.warmup):
        b.step()
    torch.cuda.synchronize()
    b.events = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        b.step()
    torch.cuda.synchronize()
    t = time.perf_counter() - t0
    ms = t / args.steps * 1e3
    value = b.sites() / (ms / 1e3) / 1e6
    ev_ms = float(np.median([a.elapsed_time(c) for a, c in b.events]))
    achieved = b.algorithmic_bytes() / (ev_ms / 1e3) / 1e9
    out = {"metric": METRIC, "value": value, "unit": "M active output sites/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "f32", "data": "synthetic", "config": b.config(),
           "roofline": {"kernel": {7: "ssconv_voxelize", 8: "ssconv_steer",
                                   9: "ssconv_interpolate + _backward"}[args.config] + " (all their launches)",
                        "bound": "hbm", "achieved": achieved,
                        "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                        "traffic_source": "not measured", "avg_launch_ms": ev_ms,
                        "algorithmic_bytes_per_launch": b.algorithmic_bytes()}}
    log(f"{b.spec.name}: {ms:.3f} ms/step, {value:.1f} M sites/s, {achieved:.0f} GB/s algorithmic")
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = {7: cpu_baseline_voxel, 8: cpu_baseline_steer, 9: cpu_baseline_interp}[args.config](
            args.config)
    print(json.dumps(out), flush=True)


def measure(args, i, steps, warmup, dev):
    """Warm up, time `steps` whole steps of workload i between two device synchronisations, and
    return the JSON fields of that measurement (value, roofline of the gather-GEMM kernel from
    the library's launch events, per-phase report, CPU oracle baseline)."""
    import torch
    import paper_2111_07383_amd as P
    from workloads import CONFIGS
    spec = CONFIGS[i]
    log(f"setting up {spec.name}")
    b = (StackBench(dev) if i == 5 else BlockBench(i, dev) if i == 6 else SingleLayer(i, dev))
    run = b.forward_only if args.only == "forward" else b.step
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    log(f"warmup done ({warmup} steps); timing {steps} steps")
    P.debug_set(4, 1)                 # HIP events around each gather-GEMM launch, on its stream
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        run()
    torch.cuda.synchronize()
    t = time.perf_counter() - t0
    P.debug_set(4, 0)
    ms = t / steps * 1e3
    value = b.sites() / (ms / 1e3) / 1e6
    log(f"{spec.name}: {ms:.3f} ms/step, {value:.2f} M sites/s")

    out = {"metric": METRIC, "value": value, "unit": "M active output sites/s", "n_gpus": 1, "steps": steps,
           "warmup": warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": spec.dtype, "data": "synthetic", "config": b.config()}
    if args.only == "forward":
        out["metric"] = METRIC + " (forward gather-GEMM only)"
        out["config"]["step"] = "forward gather-MFMA only (rule book and kernel prebuilt)"
    n_timed, kern_ms = P.debug_kernel_ms()
    flops_step, launches_step = b.gather_flops(args.only == "forward")
    if n_timed != launches_step * steps:
        log(f"warning: {n_timed} gather-GEMM launches timed, expected {launches_step * steps}")
    avg_ms = kern_ms / max(n_timed, 1)
    flops_launch = flops_step / launches_step
    achieved = flops_step * steps / (kern_ms / 1e3) / 1e12
    traffic, tsrc = traffic_from_summary(spec)
    out["roofline"] = {"kernel": kernel_name(spec.dtype), "bound": "mfma", "achieved": achieved,
                       "peak": PEAK[spec.dtype], "unit": "TFLOP/s", "frac": achieved / PEAK[spec.dtype],
                       "traffic": traffic, "traffic_source": tsrc, "avg_launch_ms": avg_ms,
                       "launches_timed": n_timed, "algorithmic_flops_per_launch": flops_launch,
                       "kernel_ms_per_step": kern_ms / steps}
    log(f"gather-GEMM: {n_timed} launches, {avg_ms:.4f} ms avg, {achieved:.1f} TFLOP/s")
    if isinstance(b, BlockBench):
        b.events = []                 # per-phase times from extra sequential steps, after the timed ones
        for _ in range(10):
            b.phase_step()
        torch.cuda.synchronize()
    if isinstance(b, SingleLayer) and args.only == "step":
        b.events = []                 # phase boundaries (torch's stream) of as many extra steps, after the
        for _ in range(steps):        # timed ones, so the timed steps carry only the gather-launch events
            b.step()
        torch.cuda.synchronize()
    if isinstance(b, StackBench) and args.only == "step":
        out["phases"] = b.serial_report()
        ph = out["phases"]
        log(f"stack serialised: {ph['stack']['ms']:.3f} ms, roofline fraction {ph['stack']['frac']:.3f}; gather "
            f"alone {ph['gather_gemm']['avg_launch_ms']:.4f} ms avg, {ph['gather_gemm']['frac']:.3f} of peak")
    if isinstance(b, (SingleLayer, BlockBench)) and b.events:
        out["phases"] = b.phase_report()
        ph = out["phases"]
        log("phases (median ms / roofline fraction): " +
            ", ".join(f"{k} {v['ms']:.3f}/{v.get('frac', float('nan')):.2f}" for k, v in ph.items() if "ms" in v))
    if not args.no_cpu_baseline and i != 5:
        log("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = (cpu_baseline_block(i) if i == 6 else cpu_baseline(i, args.cpu_budget))
    return out


def main():
    args = parse()
    if args.counter_summary:
        write_counter_summary(args)
        return
    if args.stats_summary:
        write_stats_summary(args)
        return
    if args.traffic_summary:
        write_traffic_summary(args)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the multi-GPU sharding is a design "
              "described in DESIGN.md, not a measured path.", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.copy_mb:
        n = args.copy_mb * (1 << 20) // 4
        x = torch.ones(n, device=dev)
        y = torch.empty_like(x)
        for _ in range(max(args.steps, 1)):
            y.copy_(x)
        torch.cuda.synchronize()
        log(f"copied {args.copy_mb} MiB x {max(args.steps, 1)}")
        return
    if args.variant:
        import paper_2111_07383_amd as P
        P.debug_set(3, args.variant)
    if args.only == "forward" and args.config in (5, 6, 7, 8, 9):
        raise SystemExit("--only forward applies to the single-layer workloads 1-4")
    if args.config in (7, 8, 9):
        return run_voxel_bench(args, dev)
    out = measure(args, args.config, args.steps, args.warmup, dev)
    second = args.secondary if args.secondary >= 0 else (2 if args.config == 4 and args.only == "step" else 0)
    if second:
        # a second workload in the same line: same step, its own timed region, not part of "value"
        sec = measure(args, second, max(args.steps // 2, 5), max(args.warmup // 2, 2), dev)
        out["secondary"] = {k: sec[k] for k in ("value", "unit", "ms_per_step", "steps", "warmup", "dtype", "config",
                                                 "roofline", "phases", "cpu_baseline") if k in sec}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
