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

    python bench.py [--steps K] [--warmup W] [--config {1..5}] [--no-cpu-baseline]
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


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2, help="workload index 1..5 (default: the 64^3 5x5x5 layer)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle work to aim for")
    ap.add_argument("--only", choices=["step", "forward"], default="step",
                    help="'forward' times the forward gather-GEMM alone over one prebuilt rule book")
    ap.add_argument("--variant", type=int, default=0, help="gather-GEMM tile-configuration override (tuning)")
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="instead of the benchmark, run plain device copies of this many MiB (counter calibration)")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# GPU side
# ---------------------------------------------------------------------------

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
        self.fwd_events = []
        self.grad = torch.from_numpy(make_grad(spec, self.n_out, self.L.cout)).to(dev).to(self.dt)
        rb = P.Rulebook(self.coords, spec.grid, self.L.ksize, self.L.stride, self.L.submanifold)
        ws = P.backward_workspace_size(rb, self.dt, self.L.cin, self.L.cout)
        rb.close()
        self.ws = torch.empty((ws,), dtype=torch.uint8, device=dev)
        self.fwd_ms = []

    def forward_only(self, timed=False):
        P, torch = self.P, self.torch
        if not hasattr(self, "_rb"):
            L = self.L
            self._rb = P.Rulebook(self.coords, self.spec.grid, L.ksize, L.stride, L.submanifold)
            self._W = P.synth_kernel(self.desc, self.basis, self.coeffs, self.dt)
            self._out = torch.empty((self.n_out, L.cout), dtype=self.dt, device=self.feats.device)
        if timed:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
        P.forward(self.feats, self._rb, self._W, out=self._out)
        if timed:
            e1.record()
            self.fwd_events.append((e0, e1))

    def step(self, timed=False):
        P, torch, L = self.P, self.torch, self.L
        rb = P.Rulebook(self.coords, self.spec.grid, L.ksize, L.stride, L.submanifold)
        W = P.synth_kernel(self.desc, self.basis, self.coeffs, self.dt)
        if timed:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
        out = P.forward(self.feats, rb, W)
        if timed:
            e1.record()
            self.fwd_events.append((e0, e1))
        P.backward(self.feats, self.grad, rb, W, self.desc, self.basis, n_coeff=self.n_coeff, workspace=self.ws)
        rb.close()
        return out

    def sites(self):
        return self.n_out

    def flops(self):
        return 2.0 * self.n_pairs * self.L.cin * self.L.cout

    def config(self):
        L = self.L
        return {"workload": self.spec.name, "grid": self.spec.grid, "batch": self.spec.batch, "ksize": L.ksize,
                "stride": L.stride, "submanifold": L.submanifold, "cin": L.cin, "cout": L.cout,
                "n_in": int(self.coords.shape[0]), "n_out": int(self.n_out), "pairs": int(self.n_pairs),
                "step": "rulebook+synth+forward+backward(dfeats,dcoeffs)"}


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
        self.fwd_ms = []

    def step(self, timed=False):
        self.st.forward(self.coords, self.feats)
        self.st.backward(self.grad, need_input_grad=False)

    def sites(self):
        return sum(self.n_outs)

    def flops(self):
        return sum(2.0 * p * L.cin * L.cout for p, L in zip(self.pairs, self.spec.layers))

    def config(self):
        return {"workload": self.spec.name, "grid": self.spec.grid, "batch": self.spec.batch,
                "layers": len(self.spec.layers), "n_in": int(self.coords.shape[0]), "n_out_per_layer": self.n_outs,
                "pairs_per_layer": [int(p) for p in self.pairs],
                "step": "5 x (rulebook+synth+forward+gate) + backward"}


# ---------------------------------------------------------------------------
# CPU oracle baseline (bounded sample of the same workload)
# ---------------------------------------------------------------------------

def cpu_baseline(i, budget_s):
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
    # sample: the first m output rows, sized from a short probe to the time budget
    probe = min(len(co), 256)
    t0 = time.perf_counter()
    R = orb.rulebook(coords, co[:probe], L.ksize, L.stride)
    kap = lay.kappa(w)
    oc.forward(f, R, kap, probe)
    t_probe = time.perf_counter() - t0
    m = int(min(len(co), max(probe, probe * budget_s / max(4 * t_probe, 1e-6))))
    g = make_grad(spec, len(co), L.cout)[:m]
    t0 = time.perf_counter()
    R = orb.rulebook(coords, co[:m], L.ksize, L.stride)
    kap = lay.kappa(w)
    oc.forward(f, R, kap, m)
    oc.grad_feats(g, R, kap, len(coords))
    dk = oc.grad_kappa(f, g, R, kap.shape)
    oc.synth_adjoint(L, lay.basis, dk)
    t = time.perf_counter() - t0 + t_sites * m / max(len(co), 1)
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": m / t / 1e6, "unit": "M active output sites/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{spec.name}: first {m} of {len(co)} output rows, all offsets; rulebook (dict, 1 thread) + "
                      f"synth + forward + backward (fp64 numpy), {t:.1f} s"}


def main():
    args = parse()
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
    from workloads import CONFIGS
    spec = CONFIGS[args.config]
    if args.variant:
        import paper_2111_07383_amd as P
        P.debug_set(3, args.variant)
    log(f"setting up {spec.name}")
    b = StackBench(dev) if args.config == 5 else SingleLayer(args.config, dev)
    if args.only == "forward" and args.config == 5:
        raise SystemExit("--only forward applies to the single-layer workloads 1-4")
    run = b.forward_only if args.only == "forward" else b.step
    b.fwd_events = []
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps); timing {args.steps} steps")
    b.fwd_events = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        run(timed=True)
    torch.cuda.synchronize()
    t = time.perf_counter() - t0
    ms = t / args.steps * 1e3
    value = b.sites() / (ms / 1e3) / 1e6
    log(f"{ms:.3f} ms/step, {value:.2f} M sites/s")

    out = {"metric": METRIC, "value": value, "unit": "M active output sites/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": spec.dtype, "data": "synthetic", "config": b.config()}
    if args.only == "forward":
        out["metric"] = METRIC + " (forward gather-GEMM only)"
        out["config"]["step"] = "forward gather-MFMA only (rule book and kernel prebuilt)"
    if b.fwd_events:
        fwd_ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in b.fwd_events]))
        flops = b.flops()
        achieved = flops / (fwd_ms / 1e3) / 1e12
        out["roofline"] = {"kernel": "gather_gemm (forward)", "bound": "mfma", "achieved": achieved,
                           "peak": PEAK[spec.dtype], "unit": "TFLOP/s", "frac": achieved / PEAK[spec.dtype],
                           "traffic": None, "avg_ms": fwd_ms, "algorithmic_flops": flops}
    if not args.no_cpu_baseline and args.config != 5:
        log("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(args.config, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
