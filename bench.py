#!/usr/bin/env python3
"""Benchmark of the MoE-layer forward pass on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--gpus 1]

One step is one moe_layer_forward (route, permute, grouped routed experts,
shared expert, combine) over a seeded synthetic batch already resident in
HBM. Prints ONE JSON line: whole-layer tokens/s over the K timed steps (with
the median, p10 and p90 of the per-step times), the roofline of the dominant
kernel pair (the routed grouped GEMM, fc1 + fc2), per-stage times and
algorithmic GB/s, the ViT-L and ViT-B layers (MFMA bound), the single-image
(weight-read bound) layer, the SwiGLU-expert layers (the paper's H layer and
the single-image shape), a same-box dense bf16 GEMM reference (hipBLASLt
through torch) at the routed GEMMs' shapes, and the CPU oracle timed on a
bounded sample of the same workload.
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/s + % bf16 MFMA peak (large batch) / % HBM BW (1 image)"
PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 4096 flop/clk x 2.4 GHz, dense
PEAK_HBM_GBS = 8000.0


# HBM bytes per launch pair (fc1 + fc2) of the routed grouped GEMM, from the
# FETCH_SIZE and WRITE_SIZE hardware counters, each scaled by the factor that
# makes the same counter read the known byte count of a plain 1 GiB device
# copy (fetch x2.0, write x1.0). Taken with `bench.py --mode gemm` and
# `--mode copy` under rocprofv3 --pmc; the summary under profiles/ gives the
# commands and raw figures. The figures hold for the GEMM sources whose hash is
# TRAFFIC_SOURCE_HASH: once those change, traffic is reported as null until
# the counters are taken again.
TRAFFIC_SOURCE_HASH = "35d87b3f8476f9ac"
TRAFFIC_BYTES = {"vitg_skew_bf16": 6924223038, "vitl_bf16": 3643498711, "vitb_bf16": 779626301,
                 "single_image_bf16": 1275359648, "vith_swiglu_bf16": 6605361156,
                 "single_image_swiglu_bf16": 1879607968}


# Every source that changes the GEMM pair's HBM bytes: the kernels, the tile
# size choice and workspace plan, the tile table, and the workloads (the
# skewed layer's stored bias decides its expert loads).
TRAFFIC_SOURCES = ("paper_2608_17402_amd/csrc/gemm.hip", "paper_2608_17402_amd/csrc/moe_internal.h",
                   "paper_2608_17402_amd/csrc/moe_api.cpp", "paper_2608_17402_amd/csrc/permute.hip",
                   "workloads/configs.py", "workloads/generate.py", "tests/golden/vitg_skew_bias_seed0.txt")


# HBM bytes of one expert-MLP backward call (all its kernels), from the same
# two counters and scale factors, taken with `bench.py --mode backward`; they
# hold for the sources whose hash is BACKWARD_TRAFFIC_SOURCE_HASH (those of
# the forward pair and backward.hip).
BACKWARD_TRAFFIC_SOURCE_HASH = "10192b99fe832cc7"
BACKWARD_TRAFFIC_BYTES = {"vitg_skew_bf16": 41177098056, "vith_swiglu_bf16": 47912615423}
BACKWARD_TRAFFIC_SOURCES = TRAFFIC_SOURCES + ("paper_2608_17402_amd/csrc/backward.hip",)


def source_hash(files):
    import hashlib

    m = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            m.update(fh.read())
    return m.hexdigest()[:16]


def backward_traffic_bytes(workload):
    if source_hash(BACKWARD_TRAFFIC_SOURCES) != BACKWARD_TRAFFIC_SOURCE_HASH:
        return None
    return BACKWARD_TRAFFIC_BYTES.get(workload)


def traffic_bytes(workload):
    if source_hash(TRAFFIC_SOURCES) != TRAFFIC_SOURCE_HASH:
        return None
    return TRAFFIC_BYTES.get(workload)


def stage_bytes(c):
    """Algorithmic HBM bytes of the memory-bound stages (each tensor read or
    written once): route reads x and the router weights and writes the
    indices and gates; permute reads the indices and writes the slots (plus
    counts and offsets); combine reads the K expert-output rows, the shared
    output and the gates and writes y."""
    es = 2 if c.dtype == "bf16" else 4
    T, K, d, E = c.T, c.K, c.d, c.E
    return {
        "route": T * d * es + E * d * es + T * K * 8,
        "permute": T * K * 4 * 2 + (2 * E + 1) * 4,
        "combine": T * K * d * es + (T * d * es if c.h_shared else 0) + T * K * 4 + T * d * es,
    }


def stage_gbs(c, stages_ms):
    b = stage_bytes(c)
    return {k: round(b[k] / (stages_ms[k] * 1e-3) / 1e9, 1) for k in b if k in stages_ms}


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=1000)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--config", default="vitg_skew_bf16")
    p.add_argument("--single-image-config", default="single_image_bf16")
    p.add_argument("--no-single-image", action="store_true")
    p.add_argument("--swiglu-configs", default="vith_swiglu_bf16,single_image_swiglu_bf16",
                   help="SwiGLU-expert layers measured beside the main workload (comma-separated, '' for none)")
    p.add_argument("--mfma-configs", default="vitl_bf16,vitb_bf16",
                   help="further MFMA-bound GELU layers measured beside the main workload ('' for none)")
    p.add_argument("--no-dense-reference", action="store_true",
                   help="skip the same-box hipBLASLt dense GEMM reference")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-backward", action="store_true",
                   help="skip the expert-MLP backward (training) measurement on the main workload")
    p.add_argument("--cpu-seconds", type=float, default=15.0,
                   help="target CPU time of the oracle sample")
    p.add_argument("--stage-reps", type=int, default=10)
    p.add_argument("--mode", choices=("layer", "gemm", "stages", "backward", "dense", "copy"), default="layer",
                   help="layer: the benchmark; gemm: only the routed grouped GEMMs of --config, repeated "
                        "(hardware-counter runs); stages: route, permute and combine of --config, repeated "
                        "(hardware-counter runs); backward: the expert-MLP backward of --config, repeated "
                        "(hardware-counter runs); dense: hipBLASLt (torch) dense bf16 GEMMs of the routed "
                        "GEMMs' total shapes, repeated (hardware-counter runs); copy: a plain device copy of "
                        "--copy-mib MiB (calibration of the byte counters)")
    p.add_argument("--copy-mib", type=int, default=1024)
    return p.parse_args()


def backward_call(c, L):
    """The expert-MLP backward call on layer L's own routing, with a seeded
    output gradient, and its flop count: fc1 again (SwiGLU: two products), dA,
    dx (SwiGLU: K = 2h), dW2 and dW1 (SwiGLU: two), 2 T K d h each."""
    import torch

    from paper_2608_17402_amd import binding

    T, K, E, d, h = c.T, c.K, c.E, c.d, c.h
    L.forward()
    binding.moe_permute(L.desc, L.idx, L.counts, L.offsets, L.slots, L.ws)
    bws = binding.alloc_backward_workspace(L.desc)
    gen = torch.Generator(device="cuda").manual_seed(5)
    gout = (torch.randn(T * K, d, device="cuda", generator=gen) * 0.5).to(torch.bfloat16)
    dx = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    dw1 = torch.empty(E, L.w1.shape[1], d, dtype=torch.float32, device="cuda")
    dw2 = torch.empty(E, d, L.w2.shape[2], dtype=torch.float32, device="cuda")

    def bwd():
        binding.moe_grouped_mlp_backward(L.desc, L.x, L.slots, L.offsets, L.w1, L.w2, gout, dx, dw1, dw2, bws)

    fl = (8.0 if c.act == "swiglu" else 5.0) * 2.0 * T * K * d * h
    return bwd, fl


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this MoE-layer build runs on one GPU only; the layer shards by tokens "
                                   "(data parallel) or by experts, neither of which is built here",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_17402_amd import binding
    from workloads import get_config, make_inputs, pad_last_dim

    torch.cuda.set_device(0)
    binding.load()

    def dev(a):
        if a is None:
            return None
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
        return torch.from_numpy(a).cuda()

    class Layer:
        def __init__(self, cfg):
            self.cfg = cfg
            t0 = time.perf_counter()
            inp = make_inputs(cfg)
            self.inp = inp
            swiglu = cfg.act == "swiglu"
            flags = binding.MOE_FLAG_SWIGLU if swiglu else 0
            self.desc = binding.make_desc(cfg.T, cfg.d, cfg.E, cfg.K, cfg.h, cfg.h_shared, cfg.lam, cfg.dtype,
                                          flags=flags)
            self.dt = binding.torch_dtype(self.desc)
            self.x, self.wr, self.b = dev(inp.x), dev(inp.w_router), dev(inp.bias)
            # SwiGLU: stacked gate/up rows as drawn; second layer with rows padded to 64 columns.
            pad = pad_last_dim if swiglu else (lambda a: a)
            self.w1, self.w2, self.w1s, self.w2s = dev(inp.w1), dev(pad(inp.w2)), dev(inp.w1s), dev(pad(inp.w2s))
            self.ws = binding.alloc_workspace(self.desc)
            T, K, E, d = cfg.T, cfg.K, cfg.E, cfg.d
            self.y = torch.empty(T, d, dtype=self.dt, device="cuda")
            self.idx = torch.empty(T, K, dtype=torch.int32, device="cuda")
            self.gate = torch.empty(T, K, dtype=torch.float32, device="cuda")
            self.counts = torch.empty(E, dtype=torch.int32, device="cuda")
            self.b_scratch = torch.zeros(E, dtype=torch.float32, device="cuda")
            self.offsets = torch.empty(E + 1, dtype=torch.int32, device="cuda")
            self.slots = torch.empty(T * K, dtype=torch.int32, device="cuda")
            self.eout = torch.empty(T * K, d, dtype=self.dt, device="cuda")
            self.shared = torch.empty(T, d, dtype=self.dt, device="cuda") if cfg.h_shared else None
            torch.cuda.synchronize()
            self.setup_s = time.perf_counter() - t0

        def forward(self, events=None):
            binding.moe_layer_forward(self.desc, self.x, self.wr, self.b, self.w1, self.w2, self.w1s, self.w2s,
                                      self.y, self.idx, self.gate, self.ws, events=events)

        def stages(self):
            """Stage entry points, in layer order (for per-stage timing)."""
            return {
                "route": lambda: binding.moe_route(self.desc, self.x, self.wr, self.b, self.idx, self.gate,
                                                   self.ws),
                "permute": lambda: binding.moe_permute(self.desc, self.idx, self.counts, self.offsets, self.slots,
                                                       self.ws),
                "grouped_mlp": lambda: binding.moe_grouped_mlp(self.desc, self.x, self.slots, self.offsets,
                                                               self.w1, self.w2, self.eout, self.ws),
                "combine": lambda: binding.moe_combine(self.desc, self.eout, self.gate, self.shared, self.y),
                # The balancing update (z-score rule) on a scratch copy of the bias.
                "bias_update": lambda: binding.moe_bias_update(self.desc, self.counts, self.b_scratch, 1e-3,
                                                               binding.MOE_BIAS_ZSCORE),
            }

    def time_calls(fn, reps):
        """Average ms per call, HIP events on the stream the kernels run on."""
        s = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        fn()
        torch.cuda.synchronize()
        e0.record(s)
        for _ in range(reps):
            fn()
        e1.record(s)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    def split_fc1_fc2(L, reps):
        """Average fc1 and fc2 times (ms) from a pass with all three of
        moe_layer_forward's events (the middle one's queue gap included)."""
        ev = binding.HipEvents(3 * reps)
        for i in range(reps):
            L.forward(ev.handles[3 * i:3 * i + 3])
        torch.cuda.synchronize()
        f1 = sum(ev.elapsed_ms(3 * i, 3 * i + 1) for i in range(reps)) / reps
        f2 = sum(ev.elapsed_ms(3 * i + 1, 3 * i + 2) for i in range(reps)) / reps
        ev.close()
        return f1, f2

    if args.mode == "copy":
        n = args.copy_mib << 20
        a = torch.ones(n // 2, dtype=torch.bfloat16, device="cuda")
        b = torch.empty_like(a)
        for _ in range(args.warmup):
            b.copy_(a)
        ms = time_calls(lambda: b.copy_(a), args.steps)
        print(json.dumps({"mode": "copy", "bytes_read_per_launch": n, "bytes_written_per_launch": n,
                          "avg_us": round(ms * 1e3, 2), "gbs": round(2 * n / (ms * 1e-3) / 1e9, 1)}), flush=True)
        return

    cfg = get_config(args.config)
    if args.mode == "dense":
        # fc1 [T K, d] x [d, h] and fc2 [T K, h] x [h, d], weights in the [out, in] layout.
        M = cfg.T * cfg.K
        g = torch.Generator(device="cuda").manual_seed(3)
        a1 = torch.randn(M, cfg.d, device="cuda", generator=g).to(torch.bfloat16)
        w1 = torch.randn(cfg.h, cfg.d, device="cuda", generator=g).to(torch.bfloat16)
        a2 = torch.randn(M, cfg.h, device="cuda", generator=g).to(torch.bfloat16)
        w2 = torch.randn(cfg.d, cfg.h, device="cuda", generator=g).to(torch.bfloat16)
        for _ in range(args.warmup + args.steps):
            torch.nn.functional.linear(a1, w1)
            torch.nn.functional.linear(a2, w2)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "dense", "workload": cfg.name, "shapes": [[M, cfg.d, cfg.h], [M, cfg.h, cfg.d]],
                          "launch_pairs": args.warmup + args.steps}), flush=True)
        return
    lay = Layer(cfg)

    if args.mode == "stages":
        # The non-GEMM stages, each repeated, for the byte counters: route,
        # permute and the separate combine kernel (on the layer's own routing).
        st = lay.stages()
        lay.forward()
        for name in ("route", "permute", "combine"):
            for _ in range(args.steps):
                st[name]()
        torch.cuda.synchronize()
        print(json.dumps({"mode": "stages", "workload": cfg.name, "launches_per_stage": args.steps}), flush=True)
        return

    if args.mode == "backward":
        # The expert-MLP backward alone, repeated, for the counter passes.
        bwd, _ = backward_call(cfg, lay)
        for _ in range(args.warmup + args.steps):
            bwd()
        torch.cuda.synchronize()
        print(json.dumps({"mode": "backward", "workload": cfg.name, "calls": args.warmup + args.steps}),
              flush=True)
        return

    if args.mode == "gemm":
        st = lay.stages()
        st["route"]()
        st["permute"]()
        for _ in range(args.warmup):
            st["grouped_mlp"]()
        ms = time_calls(st["grouped_mlp"], args.steps)
        print(json.dumps({"mode": "gemm", "workload": cfg.name, "launch_pairs": args.steps + 1 + args.warmup,
                          "avg_pair_us": round(ms * 1e3, 2)}), flush=True)
        return

    for _ in range(args.warmup):
        lay.forward()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    hev = binding.HipEvents(3 * args.steps)
    # One event between consecutive steps (per-step times for the median and
    # percentiles); the first and the last bracket the timed region.
    sev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    wall0 = time.perf_counter()
    sev[0].record(stream)
    for i in range(args.steps):
        # The events right before fc1 and right after fc2 (no event between
        # them, whose queue gap would count in the pair's time).
        h = hev.handles[3 * i:3 * i + 3]
        lay.forward([h[0], None, h[2]])
        sev[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = sev[0].elapsed_time(sev[-1]) / args.steps
    step_ms = np.array([sev[i].elapsed_time(sev[i + 1]) for i in range(args.steps)])
    value = cfg.T / (ms * 1e-3)
    gemm_ms = sum(hev.elapsed_ms(3 * i, 3 * i + 2) for i in range(args.steps)) / args.steps
    hev.close()
    # The fc1 / fc2 split, from a pass with the middle event as well.
    fc1_ms, fc2_ms = split_fc1_fc2(lay, min(args.steps, 100))

    # Per-stage times (the stage entry points run the same kernels).
    stages_ms = {k: time_calls(f, args.stage_reps) for k, f in lay.stages().items()}
    routed_flops = 2.0 * cfg.n_mats * cfg.T * cfg.K * cfg.d * cfg.h
    achieved = routed_flops / (gemm_ms * 1e-3) / 1e12
    roofline = {
        "kernel": "routed grouped GEMM: the fc1+GELU and fc2 kernels of one layer step",
        "bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
        "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic_bytes(cfg.name),
        "algorithmic_flops_per_launch": routed_flops, "avg_launch_us": round(gemm_ms * 1e3, 2),
        "fc1_us": round(fc1_ms * 1e3, 2), "fc2_us": round(fc2_ms * 1e3, 2),
        "timing": "HIP events recorded by moe_layer_forward on its stream right before fc1 and right after fc2, "
                  "every timed step; fc1_us / fc2_us from a further pass with an event between them as well",
    }
    layer_flops = cfg.gemm_flops()

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": cfg.name, "tokens": cfg.T, "images": cfg.images,
                   "tokens_per_image": cfg.tokens_per_image, "d_model": cfg.d, "experts": cfg.E, "top_k": cfg.K,
                   "expert_hidden": cfg.h, "shared_hidden": cfg.h_shared, "bias": cfg.bias},
        "us_per_layer": round(ms * 1e3, 1),
        "step_us": {"median": round(float(np.median(step_ms)) * 1e3, 1),
                    "p10": round(float(np.percentile(step_ms, 10)) * 1e3, 1),
                    "p90": round(float(np.percentile(step_ms, 90)) * 1e3, 1),
                    "min": round(float(step_ms.min()) * 1e3, 1), "max": round(float(step_ms.max()) * 1e3, 1)},
        "layer_gemm_tflops": round(layer_flops / (ms * 1e-3) / 1e12, 2),
        "layer_gemm_frac_of_bf16_peak": round(layer_flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "roofline": roofline,
        "stages_us": {k: round(v * 1e3, 1) for k, v in stages_ms.items()},
        "stages_gbs": stage_gbs(cfg, stages_ms),
        "timed_wall_s": round(wall, 3),
    }

    def measure(c, reps):
        """Whole-layer time of layer config c, then (a second pass of the same
        length) the routed grouped GEMM pair from the HIP events that
        moe_layer_forward records around fc1 and fc2. Each recorded event
        leaves a gap of several microseconds in the queue, which would inflate
        the layer time of these short layers, so the first pass records none."""
        L = Layer(c)
        for _ in range(3):
            L.forward()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            L.forward()
        e1.record(stream)
        torch.cuda.synchronize()
        l_ms = e0.elapsed_time(e1) / reps
        ev = binding.HipEvents(3 * reps)
        for i in range(reps):
            h = ev.handles[3 * i:3 * i + 3]
            L.forward([h[0], None, h[2]])
        torch.cuda.synchronize()
        pair = sum(ev.elapsed_ms(3 * i, 3 * i + 2) for i in range(reps)) / reps
        ev.close()
        f1, f2 = split_fc1_fc2(L, reps)
        return L, l_ms, pair, f1, f2

    def dense_reference(c, routed_tflops):
        """Same-box context for the routed grouped GEMM: hipBLASLt (through
        torch) bf16 GEMMs of the same total shape, fc1 [T K, d] x [d, h] and
        fc2 [T K, h] x [h, d] as single dense products, and as a batch of E
        equal expert blocks of T K / E rows (torch.bmm with contiguous
        operands); a square 8192^3 product (a long contraction); and the GB/s
        of a 1 GiB device copy, the context of the HBM-bound stages. Random
        operands; weights in the [out, in] layout."""
        M, d, h, E = c.T * c.K, c.d, c.h, c.E
        g = torch.Generator(device="cuda").manual_seed(3)

        def rnd(*shape):
            return torch.randn(*shape, device="cuda", generator=g).to(torch.bfloat16)

        res = {}
        a1, w1 = rnd(M, d), rnd(h, d)
        a2, w2 = rnd(M, h), rnd(d, h)
        fl = 2.0 * M * d * h
        reps = 10
        t1 = time_calls(lambda: torch.nn.functional.linear(a1, w1), reps)
        t2 = time_calls(lambda: torch.nn.functional.linear(a2, w2), reps)
        del a1, a2
        m = M // E
        b1, wb1 = rnd(E, m, d), rnd(E, d, h)
        b2, wb2 = rnd(E, m, h), rnd(E, h, d)
        fb = 2.0 * E * m * d * h
        t3 = time_calls(lambda: torch.bmm(b1, wb1), reps)
        t4 = time_calls(lambda: torch.bmm(b2, wb2), reps)
        del b1, b2, wb1, wb2
        # A long contraction (8192^3): what the library reaches on this machine
        # when the K loop is long against the tile's start-up and epilogue.
        q, wq = rnd(8192, 8192), rnd(8192, 8192)
        fq = 2.0 * 8192 ** 3
        t5 = time_calls(lambda: torch.nn.functional.linear(q, wq), reps)
        del q, wq
        # A plain device copy of 1 GiB: the HBM bandwidth a streaming kernel reaches here.
        ca = torch.empty(1 << 29, dtype=torch.bfloat16, device="cuda").fill_(1)
        cb = torch.empty_like(ca)
        tc = time_calls(lambda: cb.copy_(ca), reps)
        del ca, cb

        def tf(f, t):
            return round(f / (t * 1e-3) / 1e12, 1)

        pair = tf(2 * fl, t1 + t2)
        res = {
            "library": "hipBLASLt via torch (bf16 in, fp32 accumulate, bf16 out)",
            "dense_fc1": {"shape": [M, d, h], "us": round(t1 * 1e3, 1), "tflops": tf(fl, t1)},
            "dense_fc2": {"shape": [M, h, d], "us": round(t2 * 1e3, 1), "tflops": tf(fl, t2)},
            "dense_pair_tflops": pair, "dense_pair_frac": round(pair / PEAK_BF16_TFLOPS, 4),
            "batched_fc1": {"shape": [E, m, d, h], "us": round(t3 * 1e3, 1), "tflops": tf(fb, t3)},
            "batched_fc2": {"shape": [E, m, h, d], "us": round(t4 * 1e3, 1), "tflops": tf(fb, t4)},
            "batched_pair_tflops": tf(2 * fb, t3 + t4),
            "routed_pair_over_dense_pair": round(routed_tflops / pair, 4),
            "square_8192": {"shape": [8192, 8192, 8192], "us": round(t5 * 1e3, 1), "tflops": tf(fq, t5),
                            "frac": round(tf(fq, t5) / PEAK_BF16_TFLOPS, 4)},
            "copy_gbs": round(2 * (1 << 30) / (tc * 1e-3) / 1e9, 1),
        }
        return res

    def backward_line(c, L):
        """Expert-MLP backward on layer L's own routing: five products of
        2 T K d h (SwiGLU: the gate/up products count twice) flop."""
        bwd, fl = backward_call(c, L)
        for _ in range(2):
            bwd()
        b_ms = time_calls(bwd, max(3, min(args.steps // 2, 10)))
        tf = fl / (b_ms * 1e-3) / 1e12
        return {
            "workload": c.name, "act": c.act, "entry": "moe_grouped_mlp_backward", "us": round(b_ms * 1e3, 1),
            "tokens_per_s": round(c.T / (b_ms * 1e-3), 1),
            "roofline": {"kernel": "expert-MLP backward: fc1 again, dA, dx, dW2, dW1 products plus transposes",
                         "bound": "mfma", "achieved": round(tf, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(tf / PEAK_BF16_TFLOPS, 4), "traffic": backward_traffic_bytes(c.name),
                         "algorithmic_flops_per_launch": fl, "avg_launch_us": round(b_ms * 1e3, 2)},
        }

    def hbm_line(c, L, l_ms, g_ms, f1, f2):
        w_bytes = c.routed_weight_bytes()
        gbs = w_bytes / (g_ms * 1e-3) / 1e9
        return {
            "workload": c.name, "tokens": c.T, "act": c.act, "us_per_layer": round(l_ms * 1e3, 1),
            "tokens_per_s": round(c.T / (l_ms * 1e-3), 1),
            "roofline": {"kernel": "routed grouped GEMM (fc1+fc2), expert weights read once", "bound": "hbm",
                         "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": traffic_bytes(c.name),
                         "algorithmic_bytes_per_launch": w_bytes,
                         "avg_launch_us": round(g_ms * 1e3, 2),
                         "fc1_us": round(f1 * 1e3, 2), "fc2_us": round(f2 * 1e3, 2)},
            "layer_weight_gbs": round((w_bytes + c.shared_weight_bytes()) / (l_ms * 1e-3) / 1e9, 1),
        }

    def mfma_line(c, l_ms, pair, f1, f2):
        fl = 2.0 * c.n_mats * c.T * c.K * c.d * c.h
        tf = fl / (pair * 1e-3) / 1e12
        return {
            "workload": c.name, "tokens": c.T, "act": c.act, "us_per_layer": round(l_ms * 1e3, 1),
            "tokens_per_s": round(c.T / (l_ms * 1e-3), 1),
            "layer_gemm_tflops": round(c.gemm_flops() / (l_ms * 1e-3) / 1e12, 2),
            "roofline": {"kernel": "routed grouped GEMM (fc1 with its activation, fc2)", "bound": "mfma",
                         "achieved": round(tf, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(tf / PEAK_BF16_TFLOPS, 4), "traffic": traffic_bytes(c.name),
                         "algorithmic_flops_per_launch": fl, "avg_launch_us": round(pair * 1e3, 2),
                         "fc1_us": round(f1 * 1e3, 2), "fc2_us": round(f2 * 1e3, 2)},
        }

    if not args.no_dense_reference and cfg.dtype == "bf16":
        out["dense_reference"] = dense_reference(cfg, achieved)

    # The lines beside the main workload: 20 to 50 timed layers each.
    sec_reps = min(max(args.steps, 20), 50)
    mf_names = [n for n in args.mfma_configs.split(",") if n]
    if mf_names:
        out["mfma_layers"] = {}
        for name in mf_names:
            c = get_config(name)
            L, l_ms, pair, f1, f2 = measure(c, sec_reps)
            line = mfma_line(c, l_ms, pair, f1, f2)
            st_ms = {k: time_calls(f, args.stage_reps) for k, f in L.stages().items()}
            line["stages_us"] = {k: round(v * 1e3, 1) for k, v in st_ms.items()}
            line["stages_gbs"] = stage_gbs(c, st_ms)
            out["mfma_layers"][name] = line
            del L

    if not args.no_single_image:
        c5 = get_config(args.single_image_config)
        reps = sec_reps
        si, si_ms, pair, f1, f2 = measure(c5, reps)
        si_stages = {k: time_calls(f, max(args.stage_reps, 20)) for k, f in si.stages().items()}
        out["single_image"] = hbm_line(c5, si, si_ms, pair, f1, f2)
        out["single_image"]["stages_us"] = {k: round(v * 1e3, 1) for k, v in si_stages.items()}
        del si

    if not args.no_backward and cfg.dtype == "bf16":
        out["backward"] = backward_line(cfg, lay)

    sw_names = [n for n in args.swiglu_configs.split(",") if n]
    if sw_names:
        out["swiglu"] = {}
        for name in sw_names:
            c = get_config(name)
            L, l_ms, pair, f1, f2 = measure(c, sec_reps)
            # ~32 rows per expert is weight-read bound; large batches are MFMA bound.
            weight_bound = c.T * c.K / c.E < 256
            out["swiglu"][name] = (hbm_line(c, L, l_ms, pair, f1, f2) if weight_bound
                                   else mfma_line(c, l_ms, pair, f1, f2))
            if not weight_bound and not args.no_backward:
                out["swiglu"][name]["backward"] = backward_line(c, L)
            del L

    if not args.no_cpu_baseline:
        import oracle

        inp = lay.inp
        f = {k: inp.f32(k) for k in ("x", "w_router", "w1", "w2", "w1s", "w2s")}
        bf16 = cfg.dtype == "bf16"

        def run(n):
            t0 = time.perf_counter()
            oracle.layer(f["x"][:n], f["w_router"], inp.bias, f["w1"], f["w2"], f["w1s"], f["w2s"], cfg.K,
                         cfg.lam, bf16)
            return time.perf_counter() - t0

        n0 = 64
        t_probe = run(n0)
        n = int(min(cfg.T, max(n0, n0 * args.cpu_seconds / max(t_probe, 1e-6))))
        t = run(n)
        cpu_model = platform.processor()
        try:
            with open("/proc/cpuinfo") as fh:
                for line in fh:
                    if line.startswith("model name"):
                        cpu_model = line.split(":", 1)[1].strip()
                        break
        except OSError:
            pass
        out["cpu_baseline"] = {
            "value": round(n / t, 2), "unit": "tokens/s", "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"first {n} of {cfg.T} tokens of {cfg.name}: full layer per token (route, {cfg.K} experts, "
                      f"shared expert, combine), fp64 plain loops, {t:.1f} s",
            "cpu_model": cpu_model, "os_cpu_count": os.cpu_count(),
        }

    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
