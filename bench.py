"""Benchmark: fused 8-bit Adam step on the 1.5B-parameter LM-shaped list.

One step = one run of the fused 8-bit optimizer step over every tensor of the
list (prepare both codebooks' decision tables, then dequantize states, fp32
Adam update, block absmax, requantize), with the params, fp16 grads and 8-bit
states already resident in HBM.  By default the step goes through a step plan
(bq_step_plan_run: one launch over all 580 tensors); --path call uses
bq_optimizer8bit_step.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]

Prints one JSON line.  The CPU baseline is the oracle (plain C, OpenMP over
blocks) timed on a bounded sample of the same workload on the host cores.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "8-bit Adam step params/sec and achieved HBM GB/s (% of peak), 1.5B-param list"
HBM_PEAK_GBS = 8000.0
BLOCKSIZE = 2048

# HBM traffic of one step-kernel launch on this workload, from two rocprofv3
# --pmc runs of `bench.py --steps 3 --warmup 1 --no-cpu-baseline` (FETCH_SIZE,
# then WRITE_SIZE, KiB per dispatch), FETCH_SIZE scaled by 2.0 and WRITE_SIZE by
# 1.0: the factors that make the counters of a plain fp32->fp16 copy of known
# size read its true bytes on MI355X (profiles/step_kernel_adam_f16_b2048_lm1p5b_pmc.md).
# Valid only for the kernel sources it was taken on (sha256 below); otherwise
# the bench reports traffic null.
KERNEL_SOURCES = ["bq_oneshot.hip", "bq_device.h", "bq_internal.h"]
MEASURED_TRAFFIC = {
    "sources_sha256": "83c016a5516dcfb38bec291f30062715ae7f0aea0c8f1cfe57774de4ae422fcf",
    "fetch_kib": 6132450.0, "write_kib": 9150410.0, "fetch_scale": 2.0, "write_scale": 1.0,
}


def step_bytes(numels, blocksize, grad_bytes, nstates):
    """Algorithmic HBM bytes of one step: fp32 param read + write, grad read,
    per state one code read + write, per block and state fp32 absmax read + write."""
    n = sum(numels)
    nblocks = sum((k + blocksize - 1) // blocksize for k in numels)
    return n * (8 + grad_bytes + 2 * nstates) + nblocks * nstates * 8


def kernel_sources_sha256():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2110_02861_amd", "csrc")
    for name in KERNEL_SOURCES:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """Counter-measured HBM bytes per step-kernel launch, or None when the
    kernel sources differ from the ones the counters were taken on."""
    m = MEASURED_TRAFFIC
    if m["sources_sha256"] is None or m["sources_sha256"] != kernel_sources_sha256():
        return None
    return m["fetch_kib"] * 1024 * m["fetch_scale"] + m["write_kib"] * 1024 * m["write_scale"]


def stream_ceiling(torch, nparams, steps=20):
    """Same-byte-mix streaming rate on flat random buffers of the same size:
    loads and stores of the step's bytes with no arithmetic (libbq_stream.so),
    best of its launch-shape variants.  Returns (best GB/s, {variant: GB/s}),
    algorithmic bytes as in step_bytes()."""
    from paper_2110_02861_amd import build as pkg_build
    if not os.path.exists(pkg_build.STREAM_LIB):
        raise RuntimeError(f"{pkg_build.STREAM_LIB} is not built")
    L = ctypes.CDLL(pkg_build.STREAM_LIB)
    P = ctypes.c_void_p
    L.bq_stream_ceiling.argtypes = [ctypes.c_int] + [P] * 6 + [ctypes.c_int64, ctypes.c_int32,
                                                               ctypes.c_uint32, P, P]
    L.bq_stream_ceiling.restype = ctypes.c_int
    L.bq_stream_variants.restype = ctypes.c_int
    n = (nparams + 4095) // 4096 * 4096
    nb = n // BLOCKSIZE
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(12345)
    w = torch.empty(n, dtype=torch.float32, device=dev).normal_(0, 0.02, generator=gen)
    g = torch.empty(n, dtype=torch.float16, device=dev).normal_(0, 1e-4, generator=gen)
    c1 = torch.randint(0, 256, (n,), dtype=torch.uint8, device=dev, generator=gen)
    c2 = torch.randint(0, 256, (n,), dtype=torch.uint8, device=dev, generator=gen)
    a1 = torch.rand(nb, device=dev, generator=gen)
    a2 = torch.rand(nb, device=dev, generator=gen)
    table = torch.randint(0, 2**31 - 1, (4096,), dtype=torch.int32, device=dev, generator=gen)
    stream = torch.cuda.current_stream()
    bufs = [P(t.data_ptr()) for t in (w, g, c1, c2, a1, a2)]
    per = {}
    for v in range(L.bq_stream_variants()):
        args = [v] + bufs + [n, BLOCKSIZE, 0, P(table.data_ptr()), P(stream.cuda_stream)]
        for _ in range(3):
            if L.bq_stream_ceiling(*args) != 0:
                raise RuntimeError("bq_stream_ceiling failed")
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            L.bq_stream_ceiling(*args)
        e1.record(stream)
        torch.cuda.synchronize()
        sec = e0.elapsed_time(e1) / steps / 1e3
        per[v] = step_bytes([n], BLOCKSIZE, 2, 2) / sec / 1e9
    del w, g, c1, c2, a1, a2, table
    torch.cuda.empty_cache()
    return max(per.values()), per


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def setup_c5(torch, bq, workloads, seed=0):
    specs = workloads.lm_1p5b_specs()
    dev = torch.device("cuda:0")
    B = BLOCKSIZE
    params, grads, states = [], [[], []], []
    for i, s in enumerate(specs):
        n = s.numel
        nb = (n + B - 1) // B
        w = torch.empty(n, dtype=torch.float32, device=dev)
        workloads.init_param_device(s, w, seed, "c5", i)
        params.append(w)
        for r in range(2):
            g = torch.empty(n, dtype=torch.float16, device=dev)
            workloads.grad_device("c5", s, g, seed, i, r)
            grads[r].append(g)
        states.append((torch.full((n,), 127, dtype=torch.uint8, device=dev),
                       torch.zeros(n, dtype=torch.uint8, device=dev),
                       torch.zeros(nb, dtype=torch.float32, device=dev),
                       torch.zeros(nb, dtype=torch.float32, device=dev)))
    torch.cuda.synchronize()
    rows = [[(params[i], grads[r][i], states[i][0], states[i][1], states[i][2], states[i][3])
             for i in range(len(specs))] for r in range(2)]
    return specs, params, grads, states, rows


def cpu_baseline(specs, params, grads, layers, steps=4):
    """Time the oracle on the first `layers` transformer layers of the list
    (initial params, the first grad buffer, zero state): one warm-up step and
    `steps` timed steps on all host cores."""
    import oracle
    from paper_2110_02861_amd import workloads
    names = [f"h.{i}." for i in range(layers)]
    idx = [i for i, s in enumerate(specs) if any(s.name.startswith(p) for p in names)]
    qs = oracle.dynamic_codebook(0)
    qu = oracle.dynamic_codebook(1)
    hp = workloads.C5
    host = []
    for i in idx:
        w = params[i].cpu().numpy().copy()
        g = grads[0][i].cpu().numpy().copy()
        n = w.size
        nb = (n + BLOCKSIZE - 1) // BLOCKSIZE
        host.append([w, g, np.full(n, 127, np.uint8), np.zeros(nb, np.float32),
                     np.zeros(n, np.uint8), np.zeros(nb, np.float32)])
    cores = len(os.sched_getaffinity(0))
    n_sample = sum(h[0].size for h in host)

    def one(t):
        for w, g, c1, a1, c2, a2 in host:
            oracle.step8(oracle.ADAM, BLOCKSIZE, w, g, c1, a1, qs, c2, a2, qu, hp["lr"],
                         hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], t, nthreads=cores)

    one(1)
    t0 = time.perf_counter()
    for t in range(2, 2 + steps):
        one(t)
    dt = time.perf_counter() - t0
    return {
        "value": steps * n_sample / dt, "unit": "params/s", "cores": cores, "kind": "oracle",
        "sample": f"first {layers} transformer layers of the 1.5B list ({len(idx)} tensors, "
                  f"{n_sample} params), zero state, 1 warm-up + {steps} timed steps, "
                  f"OpenMP over blocks",
        "seconds": dt,
        "gbs": steps * step_bytes([h[0].size for h in host], BLOCKSIZE, 2, 2) / dt / 1e9,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-stream-ceiling", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=16)
    ap.add_argument("--path", choices=["plan", "call"], default="plan",
                    help="plan: bq_step_plan_run (one launch over all 580 tensors); "
                         "call: bq_optimizer8bit_step (descriptor chunks of 56 tensors)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the 8-bit step has no cross-GPU exchange, and "
              "this build runs on a single MI355X (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2110_02861_amd import bq, workloads

    torch.cuda.set_device(0)
    qs_d = torch.from_numpy(bq.bq_make_dynamic_codebook(bq.BQ_SIGNED)).cuda()
    qu_d = torch.from_numpy(bq.bq_make_dynamic_codebook(bq.BQ_UNSIGNED)).cuda()
    log("allocating the 1.5B-parameter list")
    specs, params, grads, states, rows = setup_c5(torch, bq, workloads)
    numels = [s.numel for s in specs]
    nparams = sum(numels)
    bytes_step = step_bytes(numels, BLOCKSIZE, 2, 2)
    hp = {k: workloads.C5[k] for k in ("lr", "beta1", "beta2", "eps", "wd")}

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline(specs, params, grads, args.cpu_layers)
        log(f"cpu baseline {cpu['value'] / 1e6:.1f} Mparam/s on {cpu['cores']} threads")

    ceiling = None
    if not args.no_stream_ceiling:
        log("measuring the same-byte-mix streaming ceiling")
        ceiling, ceiling_per = stream_ceiling(torch, nparams)
        log(f"stream ceiling {ceiling:.0f} GB/s (variants {ceiling_per})")

    stream = torch.cuda.current_stream()

    # a ring of two gradient buffers, one plan (or descriptor array) for each
    if args.path == "plan":
        plans = [bq.StepPlan(bq.BQ_ADAM, BLOCKSIZE, bq.BQ_F16, r) for r in rows]

        def step(t):
            plans[t % 2].run(dict(hp, step=t), qs_d, qu_d, stream=stream)
    else:
        arrays = [(bq.make_tensor_array(r), len(r)) for r in rows]

        def step(t):
            bq.bq_optimizer8bit_step(bq.BQ_ADAM, BLOCKSIZE, bq.BQ_F16, arrays[t % 2],
                                     dict(hp, step=t), qs_d, qu_d, stream=stream)

    log(f"warmup {args.warmup} steps")
    t = 1
    for _ in range(args.warmup):
        step(t)
        t += 1
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    log(f"timing {args.steps} steps")
    start.record(stream)
    for _ in range(args.steps):
        step(t)
        t += 1
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    sec = ms / 1e3
    gbs = bytes_step / sec / 1e9
    res = {
        "metric": METRIC,
        "value": nparams / sec,
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded torch Philox on the GPU; shapes of a 48-layer GPT-2-style LM)",
        "config": {
            "workload": "8-bit Adam, 1.5B-param LM-shaped list: 48 layers, d=1600, ffn 6400, "
                        "vocab 50257, ctx 1024; fp32 params N(0,0.02), fp16 grads N(0,1e-4) "
                        "with 0.01% outliers x1000, blocksize 2048",
            "tensors": len(specs), "params": nparams, "blocksize": BLOCKSIZE,
            "grad_dtype": "fp16", "state_dtype": "u8", "path": args.path,
        },
        "gbs": gbs,
        "hbm_frac": gbs / HBM_PEAK_GBS,
        "roofline": {
            "bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": gbs / HBM_PEAK_GBS, "traffic": measured_traffic(),
            "bytes_per_step": bytes_step,
            "kernel": "step_oneshot_kernel<Adam, fp16 grad, 2048> (+ prepare_kernel, ~10 us, "
                      "inside the timed launch pair)",
        },
        "stream_ceiling": None if ceiling is None else {
            "gbs": ceiling, "frac_of_peak": ceiling / HBM_PEAK_GBS,
            "step_frac_of_ceiling": gbs / ceiling,
            "per_variant": ceiling_per,
            "kind": "same byte mix, flat random buffers, no arithmetic, best of the launch "
                    "shapes in libbq_stream.so",
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
