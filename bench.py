"""Benchmark: fused 8-bit Adam step on the 1.5B-parameter LM-shaped list.

One step = one run of the fused 8-bit optimizer step over every tensor of the
list (prepare both codebooks' decision tables, then dequantize states, fp32
Adam update, block absmax, requantize), with the params, fp16 grads and 8-bit
states already resident in HBM.  By default the step goes through a step plan
(bq_step_plan_run: one launch over all 580 tensors); --path call uses
bq_optimizer8bit_step, --path optim the drop-in torch optimizer.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
                    [--workload lm1p5b-adam|gpt2m-adamw|resnet50-momentum|
                                quantize|dequantize|stream-study] [--blocksize B]

Prints one JSON line.  The CPU baseline is the oracle (plain C, OpenMP over
blocks) timed on a bounded sample of the same workload on the host cores.
The other workloads are secondary measurements of the same kernels: the
8-bit AdamW step on the GPT-2-medium list (fp16 grads), the 8-bit Momentum
step on the ResNet-50 list (fp32 grads), and standalone block-wise quantize /
dequantize of 67,108,864 Student-t values over four rotating buffers.
--workload stream-study times the step's byte mix (and its reads and writes
alone) under every launch shape, cache policy, tile order and occupancy of
libbq_stream.so's access-shape study, beside the step itself.
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

# HBM traffic of the dominant kernel per step (summed over its launches in one
# step: 11 for the call path on the 1.5B list, else 1), from two rocprofv3 --pmc
# runs of the bench command (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch),
# FETCH_SIZE scaled by 2.0 and WRITE_SIZE by 1.0: the factors that make the
# counters of kernels of known traffic (a plain fp32->fp16 copy, the
# same-byte-mix stream) read their true bytes on MI355X.  Valid only for the
# kernel sources the counters were taken on (sha256 below); otherwise the
# bench reports traffic null.  Keys: (workload, blocksize, path).
KERNEL_SOURCES = ["bq_oneshot.hip", "bq_device.h", "bq_internal.h", "bq_scalars.h"]
TRAFFIC_SOURCES_SHA256 = "40268921eca199e3ddefaddae5526de97b1e52cf37091f460c9e91e6bbf98db6"
FETCH_SCALE, WRITE_SCALE = 2.0, 1.0
MEASURED_TRAFFIC = {
    ("lm1p5b-adam", 2048, "plan"): {"fetch_kib": 6132950.734, "write_kib": 9150410.344},
    ("lm1p5b-adam", 2048, "static"): {"fetch_kib": 6109054.891, "write_kib": 9150410.578},
    # 11 launches per step: the mean per dispatch times 11
    ("lm1p5b-adam", 2048, "call"): {"fetch_kib": 11 * 555761.575, "write_kib": 11 * 831891.200},
    ("gpt2m-adamw", 2048, "plan"): {"fetch_kib": 1397257.109, "write_kib": 2084463.539},
    # the plan and prepared paths run the same step kernel on the same list
    ("resnet50-momentum", 2048, "prepared"): {"fetch_kib": 113032.703, "write_kib": 124988.266},
    ("resnet50-momentum", 2048, "plan"): {"fetch_kib": 113032.703, "write_kib": 124988.266},
    ("quantize", 2048, "plan"): {"fetch_kib": 131141.926, "write_kib": 65792.0},
    ("quantize", 2048, "call"): {"fetch_kib": 131174.500, "write_kib": 65792.0},
    ("dequantize", 2048, "call"): {"fetch_kib": 33812.742, "write_kib": 262144.0},
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


def measured_traffic(workload, blocksize, path):
    """Counter-measured HBM bytes per launch of the workload's dominant kernel,
    or None when none were taken for it or the kernel sources differ from the
    ones the counters were taken on."""
    m = MEASURED_TRAFFIC.get((workload, blocksize, path))
    if m is None or TRAFFIC_SOURCES_SHA256 != kernel_sources_sha256():
        return None
    return m["fetch_kib"] * 1024 * FETCH_SCALE + m["write_kib"] * 1024 * WRITE_SCALE


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


STUDY_MODES = {0: "mix", 1: "reads", 2: "writes"}


def run_stream_study(args, torch, bq, workloads):
    """The access-shape study of libbq_stream.so (bq_stream_study): every
    variant at the hardware's occupancy and at 2, 3 and 4 workgroups per CU,
    over buffers of the 1.5B list's size, with the fused step itself (plan,
    maps prepared once) on that list as one more case; `rounds` interleaved
    rounds of 3 launches per case, median and best GB/s of algorithmic bytes
    (mix 14 B per element + 16 B per block, reads 8 + 8, writes 6 + 8)."""
    from paper_2110_02861_amd import build as pkg_build
    L = ctypes.CDLL(pkg_build.STREAM_LIB)
    P = ctypes.c_void_p
    L.bq_stream_study_variants.restype = ctypes.c_int
    L.bq_stream_study_info.restype = ctypes.c_char_p
    L.bq_stream_study_info.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_int)]
    L.bq_stream_study.restype = ctypes.c_int
    L.bq_stream_study.argtypes = [ctypes.c_int, ctypes.POINTER(P), ctypes.POINTER(P),
                                  ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, P, ctypes.c_int,
                                  P]
    log("allocating the lm1p5b-adam list and the study buffers")
    specs, params, grads, states, rows = setup_c5(torch, bq, workloads)
    nparams = sum(p.numel() for p in params)
    n = nparams // 8192 * 8192
    nb = n // BLOCKSIZE
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(12345)

    def bufs():
        return [torch.empty(n, dtype=torch.float32, device=dev).normal_(0, 0.02, generator=gen),
                torch.empty(n, dtype=torch.float16, device=dev).normal_(0, 1e-4, generator=gen),
                torch.randint(0, 256, (n,), dtype=torch.uint8, device=dev, generator=gen),
                torch.randint(0, 256, (n,), dtype=torch.uint8, device=dev, generator=gen),
                torch.rand(nb, device=dev, generator=gen), torch.rand(nb, device=dev, generator=gen)]
    bi, bo = bufs(), bufs()
    pin = (P * 6)(*[t.data_ptr() for t in bi])
    pout = (P * 6)(*[t.data_ptr() for t in bo])
    table = torch.randint(0, 2**31 - 1, (880 * 4,), dtype=torch.int32, device=dev, generator=gen)
    stream = torch.cuda.current_stream()
    mode_bytes = {0: 14 * n + 16 * nb, 1: 8 * n + 8 * nb, 2: 6 * n + 8 * nb}
    cases = []
    for v in range(L.bq_stream_study_variants()):
        info = (ctypes.c_int * 3)()
        name = L.bq_stream_study_info(v, info).decode()
        for per_cu in (0, 2, 3, 4):
            cases.append(dict(v=v, name=name, threads=info[0], chunks=info[1],
                              mode=STUDY_MODES[info[2]], per_cu=per_cu,
                              bytes=mode_bytes[info[2]]))

    qs = torch.from_numpy(bq.bq_make_dynamic_codebook(bq.BQ_SIGNED)).to(dev)
    qu = torch.from_numpy(bq.bq_make_dynamic_codebook(bq.BQ_UNSIGNED)).to(dev)
    prepared = bq.prepare_codebook_pair(qs, qu, stream=stream)
    plans = [bq.StepPlan(bq.BQ_ADAM, BLOCKSIZE, bq.BQ_F16, r) for r in rows]
    hp = {k: workloads.C5[k] for k in ("lr", "beta1", "beta2", "eps", "wd")}
    t = [1]
    cases.append(dict(v=-1, name="the fused step (plan, maps prepared once), lm1p5b-adam list",
                      threads=512, chunks=2, mode="step", per_cu=0,
                      bytes=step_bytes([p.numel() for p in params], BLOCKSIZE, 2, 2)))

    def launch(c):
        if c["v"] < 0:
            plans[t[0] % 2].run_prepared(dict(hp, step=t[0]), prepared, stream=stream)
            t[0] += 1
            return 0
        return L.bq_stream_study(c["v"], pin, pout, n, BLOCKSIZE, 0, P(table.data_ptr()),
                                 c["per_cu"], P(stream.cuda_stream))

    live = []
    for c in cases:
        rc = launch(c)
        if rc == 0:
            live.append(c)
        elif rc != -1:
            raise RuntimeError(f"bq_stream_study variant {c['v']} per_cu {c['per_cu']}: {rc}")
    torch.cuda.synchronize()
    log(f"{len(live)} cases, {args.rounds} rounds")
    times = [[] for _ in live]
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    for r in range(args.rounds):
        for i, c in enumerate(live):
            e0.record(stream)
            for _ in range(3):
                launch(c)
            e1.record(stream)
            e1.synchronize()
            times[i].append(e0.elapsed_time(e1) / 3)
        log(f"round {r} done")
    out = []
    for c, ts in zip(live, times):
        ts = sorted(ts)
        med = ts[len(ts) // 2]
        out.append(dict(c, ms_median=med, gbs_median=c["bytes"] / med / 1e6,
                        gbs_best=c["bytes"] / ts[0] / 1e6))
        log(f"{c['name']:48s} per CU {c['per_cu'] or 'hw'}: {out[-1]['gbs_median']:7.0f} GB/s "
            f"(best {out[-1]['gbs_best']:7.0f})")
    mix = [o for o in out if o["mode"] == "mix"]
    best = max(mix, key=lambda o: o["gbs_median"])
    step = [o for o in out if o["mode"] == "step"][0]
    return {"metric": "access-shape study of the fused step's byte mix: algorithmic GB/s per "
                      "launch shape (median of interleaved rounds)",
            "value": best["gbs_median"], "unit": "GB/s", "n_gpus": 1, "rounds": args.rounds,
            "higher_is_better": True, "data": "synthetic (seeded torch Philox on the GPU)",
            "config": {"workload": f"flat buffers of {n} elements (the 1.5B list's size, "
                                   f"rounded down to 8192), blocksize {BLOCKSIZE}"},
            "best_mix": {k: best[k] for k in ("name", "per_cu", "gbs_median", "gbs_best")},
            "step_gbs_median": step["gbs_median"],
            "step_frac_of_best_mix": step["gbs_median"] / best["gbs_median"],
            "peak_gbs": HBM_PEAK_GBS, "cases": out}


def setup_list(torch, bq, workloads, config, nstates, blocksize=BLOCKSIZE, seed=0, zero1=127):
    """Params, a ring of two grad buffers and zero 8-bit states for one of the
    parameter lists, generated on the GPU (zero1: the code of 0 in state 1's
    map).  Returns (specs, params, grads, states, rows) with rows[r] the
    bq_tensor tuples that use grad buffer r."""
    specs = workloads.SPECS[config]()
    gdt = getattr(torch, workloads.GRADS[config][0])
    dev = torch.device("cuda:0")
    B = blocksize
    params, grads, states = [], [[], []], []
    for i, s in enumerate(specs):
        n = s.numel
        nb = (n + B - 1) // B
        w = torch.empty(n, dtype=torch.float32, device=dev)
        workloads.init_param_device(s, w, seed, config, i)
        params.append(w)
        for r in range(2):
            g = torch.empty(n, dtype=gdt, device=dev)
            workloads.grad_device(config, s, g, seed, i, r)
            grads[r].append(g)
        if nstates == 2:
            states.append((torch.full((n,), zero1, dtype=torch.uint8, device=dev),
                           torch.zeros(n, dtype=torch.uint8, device=dev),
                           torch.zeros(nb, dtype=torch.float32, device=dev),
                           torch.zeros(nb, dtype=torch.float32, device=dev)))
        else:
            states.append((torch.full((n,), zero1, dtype=torch.uint8, device=dev), None,
                           torch.zeros(nb, dtype=torch.float32, device=dev), None))
    torch.cuda.synchronize()
    rows = [[(params[i], grads[r][i], states[i][0], states[i][1], states[i][2], states[i][3])
             for i in range(len(specs))] for r in range(2)]
    return specs, params, grads, states, rows


def setup_c5(torch, bq, workloads, seed=0):
    return setup_list(torch, bq, workloads, "c5", 2, BLOCKSIZE, seed)


def cpu_model():
    """The host CPU's model name (first processor in /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(specs, params, grads, layers, steps=6):
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
        "cpu_model": cpu_model(), "per_core": steps * n_sample / dt / cores,
        "sample": f"first {layers} transformer layers of the 1.5B list ({len(idx)} tensors, "
                  f"{n_sample} params), zero state, 1 warm-up + {steps} timed steps, "
                  f"OpenMP over blocks",
        "seconds": dt,
        "gbs": steps * step_bytes([h[0].size for h in host], BLOCKSIZE, 2, 2) / dt / 1e9,
    }


_LM = ("1.5B-param LM-shaped list: 48 layers, d=1600, ffn 6400, vocab 50257, ctx 1024; fp32 params "
       "N(0,0.02), fp16 grads N(0,1e-4) with 0.01% outliers x1000")
LIST_WORKLOADS = {
    # name: config, optimizer, description, hyperparameters (None: the config's own),
    # extra bytes of the per-tensor norm pass besides the grad it reads again
    # (per param, per block and state)
    "lm1p5b-adam": dict(config="c5", opt="adam", desc="8-bit Adam, " + _LM, hp=None,
                        norms=(0, 0)),
    "lm1p5b-adam-bf16": dict(config="c5bf16", opt="adam", norms=(0, 0), hp=None,
                             desc="8-bit Adam, " + _LM.replace("fp16 grads", "bf16 grads")),
    "gpt2m-adamw": dict(config="c4", opt="adamw", hp=None, norms=(0, 0),
                        desc="8-bit AdamW, GPT-2-medium-shaped list: 24 layers, d=1024, ffn 4096, "
                             "vocab 50257, ctx 1024; fp32 params N(0,0.02), fp16 grads N(0,1e-4), "
                             "heavy-tailed embedding rows"),
    "resnet50-momentum": dict(config="c3", opt="momentum", hp=None, norms=(0, 0),
                              desc="8-bit Momentum, ResNet-50 v1.5 parameter list (161 tensors); "
                                   "conv/fc N(0, sqrt(2/fan_in)), BN 1/0, fp32 grads N(0,1e-3)"),
    "lm1p5b-adagrad": dict(config="c5", opt="adagrad", desc="8-bit AdaGrad, " + _LM,
                           hp=dict(lr=1e-2, beta1=0.0, beta2=0.0, eps=1e-10, wd=0.0),
                           norms=(0, 0)),
    # LAMB reads w, g and both states again for the norms of w and of the update
    "lm1p5b-lamb": dict(config="c5", opt="lamb", desc="8-bit LAMB, " + _LM,
                        hp=dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6, wd=0.01),
                        norms=(6, 4)),
    # LARS reads w and g again for their norms
    "lm1p5b-lars": dict(config="c5", opt="lars", desc="8-bit LARS, " + _LM,
                        hp=dict(lr=0.1, beta1=0.9, beta2=0.0, eps=0.0, wd=1e-4, trust=1e-3),
                        norms=(4, 0)),
}
# The setup of the paper's optimizer-runtime table (App. E): one sample of 10^9
# normal values with fp32 gradients; reported as ms per update per 10^9 params
# beside the table's number for the paper's 8-bit kernel on a V100 (context, not
# a target: other hardware, and the paper's batch of 100 updates).
_P1B = "one tensor of 10^9 N(0,1) fp32 params, fp32 grads N(0,1)"
PAPER_TABLE_MS = {"adam": 47.0, "momentum": 34.0, "lamb": 65.0, "lars": 43.0}
for _opt, _hp, _norms in (
        ("adam", dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0), (0, 0)),
        ("momentum", dict(lr=0.1, beta1=0.9, beta2=0.0, eps=0.0, wd=0.0), (0, 0)),
        ("lamb", dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6, wd=0.01), (6, 4)),
        ("lars", dict(lr=0.1, beta1=0.9, beta2=0.0, eps=0.0, wd=1e-4, trust=1e-3), (4, 0))):
    LIST_WORKLOADS["paper1b-" + _opt] = dict(config="p1b", opt=_opt, hp=_hp, norms=_norms,
                                             desc=f"8-bit {_opt}, " + _P1B)


def run_cpu_oracle(args):
    """The oracle on one host thread: C1 (8-bit Adam, one 1,048,576-element
    tensor, 10 steps from the zero state), C2 (block-wise quantize and
    dequantize of 67,108,864 Student-t values, B = 2048) and C3 (8-bit Momentum
    on the ResNet-50 list, 2 steps), all inputs from the host generators.  A
    per-core reference for the GPU figures; no GPU is used."""
    import oracle
    from paper_2110_02861_amd import workloads
    qs, qu = oracle.dynamic_codebook(0), oracle.dynamic_codebook(1)
    B = BLOCKSIZE

    def run_steps(config, opt, steps):
        specs = workloads.SPECS[config]()
        hp = getattr(workloads, config.upper())
        two = opt in (oracle.ADAM, oracle.ADAMW)
        st = []
        for i, sp in enumerate(specs):
            w = workloads.init_param_host(sp, workloads.host_rng(0, config, i, 0))
            nb = (sp.numel + B - 1) // B
            st.append([w, np.full(sp.numel, 127, np.uint8), np.zeros(nb, np.float32),
                       np.zeros(sp.numel, np.uint8) if two else None,
                       np.zeros(nb, np.float32) if two else None])
        grads = [[workloads.grad_host(config, sp, workloads.host_rng(0, config, i, t))
                  for i, sp in enumerate(specs)] for t in range(1, steps + 1)]
        t0 = time.perf_counter()
        for t in range(1, steps + 1):
            for (w, c1, a1, c2, a2), g in zip(st, grads[t - 1]):
                oracle.step8(opt, B, w, g, c1, a1, qs, c2, a2, qu, hp["lr"], hp["beta1"],
                             hp["beta2"], hp["eps"], hp["wd"], t, nthreads=1)
        dt = time.perf_counter() - t0
        n = sum(sp.numel for sp in specs)
        return n, steps, dt, [sp.numel for sp in specs]

    log("C1 on one thread")
    n1, k1, d1, e1 = run_steps("c1", oracle.ADAM, 10)
    log("C3 on one thread")
    n3, k3, d3, e3 = run_steps("c3", oracle.MOMENTUM, 2)
    log("C2 on one thread")
    x = workloads.student_t_host(QUANT_N, seed=0)
    t0 = time.perf_counter()
    codes, absmax = oracle.quantize_blockwise(qs, x, B, nthreads=1)
    dq = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.dequantize_blockwise(qs, codes, absmax, B, nthreads=1)
    dd = time.perf_counter() - t0
    qbytes = QUANT_N * 5 + (QUANT_N + B - 1) // B * 4
    c1 = {"params_per_s": n1 * k1 / d1, "gbs": k1 * step_bytes(e1, B, 2, 2) / d1 / 1e9,
          "seconds": d1, "steps": k1}
    c3 = {"params_per_s": n3 * k3 / d3, "gbs": k3 * step_bytes(e3, B, 4, 1) / d3 / 1e9,
          "seconds": d3, "steps": k3}
    c2 = {"quantize_elements_per_s": QUANT_N / dq, "quantize_gbs": qbytes / dq / 1e9,
          "dequantize_elements_per_s": QUANT_N / dd, "dequantize_gbs": qbytes / dd / 1e9,
          "seconds": dq + dd}
    return {
        "metric": "oracle (plain C, one host thread) 8-bit Adam step params/sec on C1",
        "value": c1["params_per_s"], "unit": "params/s", "n_gpus": 0, "steps": k1, "warmup": 0,
        "ms_per_step": d1 / k1 * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic (seeded numpy PCG64 on the host)",
        "config": {"workload": "the CPU oracle on one thread: C1 (8-bit Adam, 1,048,576 params, "
                               "10 steps), C2 (quantize + dequantize, 67,108,864 Student-t "
                               "values, B 2048), C3 (8-bit Momentum, ResNet-50 list, 2 steps)",
                   "threads": 1, "cpu_model": cpu_model()},
        "c1_adam": c1, "c2_quantize": c2, "c3_momentum": c3,
    }


def workload_bytes(name, numels, blocksize, grad_bytes):
    """Algorithmic HBM bytes of one step of a list workload: the fused step's
    bytes plus, for LAMB and LARS, the norm pass's reads (the grad again, and
    the listed extra bytes)."""
    W = LIST_WORKLOADS[name]
    nstates = 2 if W["opt"] in ("adam", "adamw", "lamb") else 1
    nblocks = sum((k + blocksize - 1) // blocksize for k in numels)
    norm_pass = W["opt"] in ("lamb", "lars")
    per_param = W["norms"][0] + (grad_bytes if norm_pass else 0)
    return (step_bytes(numels, blocksize, grad_bytes, nstates) + sum(numels) * per_param
            + nblocks * W["norms"][1] * nstates)


QUANT_N = 67_108_864
QUANT_BUFFERS = 4


def timed(torch, stream, fn, steps, warmup, per_event):
    """Run fn(i) warmup times, then `steps` times with a HIP event on `stream`
    every `per_event` calls.  Returns (ms per call over the whole timed region,
    sorted per-call ms of each event segment)."""
    for i in range(warmup):
        fn(i)
    # every event is created before the timed region: creating one inside it
    # is a host call that can stall the enqueue of a short step
    nev = 1 + (steps + per_event - 1) // per_event
    pool = [torch.cuda.Event(enable_timing=True) for _ in range(nev)]
    torch.cuda.synchronize()
    evs = [pool[0]]
    evs[0].record(stream)
    for i in range(steps):
        fn(warmup + i)
        if (i + 1) % per_event == 0 or i + 1 == steps:
            e = pool[len(evs)]
            e.record(stream)
            evs.append(e)
    torch.cuda.synchronize()
    total = evs[0].elapsed_time(evs[-1]) / steps
    seg = []
    done = 0
    for a, b in zip(evs[:-1], evs[1:]):
        k = min(per_event, steps - done)
        done += k
        seg.append(a.elapsed_time(b) / k)
    return total, sorted(seg)


def base_record(args, metric, value, unit, ms, seg, dtype, data, config):
    return {
        "metric": metric, "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": dtype, "data": data, "config": config,
        "ms_per_step_median": seg[len(seg) // 2], "ms_per_step_min": seg[0],
    }


def run_list(args, torch, bq, workloads):
    W = LIST_WORKLOADS[args.workload]
    config, opt_name, desc = W["config"], W["opt"], W["desc"]
    headline = args.workload == "lm1p5b-adam"
    B = args.blocksize
    opt = bq.OPTIMIZERS[opt_name]
    nstates = 2 if opt_name in ("adam", "adamw", "lamb") else 1
    gdt_name = workloads.GRADS[config][0]
    gdt = {"float16": bq.BQ_F16, "bfloat16": bq.BQ_BF16, "float32": bq.BQ_F32}[gdt_name]
    gname = {"float16": "fp16", "bfloat16": "bf16", "float32": "fp32"}[gdt_name]
    torch.cuda.set_device(0)
    qs_d = torch.from_numpy(bq.bq_make_dynamic_codebook(bq.BQ_SIGNED)).cuda()
    qu_d = torch.from_numpy(bq.bq_make_dynamic_codebook(bq.BQ_UNSIGNED)).cuda()
    # AdaGrad's one state (a sum of squares) lives on the unsigned map
    q1 = qu_d if opt_name == "adagrad" else qs_d
    zero1 = 0 if opt_name == "adagrad" else 127
    log(f"allocating the {args.workload} list")
    specs, params, grads, states, rows = setup_list(torch, bq, workloads, config, nstates, B,
                                                    zero1=zero1)
    numels = [s.numel for s in specs]
    nparams = sum(numels)
    bytes_step = workload_bytes(args.workload, numels, B, 4 if gdt == bq.BQ_F32 else 2)
    if W["hp"]:
        hp = dict(W["hp"])
    else:
        C = getattr(workloads, config.upper())
        hp = {k: C[k] for k in ("lr", "beta1", "beta2", "eps", "wd")}

    cpu = None
    if headline and not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline(specs, params, grads, args.cpu_layers)
        log(f"cpu baseline {cpu['value'] / 1e6:.1f} Mparam/s on {cpu['cores']} threads")

    ceiling = None
    if headline and not args.no_stream_ceiling:
        log("measuring the same-byte-mix streaming ceiling")
        ceiling, ceiling_per = stream_ceiling(torch, nparams)
        log(f"stream ceiling {ceiling:.0f} GB/s (variants {ceiling_per})")

    stream = torch.cuda.current_stream()
    q2 = qu_d if nstates == 2 else None
    if args.path in ("call", "static") and opt_name in ("lamb", "lars"):
        print("LAMB and LARS run through step plans only (--path plan or optim)",
              file=sys.stderr)
        sys.exit(2)

    # a ring of two gradient buffers, one plan (or descriptor array) for each
    if args.path in ("optim", "optim-graph"):
        from paper_2110_02861_amd import optim
        del states, rows
        torch.cuda.empty_cache()
        ps = [torch.nn.Parameter(w) for w in params]
        for p in ps:
            p.grad_dtype = None  # fp16 grads on fp32 params
        cap = dict(capturable=args.path == "optim-graph")
        if opt_name == "momentum":
            opt_obj = optim.SGD8bit(ps, lr=hp["lr"], momentum=hp["beta1"],
                                    weight_decay=hp["wd"], blocksize=B, **cap)
        elif opt_name == "adagrad":
            opt_obj = optim.Adagrad8bit(ps, lr=hp["lr"], eps=hp["eps"], weight_decay=hp["wd"],
                                        blocksize=B, **cap)
        elif opt_name == "lars":
            opt_obj = optim.Lars8bit(ps, lr=hp["lr"], momentum=hp["beta1"],
                                     weight_decay=hp["wd"], trust_coefficient=hp["trust"],
                                     blocksize=B, **cap)
        else:
            cls = {"adam": optim.Adam8bit, "adamw": optim.AdamW8bit,
                   "lamb": optim.Lamb8bit}[opt_name]
            opt_obj = cls(ps, lr=hp["lr"], betas=(hp["beta1"], hp["beta2"]), eps=hp["eps"],
                          weight_decay=hp["wd"], blocksize=B, **cap)

        def step(i):
            for p, g in zip(ps, grads[i % 2]):
                p.grad = g
            opt_obj.step()

        if args.path == "optim-graph":
            # one eager step per grad buffer creates the states and both plans;
            # then step() is captured once per buffer and replayed
            step(0)
            step(1)
            graphs = []
            for r in (0, 1):
                for p, g in zip(ps, grads[r]):
                    p.grad = g
                graph = torch.cuda.CUDAGraph()
                with torch.cuda.graph(graph):
                    opt_obj.step()
                graphs.append(graph)
            torch.cuda.synchronize()

            def step(i):  # noqa: F811
                graphs[i % 2].replay()
    elif args.path == "plan":
        plans = [bq.StepPlan(opt, B, gdt, r) for r in rows]

        def step(i):
            plans[i % 2].run(dict(hp, step=i + 1), q1, q2, stream=stream)
    elif args.path == "prepared":
        plans = [bq.StepPlan(opt, B, gdt, r) for r in rows]
        prepared = bq.prepare_codebook_pair(q1, q2, stream=stream)

        def step(i):
            plans[i % 2].run_prepared(dict(hp, step=i + 1), prepared, stream=stream)
    elif args.path == "device":
        plans = [bq.StepPlan(opt, B, gdt, r) for r in rows]
        prepared = bq.prepare_codebook_pair(q1, q2, stream=stream)
        hp_dev = bq.device_hparams(dict(hp, step=0))

        def step(i):
            plans[i % 2].run_device(hp_dev, prepared, advance=True, stream=stream)
    elif args.path == "static":
        arrays = [(bq.make_tensor_array(r), len(r)) for r in rows]

        def step(i):
            bq.bq_optimizer8bit_step_static(opt, B, gdt, arrays[i % 2], dict(hp, step=i + 1),
                                            q1, q2, stream=stream)
    else:
        arrays = [(bq.make_tensor_array(r), len(r)) for r in rows]

        def step(i):
            bq.bq_optimizer8bit_step(opt, B, gdt, arrays[i % 2], dict(hp, step=i + 1), q1,
                                     q2, stream=stream)

    log(f"warmup {args.warmup} steps, timing {args.steps} steps")
    ms, seg = timed(torch, stream, step, args.steps, args.warmup, 1)
    gbs = bytes_step / (ms / 1e3) / 1e9
    tag = {"adam": "Adam", "adamw": "AdamW", "momentum": "Momentum", "adagrad": "AdaGrad",
           "lamb": "LAMB", "lars": "LARS"}[opt_name]
    paper_ms = PAPER_TABLE_MS.get(opt_name) if config == "p1b" else None
    metric = METRIC if headline else (
        f"8-bit {tag} step params/sec and achieved HBM GB/s (% of peak), {args.workload} list")
    res = base_record(
        args, metric, nparams / (ms / 1e3), "params/s", ms, seg, "f32",
        f"synthetic (seeded torch Philox on the GPU; shapes of the {args.workload} list)",
        {"workload": f"{desc}, blocksize {B}", "tensors": len(specs), "params": nparams,
         "blocksize": B, "grad_dtype": gname,
         "state_dtype": "u8", "path": args.path})
    kname = {"call": f"step_persistent_kernel<{tag}, {gname} grad, {B}> (call path)",
             "static": f"step_static_kernel<{tag}, {gname} grad, {B}> (+ prepare_kernel and "
                       f"{-(-len(specs) // 56)} descriptor uploads)"}.get(
        args.path, f"step_oneshot_kernel<{tag}, {gname} grad, {B}>")
    if opt_name in ("lamb", "lars"):
        kname += " (+ norms_kernel and trust_ratio_kernel: the per-tensor norm pass)"
    if args.path == "optim":
        kname += f" via optim.{type(opt_obj).__name__}.step()"
    if args.path == "optim-graph":
        kname += (f" via optim.{type(opt_obj).__name__}(capturable=True).step() captured in a "
                  "HIP graph (+ scalars_kernel)")
    res.update({
        "gbs": gbs,
        "hbm_frac": gbs / HBM_PEAK_GBS,
        "roofline": {
            "bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": gbs / HBM_PEAK_GBS,
            "traffic": measured_traffic(args.workload, B, args.path),
            "bytes_per_step": bytes_step,
            "kernel": kname + {"plan": " (+ prepare_kernel, ~6 us, inside the timed launch pair)",
                               "device": " (+ scalars_kernel: the step's scalars from device "
                                         "hyperparameters)"}.get(args.path, ""),
        },
        "stream_ceiling": None if ceiling is None else {
            "gbs": ceiling, "frac_of_peak": ceiling / HBM_PEAK_GBS,
            "step_frac_of_ceiling": gbs / ceiling,
            "per_variant": ceiling_per,
            "kind": "same byte mix, flat random buffers, no arithmetic, best of the launch "
                    "shapes in libbq_stream.so",
        },
        "cpu_baseline": cpu,
    })
    if paper_ms is not None:
        res["ms_per_update_per_1e9_params"] = ms * 1e9 / nparams
        res["paper_table_ms_per_update_per_1e9_params_v100"] = paper_ms
    return res


def run_quant(args, torch, bq, workloads):
    """Standalone quantize or dequantize of 67,108,864 Student-t(3) x 1e-2
    values; four input / output buffer sets rotate so that no call finds its
    operands in the 256 MB last-level cache."""
    if args.path in ("optim", "optim-graph", "prepared", "device", "static"):
        print(f"--path {args.path} applies to the optimizer-step workloads (the quantize plan "
              "path already reads a codebook prepared once)", file=sys.stderr)
        sys.exit(2)
    B = args.blocksize
    n = QUANT_N
    nb = (n + B - 1) // B
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    qs_d = torch.from_numpy(bq.bq_make_dynamic_codebook(bq.BQ_SIGNED)).cuda()
    prepared = bq.bq_prepare_codebook(qs_d)
    log("generating the Student-t input on the host")
    x_h = torch.from_numpy(workloads.student_t_host(n, seed=0))
    xs = [x_h.to(dev) for _ in range(QUANT_BUFFERS)]
    codes = [torch.empty(n, dtype=torch.uint8, device=dev) for _ in range(QUANT_BUFFERS)]
    absmax = [torch.empty(nb, dtype=torch.float32, device=dev) for _ in range(QUANT_BUFFERS)]
    outs = [torch.empty(n, dtype=torch.float32, device=dev) for _ in range(QUANT_BUFFERS)]
    stream = torch.cuda.current_stream()
    for k in range(QUANT_BUFFERS):
        bq.bq_quantize_blockwise_prepared(prepared, xs[k], B, codes[k], absmax[k], stream=stream)
    torch.cuda.synchronize()
    L = bq.lib()
    path = args.path if args.workload == "quantize" else "call"
    if args.workload == "quantize":
        if args.path == "plan":
            pp = prepared.data_ptr()
            args_k = [(pp, xs[k].data_ptr(), n, B, codes[k].data_ptr(), absmax[k].data_ptr(),
                       stream.cuda_stream) for k in range(QUANT_BUFFERS)]

            def call(i):
                if L.bq_quantize_blockwise_prepared(*args_k[i % QUANT_BUFFERS]) != 0:
                    raise RuntimeError("bq_quantize_blockwise_prepared failed")
            kname = f"quantize_oneshot_kernel<{B}> (prepared codebook)"
        else:
            qp = qs_d.data_ptr()
            args_k = [(qp, xs[k].data_ptr(), n, B, codes[k].data_ptr(), absmax[k].data_ptr(),
                       stream.cuda_stream) for k in range(QUANT_BUFFERS)]

            def call(i):
                if L.bq_quantize_blockwise(*args_k[i % QUANT_BUFFERS]) != 0:
                    raise RuntimeError("bq_quantize_blockwise failed")
            kname = f"quantize_kernel<{B}> (persistent, raw codebook)"
        what = "block-wise quantize"
    else:
        qp = qs_d.data_ptr()
        args_k = [(qp, codes[k].data_ptr(), absmax[k].data_ptr(), n, B, outs[k].data_ptr(),
                   stream.cuda_stream) for k in range(QUANT_BUFFERS)]

        def call(i):
            if L.bq_dequantize_blockwise(*args_k[i % QUANT_BUFFERS]) != 0:
                raise RuntimeError("bq_dequantize_blockwise failed")
        kname = "dequantize_kernel"
        what = "block-wise dequantize"
    steps = args.steps * 20
    warmup = args.warmup * 4
    log(f"warmup {warmup} calls, timing {steps} calls")
    ms, seg = timed(torch, stream, call, steps, warmup, 20)
    nbytes = n * 5 + nb * 4
    gbs = nbytes / (ms / 1e3) / 1e9
    # round-trip error of the timed data, outside the timed region: quantize
    # buffer set 0 again, dequantize it, compare with the input
    torch.cuda.synchronize()
    bq.bq_quantize_blockwise_prepared(prepared, xs[0], B, codes[0], absmax[0], stream=stream)
    bq.bq_dequantize_blockwise(qs_d, codes[0], absmax[0], B, outs[0], stream=stream)
    err = (outs[0].double() - xs[0].double()).abs()
    round_trip = {"mean_abs_err": float(err.mean()), "max_abs_err": float(err.max()),
                  "max_rel_err_of_block_absmax": float(
                      (err.view(-1, B) / absmax[0].double().clamp_min(1e-300)[:, None]).max()
                      if n % B == 0 else float("nan")),
                  "mean_abs_value": float(xs[0].double().abs().mean())}
    del err
    res = base_record(
        args, f"{what} elements/sec and achieved HBM GB/s (% of peak), 67M Student-t values",
        n / (ms / 1e3), "elements/s", ms, seg, "f32",
        "synthetic (numpy PCG64 Student-t(3) x 1e-2, seed 0; four rotating buffer sets)",
        {"workload": f"{what}, signed dynamic map, n = {n}, blocksize {B}", "elements": n,
         "blocksize": B, "path": path})
    res["steps"] = steps
    res["warmup"] = warmup
    res.update({
        "gbs": gbs, "hbm_frac": gbs / HBM_PEAK_GBS,
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS,
                     "traffic": measured_traffic(args.workload, B, path), "bytes_per_step": nbytes,
                     "kernel": kname},
        "stream_ceiling": None, "cpu_baseline": None,
        "round_trip": round_trip,
    })
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="lm1p5b-adam",
                    choices=list(LIST_WORKLOADS) + ["quantize", "dequantize", "cpu-oracle",
                                                    "stream-study"])
    ap.add_argument("--rounds", type=int, default=5,
                    help="stream-study: interleaved rounds over all cases")
    ap.add_argument("--blocksize", type=int, default=BLOCKSIZE)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-stream-ceiling", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=16)
    ap.add_argument("--path", choices=["plan", "prepared", "device", "call", "static", "optim",
                                       "optim-graph"],
                    default="plan",
                    help="plan: bq_step_plan_run (a prepare launch from the raw maps, then one "
                         "launch over the whole list) or, for quantize, the prepared codebook; "
                         "prepared: bq_step_plan_run_prepared (the maps' tables prepared once, "
                         "before the timed steps); device: bq_step_plan_run_device (as prepared, "
                         "the hyperparameters read and the step advanced in device memory); "
                         "call: bq_optimizer8bit_step "
                         "(descriptor chunks of 56 tensors) or bq_quantize_blockwise; static: "
                         "bq_optimizer8bit_step_static (no allocation: tables and descriptors "
                         "in the library's static device array, one step launch); optim: "
                         "the drop-in torch optimizer (Adam8bit / AdamW8bit / SGD8bit) with "
                         "the grads of the ring assigned to .grad before each step; "
                         "optim-graph: the same optimizer built with capturable=True, its step() "
                         "captured into a HIP graph once per grad buffer and replayed")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the 8-bit step has no cross-GPU exchange, and "
              "the library runs on a single MI355X (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    if args.workload == "cpu-oracle":
        print(json.dumps(run_cpu_oracle(args)), flush=True)
        return

    import torch
    from paper_2110_02861_amd import bq, workloads

    if args.workload == "stream-study":
        res = run_stream_study(args, torch, bq, workloads)
    elif args.workload in LIST_WORKLOADS:
        res = run_list(args, torch, bq, workloads)
    else:
        res = run_quant(args, torch, bq, workloads)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
