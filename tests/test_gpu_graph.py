"""The step under HIP graph capture: a captured plan run (prepare + step
kernels) and a captured allocation-free call, replayed with new grads written
eagerly between replays, must give the same bytes as the same runs made
eagerly, after every replay.  The hyperparameters (step count included) are
baked into the captured launches, so every run here uses the same ones."""
import numpy as np
import pytest
import torch

from paper_2110_02861_amd import bq, optim
from tests.gpu_helpers import codebooks_on_device, host, needs_gpu, say

pytestmark = [pytest.mark.gpu, needs_gpu]

HP = dict(lr=1e-3, beta1=0.9, beta2=0.995, eps=1e-8, wd=0.0, step=3)


def make_state(sizes, seed):
    rows = []
    for i, n in enumerate(sizes):
        rng = np.random.default_rng([seed, i])
        w = torch.from_numpy(rng.uniform(-0.05, 0.05, n).astype(np.float32)).cuda()
        nb = (n + 2047) // 2048
        rows.append((w, torch.zeros(n, dtype=torch.float16, device="cuda"),
                     torch.full((n,), 127, dtype=torch.uint8, device="cuda"),
                     torch.zeros(n, dtype=torch.uint8, device="cuda"),
                     torch.zeros(nb, dtype=torch.float32, device="cuda"),
                     torch.zeros(nb, dtype=torch.float32, device="cuda")))
    return rows


def grads_for(sizes, r):
    return [torch.from_numpy((np.random.default_rng([77, i, r]).standard_normal(n) * 1e-3)
                             .astype(np.float16)).cuda() for i, n in enumerate(sizes)]


@pytest.mark.parametrize("path", ["plan", "prepared", "call"])
def test_captured_step_replays_match_eager(path):
    sizes = [5000, 3 * 4096 + 11, 300]
    _, _, qs_d, qu_d = codebooks_on_device()
    eager, graphed = make_state(sizes, 1), make_state(sizes, 1)
    plans = {}
    if path != "call":
        plans = {"e": bq.StepPlan(bq.BQ_ADAM, 2048, bq.BQ_F16, eager),
                 "g": bq.StepPlan(bq.BQ_ADAM, 2048, bq.BQ_F16, graphed)}
    prepared = bq.prepare_codebook_pair(qs_d, qu_d)

    def run(rows, key, stream=None):
        if path == "plan":
            plans[key].run(HP, qs_d, qu_d, stream=stream)
        elif path == "prepared":
            plans[key].run_prepared(HP, prepared, stream=stream)
        else:
            bq.bq_optimizer8bit_step(bq.BQ_ADAM, 2048, bq.BQ_F16, rows, HP, qs_d, qu_d,
                                     stream=stream)

    # warm up both on a side stream (as torch's graph capture expects), then
    # restore the graphed copy to the eager copy's state
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run(graphed, "g", stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for e, g in zip(eager, graphed):
        for te, tg in zip(e, g):
            tg.copy_(te)
    torch.cuda.synchronize()
    say(f"capturing the {path} step")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run(graphed, "g", stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    for r in range(4):
        gs = grads_for(sizes, r)
        for e, g, gr in zip(eager, graphed, gs):
            e[1].copy_(gr)
            g[1].copy_(gr)
        torch.cuda.synchronize()
        say(f"{path}: eager run and graph replay {r}")
        run(eager, "e")
        graph.replay()
        torch.cuda.synchronize()
        for i, (e, g) in enumerate(zip(eager, graphed)):
            for k, name in ((0, "param"), (2, "codes1"), (3, "codes2"), (4, "absmax1"),
                            (5, "absmax2")):
                a, b = host(e[k]), host(g[k])
                assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), (path, r, i, name)
    for p in plans.values():
        p.close()


@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")  # refused before any launch
def test_optimizer_step_refuses_capture():
    """A drop-in optimizer step passes its step count as a launch argument, so a
    replayed graph would repeat one step's bias correction: step() refuses to
    run under capture, before it counts the step or launches anything."""
    p = torch.nn.Parameter(torch.zeros(5000, device="cuda"))
    p.grad = torch.full_like(p, 1e-3)
    opt = optim.Adam8bit([p])
    opt.step()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    say("capturing an optimizer step (refused)")
    with pytest.raises(RuntimeError, match="cannot be captured"):
        with torch.cuda.graph(graph):
            opt.step()
    torch.cuda.synchronize()
    assert opt.state[p]["step"] == 1
    opt.step()
    torch.cuda.synchronize()
    assert opt.state[p]["step"] == 2


def test_captured_device_hparam_run_replays_as_successive_steps():
    """One captured run with device-resident hyperparameters, replayed four
    times, is four successive steps (t = 1..4): each replay advances the step
    in device memory.  The lr is rewritten in device memory between replays 2
    and 3, as a schedule would.  Every replay equals an eager run given the
    same step and lr by the host."""
    sizes = [5000, 3 * 4096 + 11, 300]
    _, _, qs_d, qu_d = codebooks_on_device()
    eager, graphed = make_state(sizes, 2), make_state(sizes, 2)
    pe = bq.StepPlan(bq.BQ_ADAM, 2048, bq.BQ_F16, eager)
    pg = bq.StepPlan(bq.BQ_ADAM, 2048, bq.BQ_F16, graphed)
    prepared = bq.prepare_codebook_pair(qs_d, qu_d)
    hp = {k: v for k, v in HP.items() if k != "step"}
    hp_dev = bq.device_hparams(dict(hp, step=0))
    # warm up on a side stream with advance off (the step stays 0), then
    # restore the graphed copy to the eager copy's state
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        warm = bq.device_hparams(dict(hp, step=1))
        pg.run_device(warm, prepared, advance=False, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for e, g in zip(eager, graphed):
        for te, tg in zip(e, g):
            tg.copy_(te)
    torch.cuda.synchronize()
    say("capturing a device-hyperparameter run")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        pg.run_device(hp_dev, prepared, advance=True, stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    assert bq.read_device_hparams(hp_dev)["step"] == 0  # capture ran nothing
    for t in range(1, 5):
        if t == 3:
            hp["lr"] = hp["lr"] * 0.25
            hp_dev.copy_(bq.device_hparams(dict(hp, step=t - 1)))
        gs = grads_for(sizes, 10 + t)
        for e, g, gr in zip(eager, graphed, gs):
            e[1].copy_(gr)
            g[1].copy_(gr)
        torch.cuda.synchronize()
        say(f"device-hyperparameter replay t={t}")
        pe.run_prepared(dict(hp, step=t), prepared)
        graph.replay()
        torch.cuda.synchronize()
        assert bq.read_device_hparams(hp_dev)["step"] == t
        for i, (e, g) in enumerate(zip(eager, graphed)):
            for k, name in ((0, "param"), (2, "codes1"), (3, "codes2"), (4, "absmax1"),
                            (5, "absmax2")):
                a, b = host(e[k]), host(g[k])
                assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), (t, i, name)
    pe.close()
    pg.close()


CAPTURABLE = {
    "adam": (optim.Adam8bit, dict(lr=1e-3, betas=(0.9, 0.995))),
    "adamw": (optim.AdamW8bit, dict(lr=1e-3, weight_decay=0.01)),
    "sgd": (optim.SGD8bit, dict(lr=0.1, momentum=0.9, weight_decay=1e-4)),
    "adagrad": (optim.Adagrad8bit, dict(lr=1e-2)),
    "lamb": (optim.Lamb8bit, dict(lr=1e-3, weight_decay=0.01)),
    "lars": (optim.Lars8bit, dict(lr=0.5, momentum=0.9, weight_decay=1e-4)),
}


@pytest.mark.parametrize("case", list(CAPTURABLE))
def test_capturable_optimizer_replays_match_eager(case):
    """capturable=True: two eager steps, one captured step() replayed three
    times (the lr halved through update_device_hparams before the last), then
    an eager step again.  Every step equals a plain optimizer's eager step on
    the same grads, bit for bit, and state_dict() reports the device count."""
    cls, kw = CAPTURABLE[case]
    sizes = [5000, 3 * 4096 + 11, 300]
    rng = np.random.default_rng(3)
    ws = [rng.uniform(-0.05, 0.05, n).astype(np.float32) for n in sizes]
    pa = [torch.nn.Parameter(torch.from_numpy(w).cuda()) for w in ws]
    pb = [torch.nn.Parameter(torch.from_numpy(w).cuda()) for w in ws]
    grads = [torch.zeros(n, dtype=torch.float16, device="cuda") for n in sizes]
    for p, q, g in zip(pa, pb, grads):
        for x in (p, q):
            if hasattr(x, "grad_dtype"):
                x.grad_dtype = None  # fp16 grads on fp32 params
            x.grad = g
    oa = cls(pa, capturable=True, **kw)
    ob = cls(pb, **kw)

    def new_grads(t):
        for i, (g, n) in enumerate(zip(grads, sizes)):
            h = (np.random.default_rng([5, i, t]).standard_normal(n) * 1e-3).astype(np.float16)
            g.copy_(torch.from_numpy(h))

    def compare(t):
        for i, (p, q) in enumerate(zip(pa, pb)):
            assert torch.equal(p.detach().view(torch.uint8), q.detach().view(torch.uint8)), \
                (case, t, i, "param")
            sa, sb = oa.state[p], ob.state[q]
            for k in ("state1", "absmax1", "state2", "absmax2"):
                if k in sb:
                    assert torch.equal(sa[k].view(torch.uint8), sb[k].view(torch.uint8)), \
                        (case, t, i, k)

    for t in (1, 2):
        new_grads(t)
        say(f"capturable {case}: eager step {t}")
        oa.step()
        ob.step()
        torch.cuda.synchronize()
        compare(t)
    graph = torch.cuda.CUDAGraph()
    say(f"capturable {case}: capturing step()")
    with torch.cuda.graph(graph):
        oa.step()
    torch.cuda.synchronize()
    for t in (3, 4, 5):
        if t == 5:
            for o in (oa, ob):
                o.param_groups[0]["lr"] *= 0.5
            oa.update_device_hparams()
        new_grads(t)
        say(f"capturable {case}: replay as step {t}")
        graph.replay()
        ob.step()
        torch.cuda.synchronize()
        compare(t)
    assert all(s["step"] == 5 for s in oa.state_dict()["state"].values())
    new_grads(6)
    oa.step()
    ob.step()
    torch.cuda.synchronize()
    compare(6)
    assert all(s["step"] == 6 for s in oa.state_dict()["state"].values())


@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")  # refused before any launch
def test_capturable_optimizer_needs_an_eager_step_first():
    p = torch.nn.Parameter(torch.zeros(5000, device="cuda"))
    p.grad = torch.full_like(p, 1e-3)
    opt = optim.Adam8bit([p], capturable=True)
    graph = torch.cuda.CUDAGraph()
    say("capturing a capturable optimizer's first step (refused)")
    with pytest.raises(RuntimeError, match="outside graph capture first"):
        with torch.cuda.graph(graph):
            opt.step()
    torch.cuda.synchronize()
    assert not opt.state[p]  # nothing was created
    opt.step()
    torch.cuda.synchronize()
    assert opt.state[p]["step"] == 1


def test_captured_plans_survive_plan_cache_eviction():
    """After a capture, eager steps on ten new grad storages overflow the plan
    cache; the captured step's plan is never evicted, and a later replay still
    equals an eager optimizer given the same sequence of grads."""
    sizes = [5000, 300]
    ws = [np.random.default_rng([8, i]).uniform(-0.05, 0.05, n).astype(np.float32)
          for i, n in enumerate(sizes)]
    pa = [torch.nn.Parameter(torch.from_numpy(w).cuda()) for w in ws]
    pb = [torch.nn.Parameter(torch.from_numpy(w).cuda()) for w in ws]
    oa = optim.Adam8bit(pa, capturable=True)
    ob = optim.Adam8bit(pb)
    static = [torch.zeros(n, device="cuda") for n in sizes]
    keep = []  # every grad buffer stays alive, so each one is a new storage

    def fill(bufs, t):
        for i, (g, n) in enumerate(zip(bufs, sizes)):
            g.copy_(torch.from_numpy(np.random.default_rng([9, i, t]).standard_normal(n)
                                     .astype(np.float32) * 1e-3))

    for p, q, g in zip(pa, pb, static):
        p.grad, q.grad = g, g
    fill(static, 0)
    oa.step()
    ob.step()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        oa.step()
    torch.cuda.synchronize()
    (pinned,) = oa._pinned
    for t in range(1, 11):
        bufs = [torch.zeros(n, device="cuda") for n in sizes]
        keep.append(bufs)
        fill(bufs, t)
        for p, q, g in zip(pa, pb, bufs):
            p.grad, q.grad = g, g
        say(f"eager step on new grad storage {t}")
        oa.step()
        ob.step()
    assert len(keep) > optim.Optimizer8bit.MAX_PLANS
    assert pinned in oa._plans and oa._plans[pinned].is_open()
    fill(static, 11)
    for q, g in zip(pb, static):
        q.grad = g
    say("replay after evictions")
    graph.replay()
    ob.step()
    torch.cuda.synchronize()
    for p, q in zip(pa, pb):
        assert torch.equal(p.detach().view(torch.uint8), q.detach().view(torch.uint8))
        for k in ("state1", "absmax1", "state2", "absmax2"):
            assert torch.equal(oa.state[p][k], ob.state[q][k]), k
