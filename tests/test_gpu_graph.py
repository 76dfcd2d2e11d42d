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
