"""The allocation-free step through the library's static device array
(bq_optimizer8bit_step_static), called through the C ABI, against the step
plan over the same list (the same kernels: bit for bit) and the
allocation-free call bq_optimizer8bit_step (codes and absmax bit-exact, params
within 1e-6 |w| + 1e-6 |update|), on calls in a row with changing lists: the
second smaller than the first, then more tensors than one upload launch
carries, one-state optimizers and every end of the blocksize range.
"""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_helpers import OPT_ID, codebooks_on_device, host, needs_gpu, param_close, say
from paper_2110_02861_amd import bq

pytestmark = [pytest.mark.gpu, needs_gpu]

HP = {"adam": dict(lr=1e-3, beta1=0.9, beta2=0.995, eps=1e-8, wd=0.0),
      "adamw": dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.01),
      "momentum": dict(lr=0.1, beta1=0.9, beta2=0.0, eps=0.0, wd=1e-4),
      "adagrad": dict(lr=0.01, beta1=0.0, beta2=0.0, eps=1e-10, wd=0.0)}
TWO = ("adam", "adamw")


def make_list(sizes, opt, B, gdt, seed):
    """Three identical copies (static call, plan, allocation-free call) of a
    list in the zero state, and per-step grads."""
    g = torch.Generator(device="cuda").manual_seed(seed)
    two = opt in TWO
    zero1 = 0 if opt == "adagrad" else 127
    base = []
    for n in sizes:
        nb = (n + B - 1) // B
        w = torch.randn(n, device="cuda", generator=g) * 0.02
        base.append((w, nb))
    copies = []
    for _ in range(3):
        rows = []
        for (w, nb) in base:
            n = w.numel()
            rows.append([w.clone(), torch.empty(n, dtype=gdt, device="cuda"),
                         torch.full((n,), zero1, dtype=torch.uint8, device="cuda"),
                         torch.zeros(n, dtype=torch.uint8, device="cuda") if two else None,
                         torch.zeros(nb, device="cuda"),
                         torch.zeros(nb, device="cuda") if two else None])
        copies.append(rows)
    return copies


def fill_grads(copies, seed, t):
    g = torch.Generator(device="cuda").manual_seed(seed * 1000 + t)
    for i in range(len(copies[0])):
        n = copies[0][i][0].numel()
        x = torch.randn(n, device="cuda", generator=g) * 1e-3
        for rows in copies:
            rows[i][1].copy_(x.to(rows[i][1].dtype))


def run_case(opt, sizes, B, gdt, seed, steps=2):
    qs, qu, qs_d, qu_d = codebooks_on_device()
    q1 = qu_d if opt == "adagrad" else qs_d
    q2 = qu_d if opt in TWO else None
    gflag = {torch.float16: bq.BQ_F16, torch.bfloat16: bq.BQ_BF16, torch.float32: bq.BQ_F32}[gdt]
    cs, cp, cc = make_list(sizes, opt, B, gdt, seed)
    plan = bq.StepPlan(opt, B, gflag, [tuple(r) for r in cp])
    for t in range(1, steps + 1):
        fill_grads((cs, cp, cc), seed, t)
        prev = [r[0].clone() for r in cc]
        hp = dict(HP[opt], step=t)
        say(f"static step {opt} B={B} {gdt} {len(sizes)} tensors t={t}")
        bq.bq_optimizer8bit_step_static(opt, B, gflag, [tuple(r) for r in cs], hp, q1, q2)
        plan.run(hp, q1, q2)
        bq.bq_optimizer8bit_step(opt, B, gflag, [tuple(r) for r in cc], hp, q1, q2)
        torch.cuda.synchronize()
        for i, (rs, rp, rc) in enumerate(zip(cs, cp, cc)):
            for k, (a, b) in enumerate(zip(rs, rp)):
                if a is not None:
                    assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), (t, i, k)
            for k in (2, 3, 4, 5):
                if rs[k] is not None:
                    assert torch.equal(rs[k], rc[k]), (t, i, k)
            w_ref = host(rc[0]).astype(np.float64)
            upd = np.abs(host(prev[i]).astype(np.float64) - w_ref)
            ok, worst = param_close(host(rs[0]), w_ref, 1e-6 * upd)
            assert ok, (t, i, worst)
        # the allocation-free call's copy continues from the static call's
        # state, so both compare one step from the same state each time
        for rs, rc in zip(cs, cc):
            rc[0].copy_(rs[0])
    return cs


def test_two_calls_in_a_row_second_smaller():
    run_case("adam", [1 << 20, 3 * 4096 + 100, 777, 0, 4096, 2048 * 5 + 1], 2048,
             torch.float16, seed=1)
    run_case("adam", [5000, 300], 2048, torch.float16, seed=2)


def test_more_tensors_than_one_upload():
    rng = np.random.default_rng(3)
    sizes = [int(x) for x in rng.integers(1, 9000, 150)]
    sizes[7] = 0
    run_case("adamw", sizes, 2048, torch.float16, seed=3)


@pytest.mark.parametrize("opt,gdt", [("momentum", torch.float32), ("adagrad", torch.bfloat16)])
def test_one_state_optimizers(opt, gdt):
    run_case(opt, [70_000, 4097, 1], 2048, gdt, seed=4)


@pytest.mark.parametrize("B", [256, 4096])
def test_blocksize_range(B):
    run_case("adam", [3 * 4096 + 5, 40_000], B, torch.float32, seed=5)


def test_first_step_matches_the_oracle():
    """One step of a ragged list from the zero state against the oracle:
    codes and absmax bit-exact, params within 1e-6 |w| + 1e-6 |update|."""
    qs, qu, qs_d, qu_d = codebooks_on_device()
    sizes = [3 * 2048 + 17, 2048, 999]
    (cs, _, _) = make_list(sizes, "adam", 2048, torch.float16, seed=6)
    w0 = [host(r[0]).copy() for r in cs]
    fill_grads((cs,), 6, 1)
    g = [host(r[1].float()).copy() for r in cs]
    hp = dict(HP["adam"], step=1)
    say("static step vs oracle")
    bq.bq_optimizer8bit_step_static("adam", 2048, bq.BQ_F16, [tuple(r) for r in cs], hp, qs_d,
                                    qu_d)
    torch.cuda.synchronize()
    for i, n in enumerate(sizes):
        nb = (n + 2047) // 2048
        w = w0[i].copy()
        c1 = np.full(n, 127, np.uint8)
        c2 = np.zeros(n, np.uint8)
        a1 = np.zeros(nb, np.float32)
        a2 = np.zeros(nb, np.float32)
        oracle.step8(OPT_ID["adam"], 2048, w, g[i], c1, a1, qs, c2, a2, qu, hp["lr"], hp["beta1"],
                     hp["beta2"], hp["eps"], hp["wd"], 1)
        np.testing.assert_array_equal(host(cs[i][2]), c1)
        np.testing.assert_array_equal(host(cs[i][3]), c2)
        np.testing.assert_array_equal(host(cs[i][4]), a1)
        np.testing.assert_array_equal(host(cs[i][5]), a2)
        upd = np.abs(w0[i].astype(np.float64) - w.astype(np.float64))
        ok, worst = param_close(host(cs[i][0]), w, 1e-6 * upd)
        assert ok, (i, worst)
