"""The drop-in optimizers (paper_2110_02861_amd.optim) against the oracle.

Each step is checked from the same state on both sides (the oracle starts from
the optimizer's state before the step): codes and absmax bit-exact, params
within 1e-6 of |w| plus 1e-6 of the update.  32-bit-state tensors (Section 3.3)
are checked against the oracle's step with fp32 states.
"""
from __future__ import annotations

import io

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import host, needs_gpu, param_close, say
from paper_2110_02861_amd import bq, optim, workloads

pytestmark = [pytest.mark.gpu, needs_gpu]

# ragged sizes: partial blocks, a tensor below one block, an exact multiple
SHAPES = [(37, 129), (5000,), (3, 2048), (300,), (1,)]
B = 2048

CASES = {
    "adam": (optim.Adam8bit, dict(lr=1e-3, betas=(0.9, 0.995), eps=1e-8, weight_decay=0.0),
             oracle.ADAM),
    "adam_l2": (optim.Adam8bit, dict(lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.01),
                oracle.ADAM),
    "adamw": (optim.AdamW8bit, dict(lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.01),
              oracle.ADAMW),
    "sgd": (optim.SGD8bit, dict(lr=0.1, momentum=0.9, weight_decay=1e-4), oracle.MOMENTUM),
    "adagrad": (optim.Adagrad8bit, dict(lr=1e-2, eps=1e-10, weight_decay=0.0), oracle.ADAGRAD),
    "lamb": (optim.Lamb8bit, dict(lr=1e-3, betas=(0.9, 0.999), eps=1e-6, weight_decay=0.01),
             oracle.LAMB),
    "lars": (optim.Lars8bit, dict(lr=0.5, momentum=0.9, weight_decay=1e-4,
                                  trust_coefficient=1e-3), oracle.LARS),
}


def oracle_hp(kw):
    if "trust_coefficient" in kw:  # LARS
        return dict(lr=kw["lr"], beta1=kw["momentum"], beta2=0.0, eps=0.0,
                    wd=kw["weight_decay"], trust=kw["trust_coefficient"])
    if "betas" not in kw and "momentum" not in kw:  # AdaGrad
        return dict(lr=kw["lr"], beta1=0.0, beta2=0.0, eps=kw["eps"], wd=kw["weight_decay"])
    if "momentum" in kw:
        return dict(lr=kw["lr"], beta1=kw["momentum"], beta2=0.0, eps=0.0, wd=kw["weight_decay"])
    return dict(lr=kw["lr"], beta1=kw["betas"][0], beta2=kw["betas"][1], eps=kw["eps"],
                wd=kw["weight_decay"])


def init_params(seed):
    out = []
    for i, s in enumerate(SHAPES):
        rng = workloads.host_rng(seed, "c1", i, 0)
        w = (rng.standard_normal(int(np.prod(s)), dtype=np.float32) * np.float32(0.02))
        out.append(torch.nn.Parameter(torch.from_numpy(w.reshape(s)).cuda()))
    return out


def grads(seed, step, dtype):
    out = []
    for i, s in enumerate(SHAPES):
        rng = workloads.host_rng(seed, "c1", i, step)
        g = rng.standard_normal(int(np.prod(s))) * 1e-3
        g[rng.random(g.size) < 1e-3] *= 100.0
        out.append(g.astype(dtype).reshape(s))
    return out


def set_grad(p, g):
    """Attach a host grad (numpy or torch); a 16-bit grad on an fp32 param
    needs grad_dtype None."""
    t = g if isinstance(g, torch.Tensor) else torch.from_numpy(np.ascontiguousarray(g))
    t = t.cuda()
    if t.dtype != p.dtype and hasattr(p, "grad_dtype"):
        p.grad_dtype = None
    p.grad = t


def grad_pair(g, gdt):
    """(grad to attach, its values for the oracle).  bf16: torch rounds the
    fp32 grad on the host and the oracle takes the exact fp32 values of the
    bf16 result."""
    if gdt == "bf16":
        gt = torch.from_numpy(np.ascontiguousarray(g, dtype=np.float32)).to(torch.bfloat16)
        return gt, gt.float().numpy()
    return g, g


def host_dtype(gdt):
    return np.float32 if gdt == "bf16" else gdt


def snapshot(opt, p):
    """Host copy of one param's optimizer state (None before its first step)."""
    s = opt.state.get(p)
    if not s:
        return None
    return {k: (host(v).copy() if isinstance(v, torch.Tensor) else v) for k, v in s.items()}


def oracle_step8(kind, hp, w, g, snap, n, two, t):
    q1 = bq.bq_make_dynamic_codebook(bq.BQ_SIGNED)
    q2 = bq.bq_make_dynamic_codebook(bq.BQ_UNSIGNED)
    if kind == oracle.ADAGRAD:  # one non-negative state: the unsigned map
        q1 = q2
    nb = (n + B - 1) // B
    if snap is None:
        c1, a1 = np.full(n, 127, np.uint8), np.zeros(nb, np.float32)
        c2 = np.zeros(n, np.uint8) if two else None
        a2 = np.zeros(nb, np.float32) if two else None
    else:
        c1, a1 = snap["state1"].copy(), snap["absmax1"].copy()
        c2 = snap["state2"].copy() if two else None
        a2 = snap["absmax2"].copy() if two else None
    w = w.copy()
    oracle.step8(kind, B, w, g, c1, a1, q1, c2, a2, q2 if two else None, hp["lr"], hp["beta1"],
                 hp["beta2"], hp["eps"], hp["wd"], t, trust=hp.get("trust", 0.0))
    return w, c1, a1, c2, a2


@pytest.mark.parametrize("use_plans", [True, False])
@pytest.mark.parametrize("gdt", [np.float32, np.float16, "bf16"])
@pytest.mark.parametrize("case", list(CASES))
def test_optimizer_matches_oracle(case, gdt, use_plans):
    cls, kw, kind = CASES[case]
    hp = oracle_hp(kw)
    two = kind in (oracle.ADAM, oracle.ADAMW, oracle.LAMB)
    params = init_params(7)
    opt = cls(params, blocksize=B, use_plans=use_plans, **kw)
    for t in range(1, 4):
        gs = grads(7, t, host_dtype(gdt))
        refs = []
        for p, g in zip(params, gs):
            g_dev, g_ref = grad_pair(g, gdt)
            refs.append(oracle_step8(kind, hp, host(p).ravel(), g_ref.ravel(),
                                     snapshot(opt, p), p.numel(), two, t))
            set_grad(p, g_dev)
        say(f"optim {case} {gdt if gdt == 'bf16' else np.dtype(gdt).name} "
            f"plans={use_plans} step {t}")
        w_before = [host(p).ravel().astype(np.float64) for p in params]
        opt.step()
        torch.cuda.synchronize()
        for i, (p, ref) in enumerate(zip(params, refs)):
            s = opt.state[p]
            w_ref, c1, a1, c2, a2 = ref
            assert s["step"] == t
            assert np.array_equal(host(s["state1"]), c1), f"{case} tensor {i} step {t}: state1"
            assert np.array_equal(host(s["absmax1"]), a1), f"{case} tensor {i} step {t}: absmax1"
            if two:
                assert np.array_equal(host(s["state2"]), c2), f"tensor {i} step {t}: state2"
                assert np.array_equal(host(s["absmax2"]), a2), f"tensor {i} step {t}: absmax2"
            upd = np.abs(w_before[i] - w_ref.astype(np.float64))
            ok, worst = param_close(host(p).ravel(), w_ref, 1e-6 * upd)
            assert ok, f"{case} tensor {i} step {t}: params off by {worst}"


@pytest.mark.parametrize("gdt", [np.float32, "bf16"])
@pytest.mark.parametrize("case", ["adam", "adamw", "sgd", "adagrad"])
def test_32bit_override_and_min_size(case, gdt):
    """override_32bit and min_8bit_size keep fp32 states, updated like the
    oracle's step with fp32 states; the other tensors stay 8-bit."""
    cls, kw, kind = CASES[case]
    hp = oracle_hp(kw)
    two = kind in (oracle.ADAM, oracle.ADAMW)
    params = init_params(11)
    opt = cls(params, blocksize=B, min_8bit_size=400, **kw)
    opt.override_32bit(params[1])
    for t in range(1, 3):
        gs = grads(11, t, np.float32)
        refs = {}
        for i, (p, g) in enumerate(zip(params, gs)):
            g_dev, g = grad_pair(g, gdt)
            snap = snapshot(opt, p)
            if i in (1, 3, 4):  # overridden, and below min_8bit_size
                w = host(p).ravel().copy()
                m = snap["exp_avg"].copy() if snap else np.zeros(p.numel(), np.float32)
                v = (snap["exp_avg_sq"].copy() if snap else np.zeros(p.numel(), np.float32)) \
                    if two else None
                oracle.step32(kind, w, g.ravel(), m, v, hp["lr"], hp["beta1"], hp["beta2"],
                              hp["eps"], hp["wd"], t)
                refs[i] = (w, m, v)
            set_grad(p, g_dev)
        say(f"optim override {case} {gdt} step {t}")
        w_before = [host(p).ravel().astype(np.float64) for p in params]
        opt.step()
        torch.cuda.synchronize()
        for i, p in enumerate(params):
            s = opt.state[p]
            if i not in refs:
                assert "state1" in s and s["state1"].dtype == torch.uint8
                continue
            assert "exp_avg" in s and "state1" not in s
            w, m, v = refs[i]
            assert np.array_equal(host(s["exp_avg"]), m), f"tensor {i} step {t}: m"
            if two:
                assert np.array_equal(host(s["exp_avg_sq"]), v), f"tensor {i} step {t}: v"
            upd = np.abs(w_before[i] - w.astype(np.float64))
            ok, worst = param_close(host(p).ravel(), w, 1e-6 * upd)
            assert ok, f"tensor {i} step {t}: params off by {worst}"
    with pytest.raises(RuntimeError):
        opt.override_32bit(params[0])


def test_state_dict_round_trip_resumes_bit_exactly():
    """Save after 2 steps, load into a fresh optimizer over copied params, and
    both continue identically (codes, absmax, params, step count)."""
    params_a = init_params(3)
    opt_a = optim.Adam8bit(params_a, lr=1e-3, betas=(0.9, 0.995))
    opt_a.override_32bit(params_a[2])
    for t in (1, 2):
        for p, g in zip(params_a, grads(3, t, np.float32)):
            set_grad(p, g)
        opt_a.step()
    buf = io.BytesIO()
    torch.save(opt_a.state_dict(), buf)
    buf.seek(0)
    sd = torch.load(buf, weights_only=True)
    params_b = [torch.nn.Parameter(p.detach().clone()) for p in params_a]
    opt_b = optim.Adam8bit(params_b, lr=1e-3, betas=(0.9, 0.995))
    opt_b.override_32bit(params_b[2])
    opt_b.load_state_dict(sd)
    for t in (3, 4):
        gs = grads(3, t, np.float32)
        for pa, pb, g in zip(params_a, params_b, gs):
            set_grad(pa, g)
            set_grad(pb, g)
        say(f"optim state_dict resume step {t}")
        opt_a.step()
        opt_b.step()
    torch.cuda.synchronize()
    for pa, pb in zip(params_a, params_b):
        assert torch.equal(pa, pb)
        sa, sb = opt_a.state[pa], opt_b.state[pb]
        assert sa["step"] == sb["step"] == 4
        for k in sa:
            if isinstance(sa[k], torch.Tensor):
                assert sa[k].dtype == sb[k].dtype, k
                assert torch.equal(sa[k], sb[k]), k


def test_plans_follow_reallocated_grads():
    """Fresh grad tensors every step (as zero_grad(set_to_none=True) gives)
    rebuild the cached plan; codes equal the plan-free path."""
    params_a = init_params(5)
    params_b = [torch.nn.Parameter(p.detach().clone()) for p in params_a]
    opt_a = optim.Adam8bit(params_a, use_plans=True)
    opt_b = optim.Adam8bit(params_b, use_plans=False)
    for t in range(1, 4):
        gs = grads(5, t, np.float16)
        for pa, pb, g in zip(params_a, params_b, gs):
            set_grad(pa, g)
            set_grad(pb, g)
        # grab a block so that the next grads land elsewhere
        keep = torch.empty(1 << 20, device="cuda")
        say(f"optim plans follow grads step {t}")
        opt_a.step()
        opt_b.step()
        del keep
    torch.cuda.synchronize()
    assert len(opt_a._plans) <= optim.Optimizer8bit.MAX_PLANS
    for pa, pb in zip(params_a, params_b):
        sa, sb = opt_a.state[pa], opt_b.state[pb]
        for k in ("state1", "absmax1", "state2", "absmax2"):
            assert torch.equal(sa[k], sb[k]), k
        upd = 1e-3 * torch.ones_like(pa)
        assert torch.all((pa - pb).abs() <= 1e-6 * pa.abs() + 1e-6 * upd)


def test_alternating_grad_buffers_reuse_plans():
    """Two grad buffer sets used in turn: one plan each, built once and reused,
    and codes equal to the plan-free path at every step."""
    params_a = init_params(5)
    params_b = [torch.nn.Parameter(p.detach().clone()) for p in params_a]
    opt_a = optim.Adam8bit(params_a, use_plans=True)
    opt_b = optim.Adam8bit(params_b, use_plans=False)
    ring = [[torch.from_numpy(g).cuda() for g in grads(5, r + 1, np.float16)] for r in range(2)]
    for p in params_a + params_b:
        p.grad_dtype = None
    seen = {}
    for t in range(1, 7):
        for pa, pb, g in zip(params_a, params_b, ring[t % 2]):
            pa.grad = g
            pb.grad = g
        say(f"optim alternating grads step {t}")
        opt_a.step()
        opt_b.step()
        assert len(opt_a._plans) == min(t, 2)
        for key, plan in opt_a._plans.items():
            assert seen.setdefault(key, plan) is plan  # never rebuilt
    torch.cuda.synchronize()
    for pa, pb in zip(params_a, params_b):
        sa, sb = opt_a.state[pa], opt_b.state[pb]
        for k in ("state1", "absmax1", "state2", "absmax2"):
            assert torch.equal(sa[k], sb[k]), k
        upd = 1e-3 * torch.ones_like(pa)
        assert torch.all((pa - pb).abs() <= 1e-6 * pa.abs() + 1e-6 * upd)


def test_training_loop_reduces_loss():
    """A least-squares fit with 8-bit Adam: the loss falls by orders of magnitude."""
    torch.manual_seed(0)
    x = torch.randn(4096, 64, device="cuda")
    w_true = torch.randn(64, 16, device="cuda")
    y = x @ w_true
    model = torch.nn.Linear(64, 16, bias=True).cuda()
    opt = optim.Adam8bit(model.parameters(), lr=3e-2)
    say("optim training loop")
    first = None
    for _ in range(300):
        opt.zero_grad(set_to_none=True)
        loss = torch.nn.functional.mse_loss(model(x), y)
        loss.backward()
        opt.step()
        first = first if first is not None else float(loss.detach())
    final = float(loss.detach())
    assert final < 1e-3 * first, (first, final)


@pytest.mark.parametrize("case", ["adam", "sgd"])
def test_state_memory(case):
    """8-bit state bytes: 1 B per param and state plus 4 B per block and state
    (2 + 8/B for Adam, 1 + 4/B for Momentum), against 8 and 4 for fp32 states."""
    B = 2048
    params = init_params(3)
    for p in params:
        p.grad = torch.zeros_like(p)
    opt = (optim.Adam8bit(params, blocksize=B) if case == "adam"
           else optim.SGD8bit(params, lr=0.1, blocksize=B))
    say(f"optim state memory {case}")
    opt.step()
    torch.cuda.synchronize()
    nstates = 2 if case == "adam" else 1
    for p in params:
        st = opt.state[p]
        nbytes = sum(t.numel() * t.element_size() for t in st.values()
                     if isinstance(t, torch.Tensor))
        n = p.numel()
        assert nbytes == nstates * (n + 4 * ((n + B - 1) // B)), (case, n, nbytes)


def test_stable_embedding_states_are_32_bit():
    """nn.StableEmbedding's weight gets fp32 states (the oracle's 32-bit step),
    the other params 8-bit states, in one optimizer step."""
    from paper_2110_02861_amd import nn
    torch.manual_seed(3)
    emb = nn.StableEmbedding(3000, 64).cuda()
    lin = torch.nn.Linear(64, 64).cuda()
    opt = optim.Adam8bit(list(emb.parameters()) + list(lin.parameters()), lr=1e-3)
    w0 = emb.weight.detach().cpu().numpy().copy()
    tokens = torch.randint(0, 3000, (16, 32), device="cuda")
    lin(emb(tokens)).square().mean().backward()
    g = emb.weight.grad.detach().cpu().numpy().copy()
    say("optim stable embedding step")
    opt.step()
    torch.cuda.synchronize()
    st = opt.state[emb.weight]
    assert "exp_avg" in st and "state1" not in st
    assert "state1" in opt.state[lin.weight]
    m = np.zeros(w0.size, np.float32)
    v = np.zeros(w0.size, np.float32)
    w = w0.reshape(-1).copy()
    oracle.step32(oracle.ADAM, w, g.reshape(-1), m, v, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1)
    np.testing.assert_array_equal(host(st["exp_avg"]).view(np.uint32), m.view(np.uint32))
    np.testing.assert_array_equal(host(st["exp_avg_sq"]).view(np.uint32), v.view(np.uint32))
    ok, worst = param_close(host(emb.weight).reshape(-1), w,
                            1e-6 * np.abs(w0.reshape(-1).astype(np.float64) - w))
    assert ok, worst


@pytest.mark.parametrize("use_plans", [True, False])
def test_param_groups_and_mixed_grad_dtypes(use_plans):
    """Two param groups with their own lr, betas and weight decay, and fp16 and
    fp32 grads inside one group: each param steps as the oracle with its group's
    hyperparameters."""
    params = init_params(11)
    g0, g1 = params[:3], params[3:]
    kw0 = dict(lr=1e-3, betas=(0.9, 0.995), eps=1e-8, weight_decay=0.0)
    kw1 = dict(lr=3e-3, betas=(0.8, 0.99), eps=1e-7, weight_decay=0.05)
    opt = optim.Adam8bit([dict(params=g0, **kw0), dict(params=g1, **kw1)], blocksize=B,
                         use_plans=use_plans)
    hps = [oracle_hp(kw0)] * 3 + [oracle_hp(kw1)] * 2
    for t in range(1, 4):
        # alternate the grad dtype per param and per step
        gs = [g.astype(np.float16 if (i + t) % 2 else np.float32)
              for i, g in enumerate(grads(11, t, np.float32))]
        refs = [oracle_step8(oracle.ADAM, hp, host(p).ravel(), g.ravel(), snapshot(opt, p),
                             p.numel(), True, t) for p, g, hp in zip(params, gs, hps)]
        for p, g in zip(params, gs):
            set_grad(p, g)
        w_before = [host(p).ravel().astype(np.float64) for p in params]
        say(f"optim two groups, mixed grad dtypes, plans={use_plans} step {t}")
        opt.step()
        torch.cuda.synchronize()
        for i, (p, ref) in enumerate(zip(params, refs)):
            s = opt.state[p]
            w_ref, c1, a1, c2, a2 = ref
            assert np.array_equal(host(s["state1"]), c1), (i, t)
            assert np.array_equal(host(s["absmax1"]), a1), (i, t)
            assert np.array_equal(host(s["state2"]), c2), (i, t)
            assert np.array_equal(host(s["absmax2"]), a2), (i, t)
            upd = np.abs(w_before[i] - w_ref.astype(np.float64))
            ok, worst = param_close(host(p).ravel(), w_ref, 1e-6 * upd)
            assert ok, (i, t, worst)


@pytest.mark.parametrize("case", ["adam", "sgd"])
def test_param_resized_after_state_raises(case):
    """A param whose storage is swapped for a larger one after its first step
    is refused before any launch: its states were sized for the old storage.
    The 32-bit-state path checks the same."""
    cls, kw, _ = CASES[case]
    for override in (False, True):
        p = torch.nn.Parameter(torch.zeros(3000, device="cuda"))
        opt = cls([p], **kw)
        if override:
            opt.override_32bit(p)
        p.grad = torch.zeros_like(p)
        say(f"optim resized param {case} 32-bit={override}: first step")
        opt.step()
        p.data = torch.zeros(5000, device="cuda")
        p.grad = torch.zeros_like(p)
        with pytest.raises(ValueError, match="changed size"):
            opt.step()
        torch.cuda.synchronize()


def test_repeated_steps_replay_and_match_oracle():
    """Steps whose params, grad storages and states equal one of the last two
    steps replay that step's launches (two grad buffers in turn, updated in
    place; one param on 32-bit states).  Every step still matches the oracle,
    a new lr takes effect in a replay, and a param moved to new storage falls
    back to the full path."""
    kind = oracle.ADAM
    kw = dict(lr=1e-3, betas=(0.9, 0.995), eps=1e-8, weight_decay=0.0)
    hp = oracle_hp(kw)
    params = init_params(13)
    opt = optim.Adam8bit(params, blocksize=B, **kw)
    opt.override_32bit(params[2])
    bufs = [[torch.zeros(p.numel(), dtype=torch.float16, device="cuda").view(p.shape)
             for p in params] for _ in range(2)]
    replays = []
    real_replay = opt._replay
    opt._replay = lambda gi, group: replays.append(real_replay(gi, group)) or replays[-1]
    for t in range(1, 7):
        if t == 4:
            hp["lr"] = kw["lr"] * 0.5
            opt.param_groups[0]["lr"] = hp["lr"]
        if t == 6:  # a param moved to new storage: the full path again
            params[0].data = params[0].data.clone()
        gs = grads(13, t, np.float16)
        buf = bufs[t % 2]
        refs = []
        for i, (p, g) in enumerate(zip(params, gs)):
            buf[i].copy_(torch.from_numpy(np.ascontiguousarray(g)))
            snap = snapshot(opt, p)
            if i == 2:
                w = host(p).ravel().copy()
                m = snap["exp_avg"].copy() if snap else np.zeros(p.numel(), np.float32)
                v = snap["exp_avg_sq"].copy() if snap else np.zeros(p.numel(), np.float32)
                oracle.step32(kind, w, g.ravel().astype(np.float32), m, v, hp["lr"],
                              hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], t)
                refs.append((w, m, v))
            else:
                refs.append(oracle_step8(kind, hp, host(p).ravel(), g.ravel(), snap, p.numel(),
                                         True, t))
            if hasattr(p, "grad_dtype"):
                p.grad_dtype = None
            p.grad = buf[i]
        say(f"optim replay step {t}")
        w_before = [host(p).ravel().astype(np.float64) for p in params]
        opt.step()
        torch.cuda.synchronize()
        for i, (p, ref) in enumerate(zip(params, refs)):
            s = opt.state[p]
            assert s["step"] == t
            if i == 2:
                w, m, v = ref
                assert np.array_equal(host(s["exp_avg"]), m), (t, "m")
                assert np.array_equal(host(s["exp_avg_sq"]), v), (t, "v")
            else:
                w, c1, a1, c2, a2 = ref
                for k, r in (("state1", c1), ("absmax1", a1), ("state2", c2), ("absmax2", a2)):
                    assert np.array_equal(host(s[k]), r), (t, i, k)
            upd = np.abs(w_before[i] - w.astype(np.float64))
            ok, worst = param_close(host(p).ravel(), w, 1e-6 * upd)
            assert ok, (t, i, worst)
    # steps 3-5 repeat the storages of steps 1-3; step 6 has a moved param
    assert replays == [False, False, True, True, True, False], replays


def test_many_param_groups_keep_their_plans():
    """Twelve param groups and two grad buffers in turn: after the first two
    steps no plan is built again (the cache makes room for every group), and
    every step equals the plan-free path."""
    ngroups = 12
    rng = np.random.default_rng(17)
    ws = [rng.uniform(-0.05, 0.05, 3000 + 500 * i).astype(np.float32) for i in range(ngroups)]
    pa = [torch.nn.Parameter(torch.from_numpy(w).cuda()) for w in ws]
    pb = [torch.nn.Parameter(torch.from_numpy(w).cuda()) for w in ws]
    opt_a = optim.Adam8bit([dict(params=[p], lr=1e-3 * (1 + i)) for i, p in enumerate(pa)])
    opt_b = optim.Adam8bit([dict(params=[p], lr=1e-3 * (1 + i)) for i, p in enumerate(pb)],
                           use_plans=False)
    bufs = [[torch.zeros_like(p) for p in pa] for _ in range(2)]
    seen = {}
    for t in range(1, 7):
        buf = bufs[t % 2]
        for i, g in enumerate(buf):
            g.copy_(torch.from_numpy(np.random.default_rng([17, i, t]).standard_normal(g.numel())
                                     .astype(np.float32) * 1e-3))
            pa[i].grad = g
            pb[i].grad = g
        say(f"optim 12 groups step {t}")
        opt_a.step()
        opt_b.step()
        torch.cuda.synchronize()
        if t > 2:
            assert set(opt_a._plans) == set(seen), "a plan was built again"
        for key, plan in opt_a._plans.items():
            assert seen.setdefault(key, plan) is plan
        for p, q in zip(pa, pb):
            sa, sb = opt_a.state[p], opt_b.state[q]
            for k in ("state1", "absmax1", "state2", "absmax2"):
                assert torch.equal(sa[k], sb[k]), (t, k)
            assert torch.all((p - q).abs() <= 1e-6 * p.abs() + 1e-8)
    assert len(opt_a._plans) == 2 * ngroups
