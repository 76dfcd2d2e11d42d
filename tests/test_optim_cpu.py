"""Host-side behaviour of the drop-in optimizers (no GPU needed)."""
from __future__ import annotations

import pytest
import torch

from paper_2110_02861_amd import optim


def test_hyperparameter_checks():
    p = [torch.nn.Parameter(torch.zeros(4))]
    with pytest.raises(ValueError):
        optim.Adam8bit(p, lr=-1.0)
    with pytest.raises(ValueError):
        optim.Adam8bit(p, betas=(0.9, 1.0))
    with pytest.raises(ValueError):
        optim.AdamW8bit(p, eps=-1e-8)
    with pytest.raises(ValueError):
        optim.SGD8bit(p, momentum=1.5)
    with pytest.raises(ValueError):
        optim.Adam8bit(p, blocksize=1000)
    with pytest.raises(ValueError):
        optim.Adam8bit(p, min_8bit_size=-1)
    with pytest.raises(ValueError, match="plans"):
        optim.Adam8bit(p, capturable=True, use_plans=False)


def test_defaults_follow_torch():
    p = [torch.nn.Parameter(torch.zeros(4))]
    a = optim.Adam8bit(p)
    assert a.defaults == dict(lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.0)
    w = optim.AdamW8bit(p)
    assert w.defaults["weight_decay"] == 1e-2
    s = optim.SGD8bit(p, lr=0.1)
    assert s.defaults == dict(lr=0.1, momentum=0.9, weight_decay=0.0)
    assert a.blocksize == 2048 and a.min_8bit_size == 0 and a.use_plans
    lamb = optim.Lamb8bit(p, weight_decay=0.01)
    assert lamb._hparams(lamb.param_groups[0], 1) == dict(lr=1e-3, beta1=0.9, beta2=0.999,
                                                          eps=1e-6, wd=0.01, step=1)
    lars = optim.Lars8bit(p, lr=0.2)
    assert lars._hparams(lars.param_groups[0], 4) == dict(lr=0.2, beta1=0.9, beta2=0.0, eps=0.0,
                                                          wd=0.0, step=4, trust=1e-3)
    with pytest.raises(ValueError):
        optim.Lars8bit(p, trust_coefficient=0.0)
    g = optim.Adagrad8bit(p)
    assert g.defaults == dict(lr=1e-2, eps=1e-10, weight_decay=0.0)
    assert g._hparams(g.param_groups[0], 2) == dict(lr=1e-2, beta1=0.0, beta2=0.0, eps=1e-10,
                                                    wd=0.0, step=2)


def test_cpu_tensors_fail_loudly():
    """No CPU fallback: a step on CPU params raises instead of computing."""
    m = torch.nn.Linear(4, 3)
    opt = optim.Adam8bit(m.parameters())
    m(torch.randn(2, 4)).sum().backward()
    with pytest.raises(TypeError, match="GPU"):
        opt.step()


def test_hparams_per_group():
    a = torch.nn.Parameter(torch.zeros(4))
    b = torch.nn.Parameter(torch.zeros(4))
    opt = optim.Adam8bit([{"params": [a]}, {"params": [b], "lr": 5e-4, "betas": (0.8, 0.99)}],
                         weight_decay=0.1)
    h0 = opt._hparams(opt.param_groups[0], 3)
    h1 = opt._hparams(opt.param_groups[1], 7)
    assert h0 == dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.1, step=3)
    assert h1 == dict(lr=5e-4, beta1=0.8, beta2=0.99, eps=1e-8, wd=0.1, step=7)
    sgd = optim.SGD8bit([a], lr=0.2, momentum=0.5, weight_decay=1e-4)
    assert sgd._hparams(sgd.param_groups[0], 1) == dict(lr=0.2, beta1=0.5, beta2=0.0, eps=0.0,
                                                        wd=1e-4, step=1)


class _FakePlan:
    """Stands in for a step plan: records whether it was closed."""

    def __init__(self):
        self.closed = False

    def close(self):
        self.closed = True


def test_load_state_dict_retires_plans_a_graph_reads():
    """Plans used under capture are not freed by load_state_dict (a graph
    captured before it may still replay them); release_graph_memory() frees
    them, and frees pinned plans still in the cache."""
    p = torch.nn.Parameter(torch.zeros(4096))
    opt = optim.Adam8bit([p], capturable=True)
    pinned, free, pinned_later = _FakePlan(), _FakePlan(), _FakePlan()
    opt._plans = {("a",): pinned, ("b",): free}
    opt._pinned = {("a",)}
    hp = torch.zeros(48, dtype=torch.uint8)
    opt._hp_dev = {(0, 1, 0): (hp, [p])}
    opt.state[p] = {"step": 3, "state1": torch.zeros(4096, dtype=torch.uint8)}
    old_state1 = opt.state[p]["state1"]
    sd = torch.optim.Optimizer.state_dict(opt)
    opt.load_state_dict(sd)
    assert free.closed and not pinned.closed
    assert opt._plans == {} and opt._pinned == set() and opt._hp_dev == {}
    assert pinned in opt._retired
    assert any(isinstance(r, tuple) and r[0] is hp for r in opt._retired)
    assert any(isinstance(r, dict) and r.get("state1") is old_state1 for r in opt._retired)
    # a later capture pins another plan in the cache
    opt._plans = {("c",): pinned_later}
    opt._pinned = {("c",)}
    opt.release_graph_memory()
    assert pinned.closed and pinned_later.closed
    assert opt._retired == [] and opt._pinned == set() and opt._plans == {}


def test_load_state_dict_without_capture_closes_every_plan():
    p = torch.nn.Parameter(torch.zeros(4096))
    opt = optim.Adam8bit([p])
    a, b = _FakePlan(), _FakePlan()
    opt._plans = {("a",): a, ("b",): b}
    opt.load_state_dict(torch.optim.Optimizer.state_dict(opt))
    assert a.closed and b.closed and opt._retired == []
