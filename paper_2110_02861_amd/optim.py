"""Drop-in PyTorch optimizers with 8-bit block-wise states, over libbq.

The paper's 8-bit optimizers replace their 32-bit counterparts without
hyperparameter changes (Section 1, Section 4): Adam (Eq. 2 with bias
correction), AdamW, SGD with momentum (Eq. 1), and AdaGrad (App. H); LAMB and
LARS, whose 8-bit versions App. E times, in their textbook forms (per-tensor
trust ratios, which need a norm pass and therefore step plans).  Each state is
stored as one uint8 code per element plus one fp32 absmax per block of
``blocksize`` elements (Section 3.1); the signed dynamic map holds the first
state and the unsigned dynamic map the second (Section 3.2); AdaGrad's single,
non-negative state (the running sum of squared gradients) uses the unsigned
map.  Tensors can keep 32-bit states instead: Section 3.3 keeps the embedding
layer's states in 32 bit (``override_32bit``, or the weight of
``nn.StableEmbedding``), and tensors below ``min_8bit_size`` elements may be
exempted as well.

Every update runs in the HIP kernels of libbq:
- 8-bit tensors go through a step plan (``bq_step_plan_run_prepared``: one
  launch over every tile of every tensor, with the fixed maps' decision tables
  prepared once per device), looked up by every storage pointer and size, or
  through ``bq_optimizer8bit_step`` when ``use_plans=False``; with
  ``capturable=True`` through ``bq_step_plan_run_device``, whose
  hyperparameters and step count live in device memory, so that ``step()``
  can be captured into a HIP graph (after one eager step) and replayed as
  successive steps;
- 32-bit tensors go through ``bq_optimizer32bit_step``.

Params must be fp32 CUDA tensors, contiguous and 16-byte aligned; grads fp32,
fp16 or bf16 of the same shape.  ``state_dict`` / ``load_state_dict`` carry the codes,
the absmax arrays and the step count of every tensor.

Graphs (``capturable=True``): a captured ``step()`` reads device memory that
the optimizer owns -- the step plans it ran, the device hyperparameters and
the state tensors.  The optimizer therefore never frees what a capture used
on its own: plans used under capture are never evicted, and
``load_state_dict`` moves them, the device hyperparameters and the replaced
state tensors to a retired list instead of freeing them.  A graph captured
before ``load_state_dict`` keeps replaying harmlessly into that retired
memory (it no longer updates the loaded states): capture again after a load.
Each capture on new grad storages pins one more plan; once every graph that
replays this optimizer's step has been dropped, ``release_graph_memory()``
frees all of it.
"""
from __future__ import annotations

import numpy as np
import torch

from . import bq

_CODEBOOKS: dict = {}


def dynamic_codebooks(device: torch.device):
    """(signed map, unsigned map) as fp32 device tensors, built once per device."""
    key = (device.type, device.index)
    if key not in _CODEBOOKS:
        qs = bq.bq_make_dynamic_codebook(bq.BQ_SIGNED)
        qu = bq.bq_make_dynamic_codebook(bq.BQ_UNSIGNED)
        _CODEBOOKS[key] = (torch.from_numpy(qs).to(device), torch.from_numpy(qu).to(device),
                           int(np.flatnonzero(qs == 0.0)[0]), int(np.flatnonzero(qu == 0.0)[0]))
    return _CODEBOOKS[key]


_GRAD_DTYPES = {torch.float32: bq.BQ_F32, torch.float16: bq.BQ_F16, torch.bfloat16: bq.BQ_BF16}

_PREPARED: dict = {}


def prepared_codebooks(device: torch.device, state1_unsigned: bool, two_states: bool):
    """The decision tables of an optimizer's fixed maps, prepared once per
    device and map pair (bq.prepare_codebook_pair) for plan runs."""
    key = (device.type, device.index, state1_unsigned, two_states)
    if key not in _PREPARED:
        qs, qu, _, _ = dynamic_codebooks(device)
        q1 = qu if state1_unsigned else qs
        prepared = bq.prepare_codebook_pair(q1, qu if two_states else None)
        # the tables are read later from whatever stream steps run on
        torch.cuda.current_stream(device).synchronize()
        _PREPARED[key] = prepared
    return _PREPARED[key]


class Optimizer8bit(torch.optim.Optimizer):
    """Base class: state management, grouping, kernel dispatch."""

    OPT: int = -1  # bq.BQ_ADAM / BQ_ADAMW / BQ_MOMENTUM
    MAX_PLANS = 8  # cached step plans per optimizer (one per param subset)

    def __init__(self, params, defaults: dict, blocksize: int = 2048, min_8bit_size: int = 0,
                 use_plans: bool = True, capturable: bool = False):
        if blocksize not in (256, 512, 1024, 2048, 4096):
            raise ValueError(f"blocksize must be a power of two in [256, 4096], got {blocksize}")
        if min_8bit_size < 0:
            raise ValueError("min_8bit_size must be >= 0")
        if capturable and not use_plans:
            raise ValueError("capturable steps run through step plans (use_plans=True)")
        self.blocksize = int(blocksize)
        self.min_8bit_size = int(min_8bit_size)
        self.use_plans = bool(use_plans)
        # capturable: the hyperparameters and step count of every (group, grad
        # dtype, device) bucket live in device memory (bq.device_hparams) and
        # every step advances the count there, so a captured step() replays as
        # successive steps
        self.capturable = bool(capturable)
        self._override32: set = set()
        self._plans: dict = {}
        self._pinned: set = set()  # keys of plans used under graph capture: never evicted
        # plans, device hyperparameters and state tensors that graphs captured
        # before a load_state_dict may still read: freed by
        # release_graph_memory() or with the optimizer
        self._retired: list = []
        self._hp_dev: dict = {}  # (group, grad dtype, device) -> (device hparams, params)
        # group index -> the last two steps' params, grad storages, pointers
        # and launches; a step equal to one of them replays its launches
        self._fast: dict = {}
        super().__init__(params, defaults)

    # -- configuration --------------------------------------------------------

    def override_32bit(self, param: torch.Tensor) -> None:
        """Keep this param's states in 32 bit (e.g. an embedding layer, Section
        3.3).  Call before the param's first step."""
        if param in self.state and self.state[param]:
            raise RuntimeError("override_32bit must be called before the param's first step")
        self._override32.add(id(param))

    def _is_8bit(self, p: torch.Tensor) -> bool:
        # a weight flagged bq_32bit_state (nn.StableEmbedding) keeps 32-bit states
        return (id(p) not in self._override32 and not getattr(p, "bq_32bit_state", False)
                and p.numel() >= self.min_8bit_size)

    # -- hyperparameters of one group (subclasses) ------------------------------

    def _hparams(self, group: dict, step: int) -> dict:
        raise NotImplementedError

    @property
    def _two_states(self) -> bool:
        return self.OPT in (bq.BQ_ADAM, bq.BQ_ADAMW, bq.BQ_LAMB)

    @property
    def _state1_unsigned(self) -> bool:
        return self.OPT == bq.BQ_ADAGRAD

    def _maps(self, device):
        """(state-1 map, state-2 map or None, state-1 zero code, state-2 zero code)."""
        qs, qu, zs, zu = dynamic_codebooks(device)
        if self._state1_unsigned:
            return qu, None, zu, zu
        return qs, (qu if self._two_states else None), zs, zu

    # -- state ------------------------------------------------------------------

    def _init_state(self, p: torch.Tensor, state: dict) -> None:
        state["step"] = 0
        if self.OPT in (bq.BQ_LAMB, bq.BQ_LARS) and not self._is_8bit(p):
            raise NotImplementedError("LAMB / LARS keep 8-bit states only (no 32-bit override)")
        if self._is_8bit(p):
            _, _, z1, z2 = self._maps(p.device)
            nb = (p.numel() + self.blocksize - 1) // self.blocksize
            state["state1"] = torch.full((p.numel(),), z1, dtype=torch.uint8, device=p.device)
            state["absmax1"] = torch.zeros(nb, dtype=torch.float32, device=p.device)
            if self._two_states:
                state["state2"] = torch.full((p.numel(),), z2, dtype=torch.uint8, device=p.device)
                state["absmax2"] = torch.zeros(nb, dtype=torch.float32, device=p.device)
        else:
            state["exp_avg"] = torch.zeros(p.numel(), dtype=torch.float32, device=p.device)
            if self._two_states:
                state["exp_avg_sq"] = torch.zeros(p.numel(), dtype=torch.float32,
                                                  device=p.device)

    @staticmethod
    def _check_param(p: torch.Tensor, g: torch.Tensor) -> None:
        # each attribute read once: this runs for every param on every step
        if not p.is_cuda:
            raise TypeError("8-bit optimizers need GPU tensors (libbq runs on the GPU only)")
        if p.dtype is not torch.float32:
            raise TypeError(f"params must be fp32, got {p.dtype}")
        if not p.is_contiguous():
            raise ValueError("params must be contiguous")
        if g.layout is not torch.strided:
            raise TypeError("sparse gradients are not supported")
        gd = g.dtype
        if gd is not torch.float32 and gd is not torch.float16 and gd is not torch.bfloat16:
            raise TypeError(f"grads must be fp32, fp16 or bf16, got {gd}")
        if g.numel() != p.numel() or not g.is_contiguous():
            raise ValueError("grads must be contiguous and shaped like their params")

    # -- the step -----------------------------------------------------------------

    @torch.no_grad()
    def step(self, closure=None):
        capturing = torch.cuda.is_available() and torch.cuda.is_current_stream_capturing()
        if capturing and not self.capturable:
            # the step count and hyperparameters travel as launch arguments: a
            # replayed graph would repeat the captured step's bias correction
            raise RuntimeError("8-bit optimizer steps cannot be captured into a graph unless the "
                               "optimizer is built with capturable=True (hyperparameters and "
                               "step count in device memory)")
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        fast = self.use_plans and not self.capturable
        for gi, group in enumerate(self.param_groups):
            if fast and self._replay(gi, group):
                continue
            # one pass over the params, bucketed by (8-bit, grad dtype, step,
            # device); every launch then covers one bucket
            buckets: dict = {}
            entries = []
            for p in group["params"]:
                g = p.grad
                if g is None:
                    continue
                self._check_param(p, g)
                state = self.state[p]
                if not state:
                    if capturing:
                        raise RuntimeError("run one step outside graph capture first: it "
                                           "creates the optimizer states and step plans")
                    self._init_state(p, state)
                dev = p.get_device()
                # the states were sized and placed for the param when they were made
                s1 = state.get("state1")
                if s1 is None:
                    s1 = state["exp_avg"]
                if s1.numel() != p.numel() or s1.get_device() != dev:
                    raise ValueError("a param changed size or device after its optimizer state "
                                     "was created")
                if self.capturable:
                    if "state1" not in state:
                        raise ValueError("capturable optimizers keep every state in 8 bit "
                                         "(no override_32bit, min_8bit_size or stable embedding)")
                    # the device count is the step; the host count follows it
                    # at eager steps and in state_dict()
                    step = 0
                    if not capturing:
                        state["step"] += 1
                else:
                    step = state["step"] + 1
                    state["step"] = step
                key = ("state1" in state, g.dtype, step, dev)
                items = buckets.get(key)
                if items is None:
                    buckets[key] = items = []
                items.append((p, g, state))
                if fast:
                    entries.append((p, state, s1, p.data_ptr(), g.data_ptr(), g.dtype,
                                    p.numel()))
            launches = []
            for (eight, gdtype, step, _), items in buckets.items():
                gdt = _GRAD_DTYPES[gdtype]
                device = items[0][0].device
                if self.capturable:
                    hp_dev = self._device_hparams(gi, group, gdt, device, items, capturing)
                    self._step8(gdt, device, items, None, hp_dev, capturing)
                    continue
                hp = self._hparams(group, step)
                if eight:
                    plan = self._step8(gdt, device, items, hp)
                    launches.append((plan, gdt, items[0][2], device))
                else:
                    rows = [(p, g, s["exp_avg"], s.get("exp_avg_sq")) for p, g, s in items]
                    bq.bq_optimizer32bit_step(self.OPT, gdt, rows, hp)
                    # params and states only: a record holds no grad
                    launches.append(([(p, s) for p, _, s in items], gdt, items[0][2], None))
            if fast:
                # most recent first; two serve alternating grad buffers
                self._fast[gi] = [(entries, launches)] + self._fast.get(gi, [])[:1]
        return loss

    def _replay(self, gi: int, group: dict) -> bool:
        """Repeat one of group gi's last two steps if this step is the same:
        the same params, each with a grad at the same storage (pointer, dtype,
        size, dense and contiguous), and the same param storages and state
        tensors.  The checks, buckets and plan lookups of that step then still
        hold, and only the step counts advance.  Returns False, having changed
        nothing, otherwise."""
        for entries, launches in self._fast.get(gi, ()):
            if self._same_step(group, entries) and all(
                    device is None or what.is_open() for what, _, _, device in launches):
                break
        else:
            return False
        for e in entries:
            e[1]["step"] += 1
        for what, gdt, ref, device in launches:
            hp = self._hparams(group, ref["step"])
            if device is None:
                rows = [(p, p.grad, s["exp_avg"], s.get("exp_avg_sq")) for p, s in what]
                bq.bq_optimizer32bit_step(self.OPT, gdt, rows, hp)
            else:
                what.run_prepared(hp, prepared_codebooks(device, self._state1_unsigned,
                                                         self._two_states))
        return True

    @staticmethod
    def _same_step(group: dict, entries) -> bool:
        n = len(entries)
        i = 0
        for p in group["params"]:
            g = p.grad
            if g is None:
                continue
            if i == n:
                return False
            q, state, s1, pp, gp, gdtype, numel = entries[i]
            if q is not p or p.data_ptr() != pp or g.dtype is not gdtype:
                return False
            if g.layout is not torch.strided or g.data_ptr() != gp:
                return False
            if g.numel() != numel or p.numel() != numel or not g.is_contiguous():
                return False
            if state.get("state1", state.get("exp_avg")) is not s1:
                return False
            i += 1
        return i == n

    def _device_hparams(self, gi, group, gdt, device, items, capturing):
        """The device hyperparameters of one bucket: made at its first step
        (from the host step count, which the run then advances), refreshed
        from the group at every eager step except for the step count."""
        key = (gi, gdt, device.index)
        entry = self._hp_dev.get(key)
        steps = {s["step"] for _, _, s in items}
        if entry is None:
            if capturing:
                raise RuntimeError("run one step outside graph capture first: it creates the "
                                   "device hyperparameters")
            if len(steps) != 1:
                raise RuntimeError("params of one capturable bucket must share their step count")
            t = bq.device_hparams(self._hparams(group, steps.pop() - 1), device)
            self._hp_dev[key] = (t, [p for p, _, _ in items])
            return t
        t, params = entry
        if len(items) != len(params) or any(p is not q for (p, _, _), q in zip(items, params)):
            raise RuntimeError("a capturable optimizer steps the same params every time")
        if not capturing:
            self._refresh(t, group)
        return t

    def _refresh(self, t, group) -> None:
        """Copy a group's hyperparameters, but not the step count, to t."""
        new = bq.device_hparams(self._hparams(group, 0), t.device)
        t[:20].copy_(new[:20])   # lr, beta1, beta2, eps, weight_decay
        t[32:].copy_(new[32:])   # trust coefficient (and padding)

    def update_device_hparams(self) -> None:
        """Capturable optimizers: copy every group's hyperparameters (e.g. a new
        lr) to device memory, for graph replays that run no eager step.  Not
        under capture."""
        for (gi, _, _), (t, _) in self._hp_dev.items():
            self._refresh(t, self.param_groups[gi])

    def _sync_steps(self) -> None:
        """Capturable optimizers: the host step counts from device memory."""
        for t, params in self._hp_dev.values():
            step = bq.read_device_hparams(t)["step"]
            for p in params:
                if self.state.get(p):
                    self.state[p]["step"] = step

    def state_dict(self):
        if self._hp_dev:
            self._sync_steps()
        return super().state_dict()

    def _step8(self, gdt: int, device, items, hp, hp_dev=None, capturing=False) -> None:
        rows = []
        key = [gdt, device.index]
        for p, g, s in items:
            s1, s2, a1, a2 = s["state1"], s.get("state2"), s["absmax1"], s.get("absmax2")
            n = p.numel()
            rows.append((p, g, s1, s2, a1, a2))
            key += (p.data_ptr(), g.data_ptr(), s1.data_ptr(), a1.data_ptr(),
                    0 if s2 is None else s2.data_ptr(), 0 if a2 is None else a2.data_ptr(), n)
        if not self.use_plans and self.OPT not in (bq.BQ_LAMB, bq.BQ_LARS):
            q1, q2, _, _ = self._maps(device)
            bq.bq_optimizer8bit_step(self.OPT, self.blocksize, gdt, rows, hp, q1, q2)
            return None
        # A plan holds device pointers and is a function of them and the sizes
        # alone: look it up by every storage pointer and size, so a plan runs
        # only on the storages it was built for.  Plans keep no references to
        # the tensors, so grads freed by zero_grad(set_to_none=True) can be
        # reallocated at the same addresses (and the plan reused); several
        # plans per param set serve alternating grad buffers.
        key = tuple(key)
        plan = self._plans.pop(key, None)
        if plan is None:
            if capturing:
                raise RuntimeError("no step plan for these tensors: run one step outside graph "
                                   "capture with the same grad tensors first")
            plan = bq.StepPlan(self.OPT, self.blocksize, gdt, rows, keep=False)
        self._plans[key] = plan  # most recently used last
        if capturing:
            self._pinned.add(key)  # a captured graph reads this plan's memory
        # at least MAX_PLANS, and room for two grad buffers per param group and
        # grad dtype, so that a step never evicts a plan it is about to reuse
        cap = max(self.MAX_PLANS, 4 * len(self.param_groups))
        while len(self._plans) - len(self._pinned) > cap:
            oldest = next(k for k in self._plans if k not in self._pinned)
            self._plans.pop(oldest).close()
            self._fast = {}  # a remembered step may hold the closed plan
        prepared = prepared_codebooks(device, self._state1_unsigned, self._two_states)
        if hp_dev is not None:
            plan.run_device(hp_dev, prepared, advance=True)
        else:
            plan.run_prepared(hp, prepared)
        return plan

    def load_state_dict(self, state_dict):
        """Load states; plans are made again.  Plans a captured graph used,
        the device hyperparameters and (when anything was captured) the
        replaced state tensors are retired, not freed: graphs captured
        before the load replay into them and must be captured again."""
        for key, plan in self._plans.items():
            if key in self._pinned:
                self._retired.append(plan)
            else:
                plan.close()
        if self._pinned or self._hp_dev:
            self._retired.extend(self._hp_dev.values())
            self._retired.extend(dict(s) for s in self.state.values())
        self._plans = {}
        self._pinned = set()
        self._hp_dev = {}  # made again from the loaded step counts
        self._fast = {}
        super().load_state_dict(state_dict)
        # torch casts every non-step state tensor to the param's dtype; the
        # codes (0..255) come through fp32 exactly and go back to uint8
        for s in self.state.values():
            for k in ("state1", "state2"):
                if k in s:
                    s[k] = s[k].to(torch.uint8)

    def release_graph_memory(self) -> None:
        """Free every plan pinned by graph capture and everything retired by
        ``load_state_dict``.  Call only once no captured graph that replays
        this optimizer's step is left: a replay afterwards would read freed
        device memory.  Later captures pin plans again."""
        for key in list(self._pinned):
            plan = self._plans.pop(key, None)
            if plan is not None:
                plan.close()
        self._pinned = set()
        for item in self._retired:
            if hasattr(item, "close"):  # a plan; tensors are dropped with the list
                item.close()
        self._retired = []
        self._fast = {}


class Adam8bit(Optimizer8bit):
    """Adam with 8-bit states (Eq. 2 with bias correction).  weight_decay adds
    an L2 term to the gradient, as torch.optim.Adam does."""

    OPT = bq.BQ_ADAM

    def __init__(self, params, lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.0,
                 **kw):
        _check_hparams(lr, betas, eps, weight_decay)
        super().__init__(params, dict(lr=lr, betas=tuple(betas), eps=eps,
                                      weight_decay=weight_decay), **kw)

    def _hparams(self, group, step):
        b1, b2 = group["betas"]
        return dict(lr=group["lr"], beta1=b1, beta2=b2, eps=group["eps"],
                    wd=group["weight_decay"], step=step)


class AdamW8bit(Adam8bit):
    """AdamW with 8-bit states: decoupled decay w *= 1 - lr * weight_decay,
    then the Adam update, as torch.optim.AdamW."""

    OPT = bq.BQ_ADAMW

    def __init__(self, params, lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=1e-2, **kw):
        super().__init__(params, lr=lr, betas=betas, eps=eps, weight_decay=weight_decay, **kw)


class SGD8bit(Optimizer8bit):
    """SGD with momentum and an 8-bit momentum buffer (Eq. 1): m = beta m + g,
    w -= lr m, with weight_decay as an L2 term; torch.optim.SGD with
    dampening 0 and nesterov False."""

    OPT = bq.BQ_MOMENTUM

    def __init__(self, params, lr=1e-2, momentum=0.9, weight_decay=0.0, **kw):
        if lr < 0.0:
            raise ValueError(f"invalid learning rate {lr}")
        if not 0.0 <= momentum < 1.0:
            raise ValueError(f"invalid momentum {momentum}")
        if weight_decay < 0.0:
            raise ValueError(f"invalid weight_decay {weight_decay}")
        super().__init__(params, dict(lr=lr, momentum=momentum, weight_decay=weight_decay), **kw)

    def _hparams(self, group, step):
        return dict(lr=group["lr"], beta1=group["momentum"], beta2=0.0, eps=0.0,
                    wd=group["weight_decay"], step=step)


class Adagrad8bit(Optimizer8bit):
    """AdaGrad with an 8-bit sum of squared gradients (App. H): r += g^2,
    w -= lr g / (sqrt(r) + eps), weight_decay as an L2 term; torch.optim.Adagrad
    with lr_decay 0 and initial_accumulator_value 0."""

    OPT = bq.BQ_ADAGRAD

    def __init__(self, params, lr=1e-2, eps=1e-10, weight_decay=0.0, **kw):
        _check_hparams(lr, (0.0, 0.0), eps, weight_decay)
        super().__init__(params, dict(lr=lr, eps=eps, weight_decay=weight_decay), **kw)

    def _hparams(self, group, step):
        return dict(lr=group["lr"], beta1=0.0, beta2=0.0, eps=group["eps"],
                    wd=group["weight_decay"], step=step)


class Lamb8bit(Optimizer8bit):
    """LAMB with 8-bit states: the Adam direction u = mhat / (sqrt(vhat) + eps)
    + weight_decay w, scaled per tensor by |w| / |u| (1 if either is zero):
    w -= lr |w| / |u| u.  Runs through step plans (a norm pass, then the step)."""

    OPT = bq.BQ_LAMB

    def __init__(self, params, lr=1e-3, betas=(0.9, 0.999), eps=1e-6, weight_decay=0.0, **kw):
        _check_hparams(lr, betas, eps, weight_decay)
        super().__init__(params, dict(lr=lr, betas=tuple(betas), eps=eps,
                                      weight_decay=weight_decay), **kw)

    def _hparams(self, group, step):
        b1, b2 = group["betas"]
        return dict(lr=group["lr"], beta1=b1, beta2=b2, eps=group["eps"],
                    wd=group["weight_decay"], step=step)


class Lars8bit(Optimizer8bit):
    """LARS with an 8-bit momentum buffer: per tensor the local rate
    trust_coefficient |w| / (|g| + weight_decay |w|) (1 if a norm is zero);
    m = momentum m + lr rate (g + weight_decay w); w -= m.  Runs through step
    plans (a norm pass, then the step)."""

    OPT = bq.BQ_LARS

    def __init__(self, params, lr=0.1, momentum=0.9, weight_decay=0.0, trust_coefficient=1e-3,
                 **kw):
        if lr < 0.0:
            raise ValueError(f"invalid learning rate {lr}")
        if not 0.0 <= momentum < 1.0:
            raise ValueError(f"invalid momentum {momentum}")
        if weight_decay < 0.0 or trust_coefficient <= 0.0:
            raise ValueError("invalid weight_decay or trust_coefficient")
        super().__init__(params, dict(lr=lr, momentum=momentum, weight_decay=weight_decay,
                                      trust_coefficient=trust_coefficient), **kw)

    def _hparams(self, group, step):
        return dict(lr=group["lr"], beta1=group["momentum"], beta2=0.0, eps=0.0,
                    wd=group["weight_decay"], step=step, trust=group["trust_coefficient"])


def _check_hparams(lr, betas, eps, weight_decay):
    if lr < 0.0:
        raise ValueError(f"invalid learning rate {lr}")
    if len(betas) != 2 or not all(0.0 <= b < 1.0 for b in betas):
        raise ValueError(f"invalid betas {betas}")
    if eps < 0.0:
        raise ValueError(f"invalid eps {eps}")
    if weight_decay < 0.0:
        raise ValueError(f"invalid weight_decay {weight_decay}")
