"""Shared helpers for the GPU parity tests (HIP path vs the CPU oracle)."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2110_02861_amd import bq

needs_gpu = pytest.mark.skipif(not torch.cuda.is_available(), reason="no GPU visible")

OPT_ID = {"adam": oracle.ADAM, "adamw": oracle.ADAMW, "momentum": oracle.MOMENTUM,
          "adagrad": oracle.ADAGRAD, "lamb": oracle.LAMB, "lars": oracle.LARS}


def say(*a):
    """Name the case before a GPU step, flushed, so a crash log shows it."""
    print("[gpu]", *a, flush=True)
    sys.stdout.flush()


def dev(x: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def codebooks_on_device():
    qs = bq.bq_make_dynamic_codebook(bq.BQ_SIGNED)
    qu = bq.bq_make_dynamic_codebook(bq.BQ_UNSIGNED)
    return qs, qu, dev(qs), dev(qu)


def param_close(got, ref, tol_extra):
    """|got - ref| <= 1e-6 |ref| + tol_extra, elementwise; returns (ok, worst excess).

    tol_extra carries the update-relative part of the bound (HostState.tol for a
    free-running comparison, 1e-6 |update| for a single step from one state).
    """
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    tol = 1e-6 * np.abs(ref) + tol_extra
    d = np.abs(got - ref)
    return bool(np.all(d <= tol)), float(np.max(d - tol)) if d.size else 0.0


def codes_agree(got, ref, min_frac=0.9999):
    """State codes: identical on >= 99.99% of elements (a single mismatch is
    allowed in a tensor too small for that fraction), others off by one."""
    got = got.astype(np.int32)
    ref = ref.astype(np.int32)
    diff = np.abs(got - ref)
    n = max(1, got.size)
    bad = np.count_nonzero(diff)
    frac = 1.0 - bad / n
    ok = diff.max(initial=0) <= 1 and (frac >= min_frac or bad <= 1)
    return bool(ok), frac, int(diff.max(initial=0))


class HostState:
    """Oracle-side copy of one tensor's param and 8-bit states.

    tol accumulates the free-running param bound: per step, 1e-6 of the
    oracle's update |w_prev - w| (the HIP path takes the hardware square root
    and reciprocal, a few ulp of the update) plus one rounding 2^-23 |w|."""

    def __init__(self, w, B, two):
        n = w.size
        nb = (n + B - 1) // B
        self.w = w.copy()
        self.c1 = np.full(n, 127, np.uint8)
        self.a1 = np.zeros(nb, np.float32)
        self.c2 = np.zeros(n, np.uint8) if two else None
        self.a2 = np.zeros(nb, np.float32) if two else None
        self.tol = np.zeros(n, np.float64)
        self.step_tol = np.zeros(n, np.float64)

    def step(self, opt, B, g, q1, q2, hp, t):
        prev = self.w.astype(np.float64)
        oracle.step8(OPT_ID[opt], B, self.w, g, self.c1, self.a1, q1, self.c2, self.a2, q2,
                     hp["lr"], hp["beta1"], hp.get("beta2", 0.0), hp.get("eps", 0.0),
                     hp.get("wd", 0.0), t, trust=hp.get("trust", 0.0))
        upd = np.abs(prev - self.w.astype(np.float64))
        self.step_tol = 1e-6 * upd
        self.tol += 1e-6 * upd + 2.0 ** -23 * np.abs(self.w.astype(np.float64))


class DevState:
    """GPU copy of one tensor's param and 8-bit states (zero state)."""

    def __init__(self, w, B, two, grad_dtype):
        n = w.size
        nb = (n + B - 1) // B
        self.w = dev(w)
        self.c1 = torch.full((n,), 127, dtype=torch.uint8, device="cuda")
        self.a1 = torch.zeros(nb, dtype=torch.float32, device="cuda")
        self.c2 = torch.zeros(n, dtype=torch.uint8, device="cuda") if two else None
        self.a2 = torch.zeros(nb, dtype=torch.float32, device="cuda") if two else None
        self.g = torch.empty(n, dtype=grad_dtype, device="cuda")

    def row(self):
        return (self.w, self.g, self.c1, self.c2, self.a1, self.a2)

    def load(self, h: "HostState"):
        """Overwrite param and states with the oracle's (oracle -> GPU only)."""
        self.w.copy_(torch.from_numpy(h.w))
        self.c1.copy_(torch.from_numpy(h.c1))
        self.a1.copy_(torch.from_numpy(h.a1))
        if self.c2 is not None:
            self.c2.copy_(torch.from_numpy(h.c2))
            self.a2.copy_(torch.from_numpy(h.a2))
