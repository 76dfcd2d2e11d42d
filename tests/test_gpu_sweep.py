"""Seeded sweeps over random configurations against the oracle: for the step,
optimizer, grad dtype, blocksize, path, codebook family, weight decay and a
ragged tensor list, two steps each; for quantize / dequantize (both quantize
paths), length, blocksize, codebook and blocks of differing character.

Every case is drawn from a fixed seed, so the sweep is the same on every run;
it looks for interactions that the per-parameter grids elsewhere do not reach.
Codes and absmax are compared bit for bit, except where the param feeds back
into a state (Momentum and LARS fold w into the gradient): there a param that
differs by an ulp after step 1 may move a state across a code boundary at step
2, so codes must agree on 99.99 % and differ by at most one.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2110_02861_amd import bq
from tests.gpu_helpers import codebooks_on_device, needs_gpu
from tests.test_gpu_quant import _other_maps, run_pair
from tests.test_gpu_step import HPS, _map_families, run_lists

pytestmark = [pytest.mark.gpu, needs_gpu]

OPTS = ["adam", "adamw", "momentum", "adagrad", "lamb", "lars"]
GRADS = [bq.BQ_F16, bq.BQ_F32, bq.BQ_BF16]
BLOCKS = [256, 512, 1024, 2048, 4096]
FAMILIES = [None, "inverse_dynamic", "linear", "quantile"]
NCASES = 40


def _cases():
    rng = np.random.default_rng(20211005)
    out = []
    for k in range(NCASES):
        opt = OPTS[rng.integers(len(OPTS))]
        gdt = GRADS[rng.integers(len(GRADS))]
        B = BLOCKS[rng.integers(len(BLOCKS))]
        paths = ["plan", "prepared"] + ([] if opt in ("lamb", "lars") else ["call"])
        path = paths[rng.integers(len(paths))]
        family = FAMILIES[rng.integers(len(FAMILIES))]
        # ragged sizes around the block and tile edges, and a few larger tensors
        sizes = []
        for _ in range(int(rng.integers(1, 9))):
            kind = rng.integers(4)
            if kind == 0:
                sizes.append(int(rng.integers(1, B + 2)))
            elif kind == 1:
                sizes.append(int(B * rng.integers(1, 5) + rng.integers(-1, 2)))
            elif kind == 2:
                sizes.append(int(rng.integers(1, 3 * 4096 + 5)))
            else:
                sizes.append(int(rng.integers(20_000, 70_000)))
        hp = dict(HPS[opt])
        if opt in ("adam", "momentum", "lamb", "lars") and rng.random() < 0.5:
            hp["wd"] = 0.0
        seed = int(rng.integers(1 << 30))
        out.append(pytest.param(opt, gdt, B, path, family, sizes, hp, seed,
                                id=f"{k:02d}-{opt}-{['f32', 'f16', 'bf16'][gdt]}-B{B}-{path}-"
                                   f"{family or 'dynamic'}"))
    return out


@pytest.mark.parametrize("opt,gdt,B,path,family,sizes,hp,seed", _cases())
def test_random_configuration(opt, gdt, B, path, family, sizes, hp, seed):
    maps = None
    if family is not None:
        q1, q2 = _map_families()[family]
        maps = (q2, q2) if opt == "adagrad" else (q1, q2)  # AdaGrad's state is non-negative
    # Adam's L2 term, Momentum's and LARS's decay put w into the state update
    feedback = hp["wd"] != 0.0 and opt in ("adam", "momentum", "lars")
    run_lists(opt, B, gdt, sizes, steps=2, seed=seed, hp=hp, exact_codes=not feedback,
              path=path, maps=maps)


# --- standalone quantize / dequantize ------------------------------------------

QMAPS = ["signed", "unsigned", "inverse_signed", "inverse_unsigned", "linear_signed",
         "linear_unsigned", "quantile_normal", "quantile_abs_t"]


def _quant_cases():
    rng = np.random.default_rng(20211006)
    out = []
    for k in range(30):
        B = BLOCKS[rng.integers(len(BLOCKS))]
        qname = QMAPS[rng.integers(len(QMAPS))]
        kind = rng.integers(3)
        if kind == 0:
            n = int(rng.integers(1, 3 * 8192 + 10))
        elif kind == 1:
            n = int(B * rng.integers(1, 40) + rng.integers(-1, 2))
        else:
            n = int(rng.integers(100_000, 600_000))
        out.append(pytest.param(B, qname, n, int(rng.integers(1 << 30)),
                                id=f"{k:02d}-B{B}-{qname}-n{n}"))
    return out


def _mixed_values(n, B, seed):
    """Blocks of differing character: normal, heavy-tailed, uniform, all zero,
    tiny and huge scales, subnormals, and repeated values."""
    rng = np.random.default_rng(seed)
    x = np.empty(n, np.float32)
    for b0 in range(0, n, B):
        m = min(B, n - b0)
        kind = rng.integers(8)
        if kind == 0:
            v = rng.standard_normal(m)
        elif kind == 1:
            v = rng.standard_t(3, m) * 1e-2
        elif kind == 2:
            v = rng.uniform(-1, 1, m)
        elif kind == 3:
            v = np.zeros(m)
        elif kind == 4:
            v = rng.standard_normal(m) * 1e-30
        elif kind == 5:
            v = rng.standard_normal(m) * 1e30
        elif kind == 6:
            v = rng.integers(-1000, 1001, m) * 2.0 ** -149  # subnormals
        else:
            v = np.repeat(rng.standard_normal(1), m)
        x[b0:b0 + m] = v.astype(np.float32)
    return x


@pytest.mark.parametrize("B,qname,n,seed", _quant_cases())
def test_random_quantize_configuration(B, qname, n, seed):
    qs, qu, qs_d, qu_d = codebooks_on_device()
    if qname in ("signed", "unsigned"):
        q_h, q_d, signed = (qs, qs_d, True) if qname == "signed" else (qu, qu_d, False)
    else:
        q_h, signed = _other_maps()[qname]
        q_d = torch.from_numpy(q_h).cuda()
    x = _mixed_values(n, B, seed)
    run_pair(q_h, q_d, x if signed else np.abs(x), B)
