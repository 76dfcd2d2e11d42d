"""A seeded sweep over random combinations of the step's parameters against the
oracle: optimizer, grad dtype, blocksize, path, codebook family, weight decay
and a ragged tensor list, two steps each.

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

from paper_2110_02861_amd import bq
from tests.gpu_helpers import needs_gpu
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
