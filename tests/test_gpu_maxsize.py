"""GPU parity on single tensors of more than 2^31 elements (64-bit indexing in
every kernel): the fused 8-bit step on both paths, the 32-bit-state step, and
block-wise quantize / dequantize.

Inputs are generated on the GPU (torch Philox, seeded) and compared with the
oracle on a sample of blocks: the first and last blocks, the blocks on either
side of element 2^31, and random blocks.  Blocks are independent (Section 3.1),
so the oracle processes each sampled block on its own; codes and absmax must
match bit for bit, params within the step tests' bound.
"""
import numpy as np
import pytest
import torch

from paper_2110_02861_amd import bq
from tests.gpu_helpers import OPT_ID, codebooks_on_device, host, needs_gpu, param_close, say

import oracle

pytestmark = [pytest.mark.gpu, needs_gpu]

TWO31 = 1 << 31
CHUNK = 1 << 27  # elements per generation chunk (keeps temporaries at 0.5 GB)


def need_free_gib(gib):
    free, _ = torch.cuda.mem_get_info()
    if free < gib * (1 << 30):
        pytest.skip(f"needs {gib} GiB of free device memory")


def student_t_(out, seed):
    """Fill the fp32 device tensor out with Student-t(3) x 1e-2 values:
    Z / sqrt((Z1^2 + Z2^2 + Z3^2) / 3), generated in chunks."""
    g = torch.Generator(device=out.device)
    g.manual_seed(seed)
    for s in range(0, out.numel(), CHUNK):
        e = min(out.numel(), s + CHUNK)
        z = torch.randn(e - s, device=out.device, generator=g)
        c = torch.randn(3, e - s, device=out.device, generator=g).square_().sum(0).div_(3.0)
        out[s:e] = z.div_(c.sqrt_()).mul_(1e-2)
    return out


def normal_(out, std, seed):
    """Fill out (fp32 or fp16, on the GPU) with N(0, std), generated in fp32 chunks."""
    g = torch.Generator(device=out.device)
    g.manual_seed(seed)
    for s in range(0, out.numel(), CHUNK):
        e = min(out.numel(), s + CHUNK)
        out[s:e] = torch.randn(e - s, device=out.device, generator=g).mul_(std)
    return out


def sample_blocks(n, B, nrandom, seed):
    nb = (n + B - 1) // B
    mid = TWO31 // B
    picks = {0, 1, nb - 2, nb - 1, mid - 2, mid - 1, mid, mid + 1}
    rng = np.random.default_rng(seed)
    picks.update(int(b) for b in rng.integers(0, nb, nrandom))
    return sorted(b for b in picks if 0 <= b < nb)


def block_slice(b, B, n):
    return slice(b * B, min((b + 1) * B, n))


@pytest.mark.parametrize("B", [256, 4096])
def test_quantize_dequantize_beyond_2_31(B):
    need_free_gib(24)
    n = TWO31 + 3 * 4096 + 1234
    qs, _, qs_d, _ = codebooks_on_device()
    say(f"max-size quantize: generating n={n}")
    x = student_t_(torch.empty(n, dtype=torch.float32, device="cuda"), seed=B)
    picks = sample_blocks(n, B, 48, seed=B)
    say(f"max-size quantize n={n} B={B} (call, prepared)")
    c_d, a_d = bq.bq_quantize_blockwise(qs_d, x, B)
    c_p, a_p = bq.bq_quantize_blockwise_prepared(bq.bq_prepare_codebook(qs_d), x, B)
    torch.cuda.synchronize()
    ref = {}
    for b in picks:
        s = block_slice(b, B, n)
        xb = host(x[s]).copy()
        cr, ar = oracle.quantize_blockwise(qs, xb, B)
        ref[b] = (cr, ar)
        for c, a in ((c_d, a_d), (c_p, a_p)):
            assert host(a[b:b + 1]).view(np.uint32)[0] == ar.view(np.uint32)[0], (B, b)
            np.testing.assert_array_equal(host(c[s]), cr)
    assert torch.equal(c_d, c_p) and torch.equal(a_d.view(torch.int32), a_p.view(torch.int32))
    del c_p, a_p, x
    torch.cuda.empty_cache()
    say(f"max-size dequantize n={n} B={B}")
    out = bq.bq_dequantize_blockwise(qs_d, c_d, a_d, B)
    torch.cuda.synchronize()
    for b in picks:
        s = block_slice(b, B, n)
        cr, ar = ref[b]
        want = oracle.dequantize_blockwise(qs, cr, ar, B)
        np.testing.assert_array_equal(host(out[s]).view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("path", ["plan", "call"])
def test_adam8bit_step_beyond_2_31(path):
    need_free_gib(24)
    B = 2048
    n = TWO31 + 3 * B + 777
    nb = (n + B - 1) // B
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.995, eps=1e-8, wd=0.0)
    qs, qu, qs_d, qu_d = codebooks_on_device()
    say(f"max-size 8-bit step ({path}): allocating n={n}")
    w = normal_(torch.empty(n, dtype=torch.float32, device="cuda"), 0.02, seed=1)
    g = torch.empty(n, dtype=torch.float16, device="cuda")
    c1 = torch.full((n,), 127, dtype=torch.uint8, device="cuda")
    c2 = torch.zeros(n, dtype=torch.uint8, device="cuda")
    a1 = torch.zeros(nb, dtype=torch.float32, device="cuda")
    a2 = torch.zeros(nb, dtype=torch.float32, device="cuda")
    rows = [(w, g, c1, c2, a1, a2)]
    plan = bq.StepPlan(bq.BQ_ADAM, B, bq.BQ_F16, rows) if path == "plan" else None
    picks = sample_blocks(n, B, 48, seed=7)
    hb = {}
    for b in picks:
        s = block_slice(b, B, n)
        k = s.stop - s.start
        hb[b] = dict(w=host(w[s]).copy(), c1=np.full(k, 127, np.uint8), c2=np.zeros(k, np.uint8),
                     a1=np.zeros(1, np.float32), a2=np.zeros(1, np.float32),
                     tol=np.zeros(k, np.float64))
    for t in (1, 2):
        normal_(g, 1e-4, seed=100 + t)
        torch.cuda.synchronize()
        gh = {b: host(g[block_slice(b, B, n)]).copy() for b in picks}
        say(f"max-size 8-bit step ({path}) t={t}")
        if plan is not None:
            plan.run(dict(hp, step=t), qs_d, qu_d)
        else:
            bq.bq_optimizer8bit_step(bq.BQ_ADAM, B, bq.BQ_F16, rows, dict(hp, step=t), qs_d, qu_d)
        torch.cuda.synchronize()
        for b in picks:
            s = block_slice(b, B, n)
            h = hb[b]
            prev = h["w"].astype(np.float64)
            oracle.step8(OPT_ID["adam"], B, h["w"], gh[b], h["c1"], h["a1"], qs, h["c2"], h["a2"],
                         qu, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], t)
            w64 = h["w"].astype(np.float64)
            h["tol"] += 1e-6 * np.abs(prev - w64) + 2.0 ** -23 * np.abs(w64)
            ok, worst = param_close(host(w[s]), h["w"], h["tol"])
            assert ok, (path, t, b, worst)
            np.testing.assert_array_equal(host(c1[s]), h["c1"])
            np.testing.assert_array_equal(host(c2[s]), h["c2"])
            assert host(a1[b:b + 1])[0] == h["a1"][0], (path, t, b)
            assert host(a2[b:b + 1])[0] == h["a2"][0], (path, t, b)
    if plan is not None:
        plan.close()


def test_adam32bit_step_beyond_2_31():
    need_free_gib(40)
    n = TWO31 + 1024 + 333
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.995, eps=1e-8, wd=0.0)
    say(f"max-size 32-bit step: allocating n={n}")
    w = normal_(torch.empty(n, dtype=torch.float32, device="cuda"), 0.02, seed=3)
    g = normal_(torch.empty(n, dtype=torch.float16, device="cuda"), 1e-4, seed=4)
    m = torch.zeros(n, dtype=torch.float32, device="cuda")
    v = torch.zeros(n, dtype=torch.float32, device="cuda")
    picks = sample_blocks(n, 1024, 48, seed=9)
    hs = {}
    for b in picks:
        s = block_slice(b, 1024, n)
        hs[b] = (host(w[s]).copy(), host(g[s]).copy())
    say("max-size 32-bit step t=1")
    bq.bq_optimizer32bit_step(bq.BQ_ADAM, bq.BQ_F16, [(w, g, m, v)], dict(hp, step=1))
    torch.cuda.synchronize()
    for b in picks:
        s = block_slice(b, 1024, n)
        wr, gr = hs[b]
        mr = np.zeros_like(wr)
        vr = np.zeros_like(wr)
        prev = wr.astype(np.float64)
        oracle.step32(oracle.ADAM, wr, gr, mr, vr, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                      hp["wd"], 1)
        np.testing.assert_array_equal(host(m[s]).view(np.uint32), mr.view(np.uint32))
        np.testing.assert_array_equal(host(v[s]).view(np.uint32), vr.view(np.uint32))
        ok, worst = param_close(host(w[s]), wr, 1e-6 * np.abs(prev - wr.astype(np.float64)))
        assert ok, (b, worst)
