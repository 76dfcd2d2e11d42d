"""Quantization error of Adam's states per data type (App. F), on synthetic states.

The paper compares the linear, quantile, inverse dynamic and dynamic maps by the
mean relative error of the Adam update computed from quantized states and by
the mean absolute quantization error of the first state (App. F, its table of
Adam errors).  Its states came from language-model training; here they come
from a synthetic run, so the numbers are this workload's, not the paper's:

1. 32-bit Adam (``bq_optimizer32bit_step``) runs ``steps`` steps on one
   ``rows x cols`` fp32 tensor with seeded LM-like gradients: N(0, 1) scaled
   per row by 1/sqrt(rank + 1) for a random rank below ``row_spread`` (a
   heavy-tailed spread of row magnitudes, as token embeddings see), with a
   Bernoulli(1e-3) mask scaling by ``outlier``.
2. The final states m and r are quantized block-wise (blocksize B) with each
   family's signed map (m) and unsigned map (r), and dequantized, all by libbq.
   Quantile maps are estimated from a sample of the block-normalized states
   (App. F.2).
3. u = m_hat / (sqrt(r_hat) + eps) with both bias corrections is compared with
   the update from the fp32 states: relative Adam error = mean (and median)
   |u_q - u| / |u| over elements with u != 0; absolute quantization error =
   mean |m - m_q|; and the share of nonzero r that quantizes to 0 (those
   elements take a step of m / eps).

    python -m paper_2110_02861_amd.analysis [--rows 8192 --cols 1024 --steps 20
                                             --row-spread 1024 --outlier 10]

``--time-quantiles N`` instead times the GPU quantile estimator
(``bq_estimate_quantile_codebook``, App. G) on N seeded normal values and
prints ns per element.
"""
from __future__ import annotations

import argparse
import json

import numpy as np
import torch

from . import bq, workloads

FAMILIES = ("linear", "quantile", "inverse_dynamic", "dynamic")


def synthetic_adam_states(rows: int, cols: int, steps: int, seed: int = 0, row_spread=1024,
                          outlier=10.0, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8):
    """fp32 m and r after ``steps`` 32-bit Adam steps (GPU), with the param."""
    dev = torch.device("cuda")
    n = rows * cols
    rng = workloads.host_rng(seed, "c4", 0, 0)
    w = torch.from_numpy((rng.standard_normal(n) * 0.02).astype(np.float32)).to(dev)
    rank = (rng.permutation(rows) % max(1, row_spread)).astype(np.float32)
    row_scale = torch.from_numpy(1.0 / np.sqrt(rank + 1.0)).to(dev).repeat_interleave(cols)
    m = torch.zeros(n, device=dev)
    r = torch.zeros(n, device=dev)
    gen = torch.Generator(device=dev)
    for t in range(1, steps + 1):
        gen.manual_seed(seed * 1000 + t)
        g = torch.randn(n, device=dev, generator=gen) * row_scale
        mask = torch.rand(n, device=dev, generator=gen) < 1e-3
        g = torch.where(mask, g * outlier, g)
        bq.bq_optimizer32bit_step(bq.BQ_ADAM, bq.BQ_F32, [(w, g, m, r)],
                                  dict(lr=lr, beta1=beta1, beta2=beta2, eps=eps, wd=0.0, step=t))
    torch.cuda.synchronize()
    return m, r


def _normalized_sample(x: torch.Tensor, blocksize: int, size: int, seed: int) -> np.ndarray:
    nb = (x.numel() + blocksize - 1) // blocksize
    pad = torch.zeros(nb * blocksize, device=x.device)
    pad[: x.numel()] = x
    blocks = pad.view(nb, blocksize)
    a = blocks.abs().amax(dim=1, keepdim=True)
    y = torch.where(a > 0, blocks / a.clamp_min(torch.finfo(torch.float32).tiny), blocks)
    y = y.reshape(-1)[: x.numel()]
    gen = torch.Generator(device=x.device)
    gen.manual_seed(seed)
    idx = torch.randint(0, x.numel(), (min(size, x.numel()),), device=x.device, generator=gen)
    return y[idx].cpu().numpy().astype(np.float32)


def maps_for(family: str, m: torch.Tensor, r: torch.Tensor, blocksize: int, seed: int = 0):
    """(signed map for m, unsigned map for r) of a family, host fp32."""
    if family == "quantile":
        return (bq.bq_make_quantile_codebook(_normalized_sample(m, blocksize, 1 << 20, seed)),
                bq.bq_make_quantile_codebook(_normalized_sample(r, blocksize, 1 << 20, seed + 1)))
    k1, k2 = bq.CODEBOOKS[family]
    return bq.bq_make_codebook(k1), bq.bq_make_codebook(k2)


def round_trip(q: np.ndarray, x: torch.Tensor, blocksize: int) -> torch.Tensor:
    q_d = torch.from_numpy(q).to(x.device)
    codes, absmax = bq.bq_quantize_blockwise(q_d, x, blocksize)
    return bq.bq_dequantize_blockwise(q_d, codes, absmax, blocksize)


def adam_errors(m, r, q1, q2, blocksize=2048, steps=20, beta1=0.9, beta2=0.999, eps=1e-8):
    mq = round_trip(q1, m, blocksize)
    rq = round_trip(q2, r, blocksize)
    bc1 = 1.0 - beta1 ** steps
    bc2 = 1.0 - beta2 ** steps

    def update(mm, rr):
        return (mm.double() / bc1) / (torch.sqrt(rr.double() / bc2) + eps)

    u = update(m, r)
    uq = update(mq, rq)
    nz = u != 0
    relv = (uq - u).abs()[nz] / u.abs()[nz]
    absq = (m.double() - mq.double()).abs().mean().item()
    r_nz = r != 0
    zero_r = ((rq == 0) & r_nz).sum().item() / max(1, r_nz.sum().item())
    return {"relative_adam_error": relv.mean().item(),
            "relative_adam_error_median": relv.median().item(),
            "absolute_quantization_error": absq, "r_quantized_to_zero": zero_r}


def run(rows=8192, cols=1024, steps=20, blocksize=2048, seed=0, row_spread=1024,
        outlier=10.0) -> dict:
    m, r = synthetic_adam_states(rows, cols, steps, seed, row_spread, outlier)
    out = {}
    for fam in FAMILIES:
        q1, q2 = maps_for(fam, m, r, blocksize, seed)
        out[fam] = adam_errors(m, r, q1, q2, blocksize, steps)
    return out


def time_quantile_estimator(n: int, reps: int = 20, seed: int = 0) -> dict:
    """Average time of bq_estimate_quantile_codebook on n normal values (HIP
    events on the launch stream), with its workspace preallocated."""
    dev = torch.device("cuda")
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    x = torch.randn(n, device=dev, generator=gen)
    ws = torch.empty(bq.lib().bq_quantile_workspace_bytes(n) // 8, dtype=torch.float64,
                     device=dev)
    out = torch.empty(256, device=dev)
    stream = torch.cuda.current_stream()
    for _ in range(3):
        bq.bq_estimate_quantile_codebook(x, out, ws)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        bq.bq_estimate_quantile_codebook(x, out, ws)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return {"n": n, "ms": ms, "ns_per_element": ms * 1e6 / n,
            "gb_per_s": n * 4 / (ms / 1e3) / 1e9}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--rows", type=int, default=8192)
    ap.add_argument("--cols", type=int, default=1024)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--blocksize", type=int, default=2048)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--row-spread", type=int, default=1024)
    ap.add_argument("--outlier", type=float, default=10.0)
    ap.add_argument("--time-quantiles", type=int, default=0, metavar="N")
    a = ap.parse_args()
    if a.time_quantiles:
        print(json.dumps(time_quantile_estimator(a.time_quantiles)))
        return
    res = run(a.rows, a.cols, a.steps, a.blocksize, a.seed, a.row_spread, a.outlier)
    print(f"{'map':16s} {'rel. Adam error':>16s} {'(median)':>10s} {'abs. quant. error':>18s} "
          f"{'r -> 0':>8s}")
    for fam, v in res.items():
        print(f"{fam:16s} {100 * v['relative_adam_error']:15.2f}% "
              f"{100 * v['relative_adam_error_median']:9.2f}% "
              f"{v['absolute_quantization_error']:18.3e} {100 * v['r_quantized_to_zero']:7.3f}%")
    print(json.dumps(res))


if __name__ == "__main__":
    main()
