"""Seeded synthetic inputs shaped like the paper's workloads.

This module holds no arithmetic of the method: only tensor shapes, value
distributions and random-number streams.  It serves both the HIP path and the
CPU oracle, which receive the same bytes.

The paper's isolated runtime measurement uses a large normal sample
(Appendix E); its training runs use GPT-2-style language models and ResNet-50
(Section 4).  Only the *shapes* of those models are reproduced here, with
random values; no dataset or trained weight is involved.

Host streams: numpy PCG64 seeded with SeedSequence([seed, config, tensor, step]).
Device streams: torch's Philox generator on the GPU, seeded from the same tuple,
used for the large lists where host generation would dominate run time.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

# Hyperparameters of the five synthetic configurations.
C1 = dict(opt="adam", lr=1e-3, beta1=0.9, beta2=0.995, eps=1e-8, wd=0.0, blocksize=2048)
C3 = dict(opt="momentum", lr=0.1, beta1=0.9, beta2=0.0, eps=0.0, wd=1e-4, blocksize=2048)
C4 = dict(opt="adamw", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.01, blocksize=2048)
C5 = dict(opt="adam", lr=1e-3, beta1=0.9, beta2=0.995, eps=1e-8, wd=0.0, blocksize=2048)
C5BF16 = C5  # the same list and optimizer with bf16 grads

CONFIG_IDS = {"c1": 1, "c2": 2, "c3": 3, "c4": 4, "c5": 5, "p1b": 6, "c5bf16": 7}


@dataclass(frozen=True)
class TensorSpec:
    name: str
    shape: tuple
    init: str          # "normal", "uniform", "ones", "zeros"
    scale: float       # std for normal, half-width for uniform
    grad_kind: str = "plain"   # "plain", "embedding" (heavy-tailed rows)

    @property
    def numel(self) -> int:
        return int(math.prod(self.shape))


def resnet50_specs() -> list[TensorSpec]:
    """ResNet-50 v1.5 parameter list: 161 tensors, 25,557,032 parameters."""
    t: list[TensorSpec] = []

    def conv(name, cout, cin, k):
        fan_in = cin * k * k
        t.append(TensorSpec(name, (cout, cin, k, k), "normal", math.sqrt(2.0 / fan_in)))

    def bn(name, c):
        t.append(TensorSpec(name + ".weight", (c,), "ones", 0.0))
        t.append(TensorSpec(name + ".bias", (c,), "zeros", 0.0))

    conv("conv1", 64, 3, 7)
    bn("bn1", 64)
    cin = 64
    for si, (width, nblocks) in enumerate([(64, 3), (128, 4), (256, 6), (512, 3)]):
        for b in range(nblocks):
            p = f"layer{si + 1}.{b}"
            conv(p + ".conv1", width, cin, 1)
            bn(p + ".bn1", width)
            conv(p + ".conv2", width, width, 3)
            bn(p + ".bn2", width)
            conv(p + ".conv3", 4 * width, width, 1)
            bn(p + ".bn3", 4 * width)
            if b == 0:
                conv(p + ".downsample", 4 * width, cin, 1)
                bn(p + ".downsample_bn", 4 * width)
            cin = 4 * width
    t.append(TensorSpec("fc.weight", (1000, 2048), "normal", math.sqrt(2.0 / 2048)))
    t.append(TensorSpec("fc.bias", (1000,), "zeros", 0.0))
    return t


def gpt2_specs(layers: int, d: int, ffn: int, vocab: int = 50257, ctx: int = 1024):
    """GPT-2-style parameter list: 12 tensors per layer plus wte, wpe, ln_f."""
    t: list[TensorSpec] = [
        TensorSpec("wte", (vocab, d), "normal", 0.02, grad_kind="embedding"),
        TensorSpec("wpe", (ctx, d), "normal", 0.02),
    ]
    for i in range(layers):
        p = f"h.{i}"
        t += [
            TensorSpec(p + ".ln_1.weight", (d,), "ones", 0.0),
            TensorSpec(p + ".ln_1.bias", (d,), "zeros", 0.0),
            TensorSpec(p + ".attn.c_attn.weight", (d, 3 * d), "normal", 0.02),
            TensorSpec(p + ".attn.c_attn.bias", (3 * d,), "zeros", 0.0),
            TensorSpec(p + ".attn.c_proj.weight", (d, d), "normal", 0.02),
            TensorSpec(p + ".attn.c_proj.bias", (d,), "zeros", 0.0),
            TensorSpec(p + ".ln_2.weight", (d,), "ones", 0.0),
            TensorSpec(p + ".ln_2.bias", (d,), "zeros", 0.0),
            TensorSpec(p + ".mlp.c_fc.weight", (d, ffn), "normal", 0.02),
            TensorSpec(p + ".mlp.c_fc.bias", (ffn,), "zeros", 0.0),
            TensorSpec(p + ".mlp.c_proj.weight", (ffn, d), "normal", 0.02),
            TensorSpec(p + ".mlp.c_proj.bias", (d,), "zeros", 0.0),
        ]
    t += [TensorSpec("ln_f.weight", (d,), "ones", 0.0),
          TensorSpec("ln_f.bias", (d,), "zeros", 0.0)]
    return t


def gpt2_medium_specs():
    """24 layers, d 1024, ffn 4096: 292 tensors, 354,823,168 parameters."""
    return gpt2_specs(24, 1024, 4096)


def lm_1p5b_specs():
    """48 layers, d 1600, ffn 6400: 580 tensors, 1,557,611,200 parameters."""
    return gpt2_specs(48, 1600, 6400)


def c1_specs():
    return [TensorSpec("w", (1_048_576,), "uniform", 0.05)]


def paper_1b_specs():
    """The setup of the paper's isolated optimizer timing (App. E): one large
    sample of a normal distribution, here 10^9 values, with fp32 gradients."""
    return [TensorSpec("w", (1_000_000_000,), "normal", 1.0)]


SPECS = {"c1": c1_specs, "c3": resnet50_specs, "c4": gpt2_medium_specs, "c5": lm_1p5b_specs,
         "p1b": paper_1b_specs, "c5bf16": lm_1p5b_specs}

# Gradient distributions per configuration: (dtype, std, outlier prob, outlier factor).
GRADS = {
    "c1": ("float16", 1e-3, 1e-3, 100.0),
    "c3": ("float32", 1e-3, 0.0, 1.0),
    "c4": ("float16", 1e-4, 0.0, 1.0),
    "c5": ("float16", 1e-4, 1e-4, 1000.0),
    "p1b": ("float32", 1.0, 0.0, 1.0),
    # the 1.5B list with bf16 grads (generated on the GPU only)
    "c5bf16": ("bfloat16", 1e-4, 1e-4, 1000.0),
}


# ---------------------------------------------------------------------------
# Host (numpy) generation
# ---------------------------------------------------------------------------

def host_rng(seed: int, config: str, tensor: int = 0, step: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence([seed, CONFIG_IDS.get(config, 0), tensor, step])
    return np.random.Generator(np.random.PCG64(ss))


def init_param_host(spec: TensorSpec, rng: np.random.Generator) -> np.ndarray:
    n = spec.numel
    if spec.init == "normal":
        g = rng.standard_normal(n, dtype=np.float32)
        return (g * np.float32(spec.scale)).astype(np.float32)
    if spec.init == "uniform":
        return rng.uniform(-spec.scale, spec.scale, n).astype(np.float32)
    if spec.init == "ones":
        return np.ones(n, np.float32)
    return np.zeros(n, np.float32)


def grad_host(config: str, spec: TensorSpec, rng: np.random.Generator) -> np.ndarray:
    """Gradient of one tensor: N(0, std) with Bernoulli(p) outliers x factor,
    embedding rows heavy-tailed, then cast to the configuration's grad dtype."""
    dtype, std, p, factor = GRADS[config]
    n = spec.numel
    g = rng.standard_normal(n, dtype=np.float32) * np.float32(std)
    if p > 0.0:
        g[rng.random(n) < p] *= np.float32(factor)
    if spec.grad_kind == "embedding":
        rows, d = spec.shape
        rank = rng.permutation(rows)
        scale = np.where(rank < 8192, 100.0 / np.sqrt(rank + 1.0), 0.0).astype(np.float32)
        g = (g.reshape(rows, d) * scale[:, None]).reshape(-1)
    return g.astype(dtype)


def student_t_host(n: int, seed: int = 0, nu: float = 3.0, scale: float = 1e-2) -> np.ndarray:
    """Heavy-tailed values for the standalone quantize / dequantize round trip."""
    rng = host_rng(seed, "c2")
    return (rng.standard_t(nu, n) * scale).astype(np.float32)


# ---------------------------------------------------------------------------
# Device (torch) generation for the large lists
# ---------------------------------------------------------------------------

def _device_seed(seed: int, config: str, tensor: int, step: int) -> int:
    ss = np.random.SeedSequence([seed, CONFIG_IDS.get(config, 0), tensor, step])
    return int(ss.generate_state(1, np.uint64)[0] & ((1 << 63) - 1))


def init_param_device(spec: TensorSpec, out, seed: int, config: str, index: int):
    """Fill the flat fp32 tensor ``out`` (on the GPU) with the spec's init."""
    import torch
    g = torch.Generator(device=out.device)
    g.manual_seed(_device_seed(seed, config, index, 0))
    if spec.init == "normal":
        out.normal_(0.0, spec.scale, generator=g)
    elif spec.init == "uniform":
        out.uniform_(-spec.scale, spec.scale, generator=g)
    elif spec.init == "ones":
        out.fill_(1.0)
    else:
        out.zero_()
    return out


def grad_device(config: str, spec: TensorSpec, out, seed: int, index: int, step: int):
    """Fill the flat grad tensor ``out`` (fp16, bf16 or fp32, on the GPU)."""
    import torch
    _, std, p, factor = GRADS[config]
    g = torch.Generator(device=out.device)
    g.manual_seed(_device_seed(seed, config, index, step + 1))
    tmp = torch.empty(out.numel(), dtype=torch.float32, device=out.device)
    tmp.normal_(0.0, std, generator=g)
    if p > 0.0:
        mask = torch.rand(out.numel(), device=out.device, generator=g) < p
        tmp[mask] *= factor
    if spec.grad_kind == "embedding":
        rows, d = spec.shape
        rank = torch.randperm(rows, device=out.device, generator=g)
        scale = torch.where(rank < 8192, 100.0 / torch.sqrt(rank.float() + 1.0),
                            torch.zeros((), device=out.device))
        tmp = (tmp.view(rows, d) * scale[:, None]).view(-1)
    out.copy_(tmp)
    return out
