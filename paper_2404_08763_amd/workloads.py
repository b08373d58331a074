"""Seeded synthetic workloads with the shapes of the paper's MLP blocks.

Input generation only: random weights, activations and calibration vectors
drawn from seeded generators (CPU; a stack's weights on the device), with no
part of the method's arithmetic.
Both the device path and the CPU oracle are fed from these buffers.

The paper times single Llama2-7B (d=4096, m=11008) and Mistral-7B (d=4096,
m=14336) MLP blocks with real weights and RefinedWeb tokens (Section 5.3);
neither is available here, so weights are N(0, 0.02^2) and activations are
synthetic with the distributions below.

Seeds (torch.Generator('cpu').manual_seed unless noted):
  W_gate, W_up, W_down of layer l   1000*l + 0, 1, 2 (stacks: the device's
                                    generator, neuron-major; stack_weights)
  calibration vectors               7   (+ 100*l for layer l of a stack)
  decode / test vectors             11
  outlier channel choice            13
  mixture scales                    17
  Q/K/V projection weight           5000
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import torch

SEED_CALIB = 7
SEED_DECODE = 11
SEED_OUTLIERS = 13
SEED_SCALES = 17
WEIGHT_STD = 0.02


@dataclass(frozen=True)
class Config:
    name: str
    d: int
    m: int
    wdtype: torch.dtype
    n_calib: int
    n_decode: int
    sparsities: tuple
    x_dist: str = "normal"          # "normal", "outliers" or "laplace_mix"
    n_layers: int = 1
    batches: tuple = (1,)
    outlier_frac: float = 0.01      # "outliers": fraction of channels scaled
    outlier_scale: float = 20.0
    mix_scales: tuple = (0.25, 0.5, 1.0)
    notes: str = ""


CONFIGS = {
    "C1": Config("C1", d=256, m=688, wdtype=torch.float32, n_calib=512, n_decode=64,
                 sparsities=(0.5,), notes="tiny single layer, fp32 weights"),
    "C2": Config("C2", d=4096, m=11008, wdtype=torch.bfloat16, n_calib=2048, n_decode=256,
                 sparsities=(0.5, 0.7, 0.9), x_dist="outliers",
                 notes="Llama2-7B-shaped MLP, 1% outlier channels x20"),
    "C3": Config("C3", d=4096, m=14336, wdtype=torch.bfloat16, n_calib=2048, n_decode=256,
                 sparsities=(0.0, 0.3, 0.5, 0.7, 0.9), x_dist="laplace_mix",
                 notes="Mistral-7B-shaped MLP, Laplace(0,1) scale mixture"),
    "C4": Config("C4", d=5120, m=13824, wdtype=torch.bfloat16, n_calib=1024, n_decode=128,
                 sparsities=(0.5,), n_layers=40, notes="Llama2-13B-shaped 40-layer stack"),
    "QKV": Config("QKV", d=4096, m=6144, wdtype=torch.bfloat16, n_calib=2048, n_decode=256,
                  sparsities=(0.5, 0.7, 0.9), x_dist="laplace_mix",
                  notes="Mistral-7B-shaped fused Q/K/V projection (4096 -> 4096 + 1024 + 1024) "
                        "behind CATS on its input; m is the output width n"),
    "C5": Config("C5", d=4096, m=11008, wdtype=torch.bfloat16, n_calib=1024, n_decode=64,
                 sparsities=(0.5, 0.7), n_layers=32, batches=(1, 2, 4, 8, 16),
                 notes="Llama2-7B-shaped 32-layer stack, small-batch decode"),
}


def generator(seed: int) -> torch.Generator:
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    return g


def weights(d: int, m: int, wdtype: torch.dtype, layer: int = 0, std: float = WEIGHT_STD):
    """Math-layout weights of one block: W_gate, W_up [d, m] and W_down [m, d].

    Drawn in fp32 from N(0, std^2) and rounded once to `wdtype`
    (round-to-nearest-even for bf16)."""
    base = 1000 * layer
    wg = (torch.randn((d, m), generator=generator(base + 0)) * std).to(wdtype)
    wu = (torch.randn((d, m), generator=generator(base + 1)) * std).to(wdtype)
    wd = (torch.randn((m, d), generator=generator(base + 2)) * std).to(wdtype)
    return wg, wu, wd


def stack_weights(d: int, m: int, wdtype: torch.dtype, layer: int, device="cpu", std: float = WEIGHT_STD):
    """Neuron-major weights of layer `layer` of a stack: W_gate^T, W_up^T and
    W_down, each [m, d], drawn in fp32 from N(0, std^2) on `device` (its own
    Philox generator on a GPU, seeds 1000*layer + 0, 1, 2) and rounded once
    to `wdtype`.  The entries are iid, so drawing them neuron-major gives the
    same distribution as drawing the math layout and transposing; a 40-layer
    stack of 5120 x 13824 blocks is generated in well under a second on a
    GPU, where the CPU generator would take minutes."""
    base = 1000 * layer
    out = []
    for k in range(3):
        g = torch.Generator(device=device)
        g.manual_seed(base + k)
        out.append((torch.randn((m, d), generator=g, device=device) * std).to(wdtype))
    return tuple(out)


def linear_weight(d: int, n: int, wdtype: torch.dtype, seed: int, std: float = WEIGHT_STD) -> torch.Tensor:
    """A linear layer's weight in channel-major layout [d, n] (row i = input
    channel i), N(0, std^2) drawn in fp32 (CPU generator) and rounded once."""
    return (torch.randn((d, n), generator=generator(seed)) * std).to(wdtype)


def outlier_channels(d: int, frac: float = 0.01) -> torch.Tensor:
    """round(frac * d) channel indices, fixed per model (seed 13)."""
    k = int(round(frac * d))
    return torch.randperm(d, generator=generator(SEED_OUTLIERS))[:k]


def laplace(shape, g: torch.Generator) -> torch.Tensor:
    """Laplace(0, 1) samples by inverting the CDF of uniform draws."""
    u = torch.rand(shape, generator=g, dtype=torch.float64) - 0.5
    u = u.clamp(-0.5 + 1e-12, 0.5 - 1e-12)
    return (-torch.sign(u) * torch.log1p(-2.0 * u.abs())).to(torch.float32)


def activations(cfg: Config, n: int, seed: int) -> torch.Tensor:
    """n synthetic hidden vectors x [n, d] fp32 for the config's distribution."""
    g = generator(seed)
    if cfg.x_dist == "normal":
        return torch.randn((n, cfg.d), generator=g)
    if cfg.x_dist == "outliers":
        x = torch.randn((n, cfg.d), generator=g)
        x[:, outlier_channels(cfg.d, cfg.outlier_frac)] *= cfg.outlier_scale
        return x
    if cfg.x_dist == "laplace_mix":
        lap = laplace((n, cfg.d), g)
        scales = torch.tensor(cfg.mix_scales, dtype=torch.float32)
        pick = torch.randint(0, len(cfg.mix_scales), (n,), generator=generator(seed + SEED_SCALES))
        return lap * scales[pick][:, None]
    raise ValueError(f"unknown x_dist {cfg.x_dist!r}")


def calib_vectors(cfg: Config, n: Optional[int] = None, layer: int = 0) -> torch.Tensor:
    return activations(cfg, cfg.n_calib if n is None else n, SEED_CALIB + 100 * layer)


def decode_vectors(cfg: Config, n: Optional[int] = None) -> torch.Tensor:
    return activations(cfg, cfg.n_decode if n is None else n, SEED_DECODE)


def shrink(cfg: Config, d: int, m: int, **kw) -> Config:
    """The same distributions at another (test-sized) shape."""
    fields = dict(cfg.__dict__)
    fields.update(d=d, m=m, **kw)
    return Config(**fields)
