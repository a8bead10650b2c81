"""Seeded synthetic inputs for the Fork-dLLM step (shapes of the paper's
LLaDA-8B-style setting: semi-autoregressive blocks over a generation region,
Section 4.1).

This module only draws random numbers and lays them out; it holds none of the
step's arithmetic.  It is the one module that both the HIP path's tests and
the oracle side read their inputs from: every tensor is a pure function of
(config, seed, step), drawn with torch's seeded generators on the requested
device, so both sides consume identical bits.

Distributions (no model weights or datasets exist here, so these stand in for
LLaDA-8B hidden states / LM head and the GSM8K, MATH-500, HumanEval, MBPP
prompts):

* W_head[v, :] ~ N(0, 1/d) i.i.d.
* hidden at step t: N(0, 1) i.i.d. (generator seeded with seed+1000+t), each
  row multiplied by a per-position scale drawn once per configuration
  (generator seed+1).  Logits are linear in the hidden row, so a scale of 1/T
  is exactly a logit temperature T and a scale of r an RMS of r.
* initial state (generator seed+2): prompt tokens uniform in [0, V), never
  masked; generation positions masked (all of them, or exactly
  round(f * G) per sequence chosen without replacement); block_start = P.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Tuple

import torch

BASE_SEED = 0x5EED


@dataclasses.dataclass(frozen=True)
class SynthConfig:
    name: str
    B: int
    P: int                 # prompt length (never masked)
    G: int                 # generation length
    block_len: int
    d: int
    V: int
    dtype: str             # "bf16" or "f32"
    tau: float             # confidence threshold (the paper's lambda)
    scale_kind: str        # how per-position scales are drawn (see row_scale)
    scale_args: Tuple[float, ...] = ()
    masked_fraction: float = 1.0
    plant_peaks: float = 0.0   # fraction of rows given one logit ~ +20
    seed: int = BASE_SEED

    @property
    def L(self) -> int:
        return self.P + self.G

    @property
    def M(self) -> int:
        return self.B * self.L

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def with_(self, **kw) -> "SynthConfig":
        return dataclasses.replace(self, **kw)


# The five workloads of the benchmark definition, plus test-only variants that
# force frequent multi-commit parallel steps.
CONFIGS = {
    "tiny": SynthConfig("tiny", B=1, P=32, G=32, block_len=8, d=256, V=1024,
                        dtype="f32", tau=0.9, scale_kind="temp_choice",
                        scale_args=(0.2, 3.0)),
    "mid": SynthConfig("mid", B=4, P=128, G=128, block_len=32, d=1024, V=32000,
                       dtype="bf16", tau=0.9, scale_kind="temp_loguniform",
                       scale_args=(0.1, 4.0), masked_fraction=0.3),
    "llada8b": SynthConfig("llada8b", B=8, P=256, G=256, block_len=32, d=4096,
                           V=126464, dtype="bf16", tau=0.9,
                           scale_kind="rms_uniform", scale_args=(0.5, 2.0)),
    "rollout": SynthConfig("rollout", B=64, P=128, G=256, block_len=32, d=4096,
                           V=126464, dtype="bf16", tau=0.95,
                           scale_kind="rms_uniform", scale_args=(0.5, 2.0)),
    "long": SynthConfig("long", B=2, P=512, G=1536, block_len=64, d=4096,
                        V=126464, dtype="bf16", tau=0.9,
                        scale_kind="hot_fraction", scale_args=(0.1, 10.0)),
}
CONFIGS["tiny_peaked"] = CONFIGS["tiny"].with_(name="tiny_peaked",
                                               scale_args=(0.05, 3.0))
CONFIGS["mid_planted"] = CONFIGS["mid"].with_(name="mid_planted", tau=0.5,
                                              plant_peaks=0.5)
# The LLaDA-8B shape with planted peaks: 30% of the rows get one logit about
# 20 above the rest (confidence near 1), so steps at d = 4096, V = 126464
# commit several positions in parallel.
CONFIGS["llada8b_planted"] = CONFIGS["llada8b"].with_(name="llada8b_planted", plant_peaks=0.3)
# ForkGRPO rollouts in the paper's shape of a batch (groups of G = 16
# rollouts per prompt, lambda = 0.8, blocks of 32), scaled down so that the
# oracle follows a whole decode: 2 prompts x 16 rollouts, 64 generated
# positions, d = 128, V = 1024; planted peaks give a mix of parallel and
# fallback steps.
CONFIGS["grpo_small"] = SynthConfig("grpo_small", B=32, P=16, G=64, block_len=32, d=128,
                                    V=1024, dtype="bf16", tau=0.8,
                                    scale_kind="temp_loguniform", scale_args=(0.1, 4.0),
                                    plant_peaks=0.15)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def weights(cfg: SynthConfig, device="cpu") -> torch.Tensor:
    """W_head [V, d], entries N(0, 1/d), stored in the config's dtype."""
    g = _gen(cfg.seed, device)
    w = torch.randn(cfg.V, cfg.d, generator=g, device=device, dtype=torch.float32)
    w.mul_(1.0 / math.sqrt(cfg.d))
    return w.to(cfg.torch_dtype).contiguous()


def row_scale(cfg: SynthConfig) -> torch.Tensor:
    """Per-position multiplier of the hidden row, [B*L] float32 on the CPU."""
    g = _gen(cfg.seed + 1, "cpu")
    n = cfg.M
    k = cfg.scale_kind
    if k == "temp_choice":            # temperature in {a, b} with p = 1/2
        a, b = cfg.scale_args
        pick = torch.rand(n, generator=g) < 0.5
        temp = torch.where(pick, torch.full((n,), a), torch.full((n,), b))
        return (1.0 / temp).float()
    if k == "temp_loguniform":        # temperature ~ LogUniform[a, b]
        a, b = cfg.scale_args
        u = torch.rand(n, generator=g, dtype=torch.float64)
        temp = torch.exp(math.log(a) + u * (math.log(b) - math.log(a)))
        return (1.0 / temp).float()
    if k == "rms_uniform":            # row RMS ~ U[a, b]
        a, b = cfg.scale_args
        u = torch.rand(n, generator=g, dtype=torch.float64)
        return (a + u * (b - a)).float()
    if k == "hot_fraction":           # fraction f of rows at temperature T
        f, temp = cfg.scale_args
        hot = torch.rand(n, generator=g) < f
        return torch.where(hot, torch.full((n,), 1.0 / temp), torch.ones(n)).float()
    if k == "const":
        (c,) = cfg.scale_args
        return torch.full((n,), float(c))
    raise ValueError("unknown scale kind %r" % k)


def hidden(cfg: SynthConfig, step: int, device="cpu",
           W: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Final hidden states [B*L, d] for denoising step ``step``."""
    g = _gen(cfg.seed + 1000 + step, device)
    h = torch.randn(cfg.M, cfg.d, generator=g, device=device, dtype=torch.float32)
    h.mul_(row_scale(cfg).to(device).unsqueeze(1))
    if cfg.plant_peaks > 0.0:
        # Add 20 * W[v] to chosen rows: the logit of v then rises by about 20
        # (|W[v]|^2 ~ 1), which makes the row's confidence close to one.
        if W is None:
            raise ValueError("planted peaks need the weights")
        gp = _gen(cfg.seed + 3000 + step, "cpu")
        chosen = torch.rand(cfg.M, generator=gp) < cfg.plant_peaks
        vocab = torch.randint(0, cfg.V, (cfg.M,), generator=gp)
        rows = torch.nonzero(chosen).flatten()
        if rows.numel():
            wf = W.to(device=device, dtype=torch.float32)
            h[rows.to(device)] += 20.0 * wf[vocab[rows].to(device)]
    return h.to(cfg.torch_dtype).contiguous()


def initial_state(cfg: SynthConfig):
    """(tokens int32 [B*L], mask uint8 [B*L], block_start int32 [B]) on CPU."""
    g = _gen(cfg.seed + 2, "cpu")
    B, P, G, L = cfg.B, cfg.P, cfg.G, cfg.L
    tokens = torch.randint(0, cfg.V, (B, L), generator=g, dtype=torch.int64).to(torch.int32)
    mask = torch.zeros(B, L, dtype=torch.uint8)
    if cfg.masked_fraction >= 1.0:
        mask[:, P:] = 1
    else:
        n = int(round(cfg.masked_fraction * G))
        for b in range(B):
            pos = torch.randperm(G, generator=g)[:n]
            mask[b, P + pos] = 1
    tokens[mask.bool()] = -1
    block_start = torch.full((B,), P, dtype=torch.int32)
    return tokens.reshape(-1).contiguous(), mask.reshape(-1).contiguous(), block_start


def to_bits(t: torch.Tensor):
    """Host numpy view of a tensor's stored bits: uint16 for bf16, float32
    for binary32 (the form the oracle reads)."""
    t = t.detach().to("cpu").contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view("uint16")
    if t.dtype == torch.float32:
        return t.numpy()
    raise TypeError("unsupported dtype %s" % t.dtype)
