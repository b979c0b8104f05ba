"""Seeded synthetic inputs for the GPT-2 FP32 training step.

This module only draws numbers and fixes the flat parameter layout; it holds
none of the training arithmetic, so both the HIP path and the float64 oracle
can be fed from it without sharing any of the method's code.

Workload recipe (Evaluation section, GPT-2 architecture figure caption and the
"Training hyperparameters" table):

* GPT-2 decoder, pre-LN blocks, tied token embedding / LM head, learned
  positional embeddings, vocabulary 50,257 padded to 50,304.
* Initialisation: weights N(0, 0.02); the two residual projections (attention
  output and MLP down-projection) N(0, 0.02/sqrt(2 L)); biases 0; LN gain 1,
  bias 0.  Values are drawn in float64 and cast to float32 once.  Padded rows
  of the token embedding are 0.
* Token ids: the paper trains on FineWeb-Edu, which is not available here; a
  Zipf(s=1.1) stream over the real vocabulary stands in for its skewed token
  frequencies.  Inputs and targets come from one stream shifted by one, as the
  double-buffered loader copies positions t and t+1 (Implementation section,
  data loader algorithm).

RNG: numpy PCG64(seed); parameters are drawn in canonical order, then data.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Tuple

import numpy as np

__all__ = [
    "GPT2Config", "TINY", "GPT2_124M", "param_specs", "num_params",
    "num_decay_params", "param_offsets", "init_params", "block_params",
    "flatten", "unflatten", "zipf_tokens", "uniform_tokens", "shifted_pair",
    "normal", "HParams", "HP_TINY", "HP_124M",
]


@dataclasses.dataclass(frozen=True)
class GPT2Config:
    """Model shape.  V = real vocabulary, Vp = padded vocabulary rows of wte."""
    V: int
    Vp: int
    max_T: int
    L: int
    H: int
    C: int
    ln_eps: float = 1e-5

    @property
    def hd(self) -> int:
        return self.C // self.H

    @property
    def F(self) -> int:
        return 4 * self.C


@dataclasses.dataclass(frozen=True)
class HParams:
    """AdamW hyper-parameters for one step (lr held constant within a step)."""
    lr: float
    beta1: float
    beta2: float
    eps: float
    weight_decay: float
    grad_clip: float  # <= 0 disables clipping


# Tiny model: 2 layers, d_model 64, 4 heads, MLP 256, vocab 256, T 32.
TINY = GPT2Config(V=256, Vp=256, max_T=32, L=2, H=4, C=64)
# GPT-2 124M as in the hyper-parameter table.
GPT2_124M = GPT2Config(V=50257, Vp=50304, max_T=1024, L=12, H=12, C=768)
# Long-context single-GPU configuration (section "Long-context training"):
# the 124M model with 16384 learned positions, run at B = 2, T = 16384.
GPT2_124M_T16K = GPT2Config(V=50257, Vp=50304, max_T=16384, L=12, H=12, C=768)
# Narrow model at long T whose whole step the float64 oracle can still run.
TINY_T4K = GPT2Config(V=256, Vp=256, max_T=4096, L=2, H=4, C=64)
# Largest-trainable-model configuration (section "Largest trainable parameter
# model"): 2.42B parameters, d_model 3072, 20 layers, 24 heads of dim 128,
# run at B = 2, T = 1024.
GPT2_2_42B = GPT2Config(V=50257, Vp=50304, max_T=1024, L=20, H=24, C=3072)
# Narrow model with the 2.42B head dim (128), small enough for the oracle.
TINY_HD128 = GPT2Config(V=256, Vp=256, max_T=64, L=2, H=2, C=256)

HP_TINY = HParams(lr=3e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1, grad_clip=0.0)
HP_124M = HParams(lr=6e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1, grad_clip=1.0)


def param_specs(cfg: GPT2Config) -> List[Tuple[str, Tuple[int, ...], bool]]:
    """Canonical flat order: (name, shape, decayed).

    Decayed (2-D) tensors come first so that weight decay applies to a prefix
    of the flat arena: wte, wpe, then per layer Wqkv, Wo, Wfc, Wfp.  Then the
    non-decayed tensors: per layer ln1g, ln1b, bqkv, bo, ln2g, ln2b, bfc, bfp,
    then lnfg, lnfb.  Linear weights are stored [in, out].
    """
    C, F, L = cfg.C, cfg.F, cfg.L
    specs: List[Tuple[str, Tuple[int, ...], bool]] = [
        ("wte", (cfg.Vp, C), True),
        ("wpe", (cfg.max_T, C), True),
    ]
    for l in range(L):
        specs += [
            (f"h{l}.Wqkv", (C, 3 * C), True),
            (f"h{l}.Wo", (C, C), True),
            (f"h{l}.Wfc", (C, F), True),
            (f"h{l}.Wfp", (F, C), True),
        ]
    for l in range(L):
        specs += [
            (f"h{l}.ln1g", (C,), False),
            (f"h{l}.ln1b", (C,), False),
            (f"h{l}.bqkv", (3 * C,), False),
            (f"h{l}.bo", (C,), False),
            (f"h{l}.ln2g", (C,), False),
            (f"h{l}.ln2b", (C,), False),
            (f"h{l}.bfc", (F,), False),
            (f"h{l}.bfp", (C,), False),
        ]
    specs += [("lnfg", (C,), False), ("lnfb", (C,), False)]
    return specs


def param_offsets(cfg: GPT2Config) -> List[int]:
    """Element offsets of each tensor in the flat arena, plus the total."""
    offs = [0]
    for _, shape, _ in param_specs(cfg):
        offs.append(offs[-1] + int(np.prod(shape)))
    return offs


def num_params(cfg: GPT2Config) -> int:
    return param_offsets(cfg)[-1]


def num_decay_params(cfg: GPT2Config) -> int:
    return sum(int(np.prod(s)) for _, s, d in param_specs(cfg) if d)


def normal(rng: np.random.Generator, shape, std: float, mean: float = 0.0) -> np.ndarray:
    """Draw in float64, cast to float32 once."""
    return (rng.standard_normal(shape) * std + mean).astype(np.float32)


def init_params(cfg: GPT2Config, seed: int, zero_wte: bool = False) -> Dict[str, np.ndarray]:
    """GPT-2 initialisation from the hyper-parameter table (float32 values)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    res_std = 0.02 / math.sqrt(2 * cfg.L)
    out: Dict[str, np.ndarray] = {}
    for name, shape, _ in param_specs(cfg):
        base = name.split(".")[-1]
        if name == "wte":
            w = np.zeros(shape, np.float32)
            real = normal(rng, (cfg.V, cfg.C), 0.02)
            if not zero_wte:
                w[: cfg.V] = real
            out[name] = w
        elif name == "wpe" or base in ("Wqkv", "Wfc"):
            out[name] = normal(rng, shape, 0.02)
        elif base in ("Wo", "Wfp"):
            out[name] = normal(rng, shape, res_std)
        elif base in ("ln1g", "ln2g") or name == "lnfg":
            out[name] = np.ones(shape, np.float32)
        else:  # biases and LN betas
            out[name] = np.zeros(shape, np.float32)
    return out


def block_params(C: int, H: int, seed: int) -> Dict[str, np.ndarray]:
    """One transformer block with every term exercised: weights and biases
    N(0, 0.02), LN gain 1 + N(0, 0.02), LN bias N(0, 0.02)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    F = 4 * C
    p = {
        "Wqkv": normal(rng, (C, 3 * C), 0.02),
        "Wo": normal(rng, (C, C), 0.02),
        "Wfc": normal(rng, (C, F), 0.02),
        "Wfp": normal(rng, (F, C), 0.02),
        "ln1g": normal(rng, (C,), 0.02, 1.0),
        "ln1b": normal(rng, (C,), 0.02),
        "bqkv": normal(rng, (3 * C,), 0.02),
        "bo": normal(rng, (C,), 0.02),
        "ln2g": normal(rng, (C,), 0.02, 1.0),
        "ln2b": normal(rng, (C,), 0.02),
        "bfc": normal(rng, (F,), 0.02),
        "bfp": normal(rng, (C,), 0.02),
    }
    return p


def flatten(cfg: GPT2Config, params: Dict[str, np.ndarray]) -> np.ndarray:
    flat = np.empty(num_params(cfg), np.float32)
    offs = param_offsets(cfg)
    for i, (name, shape, _) in enumerate(param_specs(cfg)):
        flat[offs[i]:offs[i + 1]] = np.asarray(params[name], np.float32).reshape(-1)
    return flat


def unflatten(cfg: GPT2Config, flat: np.ndarray) -> Dict[str, np.ndarray]:
    offs = param_offsets(cfg)
    return {name: np.asarray(flat[offs[i]:offs[i + 1]]).reshape(shape)
            for i, (name, shape, _) in enumerate(param_specs(cfg))}


def zipf_tokens(n: int, V: int, s: float, seed: int) -> np.ndarray:
    """n ids with P(id = k) proportional to (k+1)^-s on [0, V), by inverse CDF."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    u = rng.random(n)
    ids = np.searchsorted(cdf, u, side="right")
    return np.minimum(ids, V - 1).astype(np.int32)


def uniform_tokens(shape, V: int, rng: np.random.Generator) -> np.ndarray:
    return rng.integers(0, V, size=shape, dtype=np.int64).astype(np.int32)


def shifted_pair(stream: np.ndarray, B: int, T: int) -> Tuple[np.ndarray, np.ndarray]:
    """x = s[0:BT], y = s[1:BT+1], each reshaped (B, T)."""
    assert stream.size >= B * T + 1
    x = stream[: B * T].reshape(B, T).copy()
    y = stream[1: B * T + 1].reshape(B, T).copy()
    return x, y
