"""Shared test helpers: tensor conversion and small hand-built inputs."""
import math

import numpy as np
import torch


def to_f64(t: torch.Tensor) -> np.ndarray:
    """Exact float64 copy of a bf16 (or any float) tensor."""
    return t.detach().to("cpu").float().numpy().astype(np.float64)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 (RNE) and return them as float64."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).float().numpy().astype(np.float64)


def random_head(n, d=128, seed=0, scale=1.0):
    g = np.random.default_rng(seed)
    q = bf16_round(g.standard_normal((n, d)) * scale)
    k = bf16_round(g.standard_normal((n, d)))
    v = bf16_round(g.standard_normal((n, d)))
    return q, k, v


def sink_head(n, d=128, beta=40.0, seed=0, sinks=4):
    """Query carries only a sink tag: logits are beta on keys 0..sinks-1 and exactly 0 elsewhere."""
    q = np.zeros((n, d))
    k = np.zeros((n, d))
    k[:sinks, 0] = 8.0
    q[:, 0] = bf16_round(np.array([beta * math.sqrt(d) / 8.0]))[0]
    v = bf16_round(np.random.default_rng(seed).standard_normal((n, d)))
    return q, k, v
