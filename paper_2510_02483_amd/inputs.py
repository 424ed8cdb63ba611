"""Seeded synthetic inputs for one decoder block.

This module is shared by the GPU path's harness and by the tests that feed the
fp64 oracle; it holds none of the block's arithmetic, only random draws.

Recipe (the report trains on a text corpus; seeded normals of the same shapes
stand in for its activations, and its weights are random-initialised):
  * one torch CPU generator per tensor, seeded 1000 * cfg_id + k with k fixed in
    the order x, dy, wq, wk, wv, wo, wg, wu, wd, attn_norm, mlp_norm;
  * x, dy ~ N(0, 1); projection weights ~ N(0, 0.02^2);
  * RMSNorm gains are ones (their usual initialisation) unless ``gamma="random"``,
    which draws 1 + 0.1 * N(0, 1) so that the gain multiplies something other
    than one;
  * every draw is made in fp32 and rounded once to bf16 (round to nearest
    even); both sides then read the same bf16 values.
"""
from __future__ import annotations

import torch

from .configs import BlockConfig

WEIGHT_NAMES = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")
NORM_NAMES = ("attn_norm", "mlp_norm")


def weight_shapes(cfg: BlockConfig) -> dict:
    H, I = cfg.hidden, cfg.intermediate
    return {
        "wq": (cfg.dq, H), "wk": (cfg.dkv, H), "wv": (cfg.dkv, H),
        "wo": (H, cfg.dq),
        "wg": (I, H), "wu": (I, H), "wd": (H, I),
        "attn_norm": (H,), "mlp_norm": (H,),
    }


def _normal(shape, seed: int, std: float, mean: float = 0.0) -> torch.Tensor:
    g = torch.Generator(device="cpu").manual_seed(seed)
    t = torch.randn(shape, generator=g, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    if mean != 0.0:
        t.add_(mean)
    return t.to(torch.bfloat16)


def make_inputs(cfg: BlockConfig, *, seed_base: int | None = None, gamma: str = "ones",
                w_std: float = 0.02, wq_std: float | None = None) -> dict:
    """Return bf16 CPU tensors: x, dy [batch, seq, hidden], the seven projection
    weights (row-major [out, in]) and the two RMSNorm gains [hidden].

    ``wq_std`` overrides the std of wq only; a large value sharpens the softmax
    (logits with std of several units) so that the running max matters.
    """
    base = 1000 * cfg.cfg_id if seed_base is None else seed_base
    shapes = weight_shapes(cfg)
    act_shape = (cfg.batch, cfg.seq, cfg.hidden)
    out = {
        "x": _normal(act_shape, base + 0, 1.0),
        "dy": _normal(act_shape, base + 1, 1.0),
    }
    for k, name in enumerate(WEIGHT_NAMES):
        std = w_std
        if name == "wq" and wq_std is not None:
            std = wq_std
        out[name] = _normal(shapes[name], base + 2 + k, std)
    for k, name in enumerate(NORM_NAMES):
        if gamma == "ones":
            out[name] = torch.ones(shapes[name], dtype=torch.bfloat16)
        elif gamma == "random":
            out[name] = _normal(shapes[name], base + 9 + k, 0.1, mean=1.0)
        else:
            raise ValueError(f"gamma must be 'ones' or 'random', got {gamma!r}")
    return out


def to_f64(inputs: dict):
    """Exact upcast of the bf16 tensors to numpy float64 arrays."""
    return {k: v.to(torch.float64).numpy() for k, v in inputs.items()}
