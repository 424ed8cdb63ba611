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
    even); both sides then read the same bf16 values;
  * a stack (make_stack_inputs) draws token ids uniformly over the vocabulary,
    the tied embedding from N(0, 0.02^2) and each block's weights as above.
"""
from __future__ import annotations

import torch

from .configs import BlockConfig, StackConfig

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


def _normal(shape, seed: int, std: float, mean: float = 0.0, device="cpu") -> torch.Tensor:
    g = torch.Generator(device=device).manual_seed(seed)
    t = torch.randn(shape, generator=g, dtype=torch.float32, device=device)
    if std != 1.0:
        t.mul_(std)
    if mean != 0.0:
        t.add_(mean)
    return t.to(torch.bfloat16)


def make_inputs(cfg: BlockConfig, *, seed_base: int | None = None, gamma: str = "ones",
                w_std: float = 0.02, wq_std: float | None = None, activations: bool = True,
                device="cpu") -> dict:
    """Return bf16 CPU tensors: x, dy [batch, seq, hidden], the seven projection
    weights (row-major [out, in]) and the two RMSNorm gains [hidden].

    ``wq_std`` overrides the std of wq only; a large value sharpens the softmax
    (logits with std of several units) so that the running max matters.
    """
    base = 1000 * cfg.cfg_id if seed_base is None else seed_base
    shapes = weight_shapes(cfg)
    act_shape = (cfg.batch, cfg.seq, cfg.hidden)
    out = {}
    if activations:
        out["x"] = _normal(act_shape, base + 0, 1.0, device=device)
        out["dy"] = _normal(act_shape, base + 1, 1.0, device=device)
    for k, name in enumerate(WEIGHT_NAMES):
        std = w_std
        if name == "wq" and wq_std is not None:
            std = wq_std
        out[name] = _normal(shapes[name], base + 2 + k, std, device=device)
    for k, name in enumerate(NORM_NAMES):
        if gamma == "ones":
            out[name] = torch.ones(shapes[name], dtype=torch.bfloat16, device=device)
        elif gamma == "random":
            out[name] = _normal(shapes[name], base + 9 + k, 0.1, mean=1.0, device=device)
        else:
            raise ValueError(f"gamma must be 'ones' or 'random', got {gamma!r}")
    return out


def make_stack_inputs(sc: StackConfig, *, gamma: str = "ones", e_std: float = 0.02, w_std: float = 0.02,
                      device="cpu") -> dict:
    """Inputs of a stack (seeds from 1000 * block.cfg_id): token ids uniform
    over the vocabulary (int32, seed base + 0), the tied embedding ~ N(0,
    e_std^2) (base + 1), the final RMSNorm gain (ones, or 1 + 0.1 N(0, 1) from
    base + 2), and for block l the weights of make_inputs with seed base
    1000 * block.cfg_id + 100 * (l + 1).  ``device`` = "cuda" draws on the GPU's
    generator (other values than the CPU's, same distributions)."""
    base = 1000 * sc.block.cfg_id
    H = sc.block.hidden
    g = torch.Generator(device=device).manual_seed(base)
    ids = torch.randint(0, sc.vocab, (sc.block.batch, sc.block.seq), generator=g, device=device,
                        dtype=torch.int64).to(torch.int32)
    out = {"ids": ids, "embed": _normal((sc.vocab, H), base + 1, e_std, device=device)}
    if gamma == "ones":
        out["final_norm"] = torch.ones((H,), dtype=torch.bfloat16, device=device)
    else:
        out["final_norm"] = _normal((H,), base + 2, 0.1, mean=1.0, device=device)
    out["layers"] = [make_inputs(sc.block, seed_base=base + 100 * (l + 1), gamma=gamma, w_std=w_std,
                                 activations=False, device=device) for l in range(sc.n_layers)]
    return out


def to_f64(inputs: dict):
    """Exact upcast of the bf16 tensors to numpy float64 arrays."""
    return {k: v.to(torch.float64).numpy() for k, v in inputs.items()}
