"""Helpers shared by the GPU parity tests: tolerance metrics and oracle calls.

Tolerances (bf16 inputs, bf16 stored intermediates, fp32 accumulation):
  outputs:   max |gpu - ref| / max |ref|            <= 2e-2
  gradients: ||gpu - ref||_F / ||ref||_F  per tensor <= 3e-2
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from oracle import block as ob
from paper_2510_02483_amd import configs

OUT_TOL = 2e-2
GRAD_TOL = 3e-2


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def max_rel(gpu, ref) -> float:
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(gpu - ref)) / max(np.max(np.abs(ref)), 1e-300))


def fro_rel(gpu, ref) -> float:
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(gpu - ref) / max(np.linalg.norm(ref), 1e-300))


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def oracle_block(c, f):
    """Oracle forward + backward on float64 copies of the bf16 inputs."""
    w = {k: f[k] for k in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "attn_norm", "mlp_norm")}
    return ob.block_fwd_bwd(f["x"], w, f["dy"], n_q_heads=c.n_q_heads, n_kv_heads=c.n_kv_heads,
                            rope_theta=c.rope_theta, eps=c.rms_eps)


def bf16_randn(shape, seed, std=1.0, device="cuda"):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(shape, generator=g) * std).to(torch.bfloat16).to(device)


# Many tokens, small weights: each weight-gradient product has 1-6 output tiles
# of 256 x 256 and splits its 3000-deep contraction over 5 workgroups (the last
# slice ragged), the partial sums reduced by a second kernel.
LONG_NARROW = configs.BlockConfig("long-narrow", 18, batch=2, seq=1500, hidden=256, n_q_heads=4, n_kv_heads=2,
                                  head_dim=64, intermediate=688, rope_theta=1e4)
