"""FLOP accounting for the block and for whole-model throughput.

Model FLOPs count each multiply-add as two FLOPs, the backward pass as twice
the forward, and no recomputation.  Causal attention counts only the
S(S+1)/2 query-key pairs that the mask keeps; the non-causal convention
(the one the report's throughput tables follow, Tables 3 and 4) counts S^2.
"""
from __future__ import annotations

from .configs import BlockConfig, StackConfig


def block_params(hidden: int, dq: int, dkv: int, inter: int) -> int:
    """Weights of the seven projections of one block (norm gains excluded)."""
    return hidden * (dq + 2 * dkv) + dq * hidden + 3 * hidden * inter


def block_fwd_flops(cfg: BlockConfig, causal: bool = True) -> float:
    gemm = 2.0 * cfg.tokens * block_params(cfg.hidden, cfg.dq, cfg.dkv, cfg.intermediate)
    pairs = cfg.seq * (cfg.seq + 1) / 2 if causal else float(cfg.seq) ** 2
    attn = 4.0 * cfg.batch * cfg.n_q_heads * cfg.head_dim * pairs  # QK^T and PV
    return gemm + attn


def block_fwd_bwd_flops(cfg: BlockConfig, causal: bool = True) -> float:
    """Model FLOPs of one forward plus backward pass (backward = 2 x forward)."""
    return 3.0 * block_fwd_flops(cfg, causal)


def attention_fwd_flops(cfg: BlockConfig, causal: bool = True) -> float:
    """QK^T and PV of the attention forward pass (model FLOPs)."""
    pairs = cfg.seq * (cfg.seq + 1) / 2 if causal else float(cfg.seq) ** 2
    return 4.0 * cfg.batch * cfg.n_q_heads * cfg.head_dim * pairs


def attention_fwd_bwd_flops(cfg: BlockConfig, causal: bool = True) -> float:
    pairs = cfg.seq * (cfg.seq + 1) / 2 if causal else float(cfg.seq) ** 2
    return 3.0 * 4.0 * cfg.batch * cfg.n_q_heads * cfg.head_dim * pairs


def training_flops_per_token(n_layers: int, hidden: int, n_heads: int, n_kv_heads: int,
                             inter: int, vocab: int, seq: int) -> float:
    """Whole-model training FLOPs per token, non-causal attention convention:
    6 * (layer weights + LM head) + 12 * layers * hidden * seq."""
    d = hidden // n_heads
    n = n_layers * block_params(hidden, n_heads * d, n_kv_heads * d, inter) + vocab * hidden
    return 6.0 * n + 12.0 * n_layers * hidden * seq


def lm_head_fwd_bwd_flops(tokens: int, hidden: int, vocab: int) -> float:
    """Logits h E^T, and in the backward dh = dz E and dE = dz^T h."""
    return 3.0 * 2.0 * tokens * hidden * vocab


def stack_fwd_bwd_flops(sc: StackConfig, causal: bool = True) -> float:
    """Model FLOPs of the stack's forward plus backward pass: every block and
    the tied LM head (recomputation in the backward pass is not counted)."""
    return sc.n_layers * block_fwd_bwd_flops(sc.block, causal) + \
        lm_head_fwd_bwd_flops(sc.tokens, sc.block.hidden, sc.vocab)


# Labelled launches of one block step (forward, then the MLP and attention
# backward passes) in the order the library issues them.
BLOCK_LAUNCHES = ("rmsnorm fwd", "qkv projection", "attention fwd", "output projection", "gate/up projection",
                  "down projection", "dact", "dh2", "dWg/dWu", "dWd", "rmsnorm bwd", "dO", "dWo", "attention bwd",
                  "dh1", "dWqkv")


def launch_flops(cfg: BlockConfig) -> dict:
    """Model FLOPs of each labelled matrix-product and attention launch of one
    block step (2 M N K per product; attention backward = 2 x forward).  The
    RMSNorm launches are bandwidth-bound and carry no entry."""
    T, H, I, dq, dkv = cfg.tokens, cfg.hidden, cfg.intermediate, cfg.dq, cfg.dkv
    dqkv = dq + 2 * dkv
    att = attention_fwd_flops(cfg)
    return {"qkv projection": 2.0 * T * dqkv * H, "attention fwd": att, "output projection": 2.0 * T * H * dq,
            "gate/up projection": 2.0 * T * 2 * I * H, "down projection": 2.0 * T * H * I,
            "dact": 2.0 * T * I * H, "dWd": 2.0 * T * H * I, "dh2": 2.0 * T * 2 * I * H,
            "dWg/dWu": 2.0 * T * 2 * I * H, "dO": 2.0 * T * dq * H, "dWo": 2.0 * T * H * dq,
            "attention bwd": 2.0 * att, "dh1": 2.0 * T * dqkv * H, "dWqkv": 2.0 * T * dqkv * H}
