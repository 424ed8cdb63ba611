"""Shape presets for one Llama-style decoder block (pre-norm, RMSNorm, RoPE,
causal grouped-query attention, SwiGLU MLP), as named in the Litespark
report's model description (Section 2.4, Table 1) and in the workloads this
library is measured on.

Pure data: no arithmetic of the method lives here.
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class BlockConfig:
    name: str
    cfg_id: int          # seeds the synthetic inputs (1000 * cfg_id + k)
    batch: int
    seq: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    intermediate: int
    rope_theta: float
    rms_eps: float = 1e-5

    @property
    def tokens(self) -> int:
        return self.batch * self.seq

    @property
    def dq(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def dkv(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def with_(self, **kw) -> "BlockConfig":
        return replace(self, **kw)


# Tiny block: parity case small enough for the fp64 oracle in well under a second.
TINY = BlockConfig("tiny", 0, batch=2, seq=128, hidden=256, n_q_heads=4, n_kv_heads=2,
                   head_dim=64, intermediate=688, rope_theta=1e4)
# Llama-3.2-3B-shaped block at sequence 2048, batch 4: the measured workload.
B3 = BlockConfig("3b", 1, batch=4, seq=2048, hidden=3072, n_q_heads=24, n_kv_heads=8,
                 head_dim=128, intermediate=8192, rope_theta=5e5)
# Same block at long context (attention-dominated).
B3_8K = BlockConfig("3b_8k", 2, batch=1, seq=8192, hidden=3072, n_q_heads=24, n_kv_heads=8,
                    head_dim=128, intermediate=8192, rope_theta=5e5)
# Llama-30B-shaped block, multi-head attention (kv heads = q heads).
B30 = BlockConfig("30b", 3, batch=2, seq=2048, hidden=6656, n_q_heads=52, n_kv_heads=52,
                  head_dim=128, intermediate=17920, rope_theta=1e4)

# The report's own 3B model (Table 1: hidden 2048, 16 query / 2 kv heads of 128,
# SwiGLU 11008) at sequence 4096, micro-batch 2.
PAPER_3B = BlockConfig("paper_3b", 8, batch=2, seq=4096, hidden=2048, n_q_heads=16, n_kv_heads=2,
                       head_dim=128, intermediate=11008, rope_theta=1e4)

# The report's own 30B block (Table 1: hidden 6656, 64 heads of 104, multi-head,
# SwiGLU 17920) at sequence 4096, micro-batch 2.
PAPER_30B = BlockConfig("paper_30b", 12, batch=2, seq=4096, hidden=6656, n_q_heads=64, n_kv_heads=64,
                        head_dim=104, intermediate=17920, rope_theta=1e4)

PRESETS = {c.name: c for c in (TINY, B3, B3_8K, B30, PAPER_3B, PAPER_30B)}


@dataclass(frozen=True)
class StackConfig:
    """A stack of identical blocks between a tied token embedding and a final
    RMSNorm + LM head, trained on next-token cross-entropy (Section 2.4)."""
    name: str
    block: BlockConfig   # shape of every block; block.cfg_id seeds the inputs
    n_layers: int
    vocab: int
    recompute: bool = True  # keep only block inputs; recompute each block in the backward
    logits_chunk: int = 0   # token rows of logits formed at a time (0: as many as fit one 2047 MiB operand)

    @property
    def tokens(self) -> int:
        return self.block.tokens

    def with_(self, **kw) -> "StackConfig":
        return replace(self, **kw)


# Small stack: parity case for the fp64 oracle (a few seconds).
TINY_STACK = StackConfig("tiny_stack", TINY.with_(name="tiny_stack_block", cfg_id=10, batch=2, seq=64),
                         n_layers=2, vocab=1000)
# Llama-3.2-3B-shaped model: 28 blocks, vocabulary 128256, micro-batch 4 x 2048.
STACK_3B = StackConfig("3b_stack", B3.with_(name="3b_stack_block", cfg_id=4), n_layers=28, vocab=128256)

# The report's 3B model whole (Table 1: 28 blocks; vocabulary 32000), micro-batch 2 x 4096.
PAPER_3B_STACK = StackConfig("paper_3b_stack", PAPER_3B.with_(name="paper_3b_stack_block", cfg_id=9),
                             n_layers=28, vocab=32000)

STACK_PRESETS = {c.name: c for c in (TINY_STACK, STACK_3B, PAPER_3B_STACK)}
