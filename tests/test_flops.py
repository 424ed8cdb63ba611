"""FLOP accounting against the report's throughput tables (Tables 3 and 4)
and against direct counting on small shapes."""
import os

import pytest

from paper_2510_02483_amd import configs
from paper_2510_02483_amd.flops import (block_fwd_bwd_flops, block_fwd_flops,
                                        training_flops_per_token)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_throughput_tables.txt")
SHAPES = {"3B": (28, 2048, 16, 2, 11008), "30B": (60, 6656, 64, 64, 17920)}


def _rows():
    with open(GOLDEN) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                m, g, tps, tf, mfu = line.split()
                yield m, int(g), float(tps), float(tf), float(mfu)


@pytest.mark.parametrize("row", list(_rows()), ids=lambda r: f"{r[0]}-{r[1]}gpu")
def test_paper_flops_per_token(row):
    """TFLOP/s per GPU divided by tokens/s per GPU is the FLOPs per token the
    tables assume; it matches 6N + 12 L H s at s = 4096, vocabulary 32000."""
    m, g, tps, tf, _ = row
    implied = tf * 1e12 / (tps / g)
    ours = training_flops_per_token(*SHAPES[m], vocab=32000, seq=4096)
    tol = 2e-2 if (m, g) in (("3B", 256), ("30B", 512)) else 2e-5  # two rows carry rounding drift
    assert abs(implied / ours - 1) < tol


def test_paper_mfu_uses_h200_peak():
    for m, g, tps, tf, mfu in _rows():
        assert abs(tf / (mfu / 100) - 989) < 12  # MFU = TFLOP/s per GPU / ~989


def test_block_flops_direct_count():
    c = configs.TINY.with_(batch=1, seq=5)
    gemm = 0
    H, dq, dkv, I, T = c.hidden, c.dq, c.dkv, c.intermediate, c.tokens
    for (m, n, k) in ((T, dq, H), (T, dkv, H), (T, dkv, H), (T, H, dq), (T, I, H), (T, I, H), (T, H, I)):
        gemm += 2 * m * n * k
    pairs = sum(i + 1 for i in range(c.seq))  # causal: key j <= query i
    attn = c.n_q_heads * pairs * c.head_dim * 2 * 2
    assert block_fwd_flops(c) == gemm + attn
    assert block_fwd_bwd_flops(c) == 3 * (gemm + attn)
    assert block_fwd_flops(c, causal=False) == gemm + c.n_q_heads * c.seq ** 2 * c.head_dim * 4


def test_3b_block_total():
    assert abs(block_fwd_bwd_flops(configs.B3) / 1e12 - 5.2572) < 1e-3


def test_launch_flops_sum_to_the_block():
    """The labelled launches of a block step carry all of its model FLOPs."""
    from paper_2510_02483_amd import configs, flops
    for c in (configs.B3, configs.TINY, configs.B30, configs.PAPER_3B):
        lf = flops.launch_flops(c)
        assert set(lf) <= set(flops.BLOCK_LAUNCHES)
        assert abs(sum(lf.values()) - flops.block_fwd_bwd_flops(c)) < 1e-6 * flops.block_fwd_bwd_flops(c)
    lf = flops.launch_flops(configs.B3)
    # the three 0.82-TFLOP products of the MLP
    assert lf["gate/up projection"] == lf["dh2"] == lf["dWg/dWu"] == 2.0 * 8192 * 16384 * 3072


def test_profile_launch_labelling():
    """Dispatches of block steps are named after their launches by position,
    split-K reductions joining their product, set-up kernels left out."""
    from paper_2510_02483_amd import profiling
    g = "gemm_kernel<...>"
    step = (["rmsnorm_fwd_kernel<6>", "rope_table_kernel", g, "attn_fwd_kernel<128>", g, "rmsnorm_fwd_kernel<6>", g, g,
             g, g, g, g, "kpart_reduce_kernel", "rmsnorm_bwd_kernel<6>", "column_sum_kernel", "rope_table_kernel", g, g,
             "attn_bwd_pre_kernel<128>", "attn_bwd_dkdv_kernel<128, true>", "attn_bwd_dkdv_reduce<128>",
             "attn_bwd_dq_kernel<128>", g, g, "rmsnorm_bwd_kernel<6>", "column_sum_kernel"])
    names = ["FillFunctor"] + step + step + ["copyBuffer"]
    steps = profiling.label_steps(names)
    assert len(steps) == 2
    labels = [lab for _, lab in steps[0]]
    assert labels[2] == "qkv projection" and labels[3] == "attention fwd"
    assert labels[8:11] == ["dact", "dh2", "dWg/dWu"]
    assert labels[11:13] == ["dWd", "dWd"]  # the split-K reduction belongs to its product
    assert labels.count("attention bwd") == 4 and labels.count("rmsnorm bwd") == 4
    assert [lab for lab in labels if lab in profiling.GEMM_ORDER][-1] == "dWqkv"
    assert steps[1][0][0] == 1 + len(step)
