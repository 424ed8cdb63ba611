"""Decoder-block parity on the GPU: sub-layers and the whole forward+backward
through the C ABI against the fp64 oracle on the same seeded bf16 inputs."""
import numpy as np
import pytest
import torch

from paper_2510_02483_amd import configs, inputs, lib as L

from gpu_util import GRAD_TOL, LONG_NARROW, OUT_TOL, f64, fro_rel, max_rel, need_gpu, oracle_block, say

pytestmark = pytest.mark.gpu

GRAD_NAMES = L.WEIGHTS

# parity cases: several tiles and ragged tails in every dimension
MID_D64 = configs.BlockConfig("mid-d64", 5, batch=2, seq=320, hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=64,
                              intermediate=1400, rope_theta=1e4)
MID_D128 = configs.BlockConfig("mid-d128", 6, batch=1, seq=200, hidden=768, n_q_heads=6, n_kv_heads=3,
                               head_dim=128, intermediate=1032, rope_theta=5e5)
MHA_D128 = configs.BlockConfig("mha-d128", 7, batch=2, seq=130, hidden=512, n_q_heads=4, n_kv_heads=4,
                               head_dim=128, intermediate=520, rope_theta=1e4)

# head sizes held in 128-wide slots (104: the report's 30B model; 72: another in-between size)
D104_GQA = configs.BlockConfig("d104-gqa", 13, batch=2, seq=130, hidden=416, n_q_heads=4, n_kv_heads=2,
                               head_dim=104, intermediate=520, rope_theta=1e4)
D104_MHA = configs.BlockConfig("d104-mha", 14, batch=1, seq=200, hidden=624, n_q_heads=6, n_kv_heads=6,
                               head_dim=104, intermediate=1040, rope_theta=1e4)
# sequences of one token: attention returns each token's own value row
ONE_TOKEN = configs.BlockConfig("one-token", 16, batch=3, seq=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                                intermediate=688, rope_theta=1e4)
D72 = configs.BlockConfig("d72", 15, batch=2, seq=96, hidden=288, n_q_heads=4, n_kv_heads=1, head_dim=72,
                          intermediate=392, rope_theta=5e5)
# hidden != n_q_heads * head_dim: the query/output projections narrow (384 -> 256
# features) or widen (256 -> 768) the model width
NARROW_HEADS = configs.BlockConfig("narrow-heads", 19, batch=2, seq=136, hidden=384, n_q_heads=4, n_kv_heads=2,
                                   head_dim=64, intermediate=1040, rope_theta=1e4)
WIDE_HEADS = configs.BlockConfig("wide-heads", 20, batch=1, seq=200, hidden=256, n_q_heads=6, n_kv_heads=2,
                                 head_dim=128, intermediate=688, rope_theta=5e5)
# multi-head attention with 64-wide heads: one query head per kv head, so the
# dK/dV kernel never splits a group (its unsplit 64-wide variant, with the
# inverse RoPE on the dK store)
MHA_D64 = configs.BlockConfig("mha-d64", 21, batch=2, seq=200, hidden=256, n_q_heads=4, n_kv_heads=4, head_dim=64,
                              intermediate=520, rope_theta=1e4)

BLOCK_CASES = [
    ("d104-gqa", D104_GQA, {"gamma": "random"}),
    ("d104-mha-sharp", D104_MHA, {"wq_std": 0.3}),
    ("d72", D72, {"gamma": "random"}),
    ("one-token-sequences", ONE_TOKEN, {"gamma": "random"}),
    ("tiny", configs.TINY, {}),
    ("tiny-random-gamma", configs.TINY, {"gamma": "random"}),
    ("tiny-sharp", configs.TINY, {"wq_std": 0.6}),
    ("mid-d64", MID_D64, {"gamma": "random"}),
    ("mid-d128", MID_D128, {}),
    ("mha-d128-sharp", MHA_D128, {"wq_std": 0.3}),
    ("long-narrow", LONG_NARROW, {"gamma": "random"}),
    ("hidden-384-heads-4x64", NARROW_HEADS, {"gamma": "random"}),
    ("hidden-256-heads-6x128-sharp", WIDE_HEADS, {"wq_std": 0.3}),
    ("mha-d64", MHA_D64, {"gamma": "random"}),
    ("mha-d64-sharp", MHA_D64, {"wq_std": 0.4}),
]


def compare_block(c, blk, fwd, gr, sample=slice(None)):
    T_H = (c.batch, c.seq, c.hidden)
    y = f64(blk.y).reshape(T_H)[sample]
    dx = f64(blk.dx).reshape(T_H)[sample]
    errs = {"y": max_rel(y, fwd["y"]), "dx": fro_rel(dx, gr["dx"])}
    for n in GRAD_NAMES:
        ref = gr[n]
        if not np.any(ref):
            # A gradient that is exactly zero (one-token sequences: the softmax
            # of a single key is 1 whatever q and k are, so dWq = dWk = 0) has
            # no relative error; its norm is measured against the value
            # projection's gradient of the same sub-layer instead.
            errs[n] = float(np.linalg.norm(f64(blk.grads[n]))) / float(np.linalg.norm(gr["wv"]))
        else:
            errs[n] = fro_rel(f64(blk.grads[n]), ref)
    say("  errors:", {k: f"{v:.2e}" for k, v in errs.items()})
    assert errs["y"] < OUT_TOL, errs
    for k, v in errs.items():
        if k != "y":
            assert v < GRAD_TOL, (k, errs)


@pytest.mark.parametrize("name,c,kw", BLOCK_CASES, ids=[b[0] for b in BLOCK_CASES])
def test_block_parity(name, c, kw):
    need_gpu()
    say(f"block parity {name} {c}")
    host = inputs.make_inputs(c, **kw)
    blk = L.Block(c, host)
    blk.step()
    torch.cuda.synchronize()
    fwd, gr = oracle_block(c, inputs.to_f64(host))
    compare_block(c, blk, fwd, gr)


@pytest.mark.parametrize("c", [MID_D64, D104_GQA, LONG_NARROW, NARROW_HEADS, WIDE_HEADS],
                         ids=["d64", "d104-padded", "split-k", "hidden-384-heads-4x64", "hidden-256-heads-6x128"])
def test_sublayers_match_block_call(c):
    """ls_attn_fwd / ls_mlp_fwd / ls_mlp_bwd / ls_attn_bwd chained by hand give
    the oracle's intermediates (x2, dx2) and final results (also with heads of
    104 in padded slots, whose saved state and workspace the separate calls
    pass between them)."""
    need_gpu()
    say(f"sub-layers {c}")
    host = inputs.make_inputs(c, gamma="random")
    dev = {k: v.cuda() for k, v in host.items()}
    T, H = c.tokens, c.hidden
    x = dev["x"].reshape(T, H)
    dy = dev["dy"].reshape(T, H)
    w = {n: dev[n] for n in GRAD_NAMES}
    s = L.ls_query_sizes(c)
    asv = torch.empty(s["attn_saved"], dtype=torch.uint8, device="cuda")
    msv = torch.empty(s["mlp_saved"], dtype=torch.uint8, device="cuda")
    aws = torch.empty(s["attn_workspace"], dtype=torch.uint8, device="cuda")
    mws = torch.empty(s["mlp_workspace"], dtype=torch.uint8, device="cuda")
    x2, y, dx2, dx = (torch.empty_like(x) for _ in range(4))
    g = {n: torch.zeros(w[n].shape, dtype=torch.float32, device="cuda") for n in GRAD_NAMES}
    L.ls_attn_fwd(c, x, w, x2, asv, aws)
    L.ls_mlp_fwd(c, x2, w, y, msv, mws)
    L.ls_mlp_bwd(c, x2, w, msv, dy, dx2, g, False, mws)
    aws.fill_(255)  # the backward rebuilds whatever it needs in its workspace
    L.ls_attn_bwd(c, x, w, asv, dx2, dx, g, False, aws)
    torch.cuda.synchronize()
    fwd, gr = oracle_block(c, inputs.to_f64(host))
    shp = (c.batch, c.seq, H)
    assert max_rel(f64(x2).reshape(shp), fwd["x2"]) < OUT_TOL
    assert max_rel(f64(y).reshape(shp), fwd["y"]) < OUT_TOL
    assert fro_rel(f64(dx2).reshape(shp), gr["dx2"]) < GRAD_TOL
    assert fro_rel(f64(dx).reshape(shp), gr["dx"]) < GRAD_TOL
    for n in GRAD_NAMES:
        assert fro_rel(f64(g[n]), gr[n]) < GRAD_TOL, n


@pytest.mark.parametrize("c", [configs.TINY, LONG_NARROW], ids=["tiny", "split-k"])
def test_accumulate_and_side_stream(c):
    """accumulate=1 adds into the fp32 gradients (also where the weight
    gradients split K: the first slice adds, the others' partial sums follow);
    a non-default stream works."""
    need_gpu()
    say(f"accumulate / side stream {c.name}")
    host = inputs.make_inputs(c, gamma="random")
    blk = L.Block(c, host)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        blk.step(accumulate=False)
        first = {n: blk.grads[n].clone() for n in GRAD_NAMES}
        blk.step(accumulate=True)
    s.synchronize()
    for n in GRAD_NAMES:
        assert max_rel(f64(blk.grads[n]), 2 * f64(first[n])) < 1e-5, n
    fwd, gr = oracle_block(c, inputs.to_f64(host))
    compare_block(c, blk, fwd, {**gr, **{n: 2 * gr[n] for n in GRAD_NAMES}})


def _full_parity(c):
    """The block at its full size and launch configuration, every sequence
    with its own upstream gradient, against the oracle on the whole batch:
    y and dx of every token and each weight gradient over all batch x seq
    rows of its contraction."""
    host = inputs.make_inputs(c)
    blk = L.Block(c, host)
    blk.step()
    torch.cuda.synchronize()
    say(f"  oracle on the whole batch ({c.batch} x {c.seq}) ...")
    fwd, gr = oracle_block(c, inputs.to_f64(host))
    compare_block(c, blk, fwd, gr)


def test_block_3b_full_size():
    """The Llama-3.2-3B-shaped block at its full size (batch 4 x seq 2048):
    the benchmark's workload and launch configuration, compared in full."""
    need_gpu()
    c = configs.B3
    say(f"3b full size {c}")
    _full_parity(c)


def _prefix_parity(c, t0, sample_seq=0):
    """The block at its full size and launch configuration, checked against
    the oracle on the first t0 tokens of one sequence.  The upstream gradient
    is zero past t0 and on every other sequence, so (causality) the outputs
    of the first t0 tokens, dx of those tokens and every weight gradient are
    those of the t0-token sequence alone, and dx is exactly zero past t0."""
    host = inputs.make_inputs(c)
    full = host["dy"].clone()
    host["dy"].zero_()
    host["dy"][sample_seq, :t0] = full[sample_seq, :t0]
    blk = L.Block(c, host)
    blk.step()
    torch.cuda.synchronize()
    one = c.with_(batch=1, seq=t0)
    f = inputs.to_f64({k: (v[sample_seq:sample_seq + 1, :t0] if k in ("x", "dy") else v) for k, v in host.items()})
    say(f"  oracle on sequence {sample_seq}, tokens 0..{t0 - 1} ...")
    fwd, gr = oracle_block(one, f)
    shp = (c.batch, c.seq, c.hidden)
    y = f64(blk.y).reshape(shp)[sample_seq:sample_seq + 1, :t0]
    dx_all = f64(blk.dx).reshape(shp)
    dx = dx_all[sample_seq:sample_seq + 1, :t0]
    errs = {"y": max_rel(y, fwd["y"]), "dx": fro_rel(dx, gr["dx"])}
    for n in GRAD_NAMES:
        errs[n] = fro_rel(f64(blk.grads[n]), gr[n])
    say("  errors:", {k: f"{v:.2e}" for k, v in errs.items()})
    assert errs["y"] < OUT_TOL, errs
    for k, v in errs.items():
        if k != "y":
            assert v < GRAD_TOL, (k, errs)
    # no upstream gradient past t0 (or on the other sequences): no input gradient there
    rest = dx_all.copy()
    rest[sample_seq, :t0] = 0
    assert np.count_nonzero(rest) == 0
    return blk, host


def test_block_3b_8k_full_size_prefix():
    """The 3B block at long context (batch 1 x seq 8192), full launch
    configuration; oracle on the first 1024 tokens (the fp64 oracle of the
    whole 8k sequence takes minutes)."""
    need_gpu()
    c = configs.B3_8K
    say(f"3b_8k full size {c}")
    _prefix_parity(c, 1024)


def test_block_30b_full_size():
    """The Llama-30B-shaped block (batch 2 x seq 2048, 52 MHA heads, SwiGLU
    17920) at full size, compared in full."""
    need_gpu()
    c = configs.B30
    say(f"30b full size {c}")
    _full_parity(c)


def test_block_paper_3b_full_size_prefix():
    """The report's own 3B block (Table 1: hidden 2048, 16 query heads sharing
    2 kv heads, SwiGLU 11008) at batch 2 x seq 4096, full launch
    configuration; oracle on the first 768 tokens of sequence 1."""
    need_gpu()
    c = configs.PAPER_3B
    say(f"paper 3b full size {c}")
    _prefix_parity(c, 768, sample_seq=1)


def test_block_paper_30b_full_size_prefix():
    """The report's own 30B block (Table 1: hidden 6656, 64 heads of 104 in
    128-wide slots, SwiGLU 17920) at batch 2 x seq 4096; oracle on the first
    256 tokens of sequence 0."""
    need_gpu()
    c = configs.PAPER_30B
    say(f"paper 30b full size {c}")
    _prefix_parity(c, 256)
