"""ls_attn_core_bwd_noalloc (no workspace argument; its scratch is a device
array the library owns) against ls_attn_core_bwd with a caller workspace:
same kernels, so the gradients must agree bit for bit.  Three calls in a row
share the array, each smaller than the one before: a split dK/dV group with
128-wide heads, a split group with 64-wide heads, and multi-head attention
(unsplit)."""
import pytest
import torch

from paper_2510_02483_amd import configs, lib as L

from gpu_util import bf16_randn, need_gpu, say

pytestmark = pytest.mark.gpu

CASES = [
    # name, batch, seq, nq, nkv, d: each needs less scratch than the one before
    ("split-d128", 1, 512, 16, 4, 128),
    ("split-d64-ragged", 2, 200, 4, 2, 64),
    ("mha-d64", 1, 136, 2, 2, 64),
]


def _inputs(B, S, nq, nkv, d, seed):
    c = configs.TINY.with_(batch=B, seq=S, n_q_heads=nq, n_kv_heads=nkv, head_dim=d, hidden=nq * d)
    T = B * S
    qkv = torch.cat([bf16_randn((T, nq * d), seed, 1.5), bf16_randn((T, nkv * d), seed + 1, 1.5),
                     bf16_randn((T, nkv * d), seed + 2)], dim=1).contiguous()
    o = torch.empty((T, nq * d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((B, nq, S), dtype=torch.float32, device="cuda")
    L.ls_attn_core_fwd(c, qkv, o, lse)
    do = bf16_randn((T, nq * d), seed + 3)
    return c, qkv, o, lse, do


def test_noalloc_matches_workspace_call():
    need_gpu()
    prev = None
    for i, (name, B, S, nq, nkv, d) in enumerate(CASES):
        say(f"no-alloc attention backward, call {i + 1}: {name} B={B} S={S} nq={nq} nkv={nkv} d={d}")
        c, qkv, o, lse, do = _inputs(B, S, nq, nkv, d, 40 + 10 * i)
        need = L.ls_attn_core_bwd_workspace(c)
        assert prev is None or need < prev, "each call smaller than the last"
        prev = need
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        ref = torch.empty_like(qkv)
        L.ls_attn_core_bwd(c, qkv, o, lse, do, ref, ws)
        out = torch.full_like(qkv, float("nan"))
        L.ls_attn_core_bwd_noalloc(c, qkv, o, lse, do, out)
        torch.cuda.synchronize()
        assert torch.equal(out, ref), name


def test_noalloc_rejects_shapes_beyond_its_scratch():
    need_gpu()
    c = configs.PAPER_3B   # split dK/dV partials of ~67 MB
    assert L.ls_attn_core_bwd_workspace(c) > L.NOALLOC_SCRATCH_BYTES
    T = c.tokens
    qkv = torch.zeros((T, c.dq + 2 * c.dkv), dtype=torch.bfloat16, device="cuda")
    o = torch.zeros((T, c.dq), dtype=torch.bfloat16, device="cuda")
    lse = torch.zeros((c.batch, c.n_q_heads, c.seq), dtype=torch.float32, device="cuda")
    dqkv = torch.empty_like(qkv)
    with pytest.raises(L.LsError) as e:
        L.ls_attn_core_bwd_noalloc(c, qkv, o, lse, o, dqkv)
    assert e.value.status == 6 and "scratch" in str(e.value)
