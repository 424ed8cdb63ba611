"""Per-kernel parity on the GPU: matrix products, RMSNorm and the attention
core, each called through the C ABI and compared with the fp64 oracle (or
numpy fp64 products of the same bf16 operands) element by element."""
import math

import numpy as np
import pytest
import torch

from oracle import block as ob
from paper_2510_02483_amd import configs, lib as L

from gpu_util import GRAD_TOL, OUT_TOL, bf16_randn, f64, fro_rel, max_rel, need_gpu, say

pytestmark = pytest.mark.gpu

# the 4104 x 4200 shape has more output tiles than compute units (17 x 17 and
# more), so its products run persistent: workgroups walk several tiles, ragged
# ones included.  K takes ragged tile counts (the masked loop) and whole ones of
# 1, 2, 3, 9 and 10 tiles of 64 (the unmasked loop, which with one wave per SIMD
# runs two tiles per pass: an odd count leaves one tile for the masked loop).
GEMM_SHAPES = [(136, 264, 72), (520, 776, 1000), (256, 512, 640), (8, 8, 8), (1032, 264, 1376), (392, 584, 200),
               (4104, 4200, 264), (136, 200, 64), (264, 136, 128), (200, 264, 192), (264, 392, 576)]
# workgroup tile shapes: automatic choice, then each forced shape (products
# whose kernel has no such variant fall back to 256 x 256)
GEMM_TILES = [(0, 0), (256, 256), (256, 192), (192, 256), (192, 192)]


@pytest.fixture(params=GEMM_TILES, ids=lambda t: "auto" if t == (0, 0) else f"{t[0]}x{t[1]}")
def tile(request):
    L.ls_gemm_tile_override(*request.param)
    yield request.param
    L.ls_gemm_tile_override(0, 0)


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_gemm_nt(M, N, K, tile):
    need_gpu()
    say(f"gemm_nt M={M} N={N} K={K} tile={tile}")
    A, B = bf16_randn((M, K), 1), bf16_randn((N, K), 2)
    C = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    L.ls_gemm_nt(A, B, C)
    torch.cuda.synchronize()
    ref = f64(A) @ f64(B).T
    assert max_rel(f64(C), ref) < 1e-2


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_gemm_nn(M, N, K, tile):
    need_gpu()
    say(f"gemm_nn M={M} N={N} K={K} tile={tile}")
    A, B = bf16_randn((M, K), 3), bf16_randn((K, N), 4)
    C = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    L.ls_gemm_nn(A, B, C)
    torch.cuda.synchronize()
    assert max_rel(f64(C), f64(A) @ f64(B)) < 1e-2


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_gemm_tn_accumulate(M, N, K, tile):
    need_gpu()
    say(f"gemm_tn M={M} N={N} K={K} tile={tile}")
    A, B = bf16_randn((K, M), 5), bf16_randn((K, N), 6)
    C = torch.full((M, N), 0.5, dtype=torch.float32, device="cuda")
    L.ls_gemm_tn(A, B, C, accumulate=False)
    torch.cuda.synchronize()
    ref = f64(A).T @ f64(B)
    assert max_rel(f64(C), ref) < 1e-5
    L.ls_gemm_tn(A, B, C, accumulate=True)
    torch.cuda.synchronize()
    assert max_rel(f64(C), 2 * ref) < 1e-5


# hidden 3584 and 4096: more than 6 chunks per lane (gamma and dres read where used);
# 4104, 6656 and 8192: the one-row-per-wave kernel
@pytest.mark.parametrize("rows,hidden", [(100, 264), (37, 6656), (1000, 3072), (5, 8), (70, 3584), (45, 4096), (50, 4104),
                                         (20, 8192)])
def test_rmsnorm(rows, hidden):
    need_gpu()
    say(f"rmsnorm rows={rows} hidden={hidden}")
    x = bf16_randn((rows, hidden), 7)
    gamma = (1 + 0.1 * bf16_randn((hidden,), 8, device="cpu").float()).to(torch.bfloat16).cuda()
    h = torch.empty_like(x)
    r = torch.empty(rows, dtype=torch.float32, device="cuda")
    L.ls_rmsnorm_fwd(rows, hidden, 1e-5, x, gamma, h, r)
    dh = bf16_randn((rows, hidden), 9)
    dres = bf16_randn((rows, hidden), 10)
    dx = torch.empty_like(x)
    dg = torch.full((hidden,), 1.0, dtype=torch.float32, device="cuda")
    ws = torch.empty(L.ls_rmsnorm_bwd_workspace(rows, hidden), dtype=torch.uint8, device="cuda")
    L.ls_rmsnorm_bwd(rows, hidden, x, gamma, r, dh, dres, dx, dg, True, ws)
    torch.cuda.synchronize()
    href, rref = ob.rmsnorm_forward(f64(x), f64(gamma), 1e-5)
    assert max_rel(f64(h), href) < OUT_TOL
    assert max_rel(f64(r), rref) < 1e-5
    dxr, dgr = ob.rmsnorm_backward(f64(dh), f64(x), f64(gamma), rref)
    assert fro_rel(f64(dx), dxr + f64(dres)) < GRAD_TOL
    assert fro_rel(f64(dg), dgr + 1.0) < 1e-4


ATTN_CASES = [
    # name, batch, seq, nq, nkv, d, q/k std (sharpness)
    ("tiny-gqa-d64", 2, 128, 4, 2, 64, 1.0),
    ("ragged-d128", 1, 200, 6, 2, 128, 1.0),
    ("sharp-d128", 2, 130, 4, 4, 128, math.sqrt(3.0)),
    ("sharp-d64-long", 1, 520, 6, 3, 64, math.sqrt(3.0)),
    ("single-token", 3, 1, 2, 1, 128, 1.0),
    ("mha-d64", 2, 200, 4, 4, 64, 1.0),
    ("mha-d64-sharp", 1, 264, 3, 3, 64, math.sqrt(3.0)),
]


@pytest.mark.parametrize("name,B,S,nq,nkv,d,std", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
def test_attention_core(name, B, S, nq, nkv, d, std):
    need_gpu()
    say(f"attention core {name}")
    c = configs.TINY.with_(batch=B, seq=S, n_q_heads=nq, n_kv_heads=nkv, head_dim=d, hidden=nq * d)
    T = B * S
    Dq, Dkv = nq * d, nkv * d
    q = bf16_randn((T, Dq), 11, std)
    k = bf16_randn((T, Dkv), 12, std)
    v = bf16_randn((T, Dkv), 13)
    qkv = torch.cat([q, k, v], dim=1).contiguous()
    o = torch.empty((T, Dq), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((B, nq, S), dtype=torch.float32, device="cuda")
    L.ls_attn_core_fwd(c, qkv, o, lse)
    do = bf16_randn((T, Dq), 14)
    dqkv = torch.empty_like(qkv)
    ws = torch.empty(L.ls_attn_core_bwd_workspace(c), dtype=torch.uint8, device="cuda")
    L.ls_attn_core_bwd(c, qkv, o, lse, do, dqkv, ws)
    torch.cuda.synchronize()
    q4 = f64(q).reshape(B, S, nq, d)
    k4 = f64(k).reshape(B, S, nkv, d)
    v4 = f64(v).reshape(B, S, nkv, d)
    oref, lref = ob.attention_forward(q4, k4, v4)
    assert max_rel(f64(o), oref.reshape(T, Dq)) < OUT_TOL
    assert np.max(np.abs(f64(lse) - lref)) < 1e-3 * max(1.0, np.max(np.abs(lref)))
    dq, dk, dv = ob.attention_backward(f64(do).reshape(B, S, nq, d), q4, k4, v4)
    g = f64(dqkv)
    assert fro_rel(g[:, Dq + Dkv:], dv.reshape(T, Dkv)) < GRAD_TOL
    if S == 1:
        # one key per query: the softmax is constant, so dq and dk are exactly zero
        scale = np.linalg.norm(dv)
        assert np.linalg.norm(g[:, :Dq + Dkv]) < 1e-4 * scale
        return
    assert fro_rel(g[:, :Dq], dq.reshape(T, Dq)) < GRAD_TOL
    assert fro_rel(g[:, Dq:Dq + Dkv], dk.reshape(T, Dkv)) < GRAD_TOL


SAMPLED_GROUP_CASES = [
    # name, batch, seq, nq, nkv, d, kv head checked.  The dK/dV kernel splits a
    # kv head's query-head group over workgroups when (seq/128) * nkv * batch
    # is below 512: "8k" and "d64-unsplit" fill the chip unsplit (512
    # workgroups); "split2of4" (256 workgroups, groups of 4) sums two partials
    # of two heads each.
    ("8k", 1, 8192, 24, 8, 128, 5),
    ("split2of4", 1, 2048, 64, 16, 64, 11),
    # 64-wide heads at (2048/128) * 8 * 4 = 512 workgroups: the unsplit kernel
    ("d64-unsplit", 4, 2048, 32, 8, 64, 6),
]


@pytest.mark.parametrize("name,B,S,nq,nkv,d,kvh", SAMPLED_GROUP_CASES, ids=[c[0] for c in SAMPLED_GROUP_CASES])
def test_attention_core_sampled_group(name, B, S, nq, nkv, d, kvh):
    """Attention at a long or many-head shape in its full launch
    configuration; the oracle computes one kv group (kv head kvh and its query
    heads) over all positions."""
    need_gpu()
    G = nq // nkv
    say(f"attention core {name}, kv group {kvh}")
    c = configs.TINY.with_(batch=B, seq=S, n_q_heads=nq, n_kv_heads=nkv, head_dim=d, hidden=nq * d)
    T, Dq, Dkv = B * S, nq * d, nkv * d
    q = bf16_randn((T, Dq), 21)
    k = bf16_randn((T, Dkv), 22)
    v = bf16_randn((T, Dkv), 23)
    qkv = torch.cat([q, k, v], dim=1).contiguous()
    o = torch.empty((T, Dq), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((B, nq, S), dtype=torch.float32, device="cuda")
    L.ls_attn_core_fwd(c, qkv, o, lse)
    do = bf16_randn((T, Dq), 24)
    dqkv = torch.empty_like(qkv)
    ws = torch.empty(L.ls_attn_core_bwd_workspace(c), dtype=torch.uint8, device="cuda")
    L.ls_attn_core_bwd(c, qkv, o, lse, do, dqkv, ws)
    torch.cuda.synchronize()
    hs = slice(kvh * G, (kvh + 1) * G)
    q4 = f64(q).reshape(B, S, nq, d)[:, :, hs]
    k4 = f64(k).reshape(B, S, nkv, d)[:, :, kvh:kvh + 1]
    v4 = f64(v).reshape(B, S, nkv, d)[:, :, kvh:kvh + 1]
    oref, lref = ob.attention_forward(q4, k4, v4)
    og = f64(o).reshape(B, S, nq, d)[:, :, hs]
    assert max_rel(og, oref) < OUT_TOL
    assert np.max(np.abs(f64(lse)[:, hs] - lref)) < 1e-3 * max(1.0, np.max(np.abs(lref)))
    dq, dk, dv = ob.attention_backward(f64(do).reshape(B, S, nq, d)[:, :, hs], q4, k4, v4)
    g = f64(dqkv)
    assert fro_rel(g[:, :Dq].reshape(B, S, nq, d)[:, :, hs], dq) < GRAD_TOL
    assert fro_rel(g[:, Dq:Dq + Dkv].reshape(B, S, nkv, d)[:, :, kvh:kvh + 1], dk) < GRAD_TOL
    assert fro_rel(g[:, Dq + Dkv:].reshape(B, S, nkv, d)[:, :, kvh:kvh + 1], dv) < GRAD_TOL
