"""The C ABI library: it loads, exports every symbol include/ls.h declares, and
rejects bad arguments before touching the GPU (these run on a host with no GPU;
no call here reaches a HIP API)."""
import ctypes
import os
import re

import pytest
import torch  # noqa: F401  (load torch's HIP runtime first, as the binding does)

from paper_2510_02483_amd import configs, lib as L

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "ls.h")

pytestmark = pytest.mark.skipif(not os.path.exists(L.LIB_PATH), reason="libls.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ls_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 18
    lib = ctypes.CDLL(L.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(L.EXPORTS), "binding and header disagree"


def test_version_and_status_strings():
    assert L.ls_version() == 100
    for code in range(8):
        assert L.lib().ls_status_string(code).decode()
    assert L.lib().ls_status_string(99).decode() == "unknown status"


def cfg_of(c):
    return L.make_cfg(c)


def test_query_sizes_tiny():
    s = L.ls_query_sizes(configs.TINY)
    c = configs.TINY
    T, H, I = c.tokens, c.hidden, c.intermediate
    # saved state holds at least h1, qkv, o (bf16) and r1, lse (fp32)
    assert s["attn_saved"] >= 2 * T * (H + c.dq + 2 * c.dkv + c.dq) + 4 * (T + c.batch * c.n_q_heads * c.seq)
    assert s["mlp_saved"] >= 2 * T * (H + 3 * I) + 4 * T
    assert s["block_workspace"] >= s["attn_saved"] + s["mlp_saved"] + 4 * T * H
    assert all(v % 256 == 0 for v in s.values())


@pytest.mark.parametrize("field,value,status", [
    ("batch", 0, 2), ("seq", -1, 2), ("hidden", 0, 2), ("n_kv_heads", 3, 2),
    ("hidden", 260, 2), ("intermediate", 690, 2), ("head_dim", 100, 3), ("head_dim", 32, 3), ("head_dim", 136, 3),
    ("head_dim", 56, 3),
    ("rope_theta", 1.0, 2), ("rms_eps", -1e-5, 2), ("hidden", 16384, 3),
])
def test_query_sizes_rejects(field, value, status):
    c = configs.TINY.with_(**{field: value})
    with pytest.raises(L.LsError) as e:
        L.ls_query_sizes(c)
    assert e.value.status == status


def test_null_pointers():
    lib = L.lib()
    s = L.LsSizes()
    assert lib.ls_query_sizes(None, ctypes.byref(s)) == 1
    cfg = cfg_of(configs.TINY)
    assert lib.ls_query_sizes(ctypes.byref(cfg), None) == 1
    assert lib.ls_attn_fwd(ctypes.byref(cfg), None, None, None, None, None, 0, None) == 1
    w = L.LsBlockWeights()
    assert lib.ls_attn_fwd(ctypes.byref(cfg), ctypes.c_void_p(4096), ctypes.byref(w), ctypes.c_void_p(1 << 40),
                           ctypes.c_void_p(1 << 41), ctypes.c_void_p(1 << 42), 1 << 30, None) == 1
    assert "NULL" in lib.ls_last_error().decode()


def _fake_weights(c, base=1 << 36, stride=1 << 30):
    return L.LsBlockWeights(*[base + i * stride for i in range(9)])


def _fake_grads(c, base=1 << 44, stride=1 << 30):
    return L.LsBlockGrads(*[base + i * stride for i in range(9)])


def test_alignment_alias_and_workspace():
    lib = L.lib()
    c = configs.TINY
    cfg = cfg_of(c)
    sizes = L.ls_query_sizes(c)
    w, g = _fake_weights(c), _fake_grads(c)
    x, dy, y, dx, ws = (1 << 32), (1 << 33), (1 << 34), (1 << 35), (1 << 46)
    V = ctypes.c_void_p
    call = lambda x_, dy_, y_, dx_, ws_, n: lib.ls_block_fwd_bwd(  # noqa: E731
        ctypes.byref(cfg), V(x_), ctypes.byref(w), V(dy_), V(y_), V(dx_), ctypes.byref(g), 0, V(ws_), n, None)
    assert call(x + 2, dy, y, dx, ws, sizes["block_workspace"]) == 4  # misaligned
    assert call(x, dy, x, dx, ws, sizes["block_workspace"]) == 5      # y aliases x
    assert call(x, dy, y, y + 64, ws, sizes["block_workspace"]) == 5  # dx overlaps y
    assert call(x, dy, y, dx, ws, sizes["block_workspace"] - 256) == 6
    assert "workspace" in lib.ls_last_error().decode()
    # gradient buffer overlapping an input
    g2 = _fake_grads(c)
    g2.wq = x
    assert lib.ls_block_fwd_bwd(ctypes.byref(cfg), V(x), ctypes.byref(w), V(dy), V(y), V(dx), ctypes.byref(g2), 0,
                                V(ws), sizes["block_workspace"], None) == 5


def test_gemm_and_norm_argument_checks():
    lib = L.lib()
    V = ctypes.c_void_p
    assert lib.ls_gemm_nt(0, 8, 8, V(1 << 32), V(1 << 33), V(1 << 34), None) == 2
    assert lib.ls_gemm_nt(12, 8, 8, V(1 << 32), V(1 << 33), V(1 << 34), None) == 2
    assert lib.ls_gemm_nn(8, 8, 8, V(1 << 32), V((1 << 33) + 8), V(1 << 34), None) == 4
    assert lib.ls_gemm_tn(64, 64, 64, V(1 << 32), V(1 << 33), V(1 << 32), 0, None) == 5
    assert lib.ls_rmsnorm_fwd(4, 12, 1e-5, V(1 << 32), V(1 << 33), V(1 << 34), V(1 << 35), None) == 2
    assert lib.ls_rmsnorm_fwd(4, 16, -1.0, V(1 << 32), V(1 << 33), V(1 << 34), V(1 << 35), None) == 2
    need = lib.ls_rmsnorm_bwd_workspace(100, 64)
    assert need >= 64 * 4
    assert lib.ls_rmsnorm_bwd(100, 64, V(1 << 32), V(1 << 33), V(1 << 34), V(1 << 35), None, V(1 << 36),
                              V(1 << 37), 0, V(1 << 38), need - 4, None) == 6


def test_gemm_tile_override_arguments():
    lib = L.lib()
    assert lib.ls_gemm_tile_override(100, 256) == 2
    assert lib.ls_gemm_tile_override(256, 128) == 2
    assert lib.ls_gemm_tile_override(192, 256) == 0
    assert lib.ls_gemm_tile_override(0, 0) == 0


def _stack_args(sc, L_=None):
    """Fake, disjoint, aligned device addresses for every stack argument (the
    checks run before any HIP call, so nothing is dereferenced)."""
    n = sc.n_layers if L_ is None else L_
    lw = (L.LsBlockWeights * max(n, 1))(*[_fake_weights(sc.block, base=(1 << 36) + l * (1 << 34)) for l in range(n)])
    lg = (L.LsBlockGrads * max(n, 1))(*[_fake_grads(sc.block, base=(1 << 44) + l * (1 << 34)) for l in range(n)])
    w = L.LsStackWeights(1 << 52, (1 << 52) + (1 << 40), lw)
    g = L.LsStackGrads(1 << 53, (1 << 53) + (1 << 40), lg)
    return w, g


def test_stack_workspace_and_config_checks():
    sc = configs.TINY_STACK
    need = L.ls_stack_workspace(sc)
    c, T, H, V = sc.block, sc.tokens, sc.block.hidden, sc.vocab
    # block inputs of every layer, the logits, one block's saved state
    assert need >= 2 * T * H * (sc.n_layers + 1) + 2 * T * V + L.ls_query_sizes(c)["attn_saved"]
    assert L.ls_stack_workspace(sc.with_(recompute=False)) > need
    assert L.ls_stack_workspace(sc.with_(n_layers=0)) < need
    for bad, status in [(dict(vocab=1001), 2), (dict(vocab=0), 2), (dict(n_layers=-1), 2),
                        (dict(vocab=1 << 20, block=c.with_(hidden=512)), 2),
                        (dict(block=c.with_(head_dim=100)), 3)]:
        with pytest.raises(L.LsError) as e:
            L.ls_stack_workspace(sc.with_(**bad))
        assert e.value.status == status, bad
    lib = L.lib()
    assert L.ls_stack_workspace(sc.with_(logits_chunk=40)) < need, "smaller logits chunks need less workspace"
    cfg = L.make_stack_cfg(sc)
    cfg.logits_chunk = -1
    n0 = ctypes.c_size_t(0)
    assert L.lib().ls_stack_workspace(ctypes.byref(cfg), ctypes.byref(n0)) == 2
    cfg = L.make_stack_cfg(sc)
    cfg.recompute = 2
    n = ctypes.c_size_t(0)
    assert lib.ls_stack_workspace(ctypes.byref(cfg), ctypes.byref(n)) == 2
    assert lib.ls_stack_workspace(None, ctypes.byref(n)) == 1


def test_stack_argument_checks():
    lib = L.lib()
    sc = configs.TINY_STACK
    cfg = L.make_stack_cfg(sc)
    need = L.ls_stack_workspace(sc)
    V = ctypes.c_void_p
    ids, tgt, loss, rows, ws = (1 << 32), (1 << 33), (1 << 34), (1 << 35), (1 << 50)
    w, g = _stack_args(sc)
    call = lambda ids_, w_, g_, loss_, ws_, n: lib.ls_stack_fwd_bwd(  # noqa: E731
        ctypes.byref(cfg), V(ids_), None, ctypes.byref(w_), V(loss_), V(rows), ctypes.byref(g_), 0, V(ws_), n, None)
    assert call(None, w, g, loss, ws, need) == 1
    assert call(ids, w, g, None, ws, need) == 1
    assert call(ids + 4, w, g, loss, ws, need) == 4
    assert call(ids, w, g, ids, ws, need) == 5                 # loss aliases ids
    assert call(ids, w, g, loss, ws, need - 256) == 6
    g2 = L.LsStackGrads(g.embed, g.final_norm, g.layers)
    g2.embed = w.embed                                         # gradient over the embedding
    assert call(ids, w, g2, loss, ws, need) == 5
    w0, g0 = _stack_args(sc)
    g0.layers[1].wq = g0.layers[0].wq                          # two layers share a gradient buffer
    assert call(ids, w0, g0, loss, ws, need) == 5
    w1, g1 = _stack_args(sc)
    w1.layers[1].wq = w1.layers[0].wq                          # tied layer weights are allowed
    assert lib.ls_stack_fwd_bwd(ctypes.byref(cfg), V(ids), V(tgt), ctypes.byref(w1), V(loss), None,
                                ctypes.byref(g1), 0, V(ws), need - 1, None) == 6
    w3 = L.LsStackWeights(w.embed, w.final_norm, None)
    assert call(ids, w3, g, loss, ws, need) == 1


def test_cross_entropy_and_embedding_argument_checks():
    lib = L.lib()
    V = ctypes.c_void_p
    need = lib.ls_cross_entropy_workspace(100)
    assert need >= 400
    z, ids, loss, rows, ws = (1 << 32), (1 << 33), (1 << 34), (1 << 35), (1 << 36)
    ce = lambda T, S, Vv, n, z_=z: lib.ls_cross_entropy(T, S, Vv, V(z_), V(ids), None, V(loss), V(rows),  # noqa
                                                         V(ws), n, None)
    assert ce(100, 10, 1001, need) == 2   # vocab not a multiple of 8
    assert ce(100, 7, 1000, need) == 2    # next-token targets need whole sequences
    assert ce(100, 10, 1000, need - 4) == 6
    assert ce(100, 10, 1000, need, z_=ids) == 5
    assert lib.ls_embed_fwd(10, 12, 100, V(ids), V(z), V(rows), None) == 2
    assert lib.ls_embed_fwd(10, 16, 100, V(ids), V(z), V(ids), None) == 5
    assert lib.ls_embed_bwd(10, 16, 100, None, V(z), V(rows), None) == 1


def test_adamw_argument_checks():
    lib = L.lib()
    V = ctypes.c_void_p
    ws_need = lib.ls_adamw_workspace()
    assert ws_need >= 2048 * 8
    cfg = L.LsAdamwCfg(1e-3, 0.9, 0.95, 1e-8, 0.01, 1.0, 1)
    p, w, g, m, v, nrm, ws = (1 << 32), (1 << 33), (1 << 34), (1 << 35), (1 << 36), (1 << 37), (1 << 38)
    call = lambda n, nd, c, p_=p, g_=g, n_ws=ws_need: lib.ls_adamw_step(  # noqa: E731
        n, nd, ctypes.byref(c), V(p_), V(w), V(g_), V(m), V(v), V(nrm), V(ws), n_ws, None)
    assert call(0, 0, cfg) == 2
    assert call(100, 101, cfg) == 2
    assert call(100, -1, cfg) == 2
    assert call(100, 50, cfg, g_=p + 16) == 5        # grad overlaps master
    assert call(100, 50, cfg, p_=p + 4) == 4         # misaligned
    assert call(100, 50, cfg, n_ws=ws_need - 8) == 6
    for field, value in [("step", 0), ("beta1", 1.0), ("beta2", -0.1), ("eps", 0.0), ("lr", -1.0),
                         ("weight_decay", -0.01)]:
        bad = L.LsAdamwCfg(1e-3, 0.9, 0.95, 1e-8, 0.01, 1.0, 1)
        setattr(bad, field, value)
        assert call(100, 50, bad) == 2, field
    assert lib.ls_adamw_step(100, 50, None, V(p), V(w), V(g), V(m), V(v), None, V(ws), ws_need, None) == 1
    assert lib.ls_adamw_step(100, 50, ctypes.byref(cfg), V(p), None, V(g), V(m), None, None, V(ws), ws_need,
                             None) == 1


def test_padded_head_sizes():
    """head_dim 104 (a 64-head, 6656-wide model) runs in 128-wide slots: the
    saved q/k/v and o and the workspace hold the padded layout (and padded
    copies of the projection weights and their fp32 gradients)."""
    c = configs.TINY.with_(hidden=416, n_q_heads=4, n_kv_heads=2, head_dim=104)
    s = L.ls_query_sizes(c)
    T, H = c.tokens, c.hidden
    pq, pkv = 4 * 128, 2 * 128
    assert s["attn_saved"] >= 2 * T * (H + pq + 2 * pkv + pq)
    assert s["attn_workspace"] >= (pq + 2 * pkv) * H * (2 + 4) + H * pq * (2 + 4)
    s128 = L.ls_query_sizes(c.with_(head_dim=128, hidden=512))
    assert s128["attn_workspace"] < s["attn_workspace"] + 4 * T * H
    lib = L.lib()
    cfg = cfg_of(c)
    V = ctypes.c_void_p
    assert lib.ls_attn_core_fwd(ctypes.byref(cfg), V(1 << 32), V(1 << 33), V(1 << 34), None) == 3
    assert lib.ls_attn_core_bwd_workspace(ctypes.byref(cfg)) == 0


def test_size_limits():
    """Every matrix must stay below 2047 MiB (buffer resources address it with
    32-bit offsets): the largest shapes are rejected before any HIP call."""
    big_t = configs.B3.with_(batch=64, seq=8192)           # 512k tokens x 3072 x 2 B = 3 GiB activations
    with pytest.raises(L.LsError) as e:
        L.ls_query_sizes(big_t)
    assert e.value.status == 2 and "2047" in str(e.value)
    wide = configs.B30.with_(intermediate=163840)          # [T, 2I] gate/up output of 2.5 GiB
    with pytest.raises(L.LsError) as e:
        L.ls_query_sizes(wide)
    assert e.value.status == 2
    ok = configs.B3.with_(batch=16, seq=2048)               # 32k tokens: 192 MiB activations
    assert L.ls_query_sizes(ok)["block_workspace"] > 0
    lib = L.lib()
    V = ctypes.c_void_p
    assert lib.ls_cross_entropy(1 << 31, 1, 8, V(1 << 32), V(1 << 33), None, V(1 << 34), V(1 << 35),
                                V(1 << 36), 1 << 40, None) == 2


def test_attn_core_bwd_noalloc_argument_checks():
    """The no-allocation attention backward checks its arguments and its
    scratch limit before any HIP call (so these run without a GPU)."""
    lib = L.lib()
    V = ctypes.c_void_p
    small = cfg_of(configs.TINY)
    big = cfg_of(configs.PAPER_3B)   # its split dK/dV partials exceed the library's scratch array
    assert L.ls_attn_core_bwd_workspace(configs.PAPER_3B) > L.NOALLOC_SCRATCH_BYTES
    assert L.ls_attn_core_bwd_workspace(configs.TINY) <= L.NOALLOC_SCRATCH_BYTES
    qkv, o, lse, do, dqkv = (1 << 36), (1 << 37), (1 << 38), (1 << 39), (1 << 40)
    assert lib.ls_attn_core_bwd_noalloc(ctypes.byref(big), V(qkv), V(o), V(lse), V(do), V(dqkv), None) == 6
    assert "scratch" in lib.ls_last_error().decode()
    assert lib.ls_attn_core_bwd_noalloc(ctypes.byref(small), V(qkv), V(o), None, V(do), V(dqkv), None) == 1
    assert lib.ls_attn_core_bwd_noalloc(ctypes.byref(small), V(qkv), V(o), V(lse), V(do), V(qkv), None) == 5
    assert lib.ls_attn_core_bwd_noalloc(ctypes.byref(small), V(qkv), V(o), V(lse), V(do), V(dqkv + 8), None) == 4
    odd = cfg_of(configs.TINY.with_(head_dim=104, hidden=416))
    assert lib.ls_attn_core_bwd_noalloc(ctypes.byref(odd), V(qkv), V(o), V(lse), V(do), V(dqkv), None) == 3
