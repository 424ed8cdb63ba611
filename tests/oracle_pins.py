"""Checks that pin the fp64 oracle to facts other than itself.

Each ``check_*`` takes the oracle module (so that a test can hand in a copy
with a planted mistake) and raises AssertionError when the oracle disagrees
with what mathematics or an independent library routine fixes:

* closed forms and special cases (q = 0 attention, the first row of a causal
  softmax, RoPE at position 0, hand-evaluated RoPE frequencies, silu'(0) = 1/2);
* invariants (softmax rows sum to one, rotation preserves pair norms and
  depends only on relative position, RMSNorm scale invariance, causal masking,
  grouped-query attention equals multi-head attention with repeated kv heads,
  the identity sum_j P_ij dP_ij = <dO_i, O_i>);
* brute force on tiny inputs (a per-row pure-Python softmax);
* library routines used independently of the oracle's own code
  (torch.nn.functional.rms_norm / silu / scaled_dot_product_attention in
  float64, RoPE as complex multiplication, torch autograd for every gradient);
* central finite differences of the oracle's own forward, which pin every
  backward formula to its forward.
"""
from __future__ import annotations

import math

import numpy as np
import torch
import torch.nn.functional as F

MICRO = dict(B=1, S=5, H=8, nq=2, nkv=1, d=4, I=12, theta=1e4, eps=1e-5)
SMALL = dict(B=2, S=16, H=32, nq=4, nkv=2, d=8, I=40, theta=1e4, eps=1e-5)


def _rng(seed):
    return np.random.default_rng(seed)


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = max(np.linalg.norm(b), 1e-300)
    return float(np.linalg.norm(a - b) / den)


def make_weights(c, seed, w_std=0.3, gamma_random=True):
    r = _rng(seed)
    H, I, dq, dkv = c["H"], c["I"], c["nq"] * c["d"], c["nkv"] * c["d"]
    w = dict(wq=r.normal(0, w_std, (dq, H)), wk=r.normal(0, w_std, (dkv, H)),
             wv=r.normal(0, w_std, (dkv, H)), wo=r.normal(0, w_std, (H, dq)),
             wg=r.normal(0, w_std, (I, H)), wu=r.normal(0, w_std, (I, H)),
             wd=r.normal(0, w_std, (H, I)))
    if gamma_random:
        w["attn_norm"] = 1 + 0.2 * r.normal(size=H)
        w["mlp_norm"] = 1 + 0.2 * r.normal(size=H)
    else:
        w["attn_norm"] = np.ones(H)
        w["mlp_norm"] = np.ones(H)
    return w


def block_kw(c):
    return dict(n_q_heads=c["nq"], n_kv_heads=c["nkv"], rope_theta=c["theta"], eps=c["eps"])


# --------------------------------------------------------------------------
# RMSNorm
# --------------------------------------------------------------------------

def check_rmsnorm_library(ob):
    r = _rng(1)
    x = r.normal(size=(3, 7, 24))
    g = 1 + 0.3 * r.normal(size=24)
    h, rs = ob.rmsnorm_forward(x, g, 1e-5)
    xt = torch.tensor(x, requires_grad=True)
    gt = torch.tensor(g, requires_grad=True)
    ht = F.rms_norm(xt, (24,), weight=gt, eps=1e-5)
    assert _rel(h, ht.detach().numpy()) < 1e-13, "rmsnorm forward vs torch rms_norm"
    dh = r.normal(size=h.shape)
    ht.backward(torch.tensor(dh))
    dx, dg = ob.rmsnorm_backward(dh, x, g, rs)
    assert _rel(dx, xt.grad.numpy()) < 1e-12, "rmsnorm dx vs torch autograd"
    assert _rel(dg, gt.grad.numpy()) < 1e-12, "rmsnorm dgamma vs torch autograd"
    # r is the reciprocal root mean square
    assert np.allclose(rs, 1.0 / np.sqrt((x ** 2).mean(-1) + 1e-5), rtol=1e-14, atol=0)


def check_rmsnorm_invariants(ob):
    r = _rng(2)
    x = r.normal(size=(5, 16))
    g = 1 + 0.3 * r.normal(size=16)
    h, rs = ob.rmsnorm_forward(x, g, 0.0)
    h2, _ = ob.rmsnorm_forward(7.5 * x, g, 0.0)
    assert np.allclose(h, h2, rtol=1e-13, atol=1e-13), "scale invariance at eps=0"
    ones = np.ones(16)
    hn, _ = ob.rmsnorm_forward(x, ones, 0.0)
    assert np.allclose((hn ** 2).mean(-1), 1.0, rtol=1e-13), "unit mean square at eps=0"
    dh = r.normal(size=x.shape)
    dx, _ = ob.rmsnorm_backward(dh, x, g, rs)
    # eps = 0: the output is invariant to scaling x, so dx is orthogonal to x
    assert np.allclose((dx * x).sum(-1), 0.0, atol=1e-12), "<dx, x> = 0 at eps=0"


# --------------------------------------------------------------------------
# RoPE
# --------------------------------------------------------------------------

def check_rope_frequencies(ob):
    # d = 4, theta = 10000: the two pairs turn by p and p/100 radians
    phi = ob.rope_angles(4, 4, 1e4)
    want = np.array([[0, 0], [1, 0.01], [2, 0.02], [3, 0.03]], dtype=np.float64)
    assert np.allclose(phi, want, rtol=1e-15, atol=1e-15), "theta^(-2i/d) at d=4"
    # d = 8, theta = 16: pair i turns at 16^(-i/4) = 2^-i
    phi = ob.rope_angles(3, 8, 16.0)
    want = np.outer(np.arange(3), [1.0, 0.5, 0.25, 0.125])
    assert np.allclose(phi, want, rtol=1e-15, atol=0), "theta^(-2i/d) at d=8"


def check_rope_complex(ob):
    """Rotate-half RoPE equals multiplying x_i + 1j x_{i+d/2} by e^{1j phi}."""
    r = _rng(3)
    S, d = 9, 8
    x = r.normal(size=(2, S, 3, d))
    phi = ob.rope_angles(S, d, 500.0)
    got = ob.rope_rotate(x, phi)
    z = (x[..., : d // 2] + 1j * x[..., d // 2:]) * np.exp(1j * phi)[None, :, None, :]
    want = np.concatenate([z.real, z.imag], -1)
    assert _rel(got, want) < 1e-14, "rope vs complex multiplication"
    assert np.array_equal(got[:, 0], x[:, 0]), "position 0 is the identity"
    back = ob.rope_rotate(got, -phi)
    assert _rel(back, x) < 1e-14, "rotation by -phi undoes rotation by phi"


def check_rope_relative(ob):
    r = _rng(4)
    d = 16
    phi = ob.rope_angles(40, d, 1e4)
    q = r.normal(size=(1, 40, 1, d))
    k = r.normal(size=(1, 40, 1, d))
    qa = ob.rope_rotate(np.repeat(q[:, :1], 40, 1), phi)  # same q at every position
    ka = ob.rope_rotate(np.repeat(k[:, :1], 40, 1), phi)
    s = np.einsum("d,d->", qa[0, 20, 0], ka[0, 13, 0])
    s2 = np.einsum("d,d->", qa[0, 30, 0], ka[0, 23, 0])
    assert abs(s - s2) < 1e-12 * max(1.0, abs(s)), "score depends on m - n only"
    half = d // 2
    v0 = q[0, 0, 0]
    got = qa[0, 37, 0]
    assert np.allclose(got[:half] ** 2 + got[half:] ** 2, v0[:half] ** 2 + v0[half:] ** 2,
                       rtol=1e-13), "pair norms preserved"


# --------------------------------------------------------------------------
# Attention
# --------------------------------------------------------------------------

def _qkv(seed, B=2, S=11, nq=4, nkv=2, d=8, scale=1.0):
    r = _rng(seed)
    return (scale * r.normal(size=(B, S, nq, d)), scale * r.normal(size=(B, S, nkv, d)),
            r.normal(size=(B, S, nkv, d)))


def check_attention_bruteforce(ob):
    """A per-row pure-Python masked softmax on a tiny case."""
    q, k, v = _qkv(5, B=1, S=6, nq=2, nkv=1, d=4, scale=2.0)
    o, lse = ob.attention_forward(q, k, v)
    for h in range(2):
        for i in range(6):
            sc = [sum(q[0, i, h, c] * k[0, j, 0, c] for c in range(4)) / 2.0 for j in range(i + 1)]
            m = max(sc)
            ex = [math.exp(s - m) for s in sc]
            tot = sum(ex)
            for c in range(4):
                want = sum(ex[j] / tot * v[0, j, 0, c] for j in range(i + 1))
                assert abs(o[0, i, h, c] - want) < 1e-12, "brute-force softmax"
            assert abs(lse[0, h, i] - (m + math.log(tot))) < 1e-12, "brute-force lse"


def check_attention_library(ob):
    q, k, v = _qkv(6, scale=1.5)
    o, lse = ob.attention_forward(q, k, v)
    tq, tk, tv = (torch.tensor(a).transpose(1, 2) for a in (q, k, v))
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True, enable_gqa=True)
    assert _rel(o, ref.transpose(1, 2).numpy()) < 1e-13, "attention vs torch SDPA (causal, GQA)"
    # lse against torch.logsumexp of masked scores
    S = q.shape[1]
    sc = torch.einsum("bhid,bhjd->bhij", tq, tk.repeat_interleave(2, 1)) / math.sqrt(q.shape[-1])
    sc = sc.masked_fill(~torch.tril(torch.ones(S, S, dtype=torch.bool)), -math.inf)
    assert _rel(lse, torch.logsumexp(sc, -1).numpy()) < 1e-13, "lse vs torch logsumexp"


def check_attention_closed_forms(ob):
    q, k, v = _qkv(7)
    # q = 0: uniform weights over the prefix
    o, lse = ob.attention_forward(np.zeros_like(q), k, v)
    S = q.shape[1]
    G = q.shape[2] // k.shape[2]
    cnt = np.arange(1, S + 1)[None, :, None]
    for h in range(q.shape[2]):
        mean = np.cumsum(v[:, :, h // G], axis=1) / cnt
        assert np.allclose(o[:, :, h], mean, rtol=1e-13, atol=1e-13), "q=0 gives prefix mean"
        assert np.allclose(lse[:, h], np.log(np.arange(1, S + 1))[None], atol=1e-13), "q=0 lse = ln(t+1)"
    # row 0 sees only key 0
    o, lse = ob.attention_forward(q, k, v)
    for h in range(q.shape[2]):
        assert np.allclose(o[:, 0, h], v[:, 0, h // G], atol=1e-14), "row 0 output is v_0"
        s00 = (q[:, 0, h] * k[:, 0, h // G]).sum(-1) / math.sqrt(q.shape[-1])
        assert np.allclose(lse[:, h, 0], s00, atol=1e-13), "row 0 lse is s_00"


def check_attention_rows_and_mask(ob):
    q, k, v = _qkv(8, scale=3.0)
    # rows of P sum to one: attention of a constant value vector returns it
    o, _ = ob.attention_forward(q, k, np.ones_like(v) * 2.5)
    assert np.allclose(o, 2.5, rtol=1e-14), "softmax rows sum to one"
    # causality: changing keys/values after position t0 leaves rows <= t0 unchanged
    o, lse = ob.attention_forward(q, k, v)
    k2, v2 = k.copy(), v.copy()
    k2[:, 6:] += 5.0
    v2[:, 6:] -= 3.0
    o2, lse2 = ob.attention_forward(q, k2, v2)
    assert np.array_equal(o[:, :6], o2[:, :6]) and np.array_equal(lse[:, :, :6], lse2[:, :, :6]), "causal"
    assert not np.allclose(o[:, 6:], o2[:, 6:]), "later rows do see the change"
    # diagonal is kept: key i matters to row i
    k3 = k.copy()
    k3[:, 5] += 4.0
    o3, _ = ob.attention_forward(q, k3, v)
    assert not np.allclose(o[:, 5], o3[:, 5]), "mask keeps the diagonal"


def check_attention_gqa(ob):
    q, k, v = _qkv(9, nq=6, nkv=2)
    o, lse = ob.attention_forward(q, k, v)
    kr, vr = np.repeat(k, 3, axis=2), np.repeat(v, 3, axis=2)  # head h reads kv h // 3
    o2, lse2 = ob.attention_forward(q, kr, vr)
    assert _rel(o, o2) < 1e-15 and _rel(lse, lse2) < 1e-15, "GQA equals MHA with repeated kv"
    r = _rng(10)
    do = r.normal(size=o.shape)
    dq, dk, dv = ob.attention_backward(do, q, k, v)
    dq2, dk2, dv2 = ob.attention_backward(do, q, kr, vr)
    assert _rel(dq, dq2) < 1e-14, "GQA dq"
    assert _rel(dk, dk2.reshape(dk2.shape[0], dk2.shape[1], 2, 3, -1).sum(3)) < 1e-13, "GQA dk sums copies"
    assert _rel(dv, dv2.reshape(dv2.shape[0], dv2.shape[1], 2, 3, -1).sum(3)) < 1e-13, "GQA dv sums copies"


def check_attention_backward_library(ob):
    q, k, v = _qkv(11, scale=1.5)
    r = _rng(12)
    do = r.normal(size=q.shape)
    dq, dk, dv = ob.attention_backward(do, q, k, v)
    tq, tk, tv = (torch.tensor(a).transpose(1, 2).requires_grad_() for a in (q, k, v))
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True, enable_gqa=True)
    ref.backward(torch.tensor(do).transpose(1, 2))
    for got, t, name in ((dq, tq, "dq"), (dk, tk, "dk"), (dv, tv, "dv")):
        assert _rel(got, t.grad.transpose(1, 2).numpy()) < 1e-12, f"attention {name} vs autograd"
    # D_i = sum_j P_ij dP_ij equals <dO_i, O_i>
    o, lse = ob.attention_forward(q, k, v)
    b, h = 1, 3
    kv = h // 2
    S = q.shape[1]
    s = q[b, :, h] @ k[b, :, kv].T / math.sqrt(q.shape[-1])
    P = np.where(np.tril(np.ones((S, S), bool)), np.exp(s - lse[b, h][:, None]), 0.0)
    dP = do[b, :, h] @ v[b, :, kv].T
    assert np.allclose((P * dP).sum(1), (do[b, :, h] * o[b, :, h]).sum(1), atol=1e-12), "D identity"


# --------------------------------------------------------------------------
# SwiGLU
# --------------------------------------------------------------------------

def check_swiglu(ob):
    r = _rng(13)
    g = r.normal(size=(4, 9)) * 3
    u = r.normal(size=(4, 9))
    a = ob.swiglu_forward(g, u)
    assert _rel(a, (F.silu(torch.tensor(g)) * torch.tensor(u)).numpy()) < 1e-14, "silu vs torch"
    gt = torch.tensor(g, requires_grad=True)
    ut = torch.tensor(u, requires_grad=True)
    da = r.normal(size=g.shape)
    (F.silu(gt) * ut).backward(torch.tensor(da))
    dg, du = ob.swiglu_backward(da, g, u)
    assert _rel(dg, gt.grad.numpy()) < 1e-13 and _rel(du, ut.grad.numpy()) < 1e-13, "swiglu grads"
    z = np.array([0.0, 1000.0, -1000.0])
    assert np.array_equal(ob.swiglu_forward(z, np.ones(3)), np.array([0.0, 1000.0, -0.0])), "silu limits"
    dg0, _ = ob.swiglu_backward(np.ones(3), z, np.ones(3))
    assert dg0[0] == 0.5 and dg0[1] == 1.0 and dg0[2] == 0.0, "silu'(0)=1/2, limits 1 and 0"
    assert np.all(np.isfinite(ob.sigmoid(np.array([-800.0, 800.0])))), "stable sigmoid"


# --------------------------------------------------------------------------
# Whole block
# --------------------------------------------------------------------------

def torch_block(x, w, c):
    """Independent float64 block built from torch library routines; autograd
    provides every gradient.  RoPE is applied as complex multiplication."""
    T = {k: torch.tensor(v, requires_grad=True) for k, v in w.items()}
    xt = torch.tensor(x, requires_grad=True)
    return torch_block_t(xt, T, c), xt, T


def torch_block_t(xt, T, c):
    """The block of torch_block on torch tensors (x [B, S, H], weights T)."""
    B, S, H = xt.shape
    nq, nkv = c["nq"], c["nkv"]
    d = T["wq"].shape[0] // nq
    half = d // 2
    inv = torch.tensor([c["theta"] ** (-2.0 * i / d) for i in range(half)], dtype=torch.float64)
    rot = torch.polar(torch.ones(S, half, dtype=torch.float64),
                      torch.arange(S, dtype=torch.float64)[:, None] * inv[None])

    def rope(t):
        z = torch.complex(t[..., :half], t[..., half:]) * rot[None, :, None, :]
        return torch.cat([z.real, z.imag], -1)

    h1 = F.rms_norm(xt, (H,), weight=T["attn_norm"], eps=c["eps"])
    q = rope(F.linear(h1, T["wq"]).view(B, S, nq, d))
    k = rope(F.linear(h1, T["wk"]).view(B, S, nkv, d))
    v = F.linear(h1, T["wv"]).view(B, S, nkv, d)
    o = F.scaled_dot_product_attention(q.transpose(1, 2), k.transpose(1, 2), v.transpose(1, 2),
                                       is_causal=True, enable_gqa=True)
    o = o.transpose(1, 2).reshape(B, S, nq * d)
    x2 = xt + F.linear(o, T["wo"])
    h2 = F.rms_norm(x2, (H,), weight=T["mlp_norm"], eps=c["eps"])
    return x2 + F.linear(F.silu(F.linear(h2, T["wg"])) * F.linear(h2, T["wu"]), T["wd"])


def check_block_vs_torch(ob, c=SMALL, seed=14):
    r = _rng(seed)
    x = r.normal(size=(c["B"], c["S"], c["H"]))
    w = make_weights(c, seed + 1)
    dy = r.normal(size=x.shape)
    fwd, grads = ob.block_fwd_bwd(x, w, dy, **block_kw(c))
    y, xt, T = torch_block(x, w, c)
    y.backward(torch.tensor(dy))
    assert _rel(fwd["y"], y.detach().numpy()) < 1e-13, "block y vs torch"
    assert _rel(grads["dx"], xt.grad.numpy()) < 1e-12, "block dx vs torch autograd"
    for name in w:
        assert _rel(grads[name], T[name].grad.numpy()) < 1e-12, f"block d{name} vs torch autograd"


def check_block_finite_differences(ob, c=MICRO, seed=15):
    """Directional derivative of L = <dy, y> along random directions in x and
    every weight, central differences with h = 1e-5 (error ~ h^2)."""
    r = _rng(seed)
    x = r.normal(size=(c["B"], c["S"], c["H"]))
    w = make_weights(c, seed + 1, w_std=0.5)
    dy = r.normal(size=x.shape)
    kw = block_kw(c)
    _, grads = ob.block_fwd_bwd(x, w, dy, **kw)

    def loss(xx, ww):
        return float(np.sum(dy * ob.block_forward(xx, ww, **kw)["y"]))

    for which in ["x"] + list(w):
        for trial in range(2):
            dirn = r.normal(size=x.shape if which == "x" else w[which].shape)
            h = 1e-5
            if which == "x":
                lp, lm = loss(x + h * dirn, w), loss(x - h * dirn, w)
                an = float(np.sum(grads["dx"] * dirn))
            else:
                wp = dict(w)
                wm = dict(w)
                wp[which] = w[which] + h * dirn
                wm[which] = w[which] - h * dirn
                lp, lm = loss(x, wp), loss(x, wm)
                an = float(np.sum(grads[which] * dirn))
            fd = (lp - lm) / (2 * h)
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), f"finite difference d{which}: {fd} vs {an}"


def check_block_causal(ob, c=SMALL, seed=16):
    r = _rng(seed)
    x = r.normal(size=(c["B"], c["S"], c["H"]))
    w = make_weights(c, seed + 1)
    kw = block_kw(c)
    t0 = 9
    y = ob.block_forward(x, w, **kw)["y"]
    x2 = x.copy()
    x2[:, t0 + 1:] = r.normal(size=x2[:, t0 + 1:].shape)
    y2 = ob.block_forward(x2, w, **kw)["y"]
    assert np.array_equal(y[:, :t0 + 1], y2[:, :t0 + 1]), "future tokens leave earlier outputs unchanged"
    dy = r.normal(size=x.shape)
    dy[:, t0 + 1:] = 0.0
    _, g = ob.block_fwd_bwd(x, w, dy, **kw)
    assert np.all(g["dx"][:, t0 + 1:] == 0.0), "no gradient flows to tokens after the last nonzero dy"
    assert np.any(g["dx"][:, :t0 + 1] != 0.0)


ALL_CHECKS = [
    check_rmsnorm_library, check_rmsnorm_invariants,
    check_rope_frequencies, check_rope_complex, check_rope_relative,
    check_attention_bruteforce, check_attention_library, check_attention_closed_forms,
    check_attention_rows_and_mask, check_attention_gqa, check_attention_backward_library,
    check_swiglu,
    check_block_vs_torch, check_block_finite_differences, check_block_causal,
]
