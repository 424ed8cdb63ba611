"""fp64 CPU oracle of one Llama-style decoder block, forward and backward.

TEST INFRASTRUCTURE ONLY.  Nothing in the library's product path imports,
links or calls this module; only the tests, the smoke check and the CPU
baseline leg of the benchmark do.

What it computes.  The Litespark report (Section 1) speeds up the attention
and MLP layers of a standard transformer without changing the function they
compute (abstract; Section 5: no architecture change and no quality loss).
Section 2.4 names the block: RMSNorm, rotary position embedding, grouped-query
(3B) or multi-head (30B) attention and a SwiGLU MLP, in the Llama layout.  So
the oracle is the plain definition of that block, written out in float64:

    h1 = RMSNorm(x; g1)                      r1 = (mean_j x_j^2 + eps)^-1/2
    q, k, v = h1 Wq^T, h1 Wk^T, h1 Wv^T       (heads of width d)
    q, k   <- RoPE(q), RoPE(k)               pair (i, i + d/2), angle p * theta^(-2i/d)
    o      = causal softmax(q k^T / sqrt(d)) v   query head h reads kv head h // G
    x2     = x + o Wo^T
    h2     = RMSNorm(x2; g2)
    y      = x2 + (silu(h2 Wg^T) * (h2 Wu^T)) Wd^T

and its exact reverse-mode derivative.  Attention materialises the full S x S
score matrix per head (no tiling, no online softmax); every matrix product is
a library matmul on float64 arrays.  Readings of points the report leaves open
(norm placement, RoPE pairing and frequencies, kv-head mapping, softmax scale,
log-sum-exp units) are listed where each function is defined.
"""
from __future__ import annotations

import math

import numpy as np


# --------------------------------------------------------------------------
# RMSNorm (Section 2.4; Zhang & Sennrich 2019)
# --------------------------------------------------------------------------

def rmsnorm_forward(x: np.ndarray, gamma: np.ndarray, eps: float):
    """h = x * r * gamma with r = 1 / sqrt(mean(x^2) + eps) over the last axis.

    Returns (h, r) with r shaped like x without its last axis.
    """
    ms = np.mean(x * x, axis=-1, keepdims=True)
    r = 1.0 / np.sqrt(ms + eps)
    return x * r * gamma, r[..., 0]


def rmsnorm_backward(dh: np.ndarray, x: np.ndarray, gamma: np.ndarray, r: np.ndarray):
    """Gradient of rmsnorm_forward.

    With a = gamma * dh:  dx = r * a - x * r^3 * <a, x> / H  (the second term is
    the derivative of r, dr/dx_j = -r^3 x_j / H), and dgamma = sum over rows of
    dh * x * r.
    """
    H = x.shape[-1]
    rr = r[..., None]
    a = dh * gamma
    dx = a * rr - x * rr ** 3 * np.sum(a * x, axis=-1, keepdims=True) / H
    dgamma = np.sum(dh * x * rr, axis=tuple(range(x.ndim - 1)))
    return dx, dgamma


# --------------------------------------------------------------------------
# Rotary position embedding (Section 2.4; Su et al.)
# Reading: the "rotate-half" pairing (i, i + d/2), frequencies theta^(-2i/d)
# with no rescaling, positions 0..S-1 restarting for every sequence.
# --------------------------------------------------------------------------

def rope_angles(seq: int, head_dim: int, theta: float) -> np.ndarray:
    """phi[p, i] = p * theta^(-2i/d) for p < seq, i < d/2 (radians, float64)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = theta ** (-2.0 * i / head_dim)
    pos = np.arange(seq, dtype=np.float64)
    return np.outer(pos, inv_freq)


def rope_rotate(x: np.ndarray, phi: np.ndarray) -> np.ndarray:
    """Rotate each pair (x_i, x_{i+d/2}) of x [B, S, heads, d] by phi[s, i].

    The backward of a rotation by phi is the rotation by -phi.
    """
    half = x.shape[-1] // 2
    c = np.cos(phi)[None, :, None, :]
    s = np.sin(phi)[None, :, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


# --------------------------------------------------------------------------
# Causal grouped-query attention (Section 2.4; Ainslie et al. for GQA)
# Reading: scale 1/sqrt(d); mask keeps key j <= query i (diagonal included);
# query head h reads kv head h // G with G = n_q / n_kv; log-sum-exp in
# natural-log units.
# --------------------------------------------------------------------------

def _probs(qh: np.ndarray, kh: np.ndarray, scale: float):
    """Explicit masked softmax for one head: returns (P [S,S], lse [S])."""
    S = qh.shape[0]
    s = (qh @ kh.T) * scale
    s = np.where(np.tril(np.ones((S, S), dtype=bool)), s, -np.inf)
    m = np.max(s, axis=1, keepdims=True)
    e = np.exp(s - m)
    l = np.sum(e, axis=1, keepdims=True)
    return e / l, (m + np.log(l))[:, 0]


def attention_forward(q: np.ndarray, k: np.ndarray, v: np.ndarray):
    """q [B,S,nq,d], k and v [B,S,nkv,d] -> (o [B,S,nq,d], lse [B,nq,S])."""
    B, S, nq, d = q.shape
    G = nq // k.shape[2]
    scale = 1.0 / math.sqrt(d)
    o = np.empty_like(q)
    lse = np.empty((B, nq, S))
    for b in range(B):
        for h in range(nq):
            P, lse[b, h] = _probs(q[b, :, h], k[b, :, h // G], scale)
            o[b, :, h] = P @ v[b, :, h // G]
    return o, lse


def attention_backward(do: np.ndarray, q: np.ndarray, k: np.ndarray, v: np.ndarray):
    """Gradients of attention_forward's o with respect to q, k, v.

    Per head: dP = dO V^T; through the row softmax dS_ij = P_ij (dP_ij -
    sum_l P_il dP_il); dQ = dS K scale; dK = dS^T Q scale; dV = P^T dO.  A kv
    head's gradient is the sum over the G query heads that read it.
    """
    B, S, nq, d = q.shape
    G = nq // k.shape[2]
    scale = 1.0 / math.sqrt(d)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(B):
        for h in range(nq):
            kv = h // G
            P, _ = _probs(q[b, :, h], k[b, :, kv], scale)
            dP = do[b, :, h] @ v[b, :, kv].T
            dS = P * (dP - np.sum(P * dP, axis=1, keepdims=True))
            dq[b, :, h] = dS @ k[b, :, kv] * scale
            dk[b, :, kv] += dS.T @ q[b, :, h] * scale
            dv[b, :, kv] += P.T @ do[b, :, h]
    return dq, dk, dv


# --------------------------------------------------------------------------
# SwiGLU (Section 2.4; Shazeer 2020): act = silu(g) * u, silu(z) = z sigmoid(z)
# --------------------------------------------------------------------------

def sigmoid(z: np.ndarray) -> np.ndarray:
    """1/(1+e^-z) for z >= 0 and e^z/(1+e^z) otherwise (no overflow)."""
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    e = np.exp(z[~pos])
    out[~pos] = e / (1.0 + e)
    return out


def swiglu_forward(g: np.ndarray, u: np.ndarray) -> np.ndarray:
    return g * sigmoid(g) * u


def swiglu_backward(dact: np.ndarray, g: np.ndarray, u: np.ndarray):
    """(dg, du) with silu'(z) = sigmoid(z) (1 + z (1 - sigmoid(z)))."""
    s = sigmoid(g)
    return dact * u * s * (1.0 + g * (1.0 - s)), dact * g * s


# --------------------------------------------------------------------------
# The block (pre-norm: x2 = x + Attn(N1 x); y = x2 + MLP(N2 x2))
# --------------------------------------------------------------------------

def block_forward(x: np.ndarray, w: dict, *, n_q_heads: int, n_kv_heads: int,
                  rope_theta: float, eps: float) -> dict:
    """x [B,S,H]; w holds wq [Dq,H], wk/wv [Dkv,H], wo [H,Dq], wg/wu [I,H],
    wd [H,I], attn_norm/mlp_norm [H] (nn.Linear [out, in] layout).

    Returns every intermediate the backward uses plus the output y.
    """
    B, S, H = x.shape
    d = w["wq"].shape[0] // n_q_heads
    h1, r1 = rmsnorm_forward(x, w["attn_norm"], eps)
    q = (h1 @ w["wq"].T).reshape(B, S, n_q_heads, d)
    k = (h1 @ w["wk"].T).reshape(B, S, n_kv_heads, d)
    v = (h1 @ w["wv"].T).reshape(B, S, n_kv_heads, d)
    phi = rope_angles(S, d, rope_theta)
    q = rope_rotate(q, phi)
    k = rope_rotate(k, phi)
    o, lse = attention_forward(q, k, v)
    o = o.reshape(B, S, n_q_heads * d)
    x2 = x + o @ w["wo"].T
    h2, r2 = rmsnorm_forward(x2, w["mlp_norm"], eps)
    g = h2 @ w["wg"].T
    u = h2 @ w["wu"].T
    act = swiglu_forward(g, u)
    y = x2 + act @ w["wd"].T
    return dict(h1=h1, r1=r1, q=q, k=k, v=v, phi=phi, o=o, lse=lse, x2=x2, h2=h2,
                r2=r2, g=g, u=u, act=act, y=y)


def block_backward(x: np.ndarray, w: dict, fwd: dict, dy: np.ndarray) -> dict:
    """Reverse mode through block_forward for upstream gradient dy [B,S,H].

    Returns dx and the gradient of every weight (same names as ``w``).
    """
    B, S, H = x.shape
    T = B * S
    t2 = lambda a: a.reshape(T, a.shape[-1])  # noqa: E731  tokens-by-features view

    # MLP sub-layer
    dact = dy @ w["wd"]
    dwd = t2(dy).T @ t2(fwd["act"])
    dg, du = swiglu_backward(dact, fwd["g"], fwd["u"])
    dh2 = dg @ w["wg"] + du @ w["wu"]
    dwg = t2(dg).T @ t2(fwd["h2"])
    dwu = t2(du).T @ t2(fwd["h2"])
    dx2_n, dgamma2 = rmsnorm_backward(dh2, fwd["x2"], w["mlp_norm"], fwd["r2"])
    dx2 = dy + dx2_n

    # attention sub-layer
    dwo = t2(dx2).T @ t2(fwd["o"])
    do = (dx2 @ w["wo"]).reshape(fwd["q"].shape)
    dq, dk, dv = attention_backward(do, fwd["q"], fwd["k"], fwd["v"])
    dq = rope_rotate(dq, -fwd["phi"]).reshape(B, S, -1)
    dk = rope_rotate(dk, -fwd["phi"]).reshape(B, S, -1)
    dv = dv.reshape(B, S, -1)
    dwq = t2(dq).T @ t2(fwd["h1"])
    dwk = t2(dk).T @ t2(fwd["h1"])
    dwv = t2(dv).T @ t2(fwd["h1"])
    dh1 = dq @ w["wq"] + dk @ w["wk"] + dv @ w["wv"]
    dx1_n, dgamma1 = rmsnorm_backward(dh1, x, w["attn_norm"], fwd["r1"])
    dx = dx2 + dx1_n
    return dict(dx=dx, dx2=dx2, do=do.reshape(B, S, -1), dqkv=np.concatenate([dq, dk, dv], -1),
                dh1=dh1, dh2=dh2, dg=dg, du=du, dact=dact,
                attn_norm=dgamma1, wq=dwq, wk=dwk, wv=dwv, wo=dwo,
                mlp_norm=dgamma2, wg=dwg, wu=dwu, wd=dwd)


def block_fwd_bwd(x: np.ndarray, w: dict, dy: np.ndarray, **cfg):
    """Forward then backward; returns (forward intermediates, gradients)."""
    fwd = block_forward(x, w, **cfg)
    return fwd, block_backward(x, w, fwd, dy)
