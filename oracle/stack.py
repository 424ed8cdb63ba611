"""fp64 CPU oracle of a stack of decoder blocks with a tied token embedding, a
final RMSNorm, the LM head and next-token cross-entropy, forward and backward.

TEST INFRASTRUCTURE ONLY.  Nothing in the library's product path imports,
links or calls this module; only the tests, the smoke check and the CPU
baseline leg of the benchmark do.

What it computes.  The Litespark report trains Llama-style models (Section
2.4: token embedding, a stack of pre-norm decoder blocks, final RMSNorm, LM
head) with a next-token language-modelling loss; the 3B model of Table 1 has 28
blocks.  With the LM head tied to the embedding matrix E [V, H]:

    x_0      = E[ids]                                (row gather)
    x_{l+1}  = block(x_l; W_l)                       (oracle.block, l = 0 .. L-1)
    h, r     = RMSNorm(x_L; g_f)
    z        = h E^T                                 (logits [T, V])
    loss     = (1/N) sum over rows t with a target of  logsumexp(z_t) - z_t[target_t]

where target[b, s] = ids[b, s+1] for s < S-1 and the last position of every
sequence has no target (N = B (S-1) rows carry one).  The backward pass is the
exact chain rule: dz = (softmax(z) - onehot(target)) / N on rows with a target
and 0 elsewhere; dh = dz E; the head's part of dE is dz^T h; the final norm's
backward gives dx_L; each block's backward (oracle.block) gives dx_l from
dx_{l+1}; and the embedding's part of dE adds row dx_0[t] into row ids[t].  The
two parts of dE are summed (tied weights).  Matrix products are numpy matmuls.
"""
from __future__ import annotations

import numpy as np

from . import block as ob


def next_token_targets(ids: np.ndarray) -> np.ndarray:
    """target[b, s] = ids[b, s+1]; -1 (no target) at the last position."""
    t = np.full_like(ids, -1)
    t[:, :-1] = ids[:, 1:]
    return t


def cross_entropy(z: np.ndarray, targets: np.ndarray):
    """Per-row loss logsumexp(z_t) - z_t[target_t] (0 where target < 0), the
    mean over rows with a target, and dz = (softmax - onehot) / N (0 on rows
    without a target).  z [T, V], targets [T]."""
    m = np.max(z, axis=1, keepdims=True)
    e = np.exp(z - m)
    s = np.sum(e, axis=1, keepdims=True)
    lse = (m + np.log(s))[:, 0]
    valid = targets >= 0
    n = int(np.count_nonzero(valid))
    rows = np.zeros(z.shape[0])
    idx = np.nonzero(valid)[0]
    rows[idx] = lse[idx] - z[idx, targets[idx]]
    dz = e / s
    dz[idx, targets[idx]] -= 1.0
    dz[~valid] = 0.0
    dz /= max(n, 1)
    return rows, rows.sum() / max(n, 1), dz


def stack_fwd_bwd(ids: np.ndarray, E: np.ndarray, blocks: list, g_f: np.ndarray, *, n_q_heads: int,
                  n_kv_heads: int, rope_theta: float, eps: float, targets: np.ndarray | None = None):
    """ids [B, S] int; E [V, H]; blocks: one weight dict per block (as
    oracle.block takes them); g_f [H].  Returns (loss, per-row losses [B*S],
    grads) with grads["embed"] [V, H], grads["final_norm"] [H] and
    grads["blocks"][l] holding the block's weight gradients."""
    B, S = ids.shape
    H = E.shape[1]
    T = B * S
    cfg = dict(n_q_heads=n_q_heads, n_kv_heads=n_kv_heads, rope_theta=rope_theta, eps=eps)
    if targets is None:
        targets = next_token_targets(ids)
    # forward: keep every block's input (the backward recomputes the block)
    xs = [E[ids]]
    for w in blocks:
        xs.append(ob.block_forward(xs[-1], w, **cfg)["y"])
    h, r = ob.rmsnorm_forward(xs[-1], g_f, eps)
    z = h.reshape(T, H) @ E.T
    rows, loss, dz = cross_entropy(z, targets.reshape(T))
    # backward
    dE = dz.T @ h.reshape(T, H)
    dh = (dz @ E).reshape(B, S, H)
    dx, dg_f = ob.rmsnorm_backward(dh, xs[-1], g_f, r)
    gblocks = [None] * len(blocks)
    for l in range(len(blocks) - 1, -1, -1):
        fwd, gr = ob.block_fwd_bwd(xs[l], blocks[l], dx, **cfg)
        gblocks[l] = {k: gr[k] for k in blocks[l]}
        dx = gr["dx"]
    np.add.at(dE, ids.reshape(T), dx.reshape(T, H))
    return loss, rows, {"embed": dE, "final_norm": dg_f, "blocks": gblocks}
