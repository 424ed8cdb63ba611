"""Checks that pin the fp64 stack oracle (embedding, decoder blocks, final
RMSNorm, tied LM head, next-token cross-entropy) to facts other than itself.

Each ``check_*`` takes the stack oracle module and raises AssertionError when
it disagrees with:

* brute force: per-row pure-Python log-sum-exp and softmax gradient;
* a closed form: with a zero embedding matrix every logit is zero, so the loss
  is ln V exactly and every gradient is exactly zero;
* an independent torch float64 model (F.embedding, the torch block, F.rms_norm,
  F.linear with the tied matrix, F.cross_entropy over the shifted logits and
  ids) whose autograd gives every gradient;
* central finite differences of the oracle's own forward loss;
* causality: a row's loss depends only on the tokens up to its target.
"""
from __future__ import annotations

import math

import numpy as np
import torch
import torch.nn.functional as F

from oracle_pins import MICRO, SMALL, _rel, _rng, block_kw, make_weights, torch_block_t


def make_stack(c, V, L, seed, w_std=0.3, e_std=1.0):
    r = _rng(seed)
    E = r.normal(0, e_std, (V, c["H"]))
    blocks = [make_weights(c, seed + 1 + l, w_std=w_std) for l in range(L)]
    g_f = 1 + 0.2 * r.normal(size=c["H"])
    return E, blocks, g_f


def make_ids(c, V, seed):
    """Token ids with repeats (V is small), so that the embedding's scatter-add
    sees several rows land on one token."""
    return _rng(seed).integers(0, V, size=(c["B"], c["S"]))


def check_ce_bruteforce(os_):
    r = _rng(31)
    T, V = 7, 9
    z = r.normal(0, 3, (T, V))
    tg = r.integers(0, V, size=T)
    tg[2] = -1
    tg[5] = -1
    rows, loss, dz = os_.cross_entropy(z, tg)
    n = 5
    tot = 0.0
    for t in range(T):
        zs = [float(v) for v in z[t]]
        big = max(zs)
        se = sum(math.exp(v - big) for v in zs)
        if tg[t] < 0:
            assert rows[t] == 0.0 and np.all(dz[t] == 0.0), "rows without a target carry nothing"
            continue
        want = big + math.log(se) - zs[tg[t]]
        assert abs(rows[t] - want) < 1e-13, "per-row loss"
        tot += want
        for v in range(V):
            g = (math.exp(zs[v] - big) / se - (1.0 if v == tg[t] else 0.0)) / n
            assert abs(dz[t, v] - g) < 1e-15, "softmax gradient"
    assert abs(loss - tot / n) < 1e-13, "mean over rows with a target"


def check_ce_library(os_):
    r = _rng(32)
    T, V = 12, 17
    z = r.normal(0, 2, (T, V))
    tg = r.integers(0, V, size=T)
    tg[[0, 7]] = -1
    rows, loss, dz = os_.cross_entropy(z, tg)
    zt = torch.tensor(z, requires_grad=True)
    lt = F.cross_entropy(zt, torch.tensor(tg), ignore_index=-1)
    lt.backward()
    assert abs(loss - lt.item()) < 1e-13, "loss vs F.cross_entropy"
    assert _rel(dz, zt.grad.numpy()) < 1e-13, "dz vs autograd"
    rt = F.cross_entropy(torch.tensor(z), torch.tensor(tg), ignore_index=-1, reduction="none")
    assert _rel(rows, rt.numpy()) < 1e-13, "per-row loss vs F.cross_entropy"


def check_targets(os_):
    ids = np.array([[3, 1, 4, 1, 5], [9, 2, 6, 5, 3]])
    want = np.array([[1, 4, 1, 5, -1], [2, 6, 5, 3, -1]])
    assert np.array_equal(os_.next_token_targets(ids), want), "next-token targets"


def check_stack_zero_embedding(os_, c=SMALL, V=11, L=2):
    """E = 0: x_0 = 0, every block maps 0 to 0 (RMSNorm(0) = 0, so q = k = v =
    0 and the MLP input is 0), every logit is 0, the loss is ln V and every
    gradient vanishes (each is a product with a zero activation or with E)."""
    E, blocks, g_f = make_stack(c, V, L, 33)
    E[:] = 0.0
    ids = make_ids(c, V, 34)
    loss, rows, g = os_.stack_fwd_bwd(ids, E, blocks, g_f, **block_kw(c))
    assert abs(loss - math.log(V)) < 1e-14, "uniform logits give ln V"
    assert np.all(rows.reshape(c["B"], c["S"])[:, -1] == 0.0), "last position has no target"
    assert np.all(g["embed"] == 0.0) and np.all(g["final_norm"] == 0.0)
    for gb in g["blocks"]:
        for k, v in gb.items():
            assert np.all(v == 0.0), f"zero gradient of {k}"


def torch_stack(ids, E, blocks, g_f, c):
    """Independent float64 model: F.embedding, torch blocks, F.rms_norm, tied
    F.linear head, F.cross_entropy of logits[:, :-1] against ids[:, 1:]."""
    Et = torch.tensor(E, requires_grad=True)
    gt = torch.tensor(g_f, requires_grad=True)
    Ts = [{k: torch.tensor(v, requires_grad=True) for k, v in w.items()} for w in blocks]
    it = torch.tensor(ids)
    x = F.embedding(it, Et)
    for T in Ts:
        x = torch_block_t(x, T, c)
    h = F.rms_norm(x, (E.shape[1],), weight=gt, eps=c["eps"])
    z = F.linear(h, Et)
    V = E.shape[0]
    rows = F.cross_entropy(z[:, :-1].reshape(-1, V), it[:, 1:].reshape(-1), reduction="none")
    loss = rows.mean()
    loss.backward()
    return loss.item(), rows.detach().numpy().reshape(ids.shape[0], -1), Et.grad.numpy(), gt.grad.numpy(), \
        [{k: t.grad.numpy() for k, t in T.items()} for T in Ts]


def check_stack_vs_torch(os_, c=SMALL, V=19, L=2, seed=35):
    E, blocks, g_f = make_stack(c, V, L, seed)
    ids = make_ids(c, V, seed + 50)
    loss, rows, g = os_.stack_fwd_bwd(ids, E, blocks, g_f, **block_kw(c))
    tl, trows, tdE, tdg, tgb = torch_stack(ids, E, blocks, g_f, c)
    assert abs(loss - tl) < 1e-12 * max(1.0, abs(tl)), "loss vs torch"
    r2 = rows.reshape(ids.shape)
    assert _rel(r2[:, :-1], trows) < 1e-12 and np.all(r2[:, -1] == 0.0), "per-row loss vs torch"
    assert _rel(g["embed"], tdE) < 1e-11, "tied embedding gradient vs torch autograd"
    assert _rel(g["final_norm"], tdg) < 1e-11, "final norm gradient vs torch autograd"
    for l in range(L):
        for k in blocks[l]:
            assert _rel(g["blocks"][l][k], tgb[l][k]) < 1e-10, f"block {l} d{k} vs torch autograd"


def check_stack_no_blocks(os_, c=SMALL, V=13):
    """L = 0: the model is embedding -> RMSNorm -> tied head."""
    check_stack_vs_torch(os_, c, V, 0, seed=36)


def check_stack_finite_differences(os_, c=MICRO, V=7, L=2, seed=37):
    E, blocks, g_f = make_stack(c, V, L, seed, w_std=0.5)
    ids = make_ids(c, V, seed + 50)
    kw = block_kw(c)
    _, _, g = os_.stack_fwd_bwd(ids, E, blocks, g_f, **kw)
    r = _rng(seed + 1)

    def loss(EE, bb, gg):
        return os_.stack_fwd_bwd(ids, EE, bb, gg, **kw)[0]

    h = 1e-5
    cases = [("embed", None), ("final_norm", None)] + [(k, l) for l in range(L) for k in ("wq", "wd", "attn_norm")]
    for which, l in cases:
        if which == "embed":
            dirn = r.normal(size=E.shape)
            fd = (loss(E + h * dirn, blocks, g_f) - loss(E - h * dirn, blocks, g_f)) / (2 * h)
            an = float(np.sum(g["embed"] * dirn))
        elif which == "final_norm":
            dirn = r.normal(size=g_f.shape)
            fd = (loss(E, blocks, g_f + h * dirn) - loss(E, blocks, g_f - h * dirn)) / (2 * h)
            an = float(np.sum(g["final_norm"] * dirn))
        else:
            dirn = r.normal(size=blocks[l][which].shape)
            bp = [dict(b) for b in blocks]
            bm = [dict(b) for b in blocks]
            bp[l][which] = blocks[l][which] + h * dirn
            bm[l][which] = blocks[l][which] - h * dirn
            fd = (loss(E, bp, g_f) - loss(E, bm, g_f)) / (2 * h)
            an = float(np.sum(g["blocks"][l][which] * dirn))
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), f"finite difference {which} {l}: {fd} vs {an}"


def check_stack_causal(os_, c=SMALL, V=23, L=2, seed=38):
    """The loss of row s depends on ids[:, :s+2] only (its inputs and its
    target); later tokens leave it unchanged, bit for bit."""
    E, blocks, g_f = make_stack(c, V, L, seed)
    ids = make_ids(c, V, seed + 50)
    kw = block_kw(c)
    _, rows, _ = os_.stack_fwd_bwd(ids, E, blocks, g_f, **kw)
    t0 = 6
    ids2 = ids.copy()
    ids2[:, t0 + 2:] = (ids2[:, t0 + 2:] + 1) % V
    _, rows2, _ = os_.stack_fwd_bwd(ids2, E, blocks, g_f, **kw)
    S = ids.shape[1]
    a, b = rows.reshape(-1, S), rows2.reshape(-1, S)
    assert np.array_equal(a[:, :t0 + 1], b[:, :t0 + 1]), "earlier rows unchanged by later tokens"
    assert not np.array_equal(a[:, t0 + 1:], b[:, t0 + 1:])


STACK_CHECKS = [
    check_ce_bruteforce, check_ce_library, check_targets, check_stack_zero_embedding,
    check_stack_vs_torch, check_stack_no_blocks, check_stack_finite_differences, check_stack_causal,
]
