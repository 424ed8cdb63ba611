"""Plant plausible mistakes in the oracle (on the CPU) and check that the pin
suite catches every one of them: a dropped term, a wrong sign, a wrong index
or mapping, a transposed operand, a wrong exponent."""
import inspect
import textwrap

import numpy as np
import pytest

from oracle import block as ob

from oracle_pins import ALL_CHECKS

# (function, exact source fragment, replacement, what the mistake is)
MUTANTS = [
    ("rmsnorm_forward", "np.sqrt(ms + eps)", "np.sqrt(ms)", "eps dropped"),
    ("rmsnorm_forward", "np.mean(x * x, axis=-1, keepdims=True)", "np.sum(x * x, axis=-1, keepdims=True)",
     "sum instead of mean"),
    ("rmsnorm_backward", "dx = a * rr - x * rr ** 3", "dx = a * rr - 0 * x * rr ** 3", "r' term dropped"),
    ("rmsnorm_backward", "x * rr ** 3", "x * rr ** 2", "wrong power of r"),
    ("rmsnorm_backward", "np.sum(dh * x * rr,", "np.sum(dh * x,", "dgamma misses r"),
    ("rmsnorm_backward", "a = dh * gamma", "a = dh", "gamma dropped in backward"),
    ("rope_angles", "-2.0 * i / head_dim", "-1.0 * i / head_dim", "wrong frequency exponent"),
    ("rope_rotate", "x1 * c - x2 * s, x2 * c + x1 * s", "x1 * c + x2 * s, x2 * c - x1 * s", "rotation sign"),
    ("rope_rotate", "x1, x2 = x[..., :half], x[..., half:]", "x1, x2 = x[..., 0::2], x[..., 1::2]",
     "interleaved pairs written back as halves"),
    ("_probs", "(qh @ kh.T) * scale", "(qh @ kh.T)", "softmax scale dropped"),
    ("_probs", "np.tril(np.ones((S, S), dtype=bool))", "np.tril(np.ones((S, S), dtype=bool), -1)",
     "mask drops the diagonal"),
    ("_probs", "np.tril(np.ones((S, S), dtype=bool))", "np.ones((S, S), dtype=bool)", "mask not causal"),
    ("_probs", "(m + np.log(l))[:, 0]", "np.log(l)[:, 0]", "lse without the max"),
    ("attention_forward", "k[b, :, h // G]", "k[b, :, h % k.shape[2]]", "kv head mapping"),
    ("attention_backward", "dS = P * (dP - np.sum(P * dP, axis=1, keepdims=True))", "dS = P * dP",
     "softmax Jacobian row term dropped"),
    ("attention_backward", "dk[b, :, kv] += dS.T @ q[b, :, h] * scale", "dk[b, :, kv] += dS @ q[b, :, h] * scale",
     "dS not transposed for dk"),
    ("attention_backward", "dv[b, :, kv] += P.T @ do[b, :, h]", "dv[b, :, kv] = P.T @ do[b, :, h]",
     "GQA copies overwrite instead of summing"),
    ("attention_backward", "dq[b, :, h] = dS @ k[b, :, kv] * scale", "dq[b, :, h] = dS @ k[b, :, kv]",
     "scale dropped in dq"),
    ("swiglu_backward", "s * (1.0 + g * (1.0 - s))", "s", "silu' term dropped"),
    ("swiglu_backward", "dact * g * s", "dact * s", "du uses sigmoid, not silu"),
    ("block_forward", "x2 = x + o @ w[\"wo\"].T", "x2 = o @ w[\"wo\"].T", "attention residual dropped"),
    ("block_forward", "y = x2 + act @ w[\"wd\"].T", "y = x + act @ w[\"wd\"].T", "wrong residual source"),
    ("block_backward", "dq = rope_rotate(dq, -fwd[\"phi\"])", "dq = rope_rotate(dq, fwd[\"phi\"])",
     "rope backward with +phi"),
    ("block_backward", "dx = dx2 + dx1_n", "dx = dy + dx1_n", "residual gradient path"),
    ("block_backward", "dh1 = dq @ w[\"wq\"] + dk @ w[\"wk\"] + dv @ w[\"wv\"]",
     "dh1 = dq @ w[\"wq\"] + dk @ w[\"wk\"]", "dv contribution dropped"),
    ("block_backward", "dwd = t2(dy).T @ t2(fwd[\"act\"])", "dwd = t2(fwd[\"act\"]).T @ t2(dy)",
     "transposed weight gradient"),
    ("block_backward", "dwg = t2(dg).T @ t2(fwd[\"h2\"])", "dwg = t2(du).T @ t2(fwd[\"h2\"])",
     "gate and up gradients swapped"),
]


def _mutate(fn_name, old, new):
    src = textwrap.dedent(inspect.getsource(getattr(ob, fn_name)))
    assert src.count(old) == 1, f"fragment not found once in {fn_name}: {old}"
    ns = dict(vars(ob))
    exec(compile(src.replace(old, new), f"<mutant {fn_name}>", "exec"), ns)
    return ns[fn_name]


@pytest.mark.parametrize("fn_name,old,new,what", MUTANTS, ids=[m[3] for m in MUTANTS])
def test_pins_catch_mutant(monkeypatch, fn_name, old, new, what):
    monkeypatch.setattr(ob, fn_name, _mutate(fn_name, old, new))
    caught = []
    with np.errstate(all="ignore"):
        for check in ALL_CHECKS:
            try:
                check(ob)
            except (AssertionError, ValueError, IndexError, FloatingPointError):
                caught.append(check.__name__)
    assert caught, f"no pin catches: {what}"
