"""The fp64 stack oracle against brute force, a closed form, an independent
torch model, finite differences and causality, and planted mistakes that the
pins must catch (CPU only)."""
import inspect
import textwrap

import numpy as np
import pytest

from oracle import stack as os_

from stack_pins import STACK_CHECKS


@pytest.mark.parametrize("check", STACK_CHECKS, ids=lambda f: f.__name__)
def test_stack_pin(check):
    check(os_)


# (function, exact source fragment, replacement, what the mistake is)
MUTANTS = [
    ("next_token_targets", "t[:, :-1] = ids[:, 1:]", "t[:, :-1] = ids[:, :-1]", "target is the input token"),
    ("cross_entropy", "lse = (m + np.log(s))[:, 0]", "lse = np.log(s)[:, 0]", "lse without the max"),
    ("cross_entropy", "dz[idx, targets[idx]] -= 1.0", "dz[idx, targets[idx]] += 1.0", "one-hot sign"),
    ("cross_entropy", "dz[~valid] = 0.0", "pass", "rows without a target get a gradient"),
    ("cross_entropy", "dz /= max(n, 1)", "dz /= z.shape[0]", "mean over all rows in the gradient"),
    ("cross_entropy", "rows.sum() / max(n, 1)", "rows.sum() / z.shape[0]", "mean over all rows in the loss"),
    ("stack_fwd_bwd", "dE = dz.T @ h.reshape(T, H)", "dE = np.zeros_like(E)", "head part of the tied gradient dropped"),
    ("stack_fwd_bwd", "np.add.at(dE, ids.reshape(T), dx.reshape(T, H))", "dE[ids.reshape(T)] += dx.reshape(T, H)",
     "repeated tokens overwrite instead of summing"),
    ("stack_fwd_bwd", "np.add.at(dE, ids.reshape(T), dx.reshape(T, H))", "pass", "embedding part dropped"),
    ("stack_fwd_bwd", "dx, dg_f = ob.rmsnorm_backward(dh, xs[-1], g_f, r)",
     "dx, dg_f = ob.rmsnorm_backward(dh, xs[-2], g_f, r)", "final norm backward on the wrong input"),
    ("stack_fwd_bwd", "ob.block_fwd_bwd(xs[l], blocks[l], dx, **cfg)", "ob.block_fwd_bwd(xs[l + 1], blocks[l], dx, **cfg)",
     "block recomputed from its output"),
    ("stack_fwd_bwd", "dh = (dz @ E).reshape(B, S, H)", "dh = (dz @ E.T.T * 0).reshape(B, S, H)", "no gradient into the stack"),
    ("stack_fwd_bwd", "h, r = ob.rmsnorm_forward(xs[-1], g_f, eps)", "h, r = ob.rmsnorm_forward(xs[-1], 1.0 + 0 * g_f, eps)",
     "final norm gain ignored"),
]


def _mutate(fn_name, old, new):
    src = textwrap.dedent(inspect.getsource(getattr(os_, fn_name)))
    assert src.count(old) == 1, f"fragment not found once in {fn_name}: {old}"
    ns = dict(vars(os_))
    exec(compile(src.replace(old, new), f"<mutant {fn_name}>", "exec"), ns)
    return ns[fn_name]


@pytest.mark.parametrize("fn_name,old,new,what", MUTANTS, ids=[m[3] for m in MUTANTS])
def test_stack_pins_catch_mutant(monkeypatch, fn_name, old, new, what):
    monkeypatch.setattr(os_, fn_name, _mutate(fn_name, old, new))
    caught = []
    with np.errstate(all="ignore"):
        for check in STACK_CHECKS:
            try:
                check(os_)
            except (AssertionError, ValueError, IndexError, FloatingPointError):
                caught.append(check.__name__)
    assert caught, f"no pin catches: {what}"
