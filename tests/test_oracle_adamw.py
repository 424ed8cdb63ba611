"""The fp64 optimizer oracle (global-norm clip + AdamW) against closed forms
and torch.optim.AdamW with clip_grad_norm_, and planted mistakes that these
pins must catch (CPU only)."""
import inspect
import math
import textwrap

import numpy as np
import pytest
import torch

from oracle import adamw as oa

HP = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.01)


def check_norm_known_values(oa_):
    assert oa_.global_norm(np.array([3.0, 4.0])) == 5.0
    assert oa_.global_norm(np.ones(16)) == 4.0
    assert oa_.clip_coefficient(0.5, 1.0) == 1.0, "small gradients are never scaled up"
    assert abs(oa_.clip_coefficient(4.0, 1.0) - 1.0 / (4.0 + 1e-6)) < 1e-16


def check_first_step_closed_form(oa_):
    """t = 1, no decay, no clip: mhat = g and vhat = g^2 exactly, so the step
    is lr g / (|g| + eps) (about lr times the sign of g)."""
    r = np.random.default_rng(1)
    p, g = r.normal(size=50), r.normal(size=50)
    z = np.zeros(50)
    hp = dict(HP, weight_decay=0.0)
    p1, m1, v1, norm = oa_.adamw_step(p, g, z, z, step=1, max_norm=None, **hp)
    assert np.allclose(p1, p - hp["lr"] * g / (np.abs(g) + hp["eps"]), rtol=0, atol=1e-15)
    assert np.allclose(m1, 0.1 * g, rtol=1e-15) and np.allclose(v1, 0.05 * g * g, rtol=1e-15)
    assert abs(norm - math.sqrt(float(np.sum(g * g)))) < 1e-12


def check_constant_gradient_bias_correction(oa_):
    """A constant gradient keeps mhat = g and vhat = g^2 at every step, so
    after t steps p = p0 - t lr g / (|g| + eps) (no decay, no clip)."""
    g = np.array([0.3, -2.0, 1e-3, 5.0])
    p = np.array([1.0, -1.0, 0.5, 0.0])
    m = np.zeros(4)
    v = np.zeros(4)
    hp = dict(HP, weight_decay=0.0)
    p0 = p.copy()
    for t in range(1, 6):
        p, m, v, _ = oa_.adamw_step(p, g, m, v, step=t, max_norm=None, **hp)
        want = p0 - t * hp["lr"] * g / (np.abs(g) + hp["eps"])
        assert np.allclose(p, want, rtol=0, atol=1e-13), f"step {t}"


def check_zero_gradient_only_decays(oa_):
    r = np.random.default_rng(2)
    p = r.normal(size=20)
    z = np.zeros(20)
    p1, m1, v1, norm = oa_.adamw_step(p, z, z, z, step=1, max_norm=1.0, n_decay=12, **HP)
    assert norm == 0.0 and np.all(m1 == 0) and np.all(v1 == 0)
    assert np.array_equal(p1[:12], p[:12] - HP["lr"] * HP["weight_decay"] * p[:12]), "decoupled decay"
    assert np.array_equal(p1[12:], p[12:]), "no decay past n_decay"


def check_clip_scales_gradient(oa_):
    """With beta1 = beta2 = 0 and t = 1 the moments are the clipped gradient
    itself: m = c g with c = max_norm / (norm + 1e-6) when norm > max_norm,
    and the clipped norm is max_norm up to that 1e-6."""
    g = np.array([3.0, 4.0, 0.0, 12.0])   # norm 13
    z = np.zeros(4)
    hp = dict(HP, beta1=0.0, beta2=0.0)
    _, m1, v1, norm = oa_.adamw_step(np.ones(4), g, z, z, step=1, max_norm=1.0, **hp)
    assert norm == 13.0
    assert np.allclose(m1, g / (13.0 + 1e-6), rtol=1e-15)
    assert abs(np.linalg.norm(m1) - 13.0 / (13.0 + 1e-6)) < 1e-15
    _, m2, _, _ = oa_.adamw_step(np.ones(4), g, z, z, step=1, max_norm=20.0, **hp)
    assert np.array_equal(m2, g), "below the threshold the gradient is unchanged"


def check_vs_torch(oa_):
    """Three steps of torch.optim.AdamW (float64) with clip_grad_norm_ over two
    parameter groups (decayed, not decayed), changing gradients each step."""
    r = np.random.default_rng(3)
    n, nd = 300, 200
    p = r.normal(size=n)
    m = np.zeros(n)
    v = np.zeros(n)
    tp_d = torch.tensor(p[:nd].copy(), requires_grad=True)
    tp_n = torch.tensor(p[nd:].copy(), requires_grad=True)
    opt = torch.optim.AdamW([{"params": [tp_d], "weight_decay": HP["weight_decay"]},
                             {"params": [tp_n], "weight_decay": 0.0}],
                            lr=HP["lr"], betas=(HP["beta1"], HP["beta2"]), eps=HP["eps"])
    for t in range(1, 4):
        g = r.normal(size=n) * (0.05 if t == 2 else 1.0)  # step 2 stays below the clip threshold
        tp_d.grad = torch.tensor(g[:nd].copy())
        tp_n.grad = torch.tensor(g[nd:].copy())
        tn = torch.nn.utils.clip_grad_norm_([tp_d, tp_n], 1.0)
        opt.step()
        p, m, v, norm = oa_.adamw_step(p, g, m, v, step=t, max_norm=1.0, n_decay=nd, **HP)
        assert abs(norm - float(tn)) < 1e-12, "pre-clip norm"
        want = np.concatenate([tp_d.detach().numpy(), tp_n.detach().numpy()])
        assert np.allclose(p, want, rtol=0, atol=1e-14), f"parameters after step {t}"
        st = opt.state[tp_d]
        assert np.allclose(m[:nd], st["exp_avg"].numpy(), rtol=1e-14, atol=1e-18)
        assert np.allclose(v[:nd], st["exp_avg_sq"].numpy(), rtol=1e-14, atol=1e-20)


ADAMW_CHECKS = [check_norm_known_values, check_first_step_closed_form, check_constant_gradient_bias_correction,
                check_zero_gradient_only_decays, check_clip_scales_gradient, check_vs_torch]


@pytest.mark.parametrize("check", ADAMW_CHECKS, ids=lambda f: f.__name__)
def test_adamw_pin(check):
    check(oa)


MUTANTS = [
    ("adamw_step", "mhat = m / (1.0 - beta1 ** step)", "mhat = m", "no bias correction of m"),
    ("adamw_step", "vhat = v / (1.0 - beta2 ** step)", "vhat = v / (1.0 - beta1 ** step)", "beta1 in v's correction"),
    ("adamw_step", "p[:nd] = p[:nd] - lr * weight_decay * p[:nd]", "pass", "decoupled decay dropped"),
    ("adamw_step", "p[:nd] = p[:nd] - lr * weight_decay * p[:nd]", "p[:nd] = p[:nd] - weight_decay * p[:nd]",
     "decay not scaled by the learning rate"),
    ("adamw_step", "p[:nd] = p[:nd] - lr * weight_decay * p[:nd]", "p = p - lr * weight_decay * p",
     "decay applied to every parameter"),
    ("adamw_step", "np.sqrt(vhat) + eps", "np.sqrt(vhat + eps)", "eps inside the square root"),
    ("adamw_step", "v = beta2 * v + (1.0 - beta2) * g * g", "v = beta2 * v + (1.0 - beta2) * np.abs(g)",
     "first power in the second moment"),
    ("adamw_step", "m = beta1 * m + (1.0 - beta1) * g", "m = beta2 * m + (1.0 - beta2) * g", "betas swapped"),
    ("clip_coefficient", "min(1.0, max_norm / (norm + 1e-6))", "max_norm / (norm + 1e-6)",
     "small gradients scaled up"),
    ("global_norm", "np.sqrt(np.sum(grads * grads))", "np.sum(np.abs(grads))", "L1 norm"),
]


def _mutate(fn_name, old, new):
    src = textwrap.dedent(inspect.getsource(getattr(oa, fn_name)))
    assert src.count(old) == 1, f"fragment not found once in {fn_name}: {old}"
    ns = dict(vars(oa))
    exec(compile(src.replace(old, new), f"<mutant {fn_name}>", "exec"), ns)
    return ns[fn_name]


@pytest.mark.parametrize("fn_name,old,new,what", MUTANTS, ids=[m[3] for m in MUTANTS])
def test_adamw_pins_catch_mutant(monkeypatch, fn_name, old, new, what):
    monkeypatch.setattr(oa, fn_name, _mutate(fn_name, old, new))
    caught = []
    with np.errstate(all="ignore"):
        for check in ADAMW_CHECKS:
            try:
                check(oa)
            except (AssertionError, ValueError, IndexError, FloatingPointError):
                caught.append(check.__name__)
    assert caught, f"no pin catches: {what}"
