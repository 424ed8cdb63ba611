"""Parity of the optimizer step on the GPU (global-norm clip + AdamW over flat
fp32 arrays) against the fp64 oracle, and two whole training steps of the
small stack (forward, backward, optimizer) against the oracles chained the
same way."""
import numpy as np
import pytest
import torch

from oracle import adamw as oa
from oracle import stack as ost
from paper_2510_02483_amd import configs, inputs, lib as L

from gpu_util import OUT_TOL, f64, fro_rel, max_rel, need_gpu, say

pytestmark = pytest.mark.gpu

HP = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.01)


@pytest.mark.parametrize("max_norm", [1.0, 0.0], ids=["clip", "no-clip"])
def test_adamw_parity(max_norm):
    """n with a ragged tail (n % 4 = 3) and a decay boundary inside a 16-byte
    vector; three steps, the clip active on steps 1 and 3 only."""
    need_gpu()
    n, nd = 1_000_003, 700_001
    say(f"adamw n={n} n_decay={nd} max_norm={max_norm}")
    g = torch.Generator().manual_seed(5)
    master = (torch.randn(n, generator=g) * 0.02).cuda()
    param = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    norm = torch.zeros(1, device="cuda")
    p_ref, m_ref, v_ref = f64(master), np.zeros(n), np.zeros(n)
    for t, std in enumerate([2e-3, 5e-4, 3e-3], start=1):
        grad = (torch.randn(n, generator=g) * std).cuda()
        L.ls_adamw_step(master, param, grad, m, v, step=t, max_norm=max_norm, n_decay=nd, grad_norm=norm, **HP)
        torch.cuda.synchronize()
        p_ref, m_ref, v_ref, nrm = oa.adamw_step(p_ref, f64(grad), m_ref, v_ref, step=t,
                                                  max_norm=max_norm if max_norm > 0 else None, n_decay=nd, **HP)
        errs = dict(p=max_rel(f64(master), p_ref), m=max_rel(f64(m), m_ref), v=max_rel(f64(v), v_ref),
                    norm=abs(norm.item() - nrm) / nrm)
        say(f"  step {t} norm {nrm:.3f}: " + " ".join(f"{k} {e:.1e}" for k, e in errs.items()))
        assert all(e < 1e-5 for e in errs.values()), errs
        assert torch.equal(param, master.to(torch.bfloat16)), "bf16 copy is the RNE rounding of the master"


def test_adamw_rejects_bad_arguments_on_gpu_host():
    need_gpu()
    x = torch.zeros(64, device="cuda")
    with pytest.raises(L.LsError):
        L.ls_adamw_step(x, None, x, torch.zeros_like(x), torch.zeros_like(x), step=1, lr=1e-3)  # grad aliases master
    with pytest.raises(L.LsError):
        L.ls_adamw_step(x, None, torch.zeros_like(x), torch.zeros_like(x), torch.zeros_like(x), step=0, lr=1e-3)


def _flat_order(sc):
    return [("embed", None)] + [(n, l) for l in range(sc.n_layers) for n in L.DECAYED] + \
        [("final_norm", None)] + [(n, l) for l in range(sc.n_layers) for n in L.NOT_DECAYED]


def test_train_steps_tiny_stack():
    """Two training steps (stack forward + backward, clipped AdamW, bf16
    weights rewritten) against the fp64 oracles chained the same way: the
    loss of each step, the pre-clip gradient norm and the moments; the final
    master weights against the optimizer oracle on the GPU's gradients.  A
    large learning rate moves the step-2 loss far beyond the tolerance, so a
    wrongly wired update would show."""
    need_gpu()
    sc = configs.TINY_STACK
    lr = 2e-2
    say(f"train steps {sc} lr={lr}")
    host = inputs.make_stack_inputs(sc, gamma="random", e_std=0.1)
    st = L.Stack(sc, host)
    order = _flat_order(sc)

    def get(h, name, l):
        return h[name] if l is None else h["layers"][l][name]

    # oracle state: fp64 master from the bf16 weights, flat in the arena order
    p_ref = np.concatenate([get(host, n, l).double().numpy().ravel() for n, l in order])
    m_ref = np.zeros_like(p_ref)
    v_ref = np.zeros_like(p_ref)
    ids = host["ids"].numpy().astype(np.int64)
    c = sc.block
    kw = dict(n_q_heads=c.n_q_heads, n_kv_heads=c.n_kv_heads, rope_theta=c.rope_theta, eps=c.rms_eps)
    losses = []
    # the optimizer oracle fed with the GPU's own gradients (isolates the update)
    p_own = p_ref.copy()
    m_own = np.zeros_like(p_ref)
    v_own = np.zeros_like(p_ref)
    for t in (1, 2):
        st.step()
        torch.cuda.synchronize()
        g_gpu = f64(st.g_arena)
        st.optimizer_step(lr=lr)
        torch.cuda.synchronize()
        p_own, m_own, v_own, _ = oa.adamw_step(p_own, g_gpu, m_own, v_own, step=t, max_norm=1.0,
                                               n_decay=st.n_decay, **dict(HP, lr=lr))
        # oracle: weights = bf16 rounding of the master (what the GPU's forward reads)
        wb = torch.from_numpy(p_ref).to(torch.bfloat16).double().numpy()
        views, off = {}, 0
        for n, l in order:
            k = get(host, n, l).numel()
            views[(n, l)] = wb[off:off + k].reshape(tuple(get(host, n, l).shape))
            off += k
        blocks = [{n: views[(n, l)] for n in L.WEIGHTS} for l in range(sc.n_layers)]
        loss, _, gr = ost.stack_fwd_bwd(ids, views[("embed", None)], blocks, views[("final_norm", None)], **kw)
        flat_g = np.concatenate([(gr["embed"] if n == "embed" else gr["final_norm"] if n == "final_norm"
                                  else gr["blocks"][l][n]).ravel() for n, l in order])
        p_ref, m_ref, v_ref, nrm = oa.adamw_step(p_ref, flat_g, m_ref, v_ref, step=t, max_norm=1.0,
                                                  n_decay=st.n_decay, **dict(HP, lr=lr))
        e_loss = abs(st.loss.item() - loss) / loss
        e_norm = abs(st.grad_norm.item() - nrm) / nrm
        say(f"  step {t}: loss {loss:.5f} (gpu {st.loss.item():.5f}, {e_loss:.1e}), grad norm {nrm:.4f} "
            f"(gpu {st.grad_norm.item():.4f}, {e_norm:.1e})")
        assert e_loss < OUT_TOL and e_norm < 3e-2
        losses.append(loss)
    assert abs(losses[1] - losses[0]) / losses[0] > 10 * OUT_TOL, "the step moved the loss"
    # Against the all-oracle chain the moments (linear in the gradients) meet
    # the gradient tolerance.  The weights are not compared that way: Adam's
    # normalised step moves a weight by about +-lr whatever its gradient's
    # size, so a weight whose gradient lies below the bf16 gradient noise may
    # move the other way.  Fed the GPU's own gradients, the optimizer oracle
    # gives the weights to fp32 rounding.
    e_m, e_v = fro_rel(f64(st.m), m_ref), fro_rel(f64(st.v), v_ref)
    e_own = max_rel(f64(st.master), p_own)
    e_mown = max_rel(f64(st.m), m_own)
    say(f"  after two steps: m {e_m:.1e}, v {e_v:.1e} (all-oracle chain); master {e_own:.1e}, m {e_mown:.1e} "
        f"(optimizer oracle on the GPU's gradients)")
    assert e_m < 3e-2 and e_v < 3e-2
    assert e_own < 1e-5 and e_mown < 1e-5
    assert torch.equal(st.w_arena, st.master.to(torch.bfloat16))
