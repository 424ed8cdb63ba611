"""The library's calls under HIP graph capture and a short training run.

Capture: every call only enqueues kernels on the caller's stream (no
allocation, no host synchronisation, no memset nodes), so a block step and a
whole model step can be captured once and replayed.  Each replay, with eager
work and synchronisations between replays, must give the eager results bit
for bit (every kernel is deterministic).

Training: forward, backward and the optimizer step chained over many steps on
one fixed batch must drive the loss down (the model memorises the batch)."""
import pytest
import torch

from paper_2510_02483_amd import configs, inputs, lib as L

from gpu_util import LONG_NARROW, need_gpu, say

pytestmark = pytest.mark.gpu


def _capture(step):
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()                      # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    return g


@pytest.mark.parametrize("c", [configs.TINY.with_(batch=2, seq=200), LONG_NARROW], ids=["tiny", "split-k"])
def test_block_step_graph_replay(c):
    need_gpu()
    say(f"graph capture {c}")
    blk = L.Block(c, inputs.make_inputs(c, gamma="random"))
    blk.step()
    torch.cuda.synchronize()
    want = {"y": blk.y.clone(), "dx": blk.dx.clone(), **{n: blk.grads[n].clone() for n in L.WEIGHTS}}
    g = _capture(lambda: blk.step())
    for rep in range(3):
        for t in [blk.y, blk.dx, *blk.grads.values()]:
            t.fill_(float("nan") if t.dtype == torch.float32 else 0.0)   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = {"y": blk.y, "dx": blk.dx, **blk.grads}
        for k, v in want.items():
            assert torch.equal(got[k], v), (rep, k)


def test_stack_step_graph_replay():
    need_gpu()
    sc = configs.TINY_STACK
    say(f"graph capture {sc}")
    st = L.Stack(sc, inputs.make_stack_inputs(sc, gamma="random", e_std=0.1))
    st.step()
    torch.cuda.synchronize()
    loss, grads = st.loss.clone(), st.g_arena.clone()
    g = _capture(lambda: st.step())
    for rep in range(3):
        st.g_arena.fill_(float("nan"))
        st.loss.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(st.loss, loss) and torch.equal(st.g_arena, grads), rep


def test_training_memorises_a_batch():
    need_gpu()
    sc = configs.TINY_STACK
    say(f"training {sc}")
    st = L.Stack(sc, inputs.make_stack_inputs(sc, gamma="random", e_std=0.1))
    losses = []
    for step in range(40):
        st.step()
        st.optimizer_step(lr=3e-3, weight_decay=0.0)
        losses.append(st.loss.item())
    say("  loss: " + " ".join(f"{v:.3f}" for v in losses[::5]) + f" ... {losses[-1]:.3f}")
    assert all(torch.isfinite(torch.tensor(losses)))
    assert losses[-1] < 0.25 * losses[0], "a fixed batch is memorised"
