"""Parity of the model-level path on the GPU: token embedding, softmax
cross-entropy and the whole stack (embedding, blocks, final RMSNorm, tied LM
head, next-token loss) forward + backward through the C ABI, against the fp64
stack oracle on the same seeded bf16 inputs."""
import numpy as np
import pytest
import torch

from oracle import stack as ost
from paper_2510_02483_amd import configs, inputs, lib as L

from gpu_util import GRAD_TOL, OUT_TOL, f64, fro_rel, max_rel, need_gpu, say

pytestmark = pytest.mark.gpu


def _ids(n, V, seed, device="cuda"):
    g = torch.Generator().manual_seed(seed)
    return torch.randint(0, V, (n,), generator=g).to(torch.int32).to(device)


def test_embedding_gather_and_scatter_add():
    need_gpu()
    T, H, V = 300, 264, 50   # ragged rows per wave, ragged 16-byte columns, many repeated ids
    say(f"embedding T={T} H={H} V={V}")
    ids = _ids(T, V, 1)
    ids[7] = V       # out of range: NaN row, skipped by the backward
    ids[11] = -3
    g = torch.Generator().manual_seed(2)
    E = torch.randn(V, H, generator=g).to(torch.bfloat16).cuda()
    x = torch.empty(T, H, dtype=torch.bfloat16, device="cuda")
    L.ls_embed_fwd(ids, E, x)
    dx = torch.randn(T, H, generator=g).to(torch.bfloat16).cuda()
    dE = torch.randn(V, H, generator=g).cuda()
    dE0 = f64(dE)
    L.ls_embed_bwd(ids, dx, dE)
    torch.cuda.synchronize()
    idn = ids.cpu().numpy()
    ok = (idn >= 0) & (idn < V)
    xe = x.cpu()
    assert torch.equal(xe[torch.from_numpy(ok)], E.cpu()[torch.from_numpy(idn[ok]).long()]), "gather is a copy"
    assert torch.isnan(xe[7].float()).all() and torch.isnan(xe[11].float()).all()
    want = dE0.copy()
    np.add.at(want, idn[ok], f64(dx)[ok])
    assert fro_rel(f64(dE), want) < 1e-6, "scatter-add"
    # repeated ids are summed in token order: the same bits on every run
    dE2 = torch.from_numpy(dE0).float().cuda()
    L.ls_embed_bwd(ids, dx, dE2)
    torch.cuda.synchronize()
    assert torch.equal(dE, dE2)


CE_CASES = [  # (tokens, seq, vocab, explicit targets)
    (37 * 4, 37, 1000, False),      # one 16-byte vector per thread, ragged
    (24, 8, 8200, True),
    (16, 16, 128256, False),        # the 3B model's vocabulary: 16 vectors per thread
    (8, 4, 131088, True),           # above the register-resident size: two streaming passes
]


@pytest.mark.parametrize("T,S,V,explicit", CE_CASES, ids=[f"T{c[0]}-V{c[2]}" for c in CE_CASES])
def test_cross_entropy(T, S, V, explicit):
    need_gpu()
    say(f"cross-entropy T={T} S={S} V={V} explicit={explicit}")
    g = torch.Generator().manual_seed(V)
    z = (torch.randn(T, V, generator=g) * 2.0).to(torch.bfloat16)
    ids = _ids(T, V, 3, device="cpu")
    if explicit:
        tg = ids.clone()
        tg[::3] = -1
        tg[1] = V - 1
        tg[2] = 0
    else:
        tg = torch.from_numpy(ost.next_token_targets(ids.numpy().reshape(-1, S)).reshape(-1)).to(torch.int32)
    rows_ref, loss_ref, dz_ref = ost.cross_entropy(z.double().numpy(), tg.numpy().astype(np.int64))
    zd = z.cuda()
    loss = torch.zeros(1, device="cuda")
    rows = torch.zeros(T, device="cuda")
    ws = torch.empty(L.ls_cross_entropy_workspace(T), dtype=torch.uint8, device="cuda")
    L.ls_cross_entropy(zd, S, ids.cuda(), tg.cuda() if explicit else None, loss, rows, ws)
    torch.cuda.synchronize()
    e_rows = max_rel(f64(rows), rows_ref)
    e_loss = abs(loss.item() - loss_ref) / abs(loss_ref)
    e_dz = fro_rel(f64(zd), dz_ref)
    say(f"  row loss {e_rows:.2e}  loss {e_loss:.2e}  dz {e_dz:.2e}")
    assert e_rows < 1e-4 and e_loss < 1e-5, "loss from the same bf16 logits"
    assert e_dz < GRAD_TOL and max_rel(f64(zd), dz_ref) < OUT_TOL
    none = tg.numpy() == -1
    assert np.all(f64(rows)[none] == 0) and np.all(f64(zd)[none] == 0), "rows without a target"


def test_cross_entropy_bad_target_is_nan():
    need_gpu()
    T, V = 6, 1000
    z = torch.randn(T, V).to(torch.bfloat16).cuda()
    ids = _ids(T, V, 4)
    tg = ids.clone()
    tg[2] = V   # outside [-1, V)
    loss = torch.zeros(1, device="cuda")
    rows = torch.zeros(T, device="cuda")
    ws = torch.empty(L.ls_cross_entropy_workspace(T), dtype=torch.uint8, device="cuda")
    L.ls_cross_entropy(z, T, ids, tg, loss, rows, ws)
    torch.cuda.synchronize()
    assert torch.isnan(loss).all() and torch.isnan(rows[2]) and torch.isnan(z[2].float()).all()
    assert torch.isfinite(rows[[0, 1, 3, 4, 5]]).all() and torch.isfinite(z[[0, 1, 3, 4, 5]].float()).all()


# ---- the whole stack ------------------------------------------------------------------------


def oracle_stack(sc, host, targets=None, batch_rows=None):
    """fp64 oracle on float64 copies of the bf16 inputs (optionally on the
    first `batch_rows` = (b, t0) sub-problem: sequence b's first t0 tokens)."""
    ids = host["ids"].numpy().astype(np.int64)
    tg = None if targets is None else targets.numpy().astype(np.int64).reshape(ids.shape)
    if batch_rows is not None:
        b, t0 = batch_rows
        ids = ids[b:b + 1, :t0]
        tg = tg[b:b + 1, :t0]
    E = host["embed"].double().numpy()
    gf = host["final_norm"].double().numpy()
    blocks = [{k: v.double().numpy() for k, v in l.items()} for l in host["layers"]]
    c = sc.block
    return ost.stack_fwd_bwd(ids, E, blocks, gf, n_q_heads=c.n_q_heads, n_kv_heads=c.n_kv_heads,
                             rope_theta=c.rope_theta, eps=c.rms_eps, targets=tg)


def compare_stack(st, ref, rows_sel=None, scale=1.0):
    loss, rows, gr = ref
    # the loss and row losses are values of this step; only gradients accumulate
    errs = {"loss": abs(st.loss.item() - loss) / abs(loss)}
    r = f64(st.row_loss)
    errs["rows"] = max_rel(r if rows_sel is None else r[rows_sel], rows)
    errs["d_embed"] = fro_rel(f64(st.d_embed) / scale, gr["embed"])
    errs["d_final_norm"] = fro_rel(f64(st.d_final_norm) / scale, gr["final_norm"])
    for l, gl in enumerate(gr["blocks"]):
        for n in L.WEIGHTS:
            errs[f"{l}.{n}"] = fro_rel(f64(st.d_layers[l][n]) / scale, gl[n])
    worst = max((v, k) for k, v in errs.items() if k not in ("loss", "rows"))
    say(f"  loss {errs['loss']:.2e} rows {errs['rows']:.2e} d_embed {errs['d_embed']:.2e} "
        f"d_final_norm {errs['d_final_norm']:.2e} worst {worst[1]} {worst[0]:.2e}")
    assert errs["loss"] < OUT_TOL and errs["rows"] < OUT_TOL, errs
    for k, v in errs.items():
        assert v < GRAD_TOL, (k, errs)


@pytest.mark.parametrize("recompute", [True, False], ids=["recompute", "saved"])
def test_stack_tiny(recompute):
    need_gpu()
    sc = configs.TINY_STACK.with_(recompute=recompute)
    say(f"stack {sc}")
    host = inputs.make_stack_inputs(sc, gamma="random", e_std=0.1)
    st = L.Stack(sc, host)
    st.step()
    torch.cuda.synchronize()
    compare_stack(st, oracle_stack(sc, host))
    # accumulate = 1 adds a second copy of every gradient
    st.step(accumulate=True)
    torch.cuda.synchronize()
    compare_stack(st, oracle_stack(sc, host), scale=2.0)


def test_stack_without_blocks():
    """Zero blocks: embedding, final RMSNorm, tied head and loss alone."""
    need_gpu()
    sc = configs.TINY_STACK.with_(n_layers=0)
    say(f"stack {sc}")
    host = inputs.make_stack_inputs(sc, gamma="random", e_std=0.5)
    st = L.Stack(sc, host)
    st.step()
    torch.cuda.synchronize()
    compare_stack(st, oracle_stack(sc, host))


def test_stack_logits_in_chunks():
    """Logits formed 40 token rows at a time (4 chunks, the last one ragged):
    the head's gradient accumulates over the chunks; same results as the
    oracle.  Heads of 104 features (padded slots) in the blocks."""
    need_gpu()
    blk = configs.BlockConfig("stack-d104", 17, batch=2, seq=64, hidden=416, n_q_heads=4, n_kv_heads=4,
                              head_dim=104, intermediate=520, rope_theta=1e4)
    sc = configs.StackConfig("stack-chunks", blk, n_layers=2, vocab=1000, logits_chunk=40)
    say(f"stack {sc}")
    host = inputs.make_stack_inputs(sc, gamma="random", e_std=0.1)
    st = L.Stack(sc, host)
    st.step()
    torch.cuda.synchronize()
    compare_stack(st, oracle_stack(sc, host))


def test_stack_tiny_explicit_targets_and_depth():
    """Explicit targets with ignored rows, three blocks, d = 128 heads."""
    need_gpu()
    blk = configs.BlockConfig("stack-d128", 11, batch=3, seq=40, hidden=384, n_q_heads=6, n_kv_heads=2,
                              head_dim=128, intermediate=520, rope_theta=5e5)
    sc = configs.StackConfig("stack-d128", blk, n_layers=3, vocab=4000)
    say(f"stack {sc}")
    host = inputs.make_stack_inputs(sc, gamma="random", e_std=0.1)
    g = torch.Generator().manual_seed(12)
    tg = torch.randint(0, sc.vocab, (sc.tokens,), generator=g).to(torch.int32)
    tg[::5] = -1
    st = L.Stack(sc, host, targets=tg)
    st.step()
    torch.cuda.synchronize()
    compare_stack(st, oracle_stack(sc, host, targets=tg))


def test_stack_3b_full_size_sequence():
    """The 3B model's shapes (hidden 3072, 24/8 heads, SwiGLU 8192, vocabulary
    128256, micro-batch 4 x 2048) at depth 2, in the launch configuration of
    the full model.  Next-token targets on every position of sequence 1 (all
    2047 of them) and none elsewhere: the loss and every gradient then equal
    those of that one 2048-token sequence (the other sequences get no
    gradient), which the oracle computes in full; the other rows' losses are
    exactly zero.  The same step without recomputation gives the same loss
    and gradients bit for bit."""
    need_gpu()
    sc = configs.STACK_3B.with_(n_layers=2)
    b = 1
    S = sc.block.seq
    t0 = S - 1
    say(f"stack full-size sequence {sc} b={b}")
    host = inputs.make_stack_inputs(sc, e_std=0.1)
    tg = torch.full((sc.block.batch, S), -1, dtype=torch.int32)
    tg[b, :t0] = host["ids"][b, 1:t0 + 1]
    tg = tg.reshape(-1)
    st = L.Stack(sc, host, targets=tg)
    st.step()
    torch.cuda.synchronize()
    say("  gpu done; oracle on the whole sequence")
    ref = oracle_stack(sc, host, targets=tg, batch_rows=(b, S))
    sel = np.zeros(sc.tokens, dtype=bool)
    sel[b * S:(b + 1) * S] = True
    assert np.all(f64(st.row_loss)[~sel] == 0.0)
    compare_stack(st, ref, rows_sel=sel)
    loss1 = st.loss.clone()
    g1 = [{n: t.clone() for n, t in d.items()} for d in st.d_layers]
    dE1 = st.d_embed.clone()
    del st
    st2 = L.Stack(sc.with_(recompute=False), host, targets=tg)
    st2.step()
    torch.cuda.synchronize()
    assert torch.equal(st2.loss, loss1)
    for l in range(sc.n_layers):
        for n in L.WEIGHTS:
            assert torch.equal(st2.d_layers[l][n], g1[l][n]), (l, n)
    assert torch.equal(st2.d_embed, dE1), "the embedding gradient is deterministic too"


def test_stack_paper_3b_full_size_prefix():
    """The report's 3B model shapes (Table 1; vocabulary 32000, micro-batch
    2 x 4096) at depth 2: targets on the first 384 tokens of sequence 0,
    checked against the oracle on that prefix."""
    need_gpu()
    sc = configs.PAPER_3B_STACK.with_(n_layers=2)
    t0, b = 384, 0
    say(f"paper 3b stack full-size prefix {sc} t0={t0}")
    host = inputs.make_stack_inputs(sc, e_std=0.1, gamma="random")
    S = sc.block.seq
    tg = torch.full((sc.block.batch, S), -1, dtype=torch.int32)
    tg[b, :t0] = host["ids"][b, 1:t0 + 1]
    tg = tg.reshape(-1)
    st = L.Stack(sc, host, targets=tg)
    st.step()
    torch.cuda.synchronize()
    ref = oracle_stack(sc, host, targets=tg, batch_rows=(b, t0))
    sel = np.zeros(sc.tokens, dtype=bool)
    sel[b * S:b * S + t0] = True
    assert np.all(f64(st.row_loss)[~sel] == 0.0)
    compare_stack(st, ref, rows_sel=sel)


@pytest.mark.parametrize("case", ["one-token-sequences", "all-ignored"])
def test_stack_without_targets(case):
    """Degenerate batches with no row to predict: sequences of one token (the
    last position has no next token) or every target ignored.  The loss is 0
    (mean over an empty set taken as 0, as the oracle does) and every
    gradient is exactly zero."""
    need_gpu()
    if case == "one-token-sequences":
        sc = configs.TINY_STACK.with_(block=configs.TINY_STACK.block.with_(batch=3, seq=1))
        tg = None
    else:
        sc = configs.TINY_STACK
        tg = torch.full((sc.tokens,), -1, dtype=torch.int32)
    say(f"stack without targets: {case} {sc}")
    host = inputs.make_stack_inputs(sc, e_std=0.1, gamma="random")
    st = L.Stack(sc, host, targets=tg)
    st.g_arena.fill_(1.0)   # overwritten (accumulate = 0) with exact zeros
    st.step()
    torch.cuda.synchronize()
    ref_loss, ref_rows, _ = oracle_stack(sc, host, targets=tg)
    assert ref_loss == 0.0 and np.all(ref_rows == 0.0)
    assert st.loss.item() == 0.0 and torch.count_nonzero(st.row_loss).item() == 0
    assert torch.count_nonzero(st.g_arena).item() == 0


def test_cross_entropy_smallest_vocabulary():
    """One row of an 8-entry vocabulary (one 16-byte vector: a single lane holds the row)."""
    need_gpu()
    z = torch.tensor([[0.5, -1.0, 3.0, 0.0, 2.0, -2.5, 1.0, 0.25]]).to(torch.bfloat16)
    tg = torch.tensor([4], dtype=torch.int32)
    rows_ref, loss_ref, dz_ref = ost.cross_entropy(z.double().numpy(), tg.numpy().astype(np.int64))
    zd = z.cuda()
    loss = torch.zeros(1, device="cuda")
    rows = torch.zeros(1, device="cuda")
    ws = torch.empty(L.ls_cross_entropy_workspace(1), dtype=torch.uint8, device="cuda")
    L.ls_cross_entropy(zd, 1, tg.cuda(), tg.cuda(), loss, rows, ws)
    torch.cuda.synchronize()
    assert abs(loss.item() - loss_ref) < 1e-5 * loss_ref
    assert max_rel(f64(zd), dz_ref) < OUT_TOL
