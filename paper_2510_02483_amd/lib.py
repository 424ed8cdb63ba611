"""Python binding of the C ABI in include/ls.h (ctypes; argument marshalling only).

Every compute step runs in the HIP kernels of libls.so.  torch is used for
device memory and the current stream.  If libls.so has not been built this
module raises on first use; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

from .configs import BlockConfig, StackConfig

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libls.so")

STATUS = {0: "LS_OK", 1: "LS_ERR_NULL", 2: "LS_ERR_SHAPE", 3: "LS_ERR_UNSUPPORTED", 4: "LS_ERR_ALIGN",
          5: "LS_ERR_ALIAS", 6: "LS_ERR_WORKSPACE", 7: "LS_ERR_HIP"}
WEIGHTS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wg", "wu", "wd")


class LsError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: {STATUS.get(status, status)}: {detail}")
        self.status = status


class LsBlockCfg(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("seq", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("intermediate", ctypes.c_int32), ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float)]


class LsBlockWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in WEIGHTS]


class LsBlockGrads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in WEIGHTS]


class LsSizes(ctypes.Structure):
    _fields_ = [("attn_saved", ctypes.c_size_t), ("mlp_saved", ctypes.c_size_t),
                ("attn_workspace", ctypes.c_size_t), ("mlp_workspace", ctypes.c_size_t),
                ("block_workspace", ctypes.c_size_t)]


class LsStackCfg(ctypes.Structure):
    _fields_ = [("block", LsBlockCfg), ("n_layers", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("recompute", ctypes.c_int32), ("logits_chunk", ctypes.c_int32)]


class LsStackWeights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("layers", ctypes.POINTER(LsBlockWeights))]


class LsStackGrads(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("layers", ctypes.POINTER(LsBlockGrads))]


class LsAdamwCfg(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("weight_decay", ctypes.c_float), ("max_norm", ctypes.c_float), ("step", ctypes.c_int32)]


_lib = None
_P = ctypes.c_void_p
_PROTOS = {
    "ls_version": (ctypes.c_int, []),
    "ls_last_error": (ctypes.c_char_p, []),
    "ls_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "ls_query_sizes": (ctypes.c_int, [_P, _P]),
    "ls_attn_fwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "ls_attn_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, ctypes.c_int, _P, ctypes.c_size_t, _P]),
    "ls_mlp_fwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "ls_mlp_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, ctypes.c_int, _P, ctypes.c_size_t, _P]),
    "ls_block_fwd_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, ctypes.c_int, _P, ctypes.c_size_t, _P]),
    "ls_attn_core_fwd": (ctypes.c_int, [_P, _P, _P, _P, _P]),
    "ls_attn_core_bwd_workspace": (ctypes.c_size_t, [_P]),
    "ls_attn_core_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "ls_attn_core_bwd_noalloc": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P]),
    "ls_rmsnorm_fwd": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int32, ctypes.c_float, _P, _P, _P, _P, _P]),
    "ls_rmsnorm_bwd_workspace": (ctypes.c_size_t, [ctypes.c_int64, ctypes.c_int32]),
    "ls_rmsnorm_bwd": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P, ctypes.c_int, _P,
                                      ctypes.c_size_t, _P]),
    "ls_gemm_nt": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, _P, _P, _P, _P]),
    "ls_gemm_nn": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, _P, _P, _P, _P]),
    "ls_gemm_tn": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, _P, _P, _P, ctypes.c_int, _P]),
    "ls_gemm_tile_override": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32]),
    "ls_stack_workspace": (ctypes.c_int, [_P, _P]),
    "ls_stack_fwd_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, ctypes.c_int, _P, ctypes.c_size_t, _P]),
    "ls_cross_entropy_workspace": (ctypes.c_size_t, [ctypes.c_int64]),
    "ls_cross_entropy": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _P, _P, _P, _P, _P, _P,
                                        ctypes.c_size_t, _P]),
    "ls_embed_fwd": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _P, _P, _P, _P]),
    "ls_embed_bwd": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _P, _P, _P, _P]),
    "ls_adamw_workspace": (ctypes.c_size_t, []),
    "ls_adamw_step": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int64, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t,
                                     _P]),
    "ls_timing_begin": (ctypes.c_int, [ctypes.c_char_p, ctypes.c_int]),
    "ls_timing_end": (ctypes.c_int, [_P, _P]),
}
EXPORTS = tuple(_PROTOS)


def lib():
    """Load libls.so (after torch, so that both share one HIP runtime)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2510_02483_amd.build`")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _PROTOS.items():
            f = getattr(l, name)
            f.restype = res
            f.argtypes = args
        _lib = l
    return _lib


def _check(status: int, where: str):
    if status != 0:
        raise LsError(status, where, lib().ls_last_error().decode())


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def make_cfg(c: BlockConfig) -> LsBlockCfg:
    return LsBlockCfg(c.batch, c.seq, c.hidden, c.n_q_heads, c.n_kv_heads, c.head_dim, c.intermediate,
                      c.rope_theta, c.rms_eps)


def make_weights(w: dict) -> LsBlockWeights:
    return LsBlockWeights(*[w[n].data_ptr() if w.get(n) is not None else None for n in WEIGHTS])


def make_grads(g: dict) -> LsBlockGrads:
    return LsBlockGrads(*[g[n].data_ptr() if g.get(n) is not None else None for n in WEIGHTS])


# ---- the ABI calls, same names ----------------------------------------------------

def ls_version() -> int:
    return lib().ls_version()


def ls_query_sizes(c: BlockConfig) -> dict:
    s = LsSizes()
    cfg = make_cfg(c)
    _check(lib().ls_query_sizes(ctypes.byref(cfg), ctypes.byref(s)), "ls_query_sizes")
    return {n: getattr(s, n) for n, _ in LsSizes._fields_}


def ls_attn_fwd(c, x, w, x2, attn_saved, workspace, stream=None):
    cfg, wt = make_cfg(c), make_weights(w)
    _check(lib().ls_attn_fwd(ctypes.byref(cfg), _p(x), ctypes.byref(wt), _p(x2), _p(attn_saved), _p(workspace),
                             workspace.numel() * workspace.element_size(), _stream(stream)), "ls_attn_fwd")


def ls_attn_bwd(c, x, w, attn_saved, dx2, dx, grads, accumulate, workspace, stream=None):
    cfg, wt, gr = make_cfg(c), make_weights(w), make_grads(grads)
    _check(lib().ls_attn_bwd(ctypes.byref(cfg), _p(x), ctypes.byref(wt), _p(attn_saved), _p(dx2), _p(dx),
                             ctypes.byref(gr), int(accumulate), _p(workspace),
                             workspace.numel() * workspace.element_size(), _stream(stream)), "ls_attn_bwd")


def ls_mlp_fwd(c, x2, w, y, mlp_saved, workspace=None, stream=None):
    cfg, wt = make_cfg(c), make_weights(w)
    nb = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().ls_mlp_fwd(ctypes.byref(cfg), _p(x2), ctypes.byref(wt), _p(y), _p(mlp_saved), _p(workspace), nb,
                            _stream(stream)), "ls_mlp_fwd")


def ls_mlp_bwd(c, x2, w, mlp_saved, dy, dx2, grads, accumulate, workspace, stream=None):
    cfg, wt, gr = make_cfg(c), make_weights(w), make_grads(grads)
    _check(lib().ls_mlp_bwd(ctypes.byref(cfg), _p(x2), ctypes.byref(wt), _p(mlp_saved), _p(dy), _p(dx2),
                            ctypes.byref(gr), int(accumulate), _p(workspace),
                            workspace.numel() * workspace.element_size(), _stream(stream)), "ls_mlp_bwd")


def ls_block_fwd_bwd(c, x, w, dy, y, dx, grads, accumulate, workspace, stream=None):
    cfg, wt, gr = make_cfg(c), make_weights(w), make_grads(grads)
    _check(lib().ls_block_fwd_bwd(ctypes.byref(cfg), _p(x), ctypes.byref(wt), _p(dy), _p(y), _p(dx),
                                  ctypes.byref(gr), int(accumulate), _p(workspace),
                                  workspace.numel() * workspace.element_size(), _stream(stream)), "ls_block_fwd_bwd")


def ls_attn_core_fwd(c, qkv, o, lse, stream=None):
    cfg = make_cfg(c)
    _check(lib().ls_attn_core_fwd(ctypes.byref(cfg), _p(qkv), _p(o), _p(lse), _stream(stream)), "ls_attn_core_fwd")


def ls_attn_core_bwd_workspace(c) -> int:
    cfg = make_cfg(c)
    return lib().ls_attn_core_bwd_workspace(ctypes.byref(cfg))


def ls_attn_core_bwd(c, qkv, o, lse, dout, dqkv, workspace, stream=None):
    cfg = make_cfg(c)
    _check(lib().ls_attn_core_bwd(ctypes.byref(cfg), _p(qkv), _p(o), _p(lse), _p(dout), _p(dqkv), _p(workspace),
                                  workspace.numel() * workspace.element_size(), _stream(stream)), "ls_attn_core_bwd")


NOALLOC_SCRATCH_BYTES = 16 << 20  # LS_ATTN_CORE_BWD_NOALLOC_SCRATCH


def ls_attn_core_bwd_noalloc(c, qkv, o, lse, dout, dqkv, stream=None):
    cfg = make_cfg(c)
    _check(lib().ls_attn_core_bwd_noalloc(ctypes.byref(cfg), _p(qkv), _p(o), _p(lse), _p(dout), _p(dqkv),
                                          _stream(stream)), "ls_attn_core_bwd_noalloc")


def ls_rmsnorm_fwd(rows, hidden, eps, x, gamma, h, r, stream=None):
    _check(lib().ls_rmsnorm_fwd(rows, hidden, eps, _p(x), _p(gamma), _p(h), _p(r), _stream(stream)), "ls_rmsnorm_fwd")


def ls_rmsnorm_bwd_workspace(rows, hidden) -> int:
    return lib().ls_rmsnorm_bwd_workspace(rows, hidden)


def ls_rmsnorm_bwd(rows, hidden, x, gamma, r, dh, dres, dx, dgamma, accumulate, workspace, stream=None):
    _check(lib().ls_rmsnorm_bwd(rows, hidden, _p(x), _p(gamma), _p(r), _p(dh), _p(dres), _p(dx), _p(dgamma),
                                int(accumulate), _p(workspace), workspace.numel() * workspace.element_size(),
                                _stream(stream)), "ls_rmsnorm_bwd")


def ls_gemm_nt(A, B, C, stream=None):
    M, K = A.shape
    N = B.shape[0]
    _check(lib().ls_gemm_nt(M, N, K, _p(A), _p(B), _p(C), _stream(stream)), "ls_gemm_nt")


def ls_gemm_nn(A, B, C, stream=None):
    M, K = A.shape
    N = B.shape[1]
    _check(lib().ls_gemm_nn(M, N, K, _p(A), _p(B), _p(C), _stream(stream)), "ls_gemm_nn")


def ls_gemm_tile_override(bm=0, bn=0):
    """Force the matrix-product tile shape (256 or 192 per side); (0, 0) = automatic."""
    _check(lib().ls_gemm_tile_override(int(bm), int(bn)), "ls_gemm_tile_override")


def ls_gemm_tn(A, B, C, accumulate=False, stream=None):
    K, M = A.shape
    N = B.shape[1]
    _check(lib().ls_gemm_tn(M, N, K, _p(A), _p(B), _p(C), int(accumulate), _stream(stream)), "ls_gemm_tn")


def make_stack_cfg(sc: StackConfig) -> LsStackCfg:
    return LsStackCfg(make_cfg(sc.block), sc.n_layers, sc.vocab, int(sc.recompute), int(sc.logits_chunk))


def ls_stack_workspace(sc: StackConfig) -> int:
    cfg = make_stack_cfg(sc)
    n = ctypes.c_size_t(0)
    _check(lib().ls_stack_workspace(ctypes.byref(cfg), ctypes.byref(n)), "ls_stack_workspace")
    return n.value


def ls_stack_fwd_bwd(sc: StackConfig, ids, targets, embed, final_norm, layers, loss, row_loss, d_embed,
                     d_final_norm, d_layers, accumulate, workspace, stream=None):
    """layers / d_layers: lists of per-block weight / gradient dicts (device tensors)."""
    cfg = make_stack_cfg(sc)
    L = sc.n_layers
    lw = (LsBlockWeights * max(L, 1))(*[make_weights(w) for w in layers])
    lg = (LsBlockGrads * max(L, 1))(*[make_grads(g) for g in d_layers])
    w = LsStackWeights(embed.data_ptr(), final_norm.data_ptr(), lw)
    g = LsStackGrads(d_embed.data_ptr(), d_final_norm.data_ptr(), lg)
    _check(lib().ls_stack_fwd_bwd(ctypes.byref(cfg), _p(ids), _p(targets), ctypes.byref(w), _p(loss), _p(row_loss),
                                  ctypes.byref(g), int(accumulate), _p(workspace),
                                  workspace.numel() * workspace.element_size(), _stream(stream)), "ls_stack_fwd_bwd")


def ls_cross_entropy_workspace(tokens: int) -> int:
    return lib().ls_cross_entropy_workspace(int(tokens))


def ls_cross_entropy(logits, seq, ids, targets, loss, row_loss, workspace, stream=None):
    """logits [tokens, vocab] bf16 is overwritten with the gradient of the loss."""
    T, V = logits.shape
    _check(lib().ls_cross_entropy(T, int(seq), V, _p(logits), _p(ids), _p(targets), _p(loss), _p(row_loss),
                                  _p(workspace), workspace.numel() * workspace.element_size(), _stream(stream)),
           "ls_cross_entropy")


def ls_embed_fwd(ids, embed, x, stream=None):
    V, H = embed.shape
    _check(lib().ls_embed_fwd(ids.numel(), H, V, _p(ids), _p(embed), _p(x), _stream(stream)), "ls_embed_fwd")


def ls_embed_bwd(ids, dx, d_embed, stream=None):
    V, H = d_embed.shape
    _check(lib().ls_embed_bwd(ids.numel(), H, V, _p(ids), _p(dx), _p(d_embed), _stream(stream)), "ls_embed_bwd")


def ls_adamw_workspace() -> int:
    return lib().ls_adamw_workspace()


def ls_adamw_step(master, param, grad, m, v, *, step, lr, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.01,
                  max_norm=1.0, n_decay=None, grad_norm=None, workspace=None, stream=None):
    """One clipped AdamW step over flat fp32 tensors (param: bf16 copy or None)."""
    n = master.numel()
    nd = n if n_decay is None else int(n_decay)
    cfg = LsAdamwCfg(lr, beta1, beta2, eps, weight_decay, 0.0 if max_norm is None else max_norm, int(step))
    if workspace is None:
        workspace = torch.empty(ls_adamw_workspace(), dtype=torch.uint8, device=master.device)
    _check(lib().ls_adamw_step(n, nd, ctypes.byref(cfg), _p(master), _p(param), _p(grad), _p(m), _p(v),
                               _p(grad_norm), _p(workspace), workspace.numel() * workspace.element_size(),
                               _stream(stream)), "ls_adamw_step")


def ls_timing_begin(label: str, max_launches: int):
    _check(lib().ls_timing_begin(label.encode(), int(max_launches)), "ls_timing_begin")


def ls_timing_end():
    """Returns (number of recorded launches, mean milliseconds)."""
    n = ctypes.c_int(0)
    ms = ctypes.c_float(0.0)
    _check(lib().ls_timing_end(ctypes.byref(n), ctypes.byref(ms)), "ls_timing_end")
    return n.value, ms.value


# ---- a small harness around ls_block_fwd_bwd ------------------------------------------

class Block:
    """Device buffers for one configuration plus a call of ls_block_fwd_bwd.

    Inputs are bf16 CPU tensors from inputs.make_inputs; they are copied to the
    device once.  Gradients are fp32 device tensors."""

    def __init__(self, c: BlockConfig, host_inputs: dict, device="cuda"):
        self.cfg = c
        dev = torch.device(device)
        self.x = host_inputs["x"].to(dev).reshape(c.tokens, c.hidden).contiguous()
        self.dy = host_inputs["dy"].to(dev).reshape(c.tokens, c.hidden).contiguous()
        self.w = {n: host_inputs[n].to(dev).contiguous() for n in WEIGHTS}
        self.grads = {n: torch.zeros(self.w[n].shape, dtype=torch.float32, device=dev) for n in WEIGHTS}
        self.y = torch.empty_like(self.x)
        self.dx = torch.empty_like(self.x)
        sizes = ls_query_sizes(c)
        self.workspace = torch.empty(sizes["block_workspace"], dtype=torch.uint8, device=dev)

    def step(self, accumulate=False, stream=None):
        ls_block_fwd_bwd(self.cfg, self.x, self.w, self.dy, self.y, self.dx, self.grads, accumulate,
                         self.workspace, stream)


DECAYED = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")
NOT_DECAYED = ("attn_norm", "mlp_norm")


class Stack:
    """Device buffers for one stack configuration plus a call of ls_stack_fwd_bwd
    and an optimizer step.

    ``host`` is the dict of inputs.make_stack_inputs (CPU or device tensors);
    everything is moved to the device once.  All bf16 weights are views into
    one arena and all fp32 gradients into another, in the same order: the
    tensors that take weight decay first (embedding, then each block's seven
    projections), then the RMSNorm gains (final, then each block's two), so
    that one ls_adamw_step call updates the whole model."""

    def __init__(self, sc: StackConfig, host: dict, device="cuda", targets=None):
        self.cfg = sc
        dev = torch.device(device)
        self.ids = host["ids"].to(dev).reshape(-1).contiguous()
        self.targets = None if targets is None else targets.to(dev).reshape(-1).contiguous()
        order = [("embed", None)] + [(n, l) for l in range(sc.n_layers) for n in DECAYED]
        order_nd = [("final_norm", None)] + [(n, l) for l in range(sc.n_layers) for n in NOT_DECAYED]

        def src(name, l):
            return host[name] if l is None else host["layers"][l][name]

        sizes = [src(n, l).numel() for n, l in order + order_nd]
        self.n_params = sum(sizes)
        self.n_decay = sum(sizes[:len(order)])
        self.w_arena = torch.empty(self.n_params, dtype=torch.bfloat16, device=dev)
        self.g_arena = torch.zeros(self.n_params, dtype=torch.float32, device=dev)
        self.layers = [dict() for _ in range(sc.n_layers)]
        self.d_layers = [dict() for _ in range(sc.n_layers)]
        off = 0
        for (name, l), k in zip(order + order_nd, sizes):
            t = src(name, l)
            w = self.w_arena[off:off + k].view(t.shape)
            w.copy_(t.to(dev))
            g = self.g_arena[off:off + k].view(t.shape)
            if l is None:
                setattr(self, name, w)
                setattr(self, "d_" + name, g)
            else:
                self.layers[l][name] = w
                self.d_layers[l][name] = g
            off += k
        self.loss = torch.zeros(1, dtype=torch.float32, device=dev)
        self.row_loss = torch.zeros(sc.tokens, dtype=torch.float32, device=dev)
        self.workspace = torch.empty(ls_stack_workspace(sc), dtype=torch.uint8, device=dev)
        self.master = None

    def step(self, accumulate=False, stream=None):
        ls_stack_fwd_bwd(self.cfg, self.ids, self.targets, self.embed, self.final_norm, self.layers, self.loss,
                         self.row_loss, self.d_embed, self.d_final_norm, self.d_layers, accumulate, self.workspace,
                         stream)

    def init_optimizer(self):
        """fp32 master weights (from the bf16 weights) and zero moments."""
        self.master = self.w_arena.float()
        self.m = torch.zeros_like(self.master)
        self.v = torch.zeros_like(self.master)
        self.grad_norm = torch.zeros(1, dtype=torch.float32, device=self.master.device)
        self.opt_workspace = torch.empty(ls_adamw_workspace(), dtype=torch.uint8, device=self.master.device)
        self.opt_steps = 0

    def optimizer_step(self, lr, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.01, max_norm=1.0, stream=None):
        """Clipped AdamW over the whole model; rewrites the bf16 weights."""
        if self.master is None:
            self.init_optimizer()
        self.opt_steps += 1
        ls_adamw_step(self.master, self.w_arena, self.g_arena, self.m, self.v, step=self.opt_steps, lr=lr,
                      beta1=beta1, beta2=beta2, eps=eps, weight_decay=weight_decay, max_norm=max_norm,
                      n_decay=self.n_decay, grad_norm=self.grad_norm, workspace=self.opt_workspace, stream=stream)
