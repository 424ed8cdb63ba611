/*
 * ls.h -- C ABI of the decoder-block library for AMD Instinct MI355X (gfx950).
 *
 * The library computes the forward and backward pass of one Llama-style
 * decoder block, the part of a transformer whose attention and MLP layers the
 * Litespark report (arXiv 2510.02483) speeds up (Section 1) while keeping the
 * standard block's result (abstract, Section 5).  Around it: the whole model's
 * forward and backward pass (token embedding, a stack of blocks, final
 * RMSNorm, tied LM head, next-token cross-entropy) and the optimizer step
 * (global-norm clipping and AdamW) of the report's training setup.  The block is the one the
 * report's Section 2.4 describes: pre-norm RMSNorm, rotary position embedding,
 * causal grouped-query attention (multi-head when kv heads = query heads) and
 * a SwiGLU MLP, with residual adds:
 *
 *   x2 = x  + Wo . Attn(RoPE(Wq h1), RoPE(Wk h1), Wv h1),   h1 = RMSNorm(x;  g1)
 *   y  = x2 + Wd . (silu(Wg h2) * (Wu h2)),                 h2 = RMSNorm(x2; g2)
 *
 * Conventions shared by every call
 *   - Element types: activations, weights and upstream gradients are bf16
 *     (raw bits in ls_bf16, round-to-nearest-even); all matrix products
 *     accumulate in fp32; weight and RMSNorm-gain gradients are fp32
 *     accumulators.
 *   - Layouts: activations are row-major [batch * seq, features] (token-major);
 *     projection weights are row-major [out_features, in_features]; RMSNorm
 *     gains are [hidden].  q/k/v heads are contiguous blocks of head_dim
 *     columns; query head h reads kv head h / (n_q_heads / n_kv_heads).
 *   - RoPE: pairs (i, i + head_dim/2) of each head turn by p * theta^(-2i/d)
 *     radians, p = 0..seq-1 restarting for every sequence.  Mask: causal,
 *     key j <= query i.  Softmax scale 1/sqrt(head_dim).  LSE in natural log.
 *   - Pointers: every pointer argument is device memory owned by the caller,
 *     16-byte aligned, dense (no strides).  The library keeps no reference to
 *     any of them after a call returns and allocates no device memory in any
 *     call below; scratch space comes from the caller's workspace.
 *   - Streams: `stream` is a hipStream_t (NULL = the null stream).  Calls only
 *     enqueue work and return; device faults surface at the caller's next
 *     synchronisation.  No host synchronisation happens inside a call.
 *   - Errors: every call returns an ls_status.  Argument checks (null
 *     pointers, shapes, alignment, aliasing, workspace size) all run before
 *     any HIP call, so they behave identically on a host without a GPU.
 *     ls_last_error() returns a thread-local description of the last failure.
 *     No C++ exception crosses this interface.
 *   - Gradient accumulation: `accumulate` = 0 overwrites the fp32 gradient
 *     buffers, 1 adds into them.
 *   - Calls that overlap on one stream are ordered; the library holds no
 *     device state between calls, so calls on different streams with
 *     disjoint buffers may run concurrently.
 */
#ifndef LS_H_
#define LS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t ls_bf16;

typedef enum {
  LS_OK = 0,
  LS_ERR_NULL = 1,        /* a required pointer is NULL */
  LS_ERR_SHAPE = 2,       /* a size is non-positive, inconsistent or not a multiple of 8 */
  LS_ERR_UNSUPPORTED = 3, /* valid but not implemented (e.g. a head_dim below 64 or above 128) */
  LS_ERR_ALIGN = 4,       /* a pointer is not 16-byte aligned */
  LS_ERR_ALIAS = 5,       /* an output buffer overlaps an input or another output */
  LS_ERR_WORKSPACE = 6,   /* workspace or saved-state buffer too small */
  LS_ERR_HIP = 7          /* the HIP runtime reported an error (see ls_last_error) */
} ls_status;

/* Shape of one decoder block.  Requirements: all sizes > 0; n_q_heads is a
 * multiple of n_kv_heads; head_dim is 64, or a multiple of 8 from 72 to 128
 * (sizes other than 64 and 128, such as the 104 of a 64-head 6656-wide model,
 * run in 128-wide slots: each head's two RoPE halves are placed at slot
 * offsets 0 and 64 with zero features between, which changes no result);
 * hidden and intermediate are multiples of 8; rms_eps >= 0, rope_theta > 1.
 * hidden need not equal n_q_heads*head_dim: the query/output projections map
 * hidden <-> n_q_heads*head_dim features either way (e.g. hidden 384 with
 * 4 heads of 64 or 6 heads of 128). */
typedef struct {
  int32_t batch;
  int32_t seq;
  int32_t hidden;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t intermediate;
  float rope_theta;
  float rms_eps;
} ls_block_cfg;

/* bf16 weights, nn.Linear layout [out, in]:
 *   wq [n_q_heads*head_dim, hidden], wk and wv [n_kv_heads*head_dim, hidden],
 *   wo [hidden, n_q_heads*head_dim], wg and wu [intermediate, hidden],
 *   wd [hidden, intermediate], attn_norm and mlp_norm [hidden]. */
typedef struct {
  const ls_bf16 *attn_norm, *wq, *wk, *wv, *wo, *mlp_norm, *wg, *wu, *wd;
} ls_block_weights;

/* fp32 gradient accumulators with the shapes of ls_block_weights. */
typedef struct {
  float *attn_norm, *wq, *wk, *wv, *wo, *mlp_norm, *wg, *wu, *wd;
} ls_block_grads;

/* Byte sizes for one configuration (each rounded up to 256 bytes). */
typedef struct {
  size_t attn_saved;     /* written by ls_attn_fwd, read by ls_attn_bwd */
  size_t mlp_saved;      /* written by ls_mlp_fwd, read by ls_mlp_bwd */
  size_t attn_workspace; /* scratch for ls_attn_fwd and ls_attn_bwd */
  size_t mlp_workspace;  /* scratch for ls_mlp_fwd and ls_mlp_bwd */
  size_t block_workspace;/* scratch for ls_block_fwd_bwd (includes both saved states) */
} ls_sizes;

/* Fill *out with the buffer sizes the calls below need for *cfg. */
int ls_query_sizes(const ls_block_cfg* cfg, ls_sizes* out);

/* Attention sub-layer forward (Section 2.4: RMSNorm, RoPE, causal GQA):
 *   x2 = x + o Wo^T,  o = causal-softmax(q k^T / sqrt(d)) v,
 *   q, k = RoPE(h1 Wq^T), RoPE(h1 Wk^T), v = h1 Wv^T, h1 = RMSNorm(x; attn_norm).
 * x, x2: [batch*seq, hidden] bf16.  attn_saved: opaque, attn_saved bytes
 * (holds h1, rotated q/k, v, o, the RMSNorm scales and the softmax log-sum-exp).
 * x2 must not overlap x or attn_saved. */
int ls_attn_fwd(const ls_block_cfg* cfg, const ls_bf16* x, const ls_block_weights* w,
                ls_bf16* x2, void* attn_saved, void* workspace, size_t workspace_bytes,
                void* stream);

/* Attention sub-layer backward (Section 1: the backward pass of the attention
 * layer is one of the operations the report's algorithmic step optimises;
 * Section 2.4 names the layer).  Given dx2 = dL/dx2, writes dx = dL/dx =
 * dx2 + (d/dx of the attention branch)^T dx2 and the gradients of attn_norm,
 * wq, wk, wv, wo (other members of *g are ignored and may be NULL).  The
 * backward recomputes the softmax from the saved log-sum-exp.  x and
 * attn_saved must be the ones ls_attn_fwd saw. */
int ls_attn_bwd(const ls_block_cfg* cfg, const ls_bf16* x, const ls_block_weights* w,
                const void* attn_saved, const ls_bf16* dx2, ls_bf16* dx,
                const ls_block_grads* g, int accumulate, void* workspace,
                size_t workspace_bytes, void* stream);

/* MLP sub-layer forward (Section 2.4: RMSNorm, SwiGLU):
 *   y = x2 + (silu(h2 Wg^T) * (h2 Wu^T)) Wd^T,  h2 = RMSNorm(x2; mlp_norm).
 * mlp_saved: opaque, mlp_saved bytes (h2, gate and up outputs, their product,
 * the RMSNorm scales). */
int ls_mlp_fwd(const ls_block_cfg* cfg, const ls_bf16* x2, const ls_block_weights* w,
               ls_bf16* y, void* mlp_saved, void* workspace, size_t workspace_bytes,
               void* stream);

/* MLP sub-layer backward (Section 1: the backward pass of the MLP layer is one
 * of the operations the report's algorithmic step optimises; Section 2.4 names
 * the layer): dx2 = dy + (d/dx2 of the MLP branch)^T dy and the gradients of
 * mlp_norm, wg, wu, wd. */
int ls_mlp_bwd(const ls_block_cfg* cfg, const ls_bf16* x2, const ls_block_weights* w,
               const void* mlp_saved, const ls_bf16* dy, ls_bf16* dx2,
               const ls_block_grads* g, int accumulate, void* workspace,
               size_t workspace_bytes, void* stream);

/* Whole block, forward then backward, in one call (Section 1: the forward and
 * backward pass operations of the attention and MLP layers; Section 2.4: the
 * block): writes y, dx and all nine weight gradients for upstream gradient dy.
 * workspace: block_workspace bytes. */
int ls_block_fwd_bwd(const ls_block_cfg* cfg, const ls_bf16* x, const ls_block_weights* w,
                     const ls_bf16* dy, ls_bf16* y, ls_bf16* dx, const ls_block_grads* g,
                     int accumulate, void* workspace, size_t workspace_bytes, void* stream);

/* ---- a stack of blocks with a tied embedding and the language-model loss ----
 *
 * The models the report trains (Section 2.4; Table 1) put a stack of these
 * blocks between a token embedding and a final RMSNorm plus LM head, and train
 * them on the next-token cross-entropy.  With the LM head tied to the embedding
 * matrix E [vocab, hidden]:
 *
 *   x_0 = E[ids];  x_{l+1} = block_l(x_l);  h = RMSNorm(x_L; final_norm);
 *   z = h E^T;  loss = (1/N) sum over rows t with target[t] >= 0 of
 *                      (ln sum_v exp z[t, v]) - z[t, target[t]],
 *
 * N = number of such rows (loss = 0 when N = 0).  Without explicit targets,
 * target[b, s] = ids[b, s+1] and the last position of each sequence has none.
 * The backward pass writes the gradients of E (head part plus embedding
 * part, summed), of final_norm and of every block's weights. */
typedef struct {
  ls_block_cfg block; /* shape of each block; block.batch x block.seq tokens */
  int32_t n_layers;   /* number of blocks, 0 .. 4096 */
  int32_t vocab;      /* vocabulary size, a positive multiple of 8; vocab*hidden*4 < 2047 MiB */
  int32_t recompute;  /* 1: keep only each block's input in the forward pass and
                         recompute the block's saved state in the backward pass;
                         0: keep every block's saved state (more workspace) */
  int32_t logits_chunk; /* token rows whose logits are formed at a time: 0 = as
                           many as stay below 2047 MiB of bf16 logits; a smaller
                           positive value trades workspace for more launches */
} ls_stack_cfg;

/* embed [vocab, hidden] bf16 (input embedding and LM head); final_norm
 * [hidden] bf16; layers: HOST array of n_layers ls_block_weights (each holding
 * device pointers).  Weights of different layers may alias. */
typedef struct {
  const ls_bf16* embed;
  const ls_bf16* final_norm;
  const ls_block_weights* layers;
} ls_stack_weights;

/* fp32 gradient accumulators: embed [vocab, hidden], final_norm [hidden],
 * layers: HOST array of n_layers ls_block_grads.  None may overlap another. */
typedef struct {
  float* embed;
  float* final_norm;
  const ls_block_grads* layers;
} ls_stack_grads;

/* Workspace bytes ls_stack_fwd_bwd needs for *cfg. */
int ls_stack_workspace(const ls_stack_cfg* cfg, size_t* bytes);

/* Forward and backward pass of the whole model for one micro-batch.
 * ids: [batch*seq] int32 token ids (device).  targets: NULL (next-token
 * targets from ids) or [batch*seq] int32, -1 = no target.  loss: one fp32
 * (device).  row_loss: NULL or [batch*seq] fp32, each row's loss (0 without a
 * target).  Errors reported through the result rather than the status (the
 * library never reads ids on the host): an id outside [0, vocab) makes its
 * embedding row NaN, and a target outside [-1, vocab) makes its row's loss
 * and gradient NaN; neither reads or writes outside any buffer.  Every
 * output is deterministic (the embedding gradient sums repeated tokens in
 * token order). */
int ls_stack_fwd_bwd(const ls_stack_cfg* cfg, const int32_t* ids, const int32_t* targets,
                     const ls_stack_weights* w, float* loss, float* row_loss,
                     const ls_stack_grads* g, int accumulate, void* workspace,
                     size_t workspace_bytes, void* stream);

/* ---- optimizer step ------------------------------------------------------------
 *
 * The report trains with AdamW (beta1 0.9, beta2 0.95, weight decay 0.01) and
 * gradient clipping at global norm 1.0 (Section 2.5, optimizer settings, and Table
 * 2).  One step over
 * n parameters held in flat fp32 arrays (callers lay every tensor out in one
 * arena; the first n_decay parameters take weight decay, the rest -- RMSNorm
 * gains -- do not):
 *
 *   norm = ||grad||_2 over all n;  c = min(1, max_norm / (norm + 1e-6))
 *   m = beta1 m + (1 - beta1) c grad;  v = beta2 v + (1 - beta2) (c grad)^2
 *   master = master (1 - lr wd [i < n_decay]) - (lr / (1 - beta1^step)) m / (sqrt(v / (1 - beta2^step)) + eps)
 *   param  = bf16(master)  (round to nearest even; skipped when param is NULL)
 *
 * grad is read only; grad_norm (NULL allowed) receives the norm before
 * clipping.  The norm is summed in fp64 in a fixed order (deterministic).
 * Every array: device memory, 16-byte aligned, no overlaps. */
typedef struct {
  float lr;
  float beta1, beta2;  /* in [0, 1) */
  float eps;           /* > 0 */
  float weight_decay;  /* >= 0, lr * weight_decay < 1 */
  float max_norm;      /* <= 0: no clipping */
  int32_t step;        /* 1-based step count t */
} ls_adamw_cfg;

/* Workspace bytes of ls_adamw_step (independent of n). */
size_t ls_adamw_workspace(void);
int ls_adamw_step(int64_t n, int64_t n_decay, const ls_adamw_cfg* cfg, float* master,
                  ls_bf16* param, const float* grad, float* m, float* v, float* grad_norm,
                  void* workspace, size_t workspace_bytes, void* stream);

/* ---- single-kernel entry points (used for per-kernel parity) ---------------- */

/* Causal attention core on a packed projection buffer.
 * qkv: [batch*seq, (n_q_heads + 2*n_kv_heads)*head_dim] bf16, row = token,
 * columns = q heads, then k heads, then v heads (q and k already rotated).
 * o: [batch*seq, n_q_heads*head_dim] bf16.  lse: [batch, n_q_heads, seq] fp32.
 * Only batch, seq, n_q_heads, n_kv_heads, head_dim of *cfg are used; head_dim
 * must be 64 or 128 here (LS_ERR_UNSUPPORTED otherwise). */
int ls_attn_core_fwd(const ls_block_cfg* cfg, const ls_bf16* qkv, ls_bf16* o, float* lse,
                     void* stream);

/* Backward of ls_attn_core_fwd: dqkv (same layout as qkv) from do, o, lse.
 * The result holds gradients with respect to the rotated q and k (no inverse
 * rotation).  workspace: at least ls_attn_core_bwd_workspace(cfg) bytes. */
size_t ls_attn_core_bwd_workspace(const ls_block_cfg* cfg);
int ls_attn_core_bwd(const ls_block_cfg* cfg, const ls_bf16* qkv, const ls_bf16* o,
                     const float* lse, const ls_bf16* dout, ls_bf16* dqkv, void* workspace,
                     size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * computation and kernels as ls_attn_core_bwd, bit for bit, without a
 * workspace argument.  Its scratch is a device array the library owns,
 * LS_ATTN_CORE_BWD_NOALLOC_SCRATCH bytes on every GPU the library runs on,
 * held until the process ends.  The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine).  A shape whose workspace
 * (ls_attn_core_bwd_workspace) exceeds the array fails with
 * LS_ERR_WORKSPACE before any HIP call.  Every call on a GPU shares that GPU's
 * array (it runs on the current device): calls that overlap on one GPU, on
 * different streams or from different threads, race and give wrong results;
 * calls ordered on one stream are safe.  The first call on a device looks the
 * array's device address up (hipGetSymbolAddress); errors there return
 * LS_ERR_HIP. */
#define LS_ATTN_CORE_BWD_NOALLOC_SCRATCH ((size_t)16 << 20)
int ls_attn_core_bwd_noalloc(const ls_block_cfg* cfg, const ls_bf16* qkv, const ls_bf16* o,
                             const float* lse, const ls_bf16* dout, ls_bf16* dqkv, void* stream);

/* RMSNorm over rows of length `hidden`: h = x * r * gamma, r = (mean x^2 + eps)^-1/2.
 * x, h: [rows, hidden] bf16; r: [rows] fp32. */
int ls_rmsnorm_fwd(int64_t rows, int32_t hidden, float eps, const ls_bf16* x,
                   const ls_bf16* gamma, ls_bf16* h, float* r, void* stream);

/* RMSNorm backward plus residual: dx = dres + r*(gamma*dh) - x*r^3*<gamma*dh, x>/hidden,
 * dgamma (+)= sum over rows of dh * x * r.  dres may be NULL (treated as zero).
 * workspace: at least ls_rmsnorm_bwd_workspace(rows, hidden) bytes. */
size_t ls_rmsnorm_bwd_workspace(int64_t rows, int32_t hidden);
int ls_rmsnorm_bwd(int64_t rows, int32_t hidden, const ls_bf16* x, const ls_bf16* gamma,
                   const float* r, const ls_bf16* dh, const ls_bf16* dres, ls_bf16* dx,
                   float* dgamma, int accumulate, void* workspace, size_t workspace_bytes,
                   void* stream);

/* Dense bf16 matrix products with fp32 accumulation (row-major operands):
 *   ls_gemm_nt:  C[M,N]  = A[M,K] . B[N,K]^T          (forward projection)
 *   ls_gemm_nn:  C[M,N]  = A[M,K] . B[K,N]            (input gradient)
 *   ls_gemm_tn:  C[M,N] (+)= A[K,M]^T . B[K,N], fp32  (weight gradient)
 * M, N, K > 0 and multiples of 8.  These single products take no workspace, so
 * ls_gemm_tn never splits K over workgroups (the block and stack calls do, for
 * weight gradients with few output tiles, in their workspace). */
int ls_gemm_nt(int64_t M, int64_t N, int64_t K, const ls_bf16* A, const ls_bf16* B,
               ls_bf16* C, void* stream);
int ls_gemm_nn(int64_t M, int64_t N, int64_t K, const ls_bf16* A, const ls_bf16* B,
               ls_bf16* C, void* stream);
int ls_gemm_tn(int64_t M, int64_t N, int64_t K, const ls_bf16* A, const ls_bf16* B,
               float* C, int accumulate, void* stream);

/* Softmax cross-entropy over rows of bf16 logits [tokens, vocab], in place:
 * row_loss[t] = ln sum_v exp z[t,v] - z[t, target[t]] (0 when target[t] = -1),
 * loss = sum(row_loss) / max(N, 1), and logits are overwritten with the
 * gradient of loss, (softmax(z[t]) - onehot(target[t])) / max(N, 1) (zero rows
 * without a target).  targets: NULL (next token of ids within sequences of
 * `seq` tokens; tokens must be a multiple of seq) or [tokens] int32.  A target
 * outside [-1, vocab) makes its row NaN.  workspace: at least
 * ls_cross_entropy_workspace(tokens) bytes. */
size_t ls_cross_entropy_workspace(int64_t tokens);
int ls_cross_entropy(int64_t tokens, int32_t seq, int32_t vocab, ls_bf16* logits,
                     const int32_t* ids, const int32_t* targets, float* loss, float* row_loss,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Token embedding rows: x[t] = embed[ids[t]] ([tokens, hidden] bf16; an id
 * outside [0, vocab) gives a NaN row), and its backward, which ADDS dx[t] into
 * d_embed[ids[t]] (fp32; the rows of repeated ids summed in token order, so
 * the result is deterministic; ids outside [0, vocab) skipped; hidden at most
 * 8192 for the backward). */
int ls_embed_fwd(int64_t tokens, int32_t hidden, int32_t vocab, const int32_t* ids,
                 const ls_bf16* embed, ls_bf16* x, void* stream);
int ls_embed_bwd(int64_t tokens, int32_t hidden, int32_t vocab, const int32_t* ids,
                 const ls_bf16* dx, float* d_embed, void* stream);

/* Tile shape of the matrix products (tuning and testing).  By default every
 * product launch picks its workgroup tile (256 or 192 rows x 256 or 192
 * columns, where its epilogue allows) to minimise waves of workgroups times
 * tile area on the device's compute units.  ls_gemm_tile_override(bm, bn)
 * forces bm x bn (each 256 or 192) for every later launch in the process that
 * allows it (others, and weight gradients that split K, keep 256 x 256);
 * (0, 0) restores the automatic choice.
 * Process-wide setting, not tied to a stream.  Returns LS_ERR_SHAPE for
 * other sizes. */
int ls_gemm_tile_override(int32_t bm, int32_t bn);

/* ---- kernel timing (diagnostics) --------------------------------------------
 * Measures one named kernel launch of the calls above with HIP events on the
 * stream it runs on.  ls_timing_begin arms recording for launches whose label
 * equals `label` (labels: "rmsnorm fwd", "qkv projection", "attention fwd",
 * "output projection", "gate/up projection", "down projection", "dact",
 * "dWd", "dh2", "dWg/dWu", "rmsnorm bwd", "dO", "dWo", "attention bwd",
 * "dh1", "dWqkv", and in ls_stack_fwd_bwd also "embedding fwd", "targets",
 * "logits", "cross-entropy", "dh head", "dE head", "loss", "embedding bwd",
 * and "adamw" for ls_adamw_step),
 * creating up to max_launches event pairs up front;
 * later calls record into them without allocating.  ls_timing_end waits for
 * the recorded events, writes the number of recorded launches and their mean
 * duration in milliseconds, disarms recording and releases the events.
 * Process-wide; not meant for concurrent use from several threads. */
int ls_timing_begin(const char* label, int max_launches);
int ls_timing_end(int* launches, float* mean_ms);

/* ---- diagnostics ------------------------------------------------------------ */
const char* ls_status_string(int status);
const char* ls_last_error(void);
/* Library version as major*10000 + minor*100 + patch. */
int ls_version(void);

#ifdef __cplusplus
}
#endif
#endif /* LS_H_ */
