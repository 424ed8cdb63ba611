// Internal launch interface between the C ABI layer and the HIP kernels.
// Every launcher enqueues work on `stream` and returns the launch status.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ls {

typedef uint16_t bf16_t;

// ---- matrix products --------------------------------------------------------
// C[m,n] = sum_k A(m,k) B(k,n), bf16 operands, fp32 accumulation.
// A: a_kcontig ? A[m*lda + k] : A[k*lda + m].
// B: b_kcontig ? row n of B (element k contiguous) : row k of B (element n contiguous).
//    The rows of B may come from up to three buffers: row index r (n if
//    b_kcontig, else k) reads seg[s] for the last s with start[s] <= r, at row
//    r - start[s] of that buffer.
// With glu set (b_kcontig only), virtual column n maps to gate row (n/128)*64 + n%64
// when (n/64) is even and to the up row with the same index when odd (seg[0] =
// gate, seg[1] = up, glu_rows = rows of each).
enum Epilogue {
  EPI_BF16 = 0,     // C (bf16) = acc
  EPI_RESID = 1,    // C (bf16) = acc + R
  EPI_ROPE = 2,     // C (bf16) = rotate(acc) on columns < rope_cols, acc elsewhere
  EPI_GLU_FWD = 3,  // gu[m][i] = g, gu[m][I+i] = u (C; skipped when null), act[m][i] = silu(g) u
  EPI_GLU_BWD = 4,  // C = dgu: dgu[m][i] = acc u silu'(g), dgu[m][I+i] = acc silu(g)
  EPI_F32 = 5,      // F (fp32, rows split over up to three buffers) (+)= acc
};

struct GemmArgs {
  int M = 0, N = 0, K = 0;
  const bf16_t* A = nullptr;
  int64_t lda = 0;
  bool a_kcontig = true;
  const bf16_t* B[3] = {nullptr, nullptr, nullptr};
  int b_start[3] = {0, 1 << 30, 1 << 30};
  int64_t ldb = 0;
  bool b_kcontig = true;
  bool glu = false;
  int glu_rows = 0;
  int epi = EPI_BF16;
  bf16_t* C = nullptr;
  int64_t ldc = 0;
  const bf16_t* R = nullptr;      // EPI_RESID, leading dimension ldc
  const float* rope_cs = nullptr; // EPI_ROPE: [seq][head_dim/2] cos then [seq][head_dim/2] sin
  int seq = 1, head_dim = 128, rope_cols = 0;
  bf16_t* act = nullptr;          // EPI_GLU_FWD: [M][I]
  const bf16_t* gu_in = nullptr;  // EPI_GLU_BWD: saved [M][2I]
  int glu_I = 0;
  float* F[3] = {nullptr, nullptr, nullptr};  // EPI_F32
  int f_start[3] = {0, 1 << 30, 1 << 30};
  int64_t ldf = 0;
  int accumulate = 0;
  // EPI_F32: fp32 workspace for splitting K over workgroups when the output
  // tiles fill at most half the compute units ((slices - 1) * M * N floats,
  // see gemm_kpart_floats); null or smaller means fewer slices or none.
  float* kpart = nullptr;
  int64_t kpart_floats = 0;
  int ksplit = 1;  // slices of K (set by gemm())
  int group_m = 8;  // tile rows per group of the launch order (set by the launch)
};

hipError_t gemm(const GemmArgs& a, hipStream_t s);
// Floats of GemmArgs::kpart with which an EPI_F32 product of this shape runs
// with its full split of K (0: it is not split).
int64_t gemm_kpart_floats(int M, int N, int K);
// Force the tile shape of later gemm launches (bm, bn in {256, 192}; 0, 0 =
// automatic).  Variants that only exist as 256 x 256 ignore it.  -1 on bad sizes.
int gemm_tile_override(int bm, int bn);

// ---- RMSNorm ------------------------------------------------------------------
hipError_t rmsnorm_fwd(int64_t rows, int hidden, float eps, const bf16_t* x, const bf16_t* gamma,
                       bf16_t* h, float* r, hipStream_t s);
// Partial buffer of rmsnorm_bwd: rmsnorm_bwd_parts(rows, hidden) x hidden floats.
int rmsnorm_bwd_parts(int64_t rows, int hidden);
hipError_t rmsnorm_bwd(int64_t rows, int hidden, const bf16_t* x, const bf16_t* gamma, const float* r,
                       const bf16_t* dh, const bf16_t* dres, bf16_t* dx, float* dgamma, int accumulate,
                       float* partial, hipStream_t s);

// ---- RoPE table -------------------------------------------------------------
// cs[p][i] = cos(p theta^(-2i/d)), cs[seq*t/2 + p*t/2 + i] = sin(...), computed in
// fp64, for a table of t/2 entries per position (t = table_dim, 0 = head_dim);
// entries i >= head_dim/2 of a wider table are cos 1, sin 0.
hipError_t rope_table(int seq, int head_dim, double theta, float* cs, hipStream_t s, int table_dim = 0);

// ---- attention ----------------------------------------------------------------
struct AttnShape {
  int batch, seq, nq, nkv, d;
  int d_scale = 0;  // features per head behind the softmax scale 1/sqrt(d_scale) (0: d)
};
hipError_t attn_fwd(const AttnShape& sh, const bf16_t* qkv, bf16_t* o, float* lse, hipStream_t s);
// Workspace for attn_bwd: D and the base-2 log-sum-exp, [batch*nq*seq] fp32 each.
size_t attn_bwd_workspace(const AttnShape& sh);
// rope_cs may be null (no inverse rotation of dq and dk).
hipError_t attn_bwd(const AttnShape& sh, const bf16_t* qkv, const bf16_t* o, const float* lse,
                    const bf16_t* dout, bf16_t* dqkv, const float* rope_cs, void* ws, hipStream_t s);

// ---- padded head layout (64 < d < 128 held in 128-wide slots) -------------------
// Feature s of a head sits at slot s (s < d/2) or dp/2 + s - d/2; other slots are zero.
hipError_t pad_head_rows(const bf16_t* src, bf16_t* dst, int heads, int d, int dp, int cols, hipStream_t s);
hipError_t pad_head_cols(const bf16_t* src, bf16_t* dst, int rows, int heads, int d, int dp, hipStream_t s);
hipError_t unpad_head_rows(const float* src, float* dst, int heads, int d, int dp, int cols, int accumulate,
                           hipStream_t s);
hipError_t unpad_head_cols(const float* src, float* dst, int rows, int heads, int d, int dp, int accumulate,
                           hipStream_t s);

// ---- token embedding and cross-entropy ------------------------------------------
// x[t] = E[ids[t]] ([T, H] bf16); an id outside [0, V) gives a NaN row.
hipError_t embed_fwd(int64_t T, int H, int V, const int32_t* ids, const bf16_t* E, bf16_t* x, hipStream_t s);
// dE[ids[t]] += dx[t], repeated ids summed in token order (deterministic; ids
// outside [0, V) skipped).  H a multiple of 8, at most 8192.
hipError_t embed_bwd(int64_t T, int H, int V, const int32_t* ids, const bf16_t* dx, float* dE, hipStream_t s);
// tg[t] = targets[t], or (targets null) ids[t+1] within a sequence of S tokens
// and -1 at its last position; counts[0] = rows with a target in [0, V).
hipError_t ce_targets(int64_t T, int S, int V, const int32_t* ids, const int32_t* targets, int32_t* tg, int* counts,
                      hipStream_t s);
// Per row of z [rows, V] bf16: row_loss = lse - z[tg]; z <- (softmax - onehot) / max(counts[0], 1).
hipError_t ce_rows(int64_t rows, int V, bf16_t* z, const int32_t* tg, const int* counts, float* row_loss,
                   hipStream_t s);
// loss = sum(row_loss[0 .. T)) / max(counts[0], 1).
hipError_t ce_loss(int64_t T, const float* row_loss, const int* counts, float* loss, hipStream_t s);

// ---- optimizer ------------------------------------------------------------------
struct AdamwHyper {
  float lr, beta1, beta2, eps, weight_decay, max_norm;  // max_norm <= 0: no clipping
  int step;                                            // t >= 1
};
// Workspace bytes of adamw_step (independent of n).
size_t adamw_workspace();
// Global-norm clip + AdamW over n fp32 parameters (decay on the first n_decay);
// param (bf16 copy) and grad_norm may be null.
hipError_t adamw_step(int64_t n, int64_t n_decay, const AdamwHyper& hp, float* master, bf16_t* param,
                      const float* grad, float* m, float* v, float* grad_norm, void* ws, hipStream_t s);

}  // namespace ls
