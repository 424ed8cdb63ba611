// C ABI of the decoder-block library: argument validation (all of it before
// any HIP call) and the orchestration of the kernels for each sub-layer.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <array>
#include <atomic>
#include <initializer_list>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"
#include "ls.h"

using ls::bf16_t;

namespace {

constexpr int kVersion = 100;  // 0.1.0

thread_local char g_last_error[512];  // a fixed buffer: reporting an error allocates nothing

// Largest matrix in bytes (exclusive): the kernels' buffer resources are
// clamped to 2047 MiB.
constexpr int64_t kMaxBytes = (int64_t)0x7ff00000;

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return code;
}

int hip_fail(hipError_t e, const char* where) {
  return fail(LS_ERR_HIP, "%s: %s (%d)", where, hipGetErrorString(e), (int)e);
}

#define LS_HIP(call, where)                          \
  do {                                               \
    hipError_t e_ = (call);                          \
    if (e_ != hipSuccess) return hip_fail(e_, where); \
  } while (0)

inline size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

// ---- optional per-launch timing (ls_timing_begin / ls_timing_end) -------------
struct Timing {
  std::mutex mu;
  std::atomic<bool> armed{false};
  std::string label;
  std::vector<hipEvent_t> ev;  // start, stop per launch
  int used = 0;
};
Timing g_timing;

void timing_mark(const char* label, hipStream_t st, bool start) {
  if (!g_timing.armed) return;
  std::lock_guard<std::mutex> lk(g_timing.mu);
  if (!g_timing.armed || g_timing.label != label) return;
  const size_t idx = 2 * (size_t)g_timing.used + (start ? 0 : 1);
  if (idx >= g_timing.ev.size()) return;
  (void)hipEventRecord(g_timing.ev[idx], st);
  if (!start) ++g_timing.used;
}

// enqueue one labelled step, with timing marks around it
#define LS_STEP(label, st, call)                         \
  do {                                                  \
    timing_mark(label, st, true);                       \
    hipError_t e_ = (call);                             \
    if (e_ != hipSuccess) return hip_fail(e_, label);   \
    timing_mark(label, st, false);                      \
  } while (0)

// Head sizes the attention kernels tile natively are 64 and 128; a size in
// between is held in 128-wide slots (dp = 128, `pad`), and Pq, Pkv, Pqkv are
// the widths of q, k/v and qkv in that layout (equal to Dq, Dkv, Dqkv otherwise).
struct Dims {
  int64_t B, S, T, H, nq, nkv, d, Dq, Dkv, Dqkv, I;
  int64_t dp, Pq, Pkv, Pqkv;
  bool pad;
};

Dims dims_of(const ls_block_cfg& c) {
  Dims m;
  m.B = c.batch;
  m.S = c.seq;
  m.T = (int64_t)c.batch * c.seq;
  m.H = c.hidden;
  m.nq = c.n_q_heads;
  m.nkv = c.n_kv_heads;
  m.d = c.head_dim;
  m.Dq = m.nq * m.d;
  m.Dkv = m.nkv * m.d;
  m.Dqkv = m.Dq + 2 * m.Dkv;
  m.I = c.intermediate;
  m.dp = (m.d == 64 || m.d == 128) ? m.d : 128;
  m.pad = m.dp != m.d;
  m.Pq = m.nq * m.dp;
  m.Pkv = m.nkv * m.dp;
  m.Pqkv = m.Pq + 2 * m.Pkv;
  return m;
}

int check_cfg(const ls_block_cfg* c) {
  if (!c) return fail(LS_ERR_NULL, "cfg is NULL");
  if (c->batch <= 0 || c->seq <= 0 || c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 ||
      c->head_dim <= 0 || c->intermediate <= 0)
    return fail(LS_ERR_SHAPE, "all sizes must be positive");
  if (c->n_q_heads % c->n_kv_heads != 0)
    return fail(LS_ERR_SHAPE, "n_q_heads (%d) is not a multiple of n_kv_heads (%d)", c->n_q_heads, c->n_kv_heads);
  if (c->hidden % 8 != 0 || c->intermediate % 8 != 0)
    return fail(LS_ERR_SHAPE, "hidden (%d) and intermediate (%d) must be multiples of 8", c->hidden, c->intermediate);
  if (!(c->rope_theta > 1.0f) || !(c->rms_eps >= 0.0f))
    return fail(LS_ERR_SHAPE, "rope_theta must exceed 1 and rms_eps must be >= 0");
  if (c->head_dim != 64 && !(c->head_dim > 64 && c->head_dim <= 128 && c->head_dim % 8 == 0))
    return fail(LS_ERR_UNSUPPORTED, "head_dim %d is not supported (64, or a multiple of 8 from 72 to 128)",
                c->head_dim);
  if (c->hidden > 8192) return fail(LS_ERR_UNSUPPORTED, "hidden %d exceeds 8192", c->hidden);
  const Dims m = dims_of(*c);
  const int64_t lim = (int64_t)1 << 30;
  // every matrix is addressed with 32-bit byte offsets (buffer loads, whose
  // resources stay below 2047 MiB)
  const int64_t widest = std::max(std::max(m.Pqkv, 2 * m.I), m.H);
  if (m.T >= lim || m.Pqkv >= lim || 2 * m.I >= lim || m.T * widest * 2 >= kMaxBytes ||
      m.I * m.H * 2 >= kMaxBytes || m.Pqkv * m.H * 4 >= kMaxBytes)
    return fail(LS_ERR_SHAPE, "problem too large (a matrix reaches 2047 MiB)");
  return LS_OK;
}

bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

struct Range {
  const void* p;
  size_t n;
  const char* name;
};

bool overlaps(const Range& a, const Range& b) {
  if (!a.p || !b.p || a.n == 0 || b.n == 0) return false;
  const uintptr_t a0 = (uintptr_t)a.p, a1 = a0 + a.n, b0 = (uintptr_t)b.p, b1 = b0 + b.n;
  return a0 < b1 && b0 < a1;
}

// every output range against every input range and every other output range
int check_ranges(const Range* in, size_t nin, const Range* out, size_t nout) {
  for (size_t i = 0; i < nin; ++i) {
    if (!in[i].p) return fail(LS_ERR_NULL, "%s is NULL", in[i].name);
    if (misaligned(in[i].p)) return fail(LS_ERR_ALIGN, "%s is not 16-byte aligned", in[i].name);
  }
  for (size_t i = 0; i < nout; ++i) {
    if (!out[i].p) return fail(LS_ERR_NULL, "%s is NULL", out[i].name);
    if (misaligned(out[i].p)) return fail(LS_ERR_ALIGN, "%s is not 16-byte aligned", out[i].name);
  }
  for (size_t i = 0; i < nout; ++i) {
    for (size_t j = 0; j < nin; ++j)
      if (overlaps(out[i], in[j])) return fail(LS_ERR_ALIAS, "%s overlaps %s", out[i].name, in[j].name);
    for (size_t j = i + 1; j < nout; ++j)
      if (overlaps(out[i], out[j])) return fail(LS_ERR_ALIAS, "%s overlaps %s", out[i].name, out[j].name);
  }
  return LS_OK;
}
int check_ranges(const std::vector<Range>& in, const std::vector<Range>& out) {
  return check_ranges(in.data(), in.size(), out.data(), out.size());
}

// ---- buffer layouts ------------------------------------------------------------

struct Carver {
  size_t off = 0;
  size_t take(size_t bytes) {
    const size_t o = off;
    off += up256(bytes);
    return o;
  }
};

struct AttnSaved {
  size_t h1, qkv, o, r1, lse, total;
};
AttnSaved attn_saved_layout(const Dims& m) {
  Carver c;
  AttnSaved s;
  s.h1 = c.take(m.T * m.H * 2);
  s.qkv = c.take(m.T * m.Pqkv * 2);
  s.o = c.take(m.T * m.Pq * 2);
  s.r1 = c.take(m.T * 4);
  s.lse = c.take(m.B * m.nq * m.S * 4);
  s.total = c.off;
  return s;
}

struct MlpSaved {
  size_t h2, gu, act, r2, total;
};
MlpSaved mlp_saved_layout(const Dims& m) {
  Carver c;
  MlpSaved s;
  s.h2 = c.take(m.T * m.H * 2);
  s.gu = c.take(m.T * 2 * m.I * 2);
  s.act = c.take(m.T * m.I * 2);
  s.r2 = c.take(m.T * 4);
  s.total = c.off;
  return s;
}

size_t norm_partial_bytes(const Dims& m) { return (size_t)ls::rmsnorm_bwd_parts(m.T, (int)m.H) * m.H * 4; }

ls::AttnShape attn_shape(const Dims& m) {
  return ls::AttnShape{(int)m.B, (int)m.S, (int)m.nq, (int)m.nkv, (int)m.dp, (int)m.d};
}

// fp32 partial sums of the weight-gradient products that split K (their
// output tiles alone would leave most compute units idle)
int64_t max_kpart_floats(std::initializer_list<std::array<int64_t, 3>> shapes) {
  int64_t n = 0;
  for (const auto& mnk : shapes) n = std::max(n, ls::gemm_kpart_floats((int)mnk[0], (int)mnk[1], (int)mnk[2]));
  return n;
}

struct AttnWs {
  size_t rope, dO, dqkv, dh1, partial, core, wpad, wopad, gpad, gopad, kpart, total;
  int64_t kpart_floats;
};
AttnWs attn_ws_layout(const Dims& m) {
  Carver c;
  AttnWs w;
  w.rope = c.take(m.S * m.dp * 4);  // cos and sin, S x dp/2 each
  w.dO = c.take(m.T * m.Pq * 2);
  w.dqkv = c.take(m.T * m.Pqkv * 2);
  // padded layout only: Wq|Wk|Wv [Pqkv, H] and Wo [H, Pq] in bf16, their fp32 gradients
  w.wpad = c.take(m.pad ? m.Pqkv * m.H * 2 : 0);
  w.wopad = c.take(m.pad ? m.H * m.Pq * 2 : 0);
  w.gpad = c.take(m.pad ? m.Pqkv * m.H * 4 : 0);
  w.gopad = c.take(m.pad ? m.H * m.Pq * 4 : 0);
  w.dh1 = c.take(m.T * m.H * 2);
  w.partial = c.take(norm_partial_bytes(m));
  w.core = c.take(ls::attn_bwd_workspace(attn_shape(m)));
  w.kpart_floats = max_kpart_floats({{m.H, m.Pq, m.T}, {m.Pqkv, m.H, m.T}});  // dWo, dWqkv
  w.kpart = c.take((size_t)w.kpart_floats * 4);
  w.total = c.off;
  return w;
}

struct MlpWs {
  size_t dgu, dh2, partial, kpart, total;
  int64_t kpart_floats;
};
MlpWs mlp_ws_layout(const Dims& m) {
  Carver c;
  MlpWs w;
  w.dgu = c.take(m.T * 2 * m.I * 2);
  w.dh2 = c.take(m.T * m.H * 2);
  w.partial = c.take(norm_partial_bytes(m));
  w.kpart_floats = max_kpart_floats({{m.H, m.I, m.T}, {2 * m.I, m.H, m.T}});  // dWd, dWg/dWu
  w.kpart = c.take((size_t)w.kpart_floats * 4);
  w.total = c.off;
  return w;
}

struct BlockWs {
  size_t attn_saved, mlp_saved, x2, dx2, scratch, total;
};
BlockWs block_ws_layout(const Dims& m) {
  Carver c;
  BlockWs w;
  w.attn_saved = c.take(attn_saved_layout(m).total);
  w.mlp_saved = c.take(mlp_saved_layout(m).total);
  w.x2 = c.take(m.T * m.H * 2);
  w.dx2 = c.take(m.T * m.H * 2);
  w.scratch = c.take(std::max(attn_ws_layout(m).total, mlp_ws_layout(m).total));
  w.total = c.off;
  return w;
}

template <typename T>
T* at(void* base, size_t off) {
  return (T*)((char*)base + off);
}
template <typename T>
const T* at(const void* base, size_t off) {
  return (const T*)((const char*)base + off);
}

// ---- argument checks shared by the sub-layer calls --------------------------------

void weight_ranges(const Dims& m, const ls_block_weights* w, bool attn, bool mlp, std::vector<Range>& v) {
  if (attn) {
    v.push_back({w->attn_norm, (size_t)m.H * 2, "w.attn_norm"});
    v.push_back({w->wq, (size_t)(m.Dq * m.H * 2), "w.wq"});
    v.push_back({w->wk, (size_t)(m.Dkv * m.H * 2), "w.wk"});
    v.push_back({w->wv, (size_t)(m.Dkv * m.H * 2), "w.wv"});
    v.push_back({w->wo, (size_t)(m.H * m.Dq * 2), "w.wo"});
  }
  if (mlp) {
    v.push_back({w->mlp_norm, (size_t)m.H * 2, "w.mlp_norm"});
    v.push_back({w->wg, (size_t)(m.I * m.H * 2), "w.wg"});
    v.push_back({w->wu, (size_t)(m.I * m.H * 2), "w.wu"});
    v.push_back({w->wd, (size_t)(m.H * m.I * 2), "w.wd"});
  }
}

void grad_ranges(const Dims& m, const ls_block_grads* g, bool attn, bool mlp, std::vector<Range>& v) {
  if (attn) {
    v.push_back({g->attn_norm, (size_t)m.H * 4, "g.attn_norm"});
    v.push_back({g->wq, (size_t)(m.Dq * m.H * 4), "g.wq"});
    v.push_back({g->wk, (size_t)(m.Dkv * m.H * 4), "g.wk"});
    v.push_back({g->wv, (size_t)(m.Dkv * m.H * 4), "g.wv"});
    v.push_back({g->wo, (size_t)(m.H * m.Dq * 4), "g.wo"});
  }
  if (mlp) {
    v.push_back({g->mlp_norm, (size_t)m.H * 4, "g.mlp_norm"});
    v.push_back({g->wg, (size_t)(m.I * m.H * 4), "g.wg"});
    v.push_back({g->wu, (size_t)(m.I * m.H * 4), "g.wu"});
    v.push_back({g->wd, (size_t)(m.H * m.I * 4), "g.wd"});
  }
}

// ---- the sub-layers (arguments already checked) ------------------------------------

// The projection weights in the layout the attention kernels read: the
// caller's buffers, or (padded head layout) copies in the workspace.
struct PaddedWeights {
  const bf16_t *wq, *wk, *wv, *wo;
  int err;
};
PaddedWeights padded_weights(const Dims& m, const ls_block_weights* w, void* ws, hipStream_t st) {
  if (!m.pad) return {(const bf16_t*)w->wq, (const bf16_t*)w->wk, (const bf16_t*)w->wv, (const bf16_t*)w->wo, LS_OK};
  const AttnWs wl = attn_ws_layout(m);
  bf16_t* wp = at<bf16_t>(ws, wl.wpad);
  bf16_t* wo = at<bf16_t>(ws, wl.wopad);
  const int d = (int)m.d, dp = (int)m.dp, H = (int)m.H;
  hipError_t e = ls::pad_head_rows((const bf16_t*)w->wq, wp, (int)m.nq, d, dp, H, st);
  if (e == hipSuccess) e = ls::pad_head_rows((const bf16_t*)w->wk, wp + m.Pq * m.H, (int)m.nkv, d, dp, H, st);
  if (e == hipSuccess) e = ls::pad_head_rows((const bf16_t*)w->wv, wp + (m.Pq + m.Pkv) * m.H, (int)m.nkv, d, dp, H, st);
  if (e == hipSuccess) e = ls::pad_head_cols((const bf16_t*)w->wo, wo, H, (int)m.nq, d, dp, st);
  if (e != hipSuccess) return {nullptr, nullptr, nullptr, nullptr, hip_fail(e, "padded weights")};
  return {wp, wp + m.Pq * m.H, wp + (m.Pq + m.Pkv) * m.H, wo, LS_OK};
}

// out_proj = false: stop after the attention core (a recomputation whose x2 is
// already known).
int run_attn_fwd(const ls_block_cfg& cfg, const Dims& m, const bf16_t* x, const ls_block_weights* w, bf16_t* x2,
                 void* saved, void* ws, hipStream_t st, bool out_proj = true) {
  const AttnSaved sv = attn_saved_layout(m);
  const AttnWs wl = attn_ws_layout(m);
  bf16_t* h1 = at<bf16_t>(saved, sv.h1);
  bf16_t* qkv = at<bf16_t>(saved, sv.qkv);
  bf16_t* o = at<bf16_t>(saved, sv.o);
  float* r1 = at<float>(saved, sv.r1);
  float* lse = at<float>(saved, sv.lse);
  float* cs = at<float>(ws, wl.rope);
  const PaddedWeights pw = padded_weights(m, w, ws, st);
  if (pw.err) return pw.err;
  LS_STEP("rmsnorm fwd", st, ls::rmsnorm_fwd(m.T, (int)m.H, cfg.rms_eps, x, (const bf16_t*)w->attn_norm, h1, r1, st));
  LS_STEP("rope table", st, ls::rope_table((int)m.S, (int)m.d, (double)cfg.rope_theta, cs, st, (int)m.dp));
  ls::GemmArgs g;
  g.M = (int)m.T;
  g.N = (int)m.Pqkv;
  g.K = (int)m.H;
  g.A = h1;
  g.lda = m.H;
  g.B[0] = pw.wq;
  g.B[1] = pw.wk;
  g.B[2] = pw.wv;
  g.b_start[1] = (int)m.Pq;
  g.b_start[2] = (int)(m.Pq + m.Pkv);
  g.ldb = m.H;
  g.epi = ls::EPI_ROPE;
  g.C = qkv;
  g.ldc = m.Pqkv;
  g.rope_cs = cs;
  g.seq = (int)m.S;
  g.head_dim = (int)m.dp;
  g.rope_cols = (int)(m.Pq + m.Pkv);
  LS_STEP("qkv projection", st, ls::gemm(g, st));
  LS_STEP("attention fwd", st, ls::attn_fwd(attn_shape(m), qkv, o, lse, st));
  if (!out_proj) return LS_OK;
  ls::GemmArgs p;
  p.M = (int)m.T;
  p.N = (int)m.H;
  p.K = (int)m.Pq;
  p.A = o;
  p.lda = m.Pq;
  p.B[0] = pw.wo;
  p.ldb = m.Pq;
  p.epi = ls::EPI_RESID;
  p.R = x;
  p.C = x2;
  p.ldc = m.H;
  LS_STEP("output projection", st, ls::gemm(p, st));
  return LS_OK;
}

int run_attn_bwd(const ls_block_cfg& cfg, const Dims& m, const bf16_t* x, const ls_block_weights* w,
                 const void* saved, const bf16_t* dx2, bf16_t* dx, const ls_block_grads* gr, int accumulate, void* ws,
                 hipStream_t st) {
  const AttnSaved sv = attn_saved_layout(m);
  const AttnWs wl = attn_ws_layout(m);
  const bf16_t* h1 = at<bf16_t>(saved, sv.h1);
  const bf16_t* qkv = at<bf16_t>(saved, sv.qkv);
  const bf16_t* o = at<bf16_t>(saved, sv.o);
  const float* r1 = at<float>(saved, sv.r1);
  const float* lse = at<float>(saved, sv.lse);
  float* cs = at<float>(ws, wl.rope);
  bf16_t* dO = at<bf16_t>(ws, wl.dO);
  bf16_t* dqkv = at<bf16_t>(ws, wl.dqkv);
  bf16_t* dh1 = at<bf16_t>(ws, wl.dh1);
  float* partial = at<float>(ws, wl.partial);
  void* core = at<char>(ws, wl.core);
  const PaddedWeights pw = padded_weights(m, w, ws, st);
  if (pw.err) return pw.err;
  LS_STEP("rope table", st, ls::rope_table((int)m.S, (int)m.d, (double)cfg.rope_theta, cs, st, (int)m.dp));
  {  // dO = dx2 Wo
    ls::GemmArgs g;
    g.M = (int)m.T;
    g.N = (int)m.Pq;
    g.K = (int)m.H;
    g.A = dx2;
    g.lda = m.H;
    g.B[0] = pw.wo;
    g.ldb = m.Pq;
    g.b_kcontig = false;
    g.epi = ls::EPI_BF16;
    g.C = dO;
    g.ldc = m.Pq;
    LS_STEP("dO", st, ls::gemm(g, st));
  }
  {  // dWo (+)= dx2^T o  (padded layout: into the workspace, then folded back)
    ls::GemmArgs g;
    g.M = (int)m.H;
    g.N = (int)m.Pq;
    g.K = (int)m.T;
    g.A = dx2;
    g.lda = m.H;
    g.a_kcontig = false;
    g.B[0] = o;
    g.ldb = m.Pq;
    g.b_kcontig = false;
    g.epi = ls::EPI_F32;
    g.F[0] = m.pad ? at<float>(ws, wl.gopad) : gr->wo;
    g.ldf = m.Pq;
    g.accumulate = m.pad ? 0 : accumulate;
    g.kpart = at<float>(ws, wl.kpart);
    g.kpart_floats = wl.kpart_floats;
    LS_STEP("dWo", st, ls::gemm(g, st));
    if (m.pad)
      LS_STEP("dWo", st, ls::unpad_head_cols(at<float>(ws, wl.gopad), gr->wo, (int)m.H, (int)m.nq, (int)m.d,
                                             (int)m.dp, accumulate, st));
  }
  LS_STEP("attention bwd", st, ls::attn_bwd(attn_shape(m), qkv, o, lse, dO, dqkv, cs, core, st));
  {  // dh1 = dq Wq + dk Wk + dv Wv
    ls::GemmArgs g;
    g.M = (int)m.T;
    g.N = (int)m.H;
    g.K = (int)m.Pqkv;
    g.A = dqkv;
    g.lda = m.Pqkv;
    g.B[0] = pw.wq;
    g.B[1] = pw.wk;
    g.B[2] = pw.wv;
    g.b_start[1] = (int)m.Pq;
    g.b_start[2] = (int)(m.Pq + m.Pkv);
    g.ldb = m.H;
    g.b_kcontig = false;
    g.epi = ls::EPI_BF16;
    g.C = dh1;
    g.ldc = m.H;
    LS_STEP("dh1", st, ls::gemm(g, st));
  }
  {  // dWq, dWk, dWv (+)= dqkv^T h1  (padded layout: into the workspace, then folded back)
    ls::GemmArgs g;
    g.M = (int)m.Pqkv;
    g.N = (int)m.H;
    g.K = (int)m.T;
    g.A = dqkv;
    g.lda = m.Pqkv;
    g.a_kcontig = false;
    g.B[0] = h1;
    g.ldb = m.H;
    g.b_kcontig = false;
    g.epi = ls::EPI_F32;
    if (m.pad) {
      g.F[0] = at<float>(ws, wl.gpad);
      g.accumulate = 0;
    } else {
      g.F[0] = gr->wq;
      g.F[1] = gr->wk;
      g.F[2] = gr->wv;
      g.f_start[1] = (int)m.Dq;
      g.f_start[2] = (int)(m.Dq + m.Dkv);
      g.accumulate = accumulate;
    }
    g.ldf = m.H;
    g.kpart = at<float>(ws, wl.kpart);
    g.kpart_floats = wl.kpart_floats;
    LS_STEP("dWqkv", st, ls::gemm(g, st));
    if (m.pad) {
      const float* gp = at<float>(ws, wl.gpad);
      LS_STEP("dWqkv", st, ls::unpad_head_rows(gp, gr->wq, (int)m.nq, (int)m.d, (int)m.dp, (int)m.H, accumulate, st));
      LS_STEP("dWqkv", st, ls::unpad_head_rows(gp + m.Pq * m.H, gr->wk, (int)m.nkv, (int)m.d, (int)m.dp, (int)m.H,
                                               accumulate, st));
      LS_STEP("dWqkv", st, ls::unpad_head_rows(gp + (m.Pq + m.Pkv) * m.H, gr->wv, (int)m.nkv, (int)m.d, (int)m.dp,
                                               (int)m.H, accumulate, st));
    }
  }
  LS_STEP("rmsnorm bwd", st,
          ls::rmsnorm_bwd(m.T, (int)m.H, x, (const bf16_t*)w->attn_norm, r1, dh1, dx2, dx, gr->attn_norm, accumulate,
                          partial, st));
  return LS_OK;
}

// keep_gu = false: a forward pass whose saved state is not used (the backward
// pass recomputes it) skips writing the gate and up outputs.  down = false:
// stop before the down projection (a recomputation whose y is already known).
int run_mlp_fwd(const ls_block_cfg& cfg, const Dims& m, const bf16_t* x2, const ls_block_weights* w, bf16_t* y,
                void* saved, hipStream_t st, bool keep_gu = true, bool down = true) {
  const MlpSaved sv = mlp_saved_layout(m);
  bf16_t* h2 = at<bf16_t>(saved, sv.h2);
  bf16_t* gu = at<bf16_t>(saved, sv.gu);
  bf16_t* act = at<bf16_t>(saved, sv.act);
  float* r2 = at<float>(saved, sv.r2);
  LS_STEP("rmsnorm fwd", st, ls::rmsnorm_fwd(m.T, (int)m.H, cfg.rms_eps, x2, (const bf16_t*)w->mlp_norm, h2, r2, st));
  {
    ls::GemmArgs g;
    g.M = (int)m.T;
    g.N = (int)(2 * ((m.I + 63) / 64) * 64);
    g.K = (int)m.H;
    g.A = h2;
    g.lda = m.H;
    g.B[0] = (const bf16_t*)w->wg;
    g.B[1] = (const bf16_t*)w->wu;
    g.glu = true;
    g.glu_rows = (int)m.I;
    g.ldb = m.H;
    g.epi = ls::EPI_GLU_FWD;
    g.C = keep_gu ? gu : nullptr;
    g.ldc = 2 * m.I;
    g.act = act;
    g.glu_I = (int)m.I;
    LS_STEP("gate/up projection", st, ls::gemm(g, st));
  }
  if (!down) return LS_OK;
  {
    ls::GemmArgs g;
    g.M = (int)m.T;
    g.N = (int)m.H;
    g.K = (int)m.I;
    g.A = act;
    g.lda = m.I;
    g.B[0] = (const bf16_t*)w->wd;
    g.ldb = m.I;
    g.epi = ls::EPI_RESID;
    g.R = x2;
    g.C = y;
    g.ldc = m.H;
    LS_STEP("down projection", st, ls::gemm(g, st));
  }
  return LS_OK;
}

int run_mlp_bwd(const ls_block_cfg& cfg, const Dims& m, const bf16_t* x2, const ls_block_weights* w,
                const void* saved, const bf16_t* dy, bf16_t* dx2, const ls_block_grads* gr, int accumulate, void* ws,
                hipStream_t st) {
  (void)cfg;
  const MlpSaved sv = mlp_saved_layout(m);
  const MlpWs wl = mlp_ws_layout(m);
  const bf16_t* h2 = at<bf16_t>(saved, sv.h2);
  const bf16_t* gu = at<bf16_t>(saved, sv.gu);
  const bf16_t* act = at<bf16_t>(saved, sv.act);
  const float* r2 = at<float>(saved, sv.r2);
  bf16_t* dgu = at<bf16_t>(ws, wl.dgu);
  bf16_t* dh2 = at<bf16_t>(ws, wl.dh2);
  float* partial = at<float>(ws, wl.partial);
  {  // dact = dy Wd, then dg, du from the saved gate/up outputs
    ls::GemmArgs g;
    g.M = (int)m.T;
    g.N = (int)m.I;
    g.K = (int)m.H;
    g.A = dy;
    g.lda = m.H;
    g.B[0] = (const bf16_t*)w->wd;
    g.ldb = m.I;
    g.b_kcontig = false;
    g.epi = ls::EPI_GLU_BWD;
    g.C = dgu;
    g.ldc = 2 * m.I;
    g.gu_in = gu;
    g.glu_I = (int)m.I;
    LS_STEP("dact", st, ls::gemm(g, st));
  }
  // dh2 and dWg/dWu follow dact, which has just written dgu, so they read
  // much of it from the last-level cache; dWd (dy and act only) goes last.
  {  // dh2 = dg Wg + du Wu
    ls::GemmArgs g;
    g.M = (int)m.T;
    g.N = (int)m.H;
    g.K = (int)(2 * m.I);
    g.A = dgu;
    g.lda = 2 * m.I;
    g.B[0] = (const bf16_t*)w->wg;
    g.B[1] = (const bf16_t*)w->wu;
    g.b_start[1] = (int)m.I;
    g.ldb = m.H;
    g.b_kcontig = false;
    g.epi = ls::EPI_BF16;
    g.C = dh2;
    g.ldc = m.H;
    LS_STEP("dh2", st, ls::gemm(g, st));
  }
  {  // dWg, dWu (+)= [dg du]^T h2
    ls::GemmArgs g;
    g.M = (int)(2 * m.I);
    g.N = (int)m.H;
    g.K = (int)m.T;
    g.A = dgu;
    g.lda = 2 * m.I;
    g.a_kcontig = false;
    g.B[0] = h2;
    g.ldb = m.H;
    g.b_kcontig = false;
    g.epi = ls::EPI_F32;
    g.F[0] = gr->wg;
    g.F[1] = gr->wu;
    g.f_start[1] = (int)m.I;
    g.ldf = m.H;
    g.accumulate = accumulate;
    g.kpart = at<float>(ws, wl.kpart);
    g.kpart_floats = wl.kpart_floats;
    LS_STEP("dWg/dWu", st, ls::gemm(g, st));
  }
  {  // dWd (+)= dy^T act
    ls::GemmArgs g;
    g.M = (int)m.H;
    g.N = (int)m.I;
    g.K = (int)m.T;
    g.A = dy;
    g.lda = m.H;
    g.a_kcontig = false;
    g.B[0] = act;
    g.ldb = m.I;
    g.b_kcontig = false;
    g.epi = ls::EPI_F32;
    g.F[0] = gr->wd;
    g.ldf = m.I;
    g.accumulate = accumulate;
    g.kpart = at<float>(ws, wl.kpart);
    g.kpart_floats = wl.kpart_floats;
    LS_STEP("dWd", st, ls::gemm(g, st));
  }
  LS_STEP("rmsnorm bwd", st,
          ls::rmsnorm_bwd(m.T, (int)m.H, x2, (const bf16_t*)w->mlp_norm, r2, dh2, dy, dx2, gr->mlp_norm, accumulate,
                          partial, st));
  return LS_OK;
}

// ---- the stack of blocks with a tied embedding, LM head and cross-entropy ------------

int check_stack_cfg(const ls_stack_cfg* c) {
  if (!c) return fail(LS_ERR_NULL, "cfg is NULL");
  if (int e = check_cfg(&c->block)) return e;
  if (c->n_layers < 0 || c->n_layers > 4096) return fail(LS_ERR_SHAPE, "n_layers %d out of range [0, 4096]", c->n_layers);
  if (c->vocab <= 0 || c->vocab % 8 != 0) return fail(LS_ERR_SHAPE, "vocab (%d) must be a positive multiple of 8", c->vocab);
  if (c->recompute != 0 && c->recompute != 1) return fail(LS_ERR_SHAPE, "recompute must be 0 or 1");
  if (c->logits_chunk < 0) return fail(LS_ERR_SHAPE, "logits_chunk must be >= 0");
  if ((int64_t)c->vocab * c->block.hidden * 4 >= kMaxBytes)
    return fail(LS_ERR_SHAPE, "vocab x hidden fp32 gradient reaches 2047 MiB");
  return LS_OK;
}

// Token rows per logits chunk: the [rows, vocab] bf16 logits of one chunk stay
// below the 2047 MiB limit of one matrix-product operand (and within the
// caller's logits_chunk when set).
int64_t logits_rows(const ls_stack_cfg& c) {
  const Dims m = dims_of(c.block);
  int64_t per = (kMaxBytes - 1) / ((int64_t)c.vocab * 2);
  if (per >= 256) per &= ~(int64_t)255;
  if (c.logits_chunk > 0) per = std::min<int64_t>(per, c.logits_chunk);
  return std::min<int64_t>(m.T, per);
}

struct StackWs {
  size_t tg, counts, rows, xs, xmid, hf, rf, logits, dh, dxa, dxb, partial, sets, set_stride, dx2, scratch, total;
  size_t asv, msv, x2;  // offsets inside one set
};
StackWs stack_ws_layout(const ls_stack_cfg& c) {
  const Dims m = dims_of(c.block);
  const size_t act = (size_t)(m.T * m.H * 2);
  Carver k;
  StackWs w;
  w.tg = k.take(m.T * 4);
  w.counts = k.take(16);
  w.rows = k.take(m.T * 4);
  w.xs = k.take(act * (size_t)(c.n_layers + 1));
  // with recomputation each block's mid-residual x2 is kept too, so that the
  // recomputation stops before the output and down projections
  w.xmid = k.take(c.recompute ? act * (size_t)c.n_layers : 0);
  w.hf = k.take(act);
  w.rf = k.take(m.T * 4);
  w.logits = k.take((size_t)logits_rows(c) * c.vocab * 2);
  w.dh = k.take(act);
  w.dxa = k.take(act);
  w.dxb = k.take(act);
  w.partial = k.take(norm_partial_bytes(m));
  w.dx2 = k.take(act);
  w.scratch = k.take(std::max(attn_ws_layout(m).total, mlp_ws_layout(m).total));
  Carver one;
  w.asv = one.take(attn_saved_layout(m).total);
  w.msv = one.take(mlp_saved_layout(m).total);
  w.x2 = one.take(act);
  w.set_stride = one.off;
  const int nsets = c.recompute ? (c.n_layers > 0 ? 1 : 0) : c.n_layers;
  w.sets = k.take(w.set_stride * (size_t)nsets);
  w.total = k.off;
  return w;
}

}  // namespace

extern "C" {

int ls_version(void) { return kVersion; }

const char* ls_last_error(void) { return g_last_error; }

const char* ls_status_string(int status) {
  switch (status) {
    case LS_OK: return "ok";
    case LS_ERR_NULL: return "null pointer";
    case LS_ERR_SHAPE: return "invalid shape";
    case LS_ERR_UNSUPPORTED: return "unsupported configuration";
    case LS_ERR_ALIGN: return "misaligned pointer";
    case LS_ERR_ALIAS: return "overlapping buffers";
    case LS_ERR_WORKSPACE: return "workspace too small";
    case LS_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int ls_query_sizes(const ls_block_cfg* cfg, ls_sizes* out) {
  if (int e = check_cfg(cfg)) return e;
  if (!out) return fail(LS_ERR_NULL, "out is NULL");
  const Dims m = dims_of(*cfg);
  out->attn_saved = attn_saved_layout(m).total;
  out->mlp_saved = mlp_saved_layout(m).total;
  out->attn_workspace = attn_ws_layout(m).total;
  out->mlp_workspace = mlp_ws_layout(m).total;
  out->block_workspace = block_ws_layout(m).total;
  return LS_OK;
}

int ls_attn_fwd(const ls_block_cfg* cfg, const ls_bf16* x, const ls_block_weights* w, ls_bf16* x2, void* attn_saved,
                void* workspace, size_t workspace_bytes, void* stream) {
  if (int e = check_cfg(cfg)) return e;
  if (!w) return fail(LS_ERR_NULL, "weights is NULL");
  const Dims m = dims_of(*cfg);
  const size_t act = (size_t)(m.T * m.H * 2);
  std::vector<Range> in{{x, act, "x"}}, out{{x2, act, "x2"},
                                           {attn_saved, attn_saved_layout(m).total, "attn_saved"},
                                           {workspace, workspace_bytes, "workspace"}};
  weight_ranges(m, w, true, false, in);
  if (int e = check_ranges(in, out)) return e;
  if (workspace_bytes < attn_ws_layout(m).total)
    return fail(LS_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, attn_ws_layout(m).total);
  return run_attn_fwd(*cfg, m, (const bf16_t*)x, w, (bf16_t*)x2, attn_saved, workspace, (hipStream_t)stream);
}

int ls_attn_bwd(const ls_block_cfg* cfg, const ls_bf16* x, const ls_block_weights* w, const void* attn_saved,
                const ls_bf16* dx2, ls_bf16* dx, const ls_block_grads* g, int accumulate, void* workspace,
                size_t workspace_bytes, void* stream) {
  if (int e = check_cfg(cfg)) return e;
  if (!w || !g) return fail(LS_ERR_NULL, "weights or grads is NULL");
  const Dims m = dims_of(*cfg);
  const size_t act = (size_t)(m.T * m.H * 2);
  std::vector<Range> in{{x, act, "x"}, {attn_saved, attn_saved_layout(m).total, "attn_saved"}, {dx2, act, "dx2"}};
  std::vector<Range> out{{dx, act, "dx"}, {workspace, workspace_bytes, "workspace"}};
  weight_ranges(m, w, true, false, in);
  grad_ranges(m, g, true, false, out);
  if (int e = check_ranges(in, out)) return e;
  if (workspace_bytes < attn_ws_layout(m).total)
    return fail(LS_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, attn_ws_layout(m).total);
  return run_attn_bwd(*cfg, m, (const bf16_t*)x, w, attn_saved, (const bf16_t*)dx2, (bf16_t*)dx, g, accumulate != 0,
                      workspace, (hipStream_t)stream);
}

int ls_mlp_fwd(const ls_block_cfg* cfg, const ls_bf16* x2, const ls_block_weights* w, ls_bf16* y, void* mlp_saved,
               void* workspace, size_t workspace_bytes, void* stream) {
  if (int e = check_cfg(cfg)) return e;
  if (!w) return fail(LS_ERR_NULL, "weights is NULL");
  const Dims m = dims_of(*cfg);
  const size_t act = (size_t)(m.T * m.H * 2);
  std::vector<Range> in{{x2, act, "x2"}}, out{{y, act, "y"}, {mlp_saved, mlp_saved_layout(m).total, "mlp_saved"}};
  if (workspace) out.push_back({workspace, workspace_bytes, "workspace"});
  weight_ranges(m, w, false, true, in);
  if (int e = check_ranges(in, out)) return e;
  return run_mlp_fwd(*cfg, m, (const bf16_t*)x2, w, (bf16_t*)y, mlp_saved, (hipStream_t)stream);
}

int ls_mlp_bwd(const ls_block_cfg* cfg, const ls_bf16* x2, const ls_block_weights* w, const void* mlp_saved,
               const ls_bf16* dy, ls_bf16* dx2, const ls_block_grads* g, int accumulate, void* workspace,
               size_t workspace_bytes, void* stream) {
  if (int e = check_cfg(cfg)) return e;
  if (!w || !g) return fail(LS_ERR_NULL, "weights or grads is NULL");
  const Dims m = dims_of(*cfg);
  const size_t act = (size_t)(m.T * m.H * 2);
  std::vector<Range> in{{x2, act, "x2"}, {mlp_saved, mlp_saved_layout(m).total, "mlp_saved"}, {dy, act, "dy"}};
  std::vector<Range> out{{dx2, act, "dx2"}, {workspace, workspace_bytes, "workspace"}};
  weight_ranges(m, w, false, true, in);
  grad_ranges(m, g, false, true, out);
  if (int e = check_ranges(in, out)) return e;
  if (workspace_bytes < mlp_ws_layout(m).total)
    return fail(LS_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, mlp_ws_layout(m).total);
  return run_mlp_bwd(*cfg, m, (const bf16_t*)x2, w, mlp_saved, (const bf16_t*)dy, (bf16_t*)dx2, g, accumulate != 0,
                     workspace, (hipStream_t)stream);
}

int ls_block_fwd_bwd(const ls_block_cfg* cfg, const ls_bf16* x, const ls_block_weights* w, const ls_bf16* dy,
                     ls_bf16* y, ls_bf16* dx, const ls_block_grads* g, int accumulate, void* workspace,
                     size_t workspace_bytes, void* stream) {
  if (int e = check_cfg(cfg)) return e;
  if (!w || !g) return fail(LS_ERR_NULL, "weights or grads is NULL");
  const Dims m = dims_of(*cfg);
  const size_t act = (size_t)(m.T * m.H * 2);
  const BlockWs bl = block_ws_layout(m);
  std::vector<Range> in{{x, act, "x"}, {dy, act, "dy"}};
  std::vector<Range> out{{y, act, "y"}, {dx, act, "dx"}, {workspace, workspace_bytes, "workspace"}};
  weight_ranges(m, w, true, true, in);
  grad_ranges(m, g, true, true, out);
  if (int e = check_ranges(in, out)) return e;
  if (workspace_bytes < bl.total)
    return fail(LS_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, bl.total);
  const hipStream_t st = (hipStream_t)stream;
  void* asv = at<char>(workspace, bl.attn_saved);
  void* msv = at<char>(workspace, bl.mlp_saved);
  bf16_t* x2 = at<bf16_t>(workspace, bl.x2);
  bf16_t* dx2 = at<bf16_t>(workspace, bl.dx2);
  void* scratch = at<char>(workspace, bl.scratch);
  const int acc = accumulate != 0;
  if (int e = run_attn_fwd(*cfg, m, (const bf16_t*)x, w, x2, asv, scratch, st)) return e;
  if (int e = run_mlp_fwd(*cfg, m, x2, w, (bf16_t*)y, msv, st)) return e;
  if (int e = run_mlp_bwd(*cfg, m, x2, w, msv, (const bf16_t*)dy, dx2, g, acc, scratch, st)) return e;
  return run_attn_bwd(*cfg, m, (const bf16_t*)x, w, asv, dx2, (bf16_t*)dx, g, acc, scratch, st);
}

int ls_timing_begin(const char* label, int max_launches) {
  if (!label) return fail(LS_ERR_NULL, "label is NULL");
  if (max_launches <= 0 || max_launches > 100000) return fail(LS_ERR_SHAPE, "max_launches out of range");
  std::lock_guard<std::mutex> lk(g_timing.mu);
  for (hipEvent_t e : g_timing.ev) (void)hipEventDestroy(e);
  g_timing.ev.clear();
  g_timing.armed = false;
  for (int i = 0; i < 2 * max_launches; ++i) {
    hipEvent_t e;
    hipError_t r = hipEventCreate(&e);
    if (r != hipSuccess) {
      for (hipEvent_t x : g_timing.ev) (void)hipEventDestroy(x);
      g_timing.ev.clear();
      return hip_fail(r, "hipEventCreate");
    }
    g_timing.ev.push_back(e);
  }
  g_timing.label = label;
  g_timing.used = 0;
  g_timing.armed = true;
  return LS_OK;
}

int ls_timing_end(int* launches, float* mean_ms) {
  if (!launches || !mean_ms) return fail(LS_ERR_NULL, "output pointer is NULL");
  std::lock_guard<std::mutex> lk(g_timing.mu);
  g_timing.armed = false;
  double total = 0.0;
  int n = g_timing.used;
  int rc = LS_OK;
  for (int i = 0; i < n && rc == LS_OK; ++i) {
    float ms = 0.f;
    hipError_t r = hipEventSynchronize(g_timing.ev[2 * i + 1]);
    if (r == hipSuccess) r = hipEventElapsedTime(&ms, g_timing.ev[2 * i], g_timing.ev[2 * i + 1]);
    if (r != hipSuccess) rc = hip_fail(r, "timing events");
    total += ms;
  }
  for (hipEvent_t e : g_timing.ev) (void)hipEventDestroy(e);
  g_timing.ev.clear();
  g_timing.used = 0;
  *launches = n;
  *mean_ms = n ? (float)(total / n) : 0.f;
  return rc;
}

// ---- single-kernel entry points ------------------------------------------------------

static int check_core_cfg(const ls_block_cfg* cfg) {
  if (int e = check_cfg(cfg)) return e;
  if (cfg->head_dim != 64 && cfg->head_dim != 128)
    return fail(LS_ERR_UNSUPPORTED, "the attention core takes head_dim 64 or 128 (got %d)", cfg->head_dim);
  return LS_OK;
}

int ls_attn_core_fwd(const ls_block_cfg* cfg, const ls_bf16* qkv, ls_bf16* o, float* lse, void* stream) {
  if (int e = check_core_cfg(cfg)) return e;
  const Dims m = dims_of(*cfg);
  std::vector<Range> in{{qkv, (size_t)(m.T * m.Dqkv * 2), "qkv"}};
  std::vector<Range> out{{o, (size_t)(m.T * m.Dq * 2), "o"}, {lse, (size_t)(m.B * m.nq * m.S * 4), "lse"}};
  if (int e = check_ranges(in, out)) return e;
  LS_HIP(ls::attn_fwd(attn_shape(m), (const bf16_t*)qkv, (bf16_t*)o, lse, (hipStream_t)stream), "attention forward");
  return LS_OK;
}

size_t ls_attn_core_bwd_workspace(const ls_block_cfg* cfg) {
  if (check_core_cfg(cfg)) return 0;
  return ls::attn_bwd_workspace(attn_shape(dims_of(*cfg)));
}

int ls_attn_core_bwd(const ls_block_cfg* cfg, const ls_bf16* qkv, const ls_bf16* o, const float* lse,
                     const ls_bf16* dout, ls_bf16* dqkv, void* workspace, size_t workspace_bytes, void* stream) {
  if (int e = check_core_cfg(cfg)) return e;
  const Dims m = dims_of(*cfg);
  const size_t need = ls::attn_bwd_workspace(attn_shape(m));
  std::vector<Range> in{{qkv, (size_t)(m.T * m.Dqkv * 2), "qkv"},
                        {o, (size_t)(m.T * m.Dq * 2), "o"},
                        {lse, (size_t)(m.B * m.nq * m.S * 4), "lse"},
                        {dout, (size_t)(m.T * m.Dq * 2), "dout"}};
  std::vector<Range> out{{dqkv, (size_t)(m.T * m.Dqkv * 2), "dqkv"}, {workspace, workspace_bytes, "workspace"}};
  if (int e = check_ranges(in, out)) return e;
  if (workspace_bytes < need) return fail(LS_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, need);
  LS_HIP(ls::attn_bwd(attn_shape(m), (const bf16_t*)qkv, (const bf16_t*)o, lse, (const bf16_t*)dout, (bf16_t*)dqkv,
                      nullptr, workspace, (hipStream_t)stream),
         "attention backward");
  return LS_OK;
}

// ---- attention-core backward with library-owned scratch ----------------------------
//
// ls_attn_core_bwd_noalloc runs the kernels of ls_attn_core_bwd with their
// scratch (D, the base-2 log-sum-exp and, when the dK/dV group is split, the
// partial dK | dV rows) in this file-scope device array instead of a
// caller-provided workspace.  Every GPU the library runs on holds its own
// copy until the process ends.  In host code `scratch` names a host-side
// stand-in, not device memory: its device address is looked up once per
// device (hipGetSymbolAddress with that device current) and only that address
// is handed to kernels.  The kernels write every scratch value before they
// read it, so nothing is cleared between calls.
static __device__ __align__(256) unsigned char scratch[LS_ATTN_CORE_BWD_NOALLOC_SCRATCH];

static constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_addr[kMaxDevices] = {};

// Device address of `scratch` on the current device (looked up on the first
// call on each device).
static int scratch_address(void** out) {
  int dev = -1;
  LS_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(LS_ERR_UNSUPPORTED, "device index %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    LS_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (!p) return fail(LS_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return LS_OK;
}

int ls_attn_core_bwd_noalloc(const ls_block_cfg* cfg, const ls_bf16* qkv, const ls_bf16* o, const float* lse,
                             const ls_bf16* dout, ls_bf16* dqkv, void* stream) {
  if (int e = check_core_cfg(cfg)) return e;
  const Dims m = dims_of(*cfg);
  const size_t need = ls::attn_bwd_workspace(attn_shape(m));
  // fixed arrays: this entry point allocates nothing, on the host either
  const Range in[] = {{qkv, (size_t)(m.T * m.Dqkv * 2), "qkv"},
                      {o, (size_t)(m.T * m.Dq * 2), "o"},
                      {lse, (size_t)(m.B * m.nq * m.S * 4), "lse"},
                      {dout, (size_t)(m.T * m.Dq * 2), "dout"}};
  const Range out[] = {{dqkv, (size_t)(m.T * m.Dqkv * 2), "dqkv"}};
  if (int e = check_ranges(in, 4, out, 1)) return e;
  if (need > (size_t)LS_ATTN_CORE_BWD_NOALLOC_SCRATCH)
    return fail(LS_ERR_WORKSPACE,
                "this shape needs %zu bytes of scratch, beyond the library's %zu-byte array (use ls_attn_core_bwd "
                "with a workspace)",
                need, (size_t)LS_ATTN_CORE_BWD_NOALLOC_SCRATCH);
  void* ws = nullptr;
  if (int e = scratch_address(&ws)) return e;
  LS_HIP(ls::attn_bwd(attn_shape(m), (const bf16_t*)qkv, (const bf16_t*)o, lse, (const bf16_t*)dout, (bf16_t*)dqkv,
                      nullptr, ws, (hipStream_t)stream),
         "attention backward");
  return LS_OK;
}

static int check_norm_shape(int64_t rows, int32_t hidden) {
  if (rows <= 0 || hidden <= 0) return fail(LS_ERR_SHAPE, "rows and hidden must be positive");
  if (hidden % 8) return fail(LS_ERR_SHAPE, "hidden %d is not a multiple of 8", hidden);
  if (hidden > 8192) return fail(LS_ERR_UNSUPPORTED, "hidden %d exceeds 8192", hidden);
  if (rows >= ((int64_t)1 << 31)) return fail(LS_ERR_SHAPE, "too many rows");
  return LS_OK;
}

int ls_rmsnorm_fwd(int64_t rows, int32_t hidden, float eps, const ls_bf16* x, const ls_bf16* gamma, ls_bf16* h,
                   float* r, void* stream) {
  if (int e = check_norm_shape(rows, hidden)) return e;
  if (!(eps >= 0.0f)) return fail(LS_ERR_SHAPE, "eps must be >= 0");
  const size_t act = (size_t)rows * hidden * 2;
  std::vector<Range> in{{x, act, "x"}, {gamma, (size_t)hidden * 2, "gamma"}};
  std::vector<Range> out{{h, act, "h"}, {r, (size_t)rows * 4, "r"}};
  if (int e = check_ranges(in, out)) return e;
  LS_HIP(ls::rmsnorm_fwd(rows, hidden, eps, (const bf16_t*)x, (const bf16_t*)gamma, (bf16_t*)h, r, (hipStream_t)stream),
         "rmsnorm_fwd");
  return LS_OK;
}

size_t ls_rmsnorm_bwd_workspace(int64_t rows, int32_t hidden) {
  if (rows <= 0 || hidden <= 0) return 0;
  return (size_t)ls::rmsnorm_bwd_parts(rows, (int)hidden) * hidden * 4;
}

int ls_rmsnorm_bwd(int64_t rows, int32_t hidden, const ls_bf16* x, const ls_bf16* gamma, const float* r,
                   const ls_bf16* dh, const ls_bf16* dres, ls_bf16* dx, float* dgamma, int accumulate, void* workspace,
                   size_t workspace_bytes, void* stream) {
  if (int e = check_norm_shape(rows, hidden)) return e;
  const size_t act = (size_t)rows * hidden * 2;
  std::vector<Range> in{{x, act, "x"}, {gamma, (size_t)hidden * 2, "gamma"}, {r, (size_t)rows * 4, "r"}, {dh, act, "dh"}};
  if (dres) in.push_back({dres, act, "dres"});
  std::vector<Range> out{{dx, act, "dx"}, {dgamma, (size_t)hidden * 4, "dgamma"}, {workspace, workspace_bytes, "workspace"}};
  if (int e = check_ranges(in, out)) return e;
  const size_t need = ls_rmsnorm_bwd_workspace(rows, hidden);
  if (workspace_bytes < need) return fail(LS_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, need);
  LS_HIP(ls::rmsnorm_bwd(rows, hidden, (const bf16_t*)x, (const bf16_t*)gamma, r, (const bf16_t*)dh,
                         (const bf16_t*)dres, (bf16_t*)dx, dgamma, accumulate != 0, (float*)workspace,
                         (hipStream_t)stream),
         "rmsnorm_bwd");
  return LS_OK;
}

static int check_gemm(int64_t M, int64_t N, int64_t K) {
  if (M <= 0 || N <= 0 || K <= 0) return fail(LS_ERR_SHAPE, "M, N, K must be positive");
  if (M % 8 || N % 8 || K % 8) return fail(LS_ERR_SHAPE, "M, N, K must be multiples of 8");
  if (M >= (1 << 30) || N >= (1 << 30) || K >= (1 << 30)) return fail(LS_ERR_SHAPE, "dimension too large");
  if (M * K * 2 >= kMaxBytes || K * N * 2 >= kMaxBytes || M * N * 4 >= kMaxBytes)
    return fail(LS_ERR_SHAPE, "an operand reaches 2047 MiB");
  return LS_OK;
}

static int gemm_common(int64_t M, int64_t N, int64_t K, const void* A, const void* B, void* C, size_t c_elem,
                       ls::GemmArgs& g) {
  if (int e = check_gemm(M, N, K)) return e;
  std::vector<Range> in{{A, (size_t)(M * K * 2), "A"}, {B, (size_t)(K * N * 2), "B"}};
  std::vector<Range> out{{C, (size_t)(M * N) * c_elem, "C"}};
  if (int e = check_ranges(in, out)) return e;
  g.M = (int)M;
  g.N = (int)N;
  g.K = (int)K;
  g.A = (const bf16_t*)A;
  g.B[0] = (const bf16_t*)B;
  return LS_OK;
}

int ls_gemm_nt(int64_t M, int64_t N, int64_t K, const ls_bf16* A, const ls_bf16* B, ls_bf16* C, void* stream) {
  ls::GemmArgs g;
  if (int e = gemm_common(M, N, K, A, B, C, 2, g)) return e;
  g.lda = K;
  g.ldb = K;
  g.C = (bf16_t*)C;
  g.ldc = N;
  LS_HIP(ls::gemm(g, (hipStream_t)stream), "gemm_nt");
  return LS_OK;
}

int ls_gemm_nn(int64_t M, int64_t N, int64_t K, const ls_bf16* A, const ls_bf16* B, ls_bf16* C, void* stream) {
  ls::GemmArgs g;
  if (int e = gemm_common(M, N, K, A, B, C, 2, g)) return e;
  g.lda = K;
  g.ldb = N;
  g.b_kcontig = false;
  g.C = (bf16_t*)C;
  g.ldc = N;
  LS_HIP(ls::gemm(g, (hipStream_t)stream), "gemm_nn");
  return LS_OK;
}

int ls_gemm_tile_override(int32_t bm, int32_t bn) {
  if (ls::gemm_tile_override(bm, bn) != 0) return fail(LS_ERR_SHAPE, "tile sizes must be 256 or 192 (0, 0: automatic)");
  return LS_OK;
}

int ls_gemm_tn(int64_t M, int64_t N, int64_t K, const ls_bf16* A, const ls_bf16* B, float* C, int accumulate,
               void* stream) {
  ls::GemmArgs g;
  if (int e = gemm_common(M, N, K, A, B, C, 4, g)) return e;
  g.lda = M;
  g.a_kcontig = false;
  g.ldb = N;
  g.b_kcontig = false;
  g.epi = ls::EPI_F32;
  g.F[0] = C;
  g.ldf = N;
  g.accumulate = accumulate != 0;
  LS_HIP(ls::gemm(g, (hipStream_t)stream), "gemm_tn");
  return LS_OK;
}


int ls_stack_workspace(const ls_stack_cfg* cfg, size_t* bytes) {
  if (int e = check_stack_cfg(cfg)) return e;
  if (!bytes) return fail(LS_ERR_NULL, "bytes is NULL");
  *bytes = stack_ws_layout(*cfg).total;
  return LS_OK;
}

int ls_stack_fwd_bwd(const ls_stack_cfg* cfg, const int32_t* ids, const int32_t* targets, const ls_stack_weights* w,
                     float* loss, float* row_loss, const ls_stack_grads* g, int accumulate, void* workspace,
                     size_t workspace_bytes, void* stream) {
  if (int e = check_stack_cfg(cfg)) return e;
  if (!w || !g) return fail(LS_ERR_NULL, "weights or grads is NULL");
  const int L = cfg->n_layers;
  if (L > 0 && (!w->layers || !g->layers)) return fail(LS_ERR_NULL, "layer weights or grads array is NULL");
  const Dims m = dims_of(cfg->block);
  const int64_t V = cfg->vocab;
  const StackWs wl = stack_ws_layout(*cfg);
  std::vector<Range> in{{ids, (size_t)m.T * 4, "ids"},
                        {w->embed, (size_t)(V * m.H * 2), "w.embed"},
                        {w->final_norm, (size_t)m.H * 2, "w.final_norm"}};
  if (targets) in.push_back({targets, (size_t)m.T * 4, "targets"});
  std::vector<Range> out{{loss, 4, "loss"},
                         {g->embed, (size_t)(V * m.H * 4), "g.embed"},
                         {g->final_norm, (size_t)m.H * 4, "g.final_norm"},
                         {workspace, workspace_bytes, "workspace"}};
  if (row_loss) out.push_back({row_loss, (size_t)m.T * 4, "row_loss"});
  for (int l = 0; l < L; ++l) {
    weight_ranges(m, &w->layers[l], true, true, in);
    grad_ranges(m, &g->layers[l], true, true, out);
  }
  if (int e = check_ranges(in, out)) return e;
  if (workspace_bytes < wl.total) return fail(LS_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, wl.total);

  const hipStream_t st = (hipStream_t)stream;
  const ls_block_cfg& bc = cfg->block;
  const int acc = accumulate != 0;
  const size_t act = (size_t)(m.T * m.H * 2);
  const bf16_t* E = (const bf16_t*)w->embed;
  auto xs = [&](int l) { return at<bf16_t>(workspace, wl.xs + act * (size_t)l); };
  auto set = [&](int l) { return at<char>(workspace, wl.sets + wl.set_stride * (size_t)(cfg->recompute ? 0 : l)); };
  int32_t* tg = at<int32_t>(workspace, wl.tg);
  int* counts = at<int>(workspace, wl.counts);
  float* rows = row_loss ? row_loss : at<float>(workspace, wl.rows);
  bf16_t* hf = at<bf16_t>(workspace, wl.hf);
  float* rf = at<float>(workspace, wl.rf);
  bf16_t* logits = at<bf16_t>(workspace, wl.logits);
  bf16_t* dh = at<bf16_t>(workspace, wl.dh);
  bf16_t* dxa = at<bf16_t>(workspace, wl.dxa);
  bf16_t* dxb = at<bf16_t>(workspace, wl.dxb);
  bf16_t* dx2 = at<bf16_t>(workspace, wl.dx2);
  void* scratch = at<char>(workspace, wl.scratch);

  // forward: embedding, blocks (keeping every block's input), final norm
  LS_STEP("embedding fwd", st, ls::embed_fwd(m.T, (int)m.H, (int)V, ids, E, xs(0), st));
  // a block's mid-residual x2: kept per block with recomputation, else in the block's saved set
  auto x2_of = [&](int l) {
    return cfg->recompute ? at<bf16_t>(workspace, wl.xmid + act * (size_t)l) : at<bf16_t>(set(l), wl.x2);
  };
  for (int l = 0; l < L; ++l) {
    char* sv = set(l);
    if (int e = run_attn_fwd(bc, m, xs(l), &w->layers[l], x2_of(l), sv + wl.asv, scratch, st)) return e;
    if (int e = run_mlp_fwd(bc, m, x2_of(l), &w->layers[l], xs(l + 1), sv + wl.msv, st, !cfg->recompute)) return e;
  }
  LS_STEP("rmsnorm fwd", st,
          ls::rmsnorm_fwd(m.T, (int)m.H, bc.rms_eps, xs(L), (const bf16_t*)w->final_norm, hf, rf, st));

  // LM head and cross-entropy, chunk by chunk of token rows
  LS_STEP("targets", st, ls::ce_targets(m.T, (int)m.S, (int)V, ids, targets, tg, counts, st));
  const int64_t tc_max = logits_rows(*cfg);
  for (int64_t t0 = 0; t0 < m.T; t0 += tc_max) {
    const int64_t tc = std::min(tc_max, m.T - t0);
    {  // logits = h E^T
      ls::GemmArgs a;
      a.M = (int)tc;
      a.N = (int)V;
      a.K = (int)m.H;
      a.A = hf + t0 * m.H;
      a.lda = m.H;
      a.B[0] = E;
      a.ldb = m.H;
      a.epi = ls::EPI_BF16;
      a.C = logits;
      a.ldc = V;
      LS_STEP("logits", st, ls::gemm(a, st));
    }
    LS_STEP("cross-entropy", st, ls::ce_rows(tc, (int)V, logits, tg + t0, counts, rows + t0, st));
    {  // dh = dz E
      ls::GemmArgs a;
      a.M = (int)tc;
      a.N = (int)m.H;
      a.K = (int)V;
      a.A = logits;
      a.lda = V;
      a.B[0] = E;
      a.ldb = m.H;
      a.b_kcontig = false;
      a.epi = ls::EPI_BF16;
      a.C = dh + t0 * m.H;
      a.ldc = m.H;
      LS_STEP("dh head", st, ls::gemm(a, st));
    }
    {  // dE (+)= dz^T h
      ls::GemmArgs a;
      a.M = (int)V;
      a.N = (int)m.H;
      a.K = (int)tc;
      a.A = logits;
      a.lda = V;
      a.a_kcontig = false;
      a.B[0] = hf + t0 * m.H;
      a.ldb = m.H;
      a.b_kcontig = false;
      a.epi = ls::EPI_F32;
      a.F[0] = g->embed;
      a.ldf = m.H;
      a.accumulate = (t0 > 0) || acc;
      LS_STEP("dE head", st, ls::gemm(a, st));
    }
  }
  LS_STEP("loss", st, ls::ce_loss(m.T, rows, counts, loss, st));

  // backward through the final norm and the blocks, recomputing each block's
  // saved state from its input when asked to
  bf16_t* dcur = dxa;
  bf16_t* dnext = dxb;
  LS_STEP("rmsnorm bwd", st,
          ls::rmsnorm_bwd(m.T, (int)m.H, xs(L), (const bf16_t*)w->final_norm, rf, dh, nullptr, dcur, g->final_norm,
                          acc, at<float>(workspace, wl.partial), st));
  for (int l = L - 1; l >= 0; --l) {
    char* sv = set(l);
    bf16_t* x2 = x2_of(l);
    if (cfg->recompute) {  // the saved state of both sub-layers; x2 and y are known
      if (int e = run_attn_fwd(bc, m, xs(l), &w->layers[l], x2, sv + wl.asv, scratch, st, false)) return e;
      if (int e = run_mlp_fwd(bc, m, x2, &w->layers[l], nullptr, sv + wl.msv, st, true, false)) return e;
    }
    if (int e = run_mlp_bwd(bc, m, x2, &w->layers[l], sv + wl.msv, dcur, dx2, &g->layers[l], acc, scratch, st))
      return e;
    if (int e = run_attn_bwd(bc, m, xs(l), &w->layers[l], sv + wl.asv, dx2, dnext, &g->layers[l], acc, scratch, st))
      return e;
    std::swap(dcur, dnext);
  }
  LS_STEP("embedding bwd", st, ls::embed_bwd(m.T, (int)m.H, (int)V, ids, dcur, g->embed, st));
  return LS_OK;
}

size_t ls_cross_entropy_workspace(int64_t tokens) { return up256((size_t)(tokens > 0 ? tokens : 0) * 4) + 256; }

int ls_cross_entropy(int64_t tokens, int32_t seq, int32_t vocab, ls_bf16* logits, const int32_t* ids,
                     const int32_t* targets, float* loss, float* row_loss, void* workspace, size_t workspace_bytes,
                     void* stream) {
  if (tokens <= 0 || seq <= 0 || vocab <= 0 || vocab % 8 != 0)
    return fail(LS_ERR_SHAPE, "tokens, seq must be positive and vocab a positive multiple of 8");
  if (tokens >= ((int64_t)1 << 31)) return fail(LS_ERR_SHAPE, "tokens (%lld) reaches 2^31", (long long)tokens);
  if (!targets && tokens % seq != 0) return fail(LS_ERR_SHAPE, "tokens (%lld) is not a multiple of seq (%d)",
                                                 (long long)tokens, seq);
  std::vector<Range> in{{ids, (size_t)tokens * 4, "ids"}};
  if (targets) in.push_back({targets, (size_t)tokens * 4, "targets"});
  std::vector<Range> out{{logits, (size_t)(tokens * vocab * 2), "logits"},
                         {loss, 4, "loss"},
                         {row_loss, (size_t)tokens * 4, "row_loss"},
                         {workspace, workspace_bytes, "workspace"}};
  if (int e = check_ranges(in, out)) return e;
  if (workspace_bytes < ls_cross_entropy_workspace(tokens))
    return fail(LS_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, ls_cross_entropy_workspace(tokens));
  const hipStream_t st = (hipStream_t)stream;
  int32_t* tg = (int32_t*)workspace;
  int* counts = at<int>(workspace, up256((size_t)tokens * 4));
  LS_HIP(ls::ce_targets(tokens, seq, vocab, ids, targets, tg, counts, st), "targets");
  LS_HIP(ls::ce_rows(tokens, vocab, (bf16_t*)logits, tg, counts, row_loss, st), "cross-entropy");
  LS_HIP(ls::ce_loss(tokens, row_loss, counts, loss, st), "loss");
  return LS_OK;
}

int ls_embed_fwd(int64_t tokens, int32_t hidden, int32_t vocab, const int32_t* ids, const ls_bf16* embed, ls_bf16* x,
                 void* stream) {
  if (tokens <= 0 || hidden <= 0 || hidden % 8 != 0 || vocab <= 0)
    return fail(LS_ERR_SHAPE, "tokens, vocab must be positive and hidden a positive multiple of 8");
  std::vector<Range> in{{ids, (size_t)tokens * 4, "ids"}, {embed, (size_t)vocab * hidden * 2, "embed"}};
  std::vector<Range> out{{x, (size_t)(tokens * hidden * 2), "x"}};
  if (int e = check_ranges(in, out)) return e;
  LS_HIP(ls::embed_fwd(tokens, hidden, vocab, ids, (const bf16_t*)embed, (bf16_t*)x, (hipStream_t)stream),
         "embedding fwd");
  return LS_OK;
}

int ls_embed_bwd(int64_t tokens, int32_t hidden, int32_t vocab, const int32_t* ids, const ls_bf16* dx, float* d_embed,
                 void* stream) {
  if (tokens <= 0 || hidden <= 0 || hidden % 8 != 0 || vocab <= 0)
    return fail(LS_ERR_SHAPE, "tokens, vocab must be positive and hidden a positive multiple of 8");
  if (hidden > 8192) return fail(LS_ERR_UNSUPPORTED, "hidden %d exceeds 8192", hidden);
  if (tokens >= ((int64_t)1 << 31)) return fail(LS_ERR_SHAPE, "tokens (%lld) reaches 2^31", (long long)tokens);
  std::vector<Range> in{{ids, (size_t)tokens * 4, "ids"}, {dx, (size_t)(tokens * hidden * 2), "dx"}};
  std::vector<Range> out{{d_embed, (size_t)vocab * hidden * 4, "d_embed"}};
  if (int e = check_ranges(in, out)) return e;
  LS_HIP(ls::embed_bwd(tokens, hidden, vocab, ids, (const bf16_t*)dx, d_embed, (hipStream_t)stream), "embedding bwd");
  return LS_OK;
}


size_t ls_adamw_workspace(void) { return ls::adamw_workspace(); }

int ls_adamw_step(int64_t n, int64_t n_decay, const ls_adamw_cfg* cfg, float* master, ls_bf16* param,
                  const float* grad, float* m, float* v, float* grad_norm, void* workspace, size_t workspace_bytes,
                  void* stream) {
  if (!cfg) return fail(LS_ERR_NULL, "cfg is NULL");
  if (n <= 0 || n_decay < 0 || n_decay > n)
    return fail(LS_ERR_SHAPE, "need n > 0 and 0 <= n_decay <= n (n = %lld, n_decay = %lld)", (long long)n,
                (long long)n_decay);
  if (cfg->step < 1) return fail(LS_ERR_SHAPE, "step must be >= 1 (got %d)", cfg->step);
  if (!(cfg->beta1 >= 0.f && cfg->beta1 < 1.f) || !(cfg->beta2 >= 0.f && cfg->beta2 < 1.f) || !(cfg->eps > 0.f) ||
      !(cfg->lr >= 0.f) || !(cfg->weight_decay >= 0.f) || !(cfg->lr * cfg->weight_decay < 1.f) ||
      !(cfg->max_norm == cfg->max_norm))
    return fail(LS_ERR_SHAPE, "hyper-parameters out of range (0 <= beta < 1, eps > 0, lr >= 0, 0 <= lr*wd < 1)");
  const size_t f4 = (size_t)n * 4;
  std::vector<Range> in{{grad, f4, "grad"}};
  std::vector<Range> out{{master, f4, "master"}, {m, f4, "m"}, {v, f4, "v"}, {workspace, workspace_bytes, "workspace"}};
  if (param) out.push_back({param, (size_t)n * 2, "param"});
  if (grad_norm) out.push_back({grad_norm, 4, "grad_norm"});
  if (int e = check_ranges(in, out)) return e;
  if (workspace_bytes < ls::adamw_workspace())
    return fail(LS_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, ls::adamw_workspace());
  ls::AdamwHyper h{cfg->lr, cfg->beta1, cfg->beta2, cfg->eps, cfg->weight_decay, cfg->max_norm, cfg->step};
  const hipStream_t st = (hipStream_t)stream;
  LS_STEP("adamw", st, ls::adamw_step(n, n_decay, h, master, (bf16_t*)param, grad, m, v, grad_norm, workspace, st));
  return LS_OK;
}

}  // extern "C"
