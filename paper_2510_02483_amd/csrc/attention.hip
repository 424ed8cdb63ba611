// Causal grouped-query attention on gfx950 matrix cores: forward with an
// online softmax over key tiles (log-sum-exp saved), backward that recomputes
// the probabilities from the log-sum-exp.
//
// Layouts: qkv is [batch*seq, (nq + 2*nkv)*d] bf16 (q heads, then k heads, then
// v heads of one token in one row), o and dout are [batch*seq, nq*d], lse and
// D are [batch, nq, seq] fp32.  Query head h reads kv head h / (nq/nkv).
//
// Forward (one workgroup = 128 query rows of one head, 4 waves x 32 rows):
// each wave computes S^T = K Q^T for a 64-key tile with the keys as MFMA rows,
// so that a lane owns one query (its running max, sum and rescale factor are
// per-lane scalars; the pair of lanes l, l+32 splits the keys) and the
// probabilities it holds are already the B operand of O^T += V^T P^T.  V is
// stored transposed in LDS ([d][key]) so the A operand reads are 8-byte LDS
// loads in the key order the probabilities arrive in.  The softmax runs in
// base 2 with the 1/sqrt(d) scale folded into one multiplier.
//
// Backward, two kernels and no atomics.  dK/dV (one workgroup = 128 keys of
// one kv head, 4 waves x 32 keys): the workgroup loops over the query heads of
// its group and over 64-row query tiles from the diagonal on; per tile it
// recomputes S = Q K^T and dP = dO V^T with keys as MFMA columns (a lane owns
// one key), forms P and dS = P (dP - D) in registers and accumulates
// dV^T += dO^T P and dK^T += Q^T dS there (the sum over the group's query heads
// happens in the same registers).  dQ (one workgroup = 128 queries of one
// head): loops over key tiles like the forward, recomputing S^T and dP^T, and
// accumulates dQ^T += K^T dS^T.  Both kernels write their gradient already
// scaled and un-rotated (inverse RoPE) in bf16.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace ls {

namespace {

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

constexpr int FWD_BQ = 128, FWD_BKV = 64;
constexpr int BWD_BKV = 128, BWD_BQ = 64;

LS_DEV u32x4 load16(const bf16_t* p) { return *(const u32x4*)p; }
LS_DEV u32x4 ld_pair8(const bf16_t* p) {  // elements p[0..3] and p[8..11]
  const u32x2 lo = *(const u32x2*)p, hi = *(const u32x2*)(p + 8);
  return u32x4{lo[0], lo[1], hi[0], hi[1]};
}
LS_DEV u32x4 pack_frag(const f32x16& v, int r0) {
  return u32x4{pack_bf2(v[r0], v[r0 + 1]), pack_bf2(v[r0 + 2], v[r0 + 3]), pack_bf2(v[r0 + 4], v[r0 + 5]),
               pack_bf2(v[r0 + 6], v[r0 + 7])};
}

// Stage rows [r0, r0 + ROWS) x columns [col, col + D) of a row-major bf16
// matrix (leading dimension ld) into LDS transposed: dst[c * PITCH + r] for
// c < D, r < ROWS.  Rows at or beyond `rows` read as zero.  8x8 blocks,
// 16-byte loads, register transpose, 16-byte LDS stores.
template <int ROWS, int D, int PITCH, int NT>
LS_DEV void stage_transposed(bf16_t* dst, const bf16_t* src, int64_t ld, int r0, int rows, int col, int tid) {
  constexpr int NB = (ROWS / 8) * (D / 8);
  for (int b = tid; b < NB; b += NT) {
    const int rb = b / (D / 8), cb = b % (D / 8);
    u32x4 in[8], t[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int r = r0 + rb * 8 + j;
      in[j] = r < rows ? load16(src + (int64_t)r * ld + col + cb * 8) : u32x4{0u, 0u, 0u, 0u};
    }
    transpose8x8(in, t);
#pragma unroll
    for (int c = 0; c < 8; ++c) *(u32x4*)&dst[(cb * 8 + c) * PITCH + rb * 8] = t[c];
  }
}

// Stage rows [r0, r0 + ROWS) x columns [col, col + D) row-major: dst[r * PITCH + c].
template <int ROWS, int D, int PITCH, int NT>
LS_DEV void stage_rows(bf16_t* dst, const bf16_t* src, int64_t ld, int r0, int rows, int col, int tid) {
  constexpr int NP = ROWS * D / 8;
  for (int c = tid; c < NP; c += NT) {
    const int r = c / (D / 8), ch = c % (D / 8);
    *(u32x4*)&dst[r * PITCH + ch * 8] =
        r0 + r < rows ? load16(src + (int64_t)(r0 + r) * ld + col + ch * 8) : u32x4{0u, 0u, 0u, 0u};
  }
}

template <int D>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(AttnShape sh, const bf16_t* __restrict__ qkv,
                                                           bf16_t* __restrict__ o, float* __restrict__ lse,
                                                           float sl2) {
  constexpr int KP = D + 8, VP = FWD_BKV + 8;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[FWD_BKV * KP];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[D * VP];

  const int S = sh.seq, nq = sh.nq, nkv = sh.nkv;
  const int nqt = (S + FWD_BQ - 1) / FWD_BQ;
  const int qt = nqt - 1 - (int)blockIdx.x;  // longest rows first
  const int h = blockIdx.y, b = blockIdx.z, kvh = h / (nq / nkv);
  const int64_t ld = (int64_t)(nq + 2 * nkv) * D;
  const bf16_t* base = qkv + (int64_t)b * S * ld;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lr = lane & 31, lh = lane >> 5;
  const int q0 = qt * FWD_BQ;
  const int qrow = q0 + 32 * wave + lr;
  const int wave_qmin = q0 + 32 * wave, wave_qmax = wave_qmin + 31;

  u32x4 qf[D / 16];
#pragma unroll
  for (int s = 0; s < D / 16; ++s)
    qf[s] = qrow < S ? load16(base + (int64_t)qrow * ld + h * D + 16 * s + 8 * lh) : u32x4{0u, 0u, 0u, 0u};

  f32x16 oacc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
  float m = -INFINITY, l = 0.f;

  const int kv_end = min(S, q0 + FWD_BQ);
  const int nkt = (kv_end + FWD_BKV - 1) / FWD_BKV;
  for (int kt = 0; kt < nkt; ++kt) {
    const int kv0 = kt * FWD_BKV;
    __syncthreads();
    stage_rows<FWD_BKV, D, KP, 256>(Ks, base, ld, kv0, S, (nq + kvh) * D, tid);
    stage_transposed<FWD_BKV, D, VP, 256>(Vt, base, ld, kv0, S, (nq + nkv + kvh) * D, tid);
    __syncthreads();
    if (kv0 > wave_qmax) continue;  // every key of the tile is in this wave's future

    f32x16 sacc[FWD_BKV / 32];
#pragma unroll
    for (int bb = 0; bb < FWD_BKV / 32; ++bb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[bb][r] = 0.f;
#pragma unroll
      for (int s = 0; s < D / 16; ++s)
        sacc[bb] = mfma32(load16(&Ks[(32 * bb + lr) * KP + 16 * s + 8 * lh]), qf[s], sacc[bb]);
    }
    // lane holds query qrow, keys kv0 + 32bb + 8(r/4) + 4lh + r%4
    const bool diag = kv0 + FWD_BKV - 1 > wave_qmin;
    float mx = -INFINITY;
#pragma unroll
    for (int bb = 0; bb < FWD_BKV / 32; ++bb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kv = kv0 + 32 * bb + 8 * (r >> 2) + 4 * lh + (r & 3);
        float t = sacc[bb][r] * sl2;
        if (diag && kv > qrow) t = -INFINITY;
        sacc[bb][r] = t;
        mx = fmaxf(mx, t);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(m, mx);
    const float alpha = exp2f(m - mnew);
    float ls = 0.f;
#pragma unroll
    for (int bb = 0; bb < FWD_BKV / 32; ++bb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2f(sacc[bb][r] - mnew);
        sacc[bb][r] = p;
        ls += p;
      }
    ls += __shfl_xor(ls, 32);
    l = l * alpha + ls;
    m = mnew;
#pragma unroll
    for (int i = 0; i < D / 32; ++i) oacc[i] *= alpha;
#pragma unroll
    for (int s = 0; s < FWD_BKV / 16; ++s) {
      const u32x4 pf = pack_frag(sacc[s >> 1], 8 * (s & 1));
#pragma unroll
      for (int i = 0; i < D / 32; ++i)
        oacc[i] = mfma32(ld_pair8(&Vt[(32 * i + lr) * VP + 16 * s + 4 * lh]), pf, oacc[i]);
    }
  }

  if (qrow < S) {
    const float inv = 1.0f / l;
    bf16_t* orow = o + ((int64_t)b * S + qrow) * nq * D + h * D;
#pragma unroll
    for (int i = 0; i < D / 32; ++i)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int d = 32 * i + 8 * rq + 4 * lh;
        *(u32x2*)(orow + d) = u32x2{pack_bf2(oacc[i][4 * rq] * inv, oacc[i][4 * rq + 1] * inv),
                                    pack_bf2(oacc[i][4 * rq + 2] * inv, oacc[i][4 * rq + 3] * inv)};
      }
    if (lh == 0) lse[((int64_t)b * nq + h) * S + qrow] = (m + log2f(l)) * LN2;
  }
}

// D[b,h,s] = <dO, O> over the head's d columns (fp32).
template <int D>
__global__ __launch_bounds__(256) void attn_bwd_pre_kernel(AttnShape sh, const bf16_t* __restrict__ o,
                                                           const bf16_t* __restrict__ dout, float* __restrict__ Dv) {
  constexpr int CPH = D / 8;  // 16-byte chunks per head
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= (int64_t)sh.batch * sh.seq) return;
  const int b = (int)(t / sh.seq), s = (int)(t % sh.seq);
  const int chunks = sh.nq * CPH;
  const bf16_t* orow = o + t * sh.nq * D;
  const bf16_t* drow = dout + t * sh.nq * D;
  for (int c0 = 0; c0 < chunks; c0 += 64) {
    const int c = c0 + lane;
    float acc = 0.f;
    if (c < chunks) {
      const u32x4 a = load16(orow + c * 8), g = load16(drow + c * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc += bf_lo(a[e]) * bf_lo(g[e]) + bf_hi(a[e]) * bf_hi(g[e]);
    }
#pragma unroll
    for (int off = CPH / 2; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
    if (c < chunks && (c % CPH) == 0) Dv[((int64_t)b * sh.nq + c / CPH) * sh.seq + s] = acc;
  }
}

// Inverse rotation of a gradient held in MFMA layout: lane holds columns
// 32i + 8(r/4) + 4lh + r%4 of one row at position `pos`; the pair partner of
// column d < D/2 is d + D/2, in register block i + D/64 of the same lane.
template <int D>
LS_DEV void unrotate_store(const f32x16 (&acc)[D / 32], float scale, const float* rope_cs, int seq, int pos, int lh,
                           bf16_t* row) {
  constexpr int HALF = D / 2, IP = HALF / 32;
#pragma unroll
  for (int i = 0; i < D / 32; ++i)
#pragma unroll
    for (int rq = 0; rq < 4; ++rq) {
      const int d = 32 * i + 8 * rq + 4 * lh;
      float out[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = acc[i][4 * rq + e] * scale;
        if (rope_cs == nullptr) {
          out[e] = x;
        } else if (i < IP) {  // first half: x1' = x1 cos + x2 sin
          const float x2 = acc[i + IP][4 * rq + e] * scale;
          const float c = rope_cs[(int64_t)pos * HALF + d + e];
          const float sn = rope_cs[(int64_t)seq * HALF + (int64_t)pos * HALF + d + e];
          out[e] = x * c + x2 * sn;
        } else {  // second half: x2' = x2 cos - x1 sin
          const float x1 = acc[i - IP][4 * rq + e] * scale;
          const int dl = d - HALF + e;
          const float c = rope_cs[(int64_t)pos * HALF + dl];
          const float sn = rope_cs[(int64_t)seq * HALF + (int64_t)pos * HALF + dl];
          out[e] = x * c - x1 * sn;
        }
      }
      *(u32x2*)(row + d) = u32x2{pack_bf2(out[0], out[1]), pack_bf2(out[2], out[3])};
    }
}

// dK and dV for 128 keys of one kv head (4 waves x 32 keys), summed over the
// query heads of the group, no atomics.
template <int D>
__global__ __launch_bounds__(256, 1) void attn_bwd_dkdv_kernel(AttnShape sh, const bf16_t* __restrict__ qkv,
                                                                const bf16_t* __restrict__ dout,
                                                                const float* __restrict__ lse,
                                                                const float* __restrict__ Dv, bf16_t* __restrict__ dqkv,
                                                                const float* __restrict__ rope_cs, float scale,
                                                                float sl2) {
  constexpr int QP = D + 8, TP = BWD_BQ + 8;
  __shared__ __attribute__((aligned(16))) bf16_t Qs[BWD_BQ * QP];
  __shared__ __attribute__((aligned(16))) bf16_t dOs[BWD_BQ * QP];
  __shared__ __attribute__((aligned(16))) bf16_t Qt[D * TP];
  __shared__ __attribute__((aligned(16))) bf16_t dOt[D * TP];
  __shared__ __attribute__((aligned(16))) float lse_s[BWD_BQ];
  __shared__ __attribute__((aligned(16))) float D_s[BWD_BQ];

  const int S = sh.seq, nq = sh.nq, nkv = sh.nkv, G = nq / nkv;
  const int kvt = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int64_t ld = (int64_t)(nq + 2 * nkv) * D;
  const int64_t ldo = (int64_t)nq * D;
  const bf16_t* base = qkv + (int64_t)b * S * ld;
  const bf16_t* dbase = dout + (int64_t)b * S * ldo;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lr = lane & 31, lh = lane >> 5;
  const int kv0 = kvt * BWD_BKV;
  const int kvrow = kv0 + 32 * wave + lr;

  u32x4 kf[D / 16], vf[D / 16];
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    const bool ok = kvrow < S;
    kf[s] = ok ? load16(base + (int64_t)kvrow * ld + (nq + kvh) * D + 16 * s + 8 * lh) : u32x4{0u, 0u, 0u, 0u};
    vf[s] = ok ? load16(base + (int64_t)kvrow * ld + (nq + nkv + kvh) * D + 16 * s + 8 * lh) : u32x4{0u, 0u, 0u, 0u};
  }

  f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[i][r] = dv[i][r] = 0.f;

  const int q_begin = (kv0 / BWD_BQ) * BWD_BQ;
  for (int g = 0; g < G; ++g) {
    const int h = kvh * G + g;
    const float* lse_h = lse + ((int64_t)b * nq + h) * S;
    const float* D_h = Dv + ((int64_t)b * nq + h) * S;
    for (int q0 = q_begin; q0 < S; q0 += BWD_BQ) {
      __syncthreads();
      stage_rows<BWD_BQ, D, QP, 256>(Qs, base, ld, q0, S, h * D, tid);
      stage_rows<BWD_BQ, D, QP, 256>(dOs, dbase, ldo, q0, S, h * D, tid);
      stage_transposed<BWD_BQ, D, TP, 256>(Qt, base, ld, q0, S, h * D, tid);
      stage_transposed<BWD_BQ, D, TP, 256>(dOt, dbase, ldo, q0, S, h * D, tid);
      if (tid < BWD_BQ) {
        const int q = q0 + tid;
        lse_s[tid] = q < S ? lse_h[q] * LOG2E : 0.f;
        D_s[tid] = q < S ? D_h[q] : 0.f;
      }
      __syncthreads();
      if (kv0 + 32 * wave > q0 + BWD_BQ - 1) continue;  // every query of the tile precedes this wave's keys

      f32x16 sacc[2], pacc[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[qb][r] = pacc[qb][r] = 0.f;
#pragma unroll
        for (int s = 0; s < D / 16; ++s) {
          sacc[qb] = mfma32(load16(&Qs[(32 * qb + lr) * QP + 16 * s + 8 * lh]), kf[s], sacc[qb]);
          pacc[qb] = mfma32(load16(&dOs[(32 * qb + lr) * QP + 16 * s + 8 * lh]), vf[s], pacc[qb]);
        }
      }
      // lane holds key kvrow, queries q0 + 32qb + 8(r/4) + 4lh + r%4
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          const int ql = 32 * qb + 8 * rq + 4 * lh;
          const f32x4 L = *(const f32x4*)&lse_s[ql];
          const f32x4 Dd = *(const f32x4*)&D_s[ql];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = 4 * rq + e, q = q0 + ql + e;
            const float p = (kvrow <= q && q < S) ? exp2f(sacc[qb][r] * sl2 - L[e]) : 0.f;
            pacc[qb][r] = p * (pacc[qb][r] - Dd[e]);
            sacc[qb][r] = p;
          }
        }
#pragma unroll
      for (int s = 0; s < BWD_BQ / 16; ++s) {
        const u32x4 pf = pack_frag(sacc[s >> 1], 8 * (s & 1));
        const u32x4 sf = pack_frag(pacc[s >> 1], 8 * (s & 1));
#pragma unroll
        for (int i = 0; i < D / 32; ++i) {
          dv[i] = mfma32(ld_pair8(&dOt[(32 * i + lr) * TP + 16 * s + 4 * lh]), pf, dv[i]);
          dk[i] = mfma32(ld_pair8(&Qt[(32 * i + lr) * TP + 16 * s + 4 * lh]), sf, dk[i]);
        }
      }
    }
  }

  // dK = scale * dS^T Q (un-rotated), dV = P^T dO.  Lane holds key kvrow.
  if (kvrow >= S) return;
  const int pos = kvrow;
  unrotate_store<D>(dk, scale, rope_cs, S, pos, lh, dqkv + ((int64_t)b * S + kvrow) * ld + (nq + kvh) * D);
  unrotate_store<D>(dv, 1.0f, nullptr, S, pos, lh, dqkv + ((int64_t)b * S + kvrow) * ld + (nq + nkv + kvh) * D);
}

// dQ for 128 queries of one head (4 waves x 32 queries): loops over the key
// tiles up to the diagonal, recomputes S^T and dP^T with keys as MFMA rows (a
// lane owns one query, as in the forward), forms dS^T in registers and
// accumulates dQ^T += K^T dS^T; K is staged row-major (for S^T) and transposed
// (for dQ^T), V row-major (for dP^T).
template <int D>
__global__ __launch_bounds__(256, 1) void attn_bwd_dq_kernel(AttnShape sh, const bf16_t* __restrict__ qkv,
                                                              const bf16_t* __restrict__ dout,
                                                              const float* __restrict__ lse,
                                                              const float* __restrict__ Dv, bf16_t* __restrict__ dqkv,
                                                              const float* __restrict__ rope_cs, float scale,
                                                              float sl2) {
  constexpr int KP = D + 8, TP = FWD_BKV + 8;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[FWD_BKV * KP];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[FWD_BKV * KP];
  __shared__ __attribute__((aligned(16))) bf16_t Kt[D * TP];

  const int S = sh.seq, nq = sh.nq, nkv = sh.nkv;
  const int nqt = (S + FWD_BQ - 1) / FWD_BQ;
  const int qt = nqt - 1 - (int)blockIdx.x;  // longest rows first
  const int h = blockIdx.y, b = blockIdx.z, kvh = h / (nq / nkv);
  const int64_t ld = (int64_t)(nq + 2 * nkv) * D;
  const int64_t ldo = (int64_t)nq * D;
  const bf16_t* base = qkv + (int64_t)b * S * ld;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lr = lane & 31, lh = lane >> 5;
  const int q0 = qt * FWD_BQ;
  const int qrow = q0 + 32 * wave + lr;
  const int wave_qmin = q0 + 32 * wave, wave_qmax = wave_qmin + 31;
  const bool qok = qrow < S;

  u32x4 qf[D / 16], df[D / 16];
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    qf[s] = qok ? load16(base + (int64_t)qrow * ld + h * D + 16 * s + 8 * lh) : u32x4{0u, 0u, 0u, 0u};
    df[s] = qok ? load16(dout + ((int64_t)b * S + qrow) * ldo + h * D + 16 * s + 8 * lh) : u32x4{0u, 0u, 0u, 0u};
  }
  const float lse2 = qok ? lse[((int64_t)b * nq + h) * S + qrow] * LOG2E : 0.f;
  const float Dq = qok ? Dv[((int64_t)b * nq + h) * S + qrow] : 0.f;

  f32x16 dq[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dq[i][r] = 0.f;

  const int kv_end = min(S, q0 + FWD_BQ);
  const int nkt = (kv_end + FWD_BKV - 1) / FWD_BKV;
  for (int kt = 0; kt < nkt; ++kt) {
    const int kv0 = kt * FWD_BKV;
    __syncthreads();
    stage_rows<FWD_BKV, D, KP, 256>(Ks, base, ld, kv0, S, (nq + kvh) * D, tid);
    stage_rows<FWD_BKV, D, KP, 256>(Vs, base, ld, kv0, S, (nq + nkv + kvh) * D, tid);
    stage_transposed<FWD_BKV, D, TP, 256>(Kt, base, ld, kv0, S, (nq + kvh) * D, tid);
    __syncthreads();
    if (kv0 > wave_qmax) continue;

    f32x16 sacc[FWD_BKV / 32], pacc[FWD_BKV / 32];
#pragma unroll
    for (int bb = 0; bb < FWD_BKV / 32; ++bb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[bb][r] = pacc[bb][r] = 0.f;
#pragma unroll
      for (int s = 0; s < D / 16; ++s) {
        sacc[bb] = mfma32(load16(&Ks[(32 * bb + lr) * KP + 16 * s + 8 * lh]), qf[s], sacc[bb]);
        pacc[bb] = mfma32(load16(&Vs[(32 * bb + lr) * KP + 16 * s + 8 * lh]), df[s], pacc[bb]);
      }
    }
    // lane holds query qrow, keys kv0 + 32bb + 8(r/4) + 4lh + r%4
#pragma unroll
    for (int bb = 0; bb < FWD_BKV / 32; ++bb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kv = kv0 + 32 * bb + 8 * (r >> 2) + 4 * lh + (r & 3);
        const float p = (kv <= qrow && kv < S) ? exp2f(sacc[bb][r] * sl2 - lse2) : 0.f;
        pacc[bb][r] = p * (pacc[bb][r] - Dq);
      }
#pragma unroll
    for (int s = 0; s < FWD_BKV / 16; ++s) {
      const u32x4 sf = pack_frag(pacc[s >> 1], 8 * (s & 1));
#pragma unroll
      for (int i = 0; i < D / 32; ++i)
        dq[i] = mfma32(ld_pair8(&Kt[(32 * i + lr) * TP + 16 * s + 4 * lh]), sf, dq[i]);
    }
  }
  if (!qok) return;
  unrotate_store<D>(dq, scale, rope_cs, S, qrow, lh, dqkv + ((int64_t)b * S + qrow) * ld + h * D);
}

template <int D>
hipError_t attn_fwd_t(const AttnShape& sh, const bf16_t* qkv, bf16_t* o, float* lse, hipStream_t s) {
  const dim3 grid((sh.seq + FWD_BQ - 1) / FWD_BQ, sh.nq, sh.batch);
  const float sl2 = LOG2E / sqrtf((float)D);
  hipLaunchKernelGGL((attn_fwd_kernel<D>), grid, dim3(256), 0, s, sh, qkv, o, lse, sl2);
  return hipGetLastError();
}

template <int D>
hipError_t attn_bwd_t(const AttnShape& sh, const bf16_t* qkv, const bf16_t* o, const float* lse, const bf16_t* dout,
                      bf16_t* dqkv, const float* rope_cs, void* ws, hipStream_t s) {
  const int64_t T = (int64_t)sh.batch * sh.seq;
  float* Dv = (float*)ws;
  hipLaunchKernelGGL((attn_bwd_pre_kernel<D>), dim3((unsigned)((T + 3) / 4)), dim3(256), 0, s, sh, o, dout, Dv);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const float scale = 1.0f / sqrtf((float)D);
  const dim3 gkv((sh.seq + BWD_BKV - 1) / BWD_BKV, sh.nkv, sh.batch);
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D>), gkv, dim3(256), 0, s, sh, qkv, dout, lse, (const float*)Dv, dqkv,
                     rope_cs, scale, scale * LOG2E);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 gq((sh.seq + FWD_BQ - 1) / FWD_BQ, sh.nq, sh.batch);
  hipLaunchKernelGGL((attn_bwd_dq_kernel<D>), gq, dim3(256), 0, s, sh, qkv, dout, lse, (const float*)Dv, dqkv,
                     rope_cs, scale, scale * LOG2E);
  return hipGetLastError();
}

}  // namespace

hipError_t attn_fwd(const AttnShape& sh, const bf16_t* qkv, bf16_t* o, float* lse, hipStream_t s) {
  if (sh.d == 128) return attn_fwd_t<128>(sh, qkv, o, lse, s);
  if (sh.d == 64) return attn_fwd_t<64>(sh, qkv, o, lse, s);
  return hipErrorInvalidValue;
}

size_t attn_bwd_workspace(const AttnShape& sh) {
  const int64_t T = (int64_t)sh.batch * sh.seq;
  return (size_t)(T * sh.nq) * sizeof(float);
}

hipError_t attn_bwd(const AttnShape& sh, const bf16_t* qkv, const bf16_t* o, const float* lse, const bf16_t* dout,
                    bf16_t* dqkv, const float* rope_cs, void* ws, hipStream_t s) {
  if (sh.d == 128) return attn_bwd_t<128>(sh, qkv, o, lse, dout, dqkv, rope_cs, ws, s);
  if (sh.d == 64) return attn_bwd_t<64>(sh, qkv, o, lse, dout, dqkv, rope_cs, ws, s);
  return hipErrorInvalidValue;
}

}  // namespace ls
