// Token embedding (row gather and its deterministic scatter-add backward) and the softmax
// cross-entropy over rows of vocabulary logits, with its gradient written in
// place of the logits.
//
// All of these are bound by HBM bandwidth.  A cross-entropy row of V bf16
// logits is read once into the registers of one 1024-thread workgroup (up to
// 131072 entries; 16 bytes per thread and step), reduced to its max and
// sum-exp, and overwritten once with the gradient; larger vocabularies stream
// the row twice.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace ls {

namespace {

constexpr uint32_t kNan2 = 0x7fc07fc0u;  // two bf16 quiet NaNs
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int CE_THREADS = 1024;
constexpr int CE_WAVES = CE_THREADS / 64;

// x[t] = E[ids[t]]: one wave per row, 16-byte copies.  An id outside [0, V)
// writes a row of NaN (no read outside E).
__global__ __launch_bounds__(256) void embed_fwd_kernel(int64_t T, int H, int V, const int32_t* __restrict__ ids,
                                                        const bf16_t* __restrict__ E, bf16_t* __restrict__ x) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const int id = ids[t];
  const bool ok = id >= 0 && id < V;
  const u32x4* src = (const u32x4*)(E + (int64_t)(ok ? id : 0) * H);
  u32x4* dst = (u32x4*)(x + t * H);
  const u32x4 nan4{kNan2, kNan2, kNan2, kNan2};
  for (int c = lane; c < H / 8; c += 64) dst[c] = ok ? src[c] : nan4;
}

// dE[ids[t]] += dx[t], deterministically: workgroup t handles token t, and
// only if t is the first occurrence of its id; it then sums the dx rows of
// every occurrence in increasing token order and adds the sum into the id's
// row with one plain read-modify-write (no other workgroup touches that row).
// Occurrences are found by comparing ids 64 at a time (a ballot per wave), so
// the scan costs O(T) id reads per token, all L2-resident.  Rows with an id
// outside [0, V) are skipped.  hidden <= 8192.
constexpr int EMB_THREADS = 256;
constexpr int EMB_CHUNKS = 4;  // 8-column chunks per thread (hidden / 8 <= 4 * 256)

__global__ __launch_bounds__(EMB_THREADS) void embed_bwd_kernel(int64_t T, int H, int V,
                                                               const int32_t* __restrict__ ids,
                                                               const bf16_t* __restrict__ dx,
                                                               float* __restrict__ dE) {
  __shared__ unsigned long long match[EMB_THREADS / 64];
  const int64_t t = blockIdx.x;
  const int id = ids[t];
  if (id < 0 || id >= V) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // an earlier occurrence owns the row
  int earlier = 0;
  for (int64_t j = tid; j < t; j += EMB_THREADS) earlier |= ids[j] == id;
  if (__syncthreads_or(earlier)) return;
  const int nch = H / 8;
  float acc[EMB_CHUNKS][8];
#pragma unroll
  for (int r = 0; r < EMB_CHUNKS; ++r) {
    const int c = tid + EMB_THREADS * r;
    u32x4 w = c < nch ? *(const u32x4*)(dx + t * H + 8 * c) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[r][2 * e] = bf_lo(w[e]);
      acc[r][2 * e + 1] = bf_hi(w[e]);
    }
  }
  // later occurrences, 256 ids per round, added in token order
  for (int64_t j0 = t + 1; j0 < T; j0 += EMB_THREADS) {
    const int64_t j = j0 + tid;
    const unsigned long long m = __ballot(j < T && ids[j] == id);
    if (lane == 0) match[wave] = m;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < EMB_THREADS / 64; ++w) {
      unsigned long long mw = match[w];
      while (mw) {
        const int b = __builtin_ctzll(mw);
        mw &= mw - 1;
        const int64_t row = j0 + 64 * w + b;
#pragma unroll
        for (int r = 0; r < EMB_CHUNKS; ++r) {
          const int c = tid + EMB_THREADS * r;
          if (c >= nch) continue;
          const u32x4 x = *(const u32x4*)(dx + row * H + 8 * c);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[r][2 * e] += bf_lo(x[e]);
            acc[r][2 * e + 1] += bf_hi(x[e]);
          }
        }
      }
    }
    __syncthreads();
  }
  float* dst = dE + (int64_t)id * H;
#pragma unroll
  for (int r = 0; r < EMB_CHUNKS; ++r) {
    const int c = tid + EMB_THREADS * r;
    if (c >= nch) continue;
    f32x4* d4 = (f32x4*)(dst + 8 * c);
    const f32x4 a = d4[0], b = d4[1];
    d4[0] = f32x4{a[0] + acc[r][0], a[1] + acc[r][1], a[2] + acc[r][2], a[3] + acc[r][3]};
    d4[1] = f32x4{b[0] + acc[r][4], b[1] + acc[r][5], b[2] + acc[r][6], b[3] + acc[r][7]};
  }
}

// One workgroup: tg[t] = targets[t] if given, else the next token of the same
// sequence (ids[t+1]) or -1 at a sequence's last position; counts[0] = number
// of rows whose target lies in [0, V).
__global__ __launch_bounds__(CE_THREADS) void ce_targets_kernel(int64_t T, int S, int V,
                                                                const int32_t* __restrict__ ids,
                                                                const int32_t* __restrict__ targets,
                                                                int32_t* __restrict__ tg, int* __restrict__ counts) {
  __shared__ int part[CE_WAVES];
  int n = 0;
  for (int64_t t = threadIdx.x; t < T; t += CE_THREADS) {
    const int g = targets ? targets[t] : ((t % S) != S - 1 ? ids[t + 1] : -1);
    tg[t] = g;
    n += (g >= 0 && g < V) ? 1 : 0;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) n += __shfl_xor(n, o);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = n;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int w = 0; w < CE_WAVES; ++w) s += part[w];
    counts[0] = s;
  }
}

LS_DEV float block_max(float v, float* red) {
  v = wave_max(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float m = red[0];
#pragma unroll
  for (int w = 1; w < CE_WAVES; ++w) m = fmaxf(m, red[w]);
  __syncthreads();
  return m;
}

LS_DEV float block_sum(float v, float* red) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < CE_WAVES; ++w) s += red[w];
  __syncthreads();
  return s;
}

// Row `blockIdx.x` of z [rows, V] (bf16): lse = ln sum exp z; row_loss = lse -
// z[target]; z is overwritten with dz = (softmax(z) - onehot(target)) / n,
// n = max(counts[0], 1).  Target -1: loss 0 and dz = 0.  A target outside
// [-1, V): loss and dz NaN.  NV > 0: each thread holds NV 16-byte vectors of
// the row in registers (V <= NV * 8 * 1024); NV = 0: two streaming passes.
template <int NV>
__global__ __launch_bounds__(CE_THREADS) void ce_rows_kernel(int V, bf16_t* __restrict__ z,
                                                             const int32_t* __restrict__ tg,
                                                             const int* __restrict__ counts,
                                                             float* __restrict__ row_loss) {
  __shared__ float red[CE_WAVES];
  const int64_t row = blockIdx.x;
  bf16_t* zr = z + row * (int64_t)V;
  u32x4* zv = (u32x4*)zr;
  const int nvec = V / 8;
  const int g = tg[row];
  const int tid = threadIdx.x;
  if (g == -1) {
    const u32x4 zero{0u, 0u, 0u, 0u};
    for (int c = tid; c < nvec; c += CE_THREADS) zv[c] = zero;
    if (tid == 0) row_loss[row] = 0.f;
    return;
  }
  const bool bad = g < -1 || g >= V;
  // max
  float m = -INFINITY;
  u32x4 v[NV > 0 ? NV : 1];
  if constexpr (NV > 0) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = tid + CE_THREADS * i;
      v[i] = c < nvec ? zv[c] : u32x4{0xff80ff80u, 0xff80ff80u, 0xff80ff80u, 0xff80ff80u};
#pragma unroll
      for (int e = 0; e < 4; ++e) m = fmaxf(m, fmaxf(bf_lo(v[i][e]), bf_hi(v[i][e])));
    }
  } else {
    for (int c = tid; c < nvec; c += CE_THREADS) {
      const u32x4 w = zv[c];
#pragma unroll
      for (int e = 0; e < 4; ++e) m = fmaxf(m, fmaxf(bf_lo(w[e]), bf_hi(w[e])));
    }
  }
  m = block_max(m, red);
  const float mb = m * kLog2e;
  // keep only the packed row live between the passes (its fp32 values would
  // not fit in the registers of a 1024-thread workgroup)
  if constexpr (NV > 0) {
#pragma unroll
    for (int i = 0; i < NV; ++i) asm volatile("" : "+v"(v[i]));
  }
  // sum of exp(z - m)
  float s = 0.f;
  if constexpr (NV > 0) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      if (tid + CE_THREADS * i >= nvec) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        s += exp2f(fmaf(bf_lo(v[i][e]), kLog2e, -mb)) + exp2f(fmaf(bf_hi(v[i][e]), kLog2e, -mb));
    }
  } else {
    for (int c = tid; c < nvec; c += CE_THREADS) {
      const u32x4 w = zv[c];
#pragma unroll
      for (int e = 0; e < 4; ++e) s += exp2f(fmaf(bf_lo(w[e]), kLog2e, -mb)) + exp2f(fmaf(bf_hi(w[e]), kLog2e, -mb));
    }
  }
  s = block_sum(s, red);
  if constexpr (NV > 0) {
#pragma unroll
    for (int i = 0; i < NV; ++i) asm volatile("" : "+v"(v[i]));
  }
  // log2 of the normaliser in base-2 units: p = exp2(z log2e - lb)
  const float lb = mb + __log2f(s);
  const float inv_n = 1.0f / (float)max(counts[0], 1);
  // the thread holding z[target] writes the row's loss
  if (bad && tid == 0) row_loss[row] = NAN;
  auto grad = [&](u32x4 w, int c) {
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int k = 8 * c + 2 * e;
      if (k == g) row_loss[row] = lb * kLn2 - bf_lo(w[e]);
      if (k + 1 == g) row_loss[row] = lb * kLn2 - bf_hi(w[e]);
      float a = exp2f(fmaf(bf_lo(w[e]), kLog2e, -lb)) - (k == g ? 1.f : 0.f);
      float b = exp2f(fmaf(bf_hi(w[e]), kLog2e, -lb)) - (k + 1 == g ? 1.f : 0.f);
      o[e] = bad ? kNan2 : pack_bf2(a * inv_n, b * inv_n);
    }
    return o;
  };
  if constexpr (NV > 0) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = tid + CE_THREADS * i;
      if (c < nvec) zv[c] = grad(v[i], c);
    }
  } else {
    for (int c = tid; c < nvec; c += CE_THREADS) zv[c] = grad(zv[c], c);
  }
}

// One workgroup: loss = sum(row_loss) / max(counts[0], 1), summed in fp64 in a
// fixed order (deterministic).
__global__ __launch_bounds__(CE_THREADS) void ce_loss_kernel(int64_t T, const float* __restrict__ row_loss,
                                                             const int* __restrict__ counts, float* __restrict__ loss) {
  __shared__ double part[CE_WAVES];
  double acc = 0.0;
  for (int64_t t = threadIdx.x; t < T; t += CE_THREADS) acc += (double)row_loss[t];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int w = 0; w < CE_WAVES; ++w) s += part[w];
    loss[0] = (float)(s / (double)max(counts[0], 1));
  }
}

}  // namespace

hipError_t embed_fwd(int64_t T, int H, int V, const int32_t* ids, const bf16_t* E, bf16_t* x, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  embed_fwd_kernel<<<dim3((unsigned)((T + 3) / 4)), dim3(256), 0, s>>>(T, H, V, ids, E, x);
  return hipGetLastError();
}

hipError_t embed_bwd(int64_t T, int H, int V, const int32_t* ids, const bf16_t* dx, float* dE, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (H % 8 != 0 || H / 8 > EMB_CHUNKS * EMB_THREADS || T >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  embed_bwd_kernel<<<dim3((unsigned)T), dim3(EMB_THREADS), 0, s>>>(T, H, V, ids, dx, dE);
  return hipGetLastError();
}

hipError_t ce_targets(int64_t T, int S, int V, const int32_t* ids, const int32_t* targets, int32_t* tg, int* counts,
                      hipStream_t s) {
  ce_targets_kernel<<<dim3(1), dim3(CE_THREADS), 0, s>>>(T, S, V, ids, targets, tg, counts);
  return hipGetLastError();
}

hipError_t ce_rows(int64_t rows, int V, bf16_t* z, const int32_t* tg, const int* counts, float* row_loss,
                   hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int nvec = V / 8;
  const int nv = (nvec + CE_THREADS - 1) / CE_THREADS;
  const dim3 grid((unsigned)rows), block(CE_THREADS);
  if (nv <= 1) ce_rows_kernel<1><<<grid, block, 0, s>>>(V, z, tg, counts, row_loss);
  else if (nv <= 2) ce_rows_kernel<2><<<grid, block, 0, s>>>(V, z, tg, counts, row_loss);
  else if (nv <= 4) ce_rows_kernel<4><<<grid, block, 0, s>>>(V, z, tg, counts, row_loss);
  else if (nv <= 8) ce_rows_kernel<8><<<grid, block, 0, s>>>(V, z, tg, counts, row_loss);
  else if (nv <= 16) ce_rows_kernel<16><<<grid, block, 0, s>>>(V, z, tg, counts, row_loss);
  else ce_rows_kernel<0><<<grid, block, 0, s>>>(V, z, tg, counts, row_loss);
  return hipGetLastError();
}

hipError_t ce_loss(int64_t T, const float* row_loss, const int* counts, float* loss, hipStream_t s) {
  ce_loss_kernel<<<dim3(1), dim3(CE_THREADS), 0, s>>>(T, row_loss, counts, loss);
  return hipGetLastError();
}

}  // namespace ls
