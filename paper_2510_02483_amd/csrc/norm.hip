// RMSNorm forward / backward (with the residual gradient and a deterministic
// gain-gradient reduction) and the RoPE cos/sin table.
//
// These kernels are bound by HBM bandwidth: each row is read with 16-byte
// coalesced loads (one wave per row) and reduced with wave shuffles.
#include "common.h"
#include "kernels.h"

namespace ls {

namespace {

constexpr int NORM_WAVES = 4;           // forward: waves per workgroup, one row per wave
constexpr int BWD_WAVES = 8;            // backward: waves per workgroup, two rows per wave at a time
constexpr int BWD_ROWS_PER_BLOCK = 32;  // rows whose gain gradient one workgroup sums
constexpr int SUM_GROUPS = 8;           // column sum: part groups per workgroup

LS_DEV void unpack8(const u32x4 w, float f[8]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f[2 * e] = bf_lo(w[e]);
    f[2 * e + 1] = bf_hi(w[e]);
  }
}

LS_DEV u32x4 pack8(const float f[8]) {
  return u32x4{pack_bf2(f[0], f[1]), pack_bf2(f[2], f[3]), pack_bf2(f[4], f[5]), pack_bf2(f[6], f[7])};
}

// h = x * r * gamma, r = 1/sqrt(mean(x^2) + eps); CH = ceil(hidden / 512) chunks per lane.
template <int CH>
__global__ __launch_bounds__(64 * NORM_WAVES) void rmsnorm_fwd_kernel(int64_t rows, int hidden, float eps,
                                                                      const bf16_t* __restrict__ x,
                                                                      const bf16_t* __restrict__ gamma,
                                                                      bf16_t* __restrict__ h, float* __restrict__ r) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * NORM_WAVES + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int chunks = hidden / 8;
  const bf16_t* xr = x + row * hidden;
  u32x4 xv[CH];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int c = lane + 64 * i;
    xv[i] = c < chunks ? *(const u32x4*)(xr + c * 8) : u32x4{0u, 0u, 0u, 0u};
    float f[8];
    unpack8(xv[i], f);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += f[e] * f[e];
  }
  ss = wave_sum(ss);
  const float rs = 1.0f / sqrtf(ss / (float)hidden + eps);
  if (lane == 0) r[row] = rs;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int c = lane + 64 * i;
    if (c >= chunks) continue;
    float f[8], g[8];
    unpack8(xv[i], f);
    unpack8(*(const u32x4*)(gamma + c * 8), g);
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = f[e] * rs * g[e];
    *(u32x4*)(h + row * hidden + c * 8) = pack8(f);
  }
}

// dx = dres + r*a - x*r^3*<a,x>/hidden with a = gamma*dh; per-workgroup
// partial sums of dh*x*r over its rows go to partial[blockIdx.x][hidden].
// Wave w handles rows w, w+8, w+16, w+24 of the workgroup's 32, each with all
// its loads (x, dh, dres) issued in one phase; gamma is loaded once.
template <int CH>
__global__ __launch_bounds__(64 * BWD_WAVES) void rmsnorm_bwd_kernel(int64_t rows, int hidden,
                                                                     const bf16_t* __restrict__ x,
                                                                     const bf16_t* __restrict__ gamma,
                                                                     const float* __restrict__ r,
                                                                     const bf16_t* __restrict__ dh,
                                                                     const bf16_t* __restrict__ dres,
                                                                     bf16_t* __restrict__ dx,
                                                                     float* __restrict__ partial) {
  __shared__ float red[CH * 512];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int chunks = hidden / 8;
  // Rows wider than 3072 (more than 6 chunks per lane): gamma and the
  // residual gradient are read where they are used instead of being held for
  // the whole row, so that x, dh and the gain-gradient sums fit the registers
  // (holding all five spills from 7 chunks on; past 8 chunks the wide kernel
  // below takes over).
  constexpr bool WIDE = CH > 6;
  auto gamma_chunk = [&](int c) { return c < chunks ? *(const u32x4*)(gamma + c * 8) : u32x4{0u, 0u, 0u, 0u}; };
  u32x4 gv[WIDE ? 1 : CH];
  float gsum[CH][8];
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    if constexpr (!WIDE) gv[i] = gamma_chunk(lane + 64 * i);
#pragma unroll
    for (int e = 0; e < 8; ++e) gsum[i][e] = 0.f;
  }
  const int64_t row_begin = (int64_t)blockIdx.x * BWD_ROWS_PER_BLOCK;
#pragma unroll 1
  for (int rr = wave; rr < BWD_ROWS_PER_BLOCK; rr += BWD_WAVES) {
    const int64_t row = row_begin + rr;
    if (row >= rows) break;
    const float rs = r[row];
    u32x4 xv[CH], dv[CH], rv[WIDE ? 1 : CH];
    auto dres_chunk = [&](int c) {
      return c < chunks && dres ? *(const u32x4*)(dres + row * hidden + c * 8) : u32x4{0u, 0u, 0u, 0u};
    };
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = lane + 64 * i;
      const bool in = c < chunks;
      xv[i] = in ? *(const u32x4*)(x + row * hidden + c * 8) : u32x4{0u, 0u, 0u, 0u};
      dv[i] = in ? *(const u32x4*)(dh + row * hidden + c * 8) : u32x4{0u, 0u, 0u, 0u};
      if constexpr (!WIDE) rv[i] = dres_chunk(c);
    }
    float dot = 0.f;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      float xf[8], df[8], g[8];
      unpack8(xv[i], xf);
      unpack8(dv[i], df);
      unpack8(WIDE ? gamma_chunk(lane + 64 * i) : gv[i], g);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        dot += g[e] * df[e] * xf[e];
        gsum[i][e] += df[e] * xf[e] * rs;
      }
    }
    dot = wave_sum(dot);
    const float coef = rs * rs * rs * dot / (float)hidden;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = lane + 64 * i;
      if (c >= chunks) continue;
      float xf[8], df[8], g[8], o[8], rf[8];
      unpack8(xv[i], xf);
      unpack8(dv[i], df);
      unpack8(WIDE ? gamma_chunk(c) : gv[i], g);
      unpack8(WIDE ? dres_chunk(c) : rv[i], rf);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = rf[e] + rs * g[e] * df[e] - xf[e] * coef;
      *(u32x4*)(dx + row * hidden + c * 8) = pack8(o);
    }
  }
  // combine the waves' column sums in a fixed order (deterministic)
  for (int w = 0; w < BWD_WAVES; ++w) {
    if (wave == w) {
#pragma unroll
      for (int i = 0; i < CH; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int j = (lane + 64 * i) * 8 + e;
          red[j] = w == 0 ? gsum[i][e] : red[j] + gsum[i][e];
        }
    }
    __syncthreads();
  }
  for (int j = threadIdx.x; j < hidden; j += 64 * BWD_WAVES) partial[(int64_t)blockIdx.x * hidden + j] = red[j];
}

// The same for rows of more than 8 chunks per lane (hidden > 4096): one row
// per wave, so that no gain-gradient sums are carried from row to row (with
// them the kernel above spills): each wave adds its row's dh*x*r into the
// workgroup's sums in wave order, straight from the row's registers.
template <int CH>
__global__ __launch_bounds__(64 * BWD_WAVES) void rmsnorm_bwd_wide_kernel(int64_t rows, int hidden,
                                                                          const bf16_t* __restrict__ x,
                                                                          const bf16_t* __restrict__ gamma,
                                                                          const float* __restrict__ r,
                                                                          const bf16_t* __restrict__ dh,
                                                                          const bf16_t* __restrict__ dres,
                                                                          bf16_t* __restrict__ dx,
                                                                          float* __restrict__ partial) {
  __shared__ float red[CH * 512];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int chunks = hidden / 8;
  const int64_t row = (int64_t)blockIdx.x * BWD_WAVES + wave;
  const bool valid = row < rows;
  const float rs = valid ? r[row] : 0.f;
  u32x4 xv[CH], dv[CH];
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int c = lane + 64 * i;
    const bool in = valid && c < chunks;
    xv[i] = in ? *(const u32x4*)(x + row * hidden + c * 8) : u32x4{0u, 0u, 0u, 0u};
    dv[i] = in ? *(const u32x4*)(dh + row * hidden + c * 8) : u32x4{0u, 0u, 0u, 0u};
  }
  float dot = 0.f;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int c = lane + 64 * i;
    float xf[8], df[8], g[8];
    unpack8(xv[i], xf);
    unpack8(dv[i], df);
    unpack8(c < chunks ? *(const u32x4*)(gamma + c * 8) : u32x4{0u, 0u, 0u, 0u}, g);
#pragma unroll
    for (int e = 0; e < 8; ++e) dot += g[e] * df[e] * xf[e];
  }
  dot = wave_sum(dot);
  const float coef = rs * rs * rs * dot / (float)hidden;
  if (valid) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = lane + 64 * i;
      if (c >= chunks) continue;
      float xf[8], df[8], g[8], o[8], rf[8];
      unpack8(xv[i], xf);
      unpack8(dv[i], df);
      unpack8(*(const u32x4*)(gamma + c * 8), g);
      unpack8(dres ? *(const u32x4*)(dres + row * hidden + c * 8) : u32x4{0u, 0u, 0u, 0u}, rf);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = rf[e] + rs * g[e] * df[e] - xf[e] * coef;
      *(u32x4*)(dx + row * hidden + c * 8) = pack8(o);
    }
  }
  // the workgroup's column sums, the waves' rows added in wave order (deterministic)
  for (int w = 0; w < BWD_WAVES; ++w) {
    if (wave == w) {
#pragma unroll
      for (int i = 0; i < CH; ++i) {
        float xf[8], df[8];
        unpack8(xv[i], xf);
        unpack8(dv[i], df);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int j = (lane + 64 * i) * 8 + e;
          const float v = df[e] * xf[e] * rs;
          red[j] = w == 0 ? v : red[j] + v;
        }
      }
    }
    __syncthreads();
  }
  for (int j = threadIdx.x; j < hidden; j += 64 * BWD_WAVES) partial[(int64_t)blockIdx.x * hidden + j] = red[j];
}

// dgamma[j] (+)= sum over parts of partial[p][j]: 64 columns per workgroup,
// SUM_GROUPS groups of threads sum interleaved parts, and the group sums are
// added in group order (deterministic).
__global__ __launch_bounds__(64 * SUM_GROUPS) void column_sum_kernel(int parts, int hidden,
                                                                     const float* __restrict__ partial,
                                                                     float* __restrict__ out, int accumulate) {
  __shared__ float red[SUM_GROUPS][64];
  const int c = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int j = blockIdx.x * 64 + c;
  float s = 0.f;
  if (j < hidden) {
#pragma unroll 8
    for (int p = g; p < parts; p += SUM_GROUPS) s += partial[(int64_t)p * hidden + j];
  }
  red[g][c] = s;
  __syncthreads();
  if (g == 0 && j < hidden) {
    float t = red[0][c];
#pragma unroll
    for (int k = 1; k < SUM_GROUPS; ++k) t += red[k][c];
    out[j] = accumulate ? out[j] + t : t;
  }
}

__global__ void rope_table_kernel(int seq, int head_dim, int table_dim, double theta, float* __restrict__ cs) {
  const int half = table_dim / 2;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)seq * half) return;
  const int p = (int)(idx / half), i = (int)(idx % half);
  const double ang = i < head_dim / 2 ? (double)p * pow(theta, -2.0 * (double)i / (double)head_dim) : 0.0;
  cs[idx] = (float)cos(ang);
  cs[(int64_t)seq * half + idx] = (float)sin(ang);
}

}  // namespace

hipError_t rmsnorm_fwd(int64_t rows, int hidden, float eps, const bf16_t* x, const bf16_t* gamma, bf16_t* h,
                       float* r, hipStream_t s) {
  const int ch = (hidden / 8 + 63) / 64;
  const dim3 grid((unsigned)((rows + NORM_WAVES - 1) / NORM_WAVES)), block(64 * NORM_WAVES);
#define LS_F(CHV) \
  case CHV: hipLaunchKernelGGL((rmsnorm_fwd_kernel<CHV>), grid, block, 0, s, rows, hidden, eps, x, gamma, h, r); break;
  switch (ch) {
    LS_F(1) LS_F(2) LS_F(3) LS_F(4) LS_F(5) LS_F(6) LS_F(7) LS_F(8)
    LS_F(9) LS_F(10) LS_F(11) LS_F(12) LS_F(13) LS_F(14) LS_F(15) LS_F(16)
    default: return hipErrorInvalidValue;
  }
#undef LS_F
  return hipGetLastError();
}

// More than 8 chunks per lane: one row per wave (rmsnorm_bwd_wide_kernel).
bool rmsnorm_bwd_wide(int hidden) { return (hidden / 8 + 63) / 64 > 8; }

int rmsnorm_bwd_parts(int64_t rows, int hidden) {
  const int per = rmsnorm_bwd_wide(hidden) ? BWD_WAVES : BWD_ROWS_PER_BLOCK;
  return (int)((rows + per - 1) / per);
}

hipError_t rmsnorm_bwd(int64_t rows, int hidden, const bf16_t* x, const bf16_t* gamma, const float* r,
                       const bf16_t* dh, const bf16_t* dres, bf16_t* dx, float* dgamma, int accumulate,
                       float* partial, hipStream_t s) {
  const int ch = (hidden / 8 + 63) / 64;
  const int parts = rmsnorm_bwd_parts(rows, hidden);
  const dim3 grid((unsigned)parts), block(64 * BWD_WAVES);
#define LS_B(CHV)                                                                                       \
  case CHV:                                                                                             \
    hipLaunchKernelGGL((rmsnorm_bwd_kernel<CHV>), grid, block, 0, s, rows, hidden, x, gamma, r, dh, dres, dx, \
                       partial);                                                                        \
    break;
#define LS_W(CHV)                                                                                            \
  case CHV:                                                                                                  \
    hipLaunchKernelGGL((rmsnorm_bwd_wide_kernel<CHV>), grid, block, 0, s, rows, hidden, x, gamma, r, dh, dres, dx, \
                       partial);                                                                             \
    break;
  switch (ch) {
    LS_B(1) LS_B(2) LS_B(3) LS_B(4) LS_B(5) LS_B(6) LS_B(7) LS_B(8)
    LS_W(9) LS_W(10) LS_W(11) LS_W(12) LS_W(13) LS_W(14) LS_W(15) LS_W(16)
    default: return hipErrorInvalidValue;
  }
#undef LS_B
#undef LS_W
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(column_sum_kernel, dim3((hidden + 63) / 64), dim3(64 * SUM_GROUPS), 0, s, parts, hidden,
                     (const float*)partial, dgamma, accumulate);
  return hipGetLastError();
}

hipError_t rope_table(int seq, int head_dim, double theta, float* cs, hipStream_t s, int table_dim) {
  if (table_dim == 0) table_dim = head_dim;
  const int64_t n = (int64_t)seq * (table_dim / 2);
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, seq, head_dim, table_dim,
                     theta, cs);
  return hipGetLastError();
}

}  // namespace ls
