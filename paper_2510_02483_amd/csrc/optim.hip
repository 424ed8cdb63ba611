// One optimizer step over flat fp32 arrays: the global L2 norm of the
// gradients, the clip coefficient min(1, max_norm / (norm + 1e-6)), and AdamW
// with decoupled weight decay on the first n_decay parameters, writing the
// fp32 master weights, both moments and a bf16 copy of the weights.
//
// Bound by HBM bandwidth: the norm pass reads 4 bytes per parameter, the
// update reads 16 (master, gradient, m, v) and writes 14 (master, m, v, bf16).
// Both passes use 16-byte accesses in grid-stride loops over a fixed grid, and
// the norm is summed in fp64 in a fixed order (deterministic).
#include <math.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace ls {

namespace {

constexpr int OPT_THREADS = 256;
constexpr int NORM_BLOCKS = 2048;  // partial sums of the norm pass (fixed: the sum order does not depend on n)

// partial[b] = sum of g^2 over the elements block b visits (fp64).
__global__ __launch_bounds__(OPT_THREADS) void sumsq_kernel(int64_t n, const float* __restrict__ g,
                                                           double* __restrict__ partial) {
  __shared__ double red[OPT_THREADS / 64];
  const int64_t nv = n / 4;
  const int64_t stride = (int64_t)gridDim.x * OPT_THREADS;
  const int64_t t0 = (int64_t)blockIdx.x * OPT_THREADS + threadIdx.x;
  double acc = 0.0;
  const f32x4* g4 = (const f32x4*)g;
  for (int64_t i = t0; i < nv; i += stride) {
    const f32x4 x = __builtin_nontemporal_load(g4 + i);
    acc += (double)x[0] * x[0] + (double)x[1] * x[1] + (double)x[2] * x[2] + (double)x[3] * x[3];
  }
  for (int64_t i = 4 * nv + t0; i < n; i += stride) acc += (double)g[i] * g[i];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < OPT_THREADS / 64; ++w) s += red[w];
    partial[blockIdx.x] = s;
  }
}

// One workgroup: norm = sqrt(sum partial); scal[0] = norm, scal[1] = clip
// coefficient (1 when max_norm <= 0); norm_out (if given) = norm.
__global__ __launch_bounds__(OPT_THREADS) void clip_kernel(int parts, const double* __restrict__ partial,
                                                          float max_norm, float* __restrict__ scal,
                                                          float* __restrict__ norm_out) {
  __shared__ double red[OPT_THREADS / 64];
  double acc = 0.0;
  for (int i = threadIdx.x; i < parts; i += OPT_THREADS) acc += partial[i];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < OPT_THREADS / 64; ++w) s += red[w];
    const double norm = sqrt(s);
    const double c = max_norm > 0.f ? fmin(1.0, (double)max_norm / (norm + 1e-6)) : 1.0;
    scal[0] = (float)norm;
    scal[1] = (float)c;
    if (norm_out) norm_out[0] = (float)norm;
  }
}

struct AdamwScalars {
  float b1, b2, one_m_b1, one_m_b2, step_size, inv_sqrt_bc2, eps, decay;  // decay = 1 - lr wd
};

LS_DEV void adamw_one(float& p, float& m, float& v, float g, float c, float decay, const AdamwScalars& h) {
  g *= c;
  m = h.b1 * m + h.one_m_b1 * g;
  v = h.b2 * v + h.one_m_b2 * g * g;
  const float denom = sqrtf(v) * h.inv_sqrt_bc2 + h.eps;
  p = p * decay - h.step_size * (m / denom);
}

__global__ __launch_bounds__(OPT_THREADS) void adamw_kernel(int64_t n, int64_t n_decay, AdamwScalars h,
                                                           const float* __restrict__ scal, float* __restrict__ master,
                                                           bf16_t* __restrict__ param, const float* __restrict__ grad,
                                                           float* __restrict__ m, float* __restrict__ v) {
  const float c = scal[1];
  const int64_t nv = n / 4;
  const int64_t stride = (int64_t)gridDim.x * OPT_THREADS;
  const int64_t t0 = (int64_t)blockIdx.x * OPT_THREADS + threadIdx.x;
  f32x4* p4 = (f32x4*)master;
  const f32x4* g4 = (const f32x4*)grad;
  f32x4* m4 = (f32x4*)m;
  f32x4* v4 = (f32x4*)v;
  for (int64_t i = t0; i < nv; i += stride) {
    f32x4 p = p4[i], mm = m4[i], vv = v4[i];
    const f32x4 g = __builtin_nontemporal_load(g4 + i);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float decay = 4 * i + e < n_decay ? h.decay : 1.0f;
      float pe = p[e], me = mm[e], ve = vv[e];
      adamw_one(pe, me, ve, g[e], c, decay, h);
      p[e] = pe;
      mm[e] = me;
      vv[e] = ve;
    }
    p4[i] = p;
    m4[i] = mm;
    v4[i] = vv;
    if (param) *(u32x2*)(param + 4 * i) = u32x2{pack_bf2(p[0], p[1]), pack_bf2(p[2], p[3])};
  }
  for (int64_t i = 4 * nv + t0; i < n; i += stride) {
    float pe = master[i], me = m[i], ve = v[i];
    adamw_one(pe, me, ve, grad[i], c, i < n_decay ? h.decay : 1.0f, h);
    master[i] = pe;
    m[i] = me;
    v[i] = ve;
    if (param) param[i] = (bf16_t)f2bf(pe);
  }
}

}  // namespace

size_t adamw_workspace() { return NORM_BLOCKS * sizeof(double) + 256; }

hipError_t adamw_step(int64_t n, int64_t n_decay, const AdamwHyper& hp, float* master, bf16_t* param,
                      const float* grad, float* m, float* v, float* grad_norm, void* ws, hipStream_t s) {
  double* partial = (double*)ws;
  float* scal = (float*)((char*)ws + NORM_BLOCKS * sizeof(double));
  sumsq_kernel<<<dim3(NORM_BLOCKS), dim3(OPT_THREADS), 0, s>>>(n, grad, partial);
  clip_kernel<<<dim3(1), dim3(OPT_THREADS), 0, s>>>(NORM_BLOCKS, partial, hp.max_norm, scal, grad_norm);
  AdamwScalars h;
  h.b1 = hp.beta1;
  h.b2 = hp.beta2;
  h.one_m_b1 = (float)(1.0 - (double)hp.beta1);
  h.one_m_b2 = (float)(1.0 - (double)hp.beta2);
  const double bc1 = 1.0 - pow((double)hp.beta1, (double)hp.step);
  const double bc2 = 1.0 - pow((double)hp.beta2, (double)hp.step);
  h.step_size = (float)((double)hp.lr / bc1);
  h.inv_sqrt_bc2 = (float)(1.0 / sqrt(bc2));
  h.eps = hp.eps;
  h.decay = (float)(1.0 - (double)hp.lr * (double)hp.weight_decay);
  // a few workgroups per compute unit keep enough 16-byte loads in flight
  const int64_t nv = (n + 3) / 4;
  const int64_t blocks = std::min<int64_t>((nv + OPT_THREADS - 1) / OPT_THREADS, 256 * 16);
  adamw_kernel<<<dim3((unsigned)std::max<int64_t>(blocks, 1)), dim3(OPT_THREADS), 0, s>>>(
      n, n_decay, h, scal, master, param, grad, m, v);
  return hipGetLastError();
}

}  // namespace ls
