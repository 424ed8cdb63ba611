// Layout changes for head sizes that the attention kernels do not tile
// natively (64 < d < 128): each head of d features is held in a slot of dp =
// 128, its first half at slot positions 0 .. d/2-1 and its second half at
// dp/2 .. dp/2 + d/2 - 1, zeros elsewhere.  With the RoPE pairs (i, i + d/2)
// so placed at (i, i + dp/2), the 128-wide kernels rotate the right pairs, and
// the zero features add exact zeros to every product.
//
// Weights are padded into that layout (rows of Wq, Wk, Wv; columns of Wo) and
// weight gradients taken in it are folded back (with the caller's accumulate
// flag).  All of these are HBM-bound copies, four elements per thread.
#include "common.h"
#include "kernels.h"

namespace ls {

namespace {

constexpr int PAD_THREADS = 256;

// Slot of feature s (0 <= s < d) of a head.
LS_DEV int slot_of(int s, int d, int dp) { return s < d / 2 ? s : dp / 2 + (s - d / 2); }
// Feature of slot j (0 <= j < dp), or -1 for a zero slot.
LS_DEV int feature_of(int j, int d, int dp) {
  if (j < d / 2) return j;
  if (j >= dp / 2 && j < dp / 2 + d / 2) return d / 2 + (j - dp / 2);
  return -1;
}

// dst [heads*dp, cols] from src [heads*d, cols] (bf16), zero rows in the gaps.
__global__ __launch_bounds__(PAD_THREADS) void pad_rows_kernel(const bf16_t* __restrict__ src, bf16_t* __restrict__ dst,
                                                              int heads, int d, int dp, int cols) {
  const int64_t n4 = (int64_t)heads * dp * cols / 4;
  for (int64_t i = (int64_t)blockIdx.x * PAD_THREADS + threadIdx.x; i < n4; i += (int64_t)gridDim.x * PAD_THREADS) {
    const int64_t e = 4 * i;
    const int64_t row = e / cols;
    const int col = (int)(e - row * cols);
    const int h = (int)(row / dp), f = feature_of((int)(row % dp), d, dp);
    u32x2 v{0u, 0u};
    if (f >= 0) v = *(const u32x2*)(src + ((int64_t)h * d + f) * cols + col);
    *(u32x2*)(dst + e) = v;
  }
}

// dst [rows, heads*dp] from src [rows, heads*d] (bf16), zero columns in the gaps.
__global__ __launch_bounds__(PAD_THREADS) void pad_cols_kernel(const bf16_t* __restrict__ src, bf16_t* __restrict__ dst,
                                                              int rows, int heads, int d, int dp) {
  const int wd = heads * dp, ws = heads * d;
  const int64_t n4 = (int64_t)rows * wd / 4;
  for (int64_t i = (int64_t)blockIdx.x * PAD_THREADS + threadIdx.x; i < n4; i += (int64_t)gridDim.x * PAD_THREADS) {
    const int64_t e = 4 * i;
    const int64_t r = e / wd;
    const int c = (int)(e - r * wd);
    const int h = c / dp, f = feature_of(c % dp, d, dp);
    u32x2 v{0u, 0u};
    if (f >= 0) v = *(const u32x2*)(src + r * ws + (int64_t)h * d + f);
    *(u32x2*)(dst + e) = v;
  }
}

// dst [heads*d, cols] (+)= src rows in the padded layout (fp32).
__global__ __launch_bounds__(PAD_THREADS) void unpad_rows_kernel(const float* __restrict__ src, float* __restrict__ dst,
                                                                int heads, int d, int dp, int cols, int accumulate) {
  const int64_t n4 = (int64_t)heads * d * cols / 4;
  for (int64_t i = (int64_t)blockIdx.x * PAD_THREADS + threadIdx.x; i < n4; i += (int64_t)gridDim.x * PAD_THREADS) {
    const int64_t e = 4 * i;
    const int64_t row = e / cols;
    const int col = (int)(e - row * cols);
    const int h = (int)(row / d), s = (int)(row % d);
    f32x4 v = *(const f32x4*)(src + ((int64_t)h * dp + slot_of(s, d, dp)) * cols + col);
    if (accumulate) v += *(const f32x4*)(dst + e);
    *(f32x4*)(dst + e) = v;
  }
}

// dst [rows, heads*d] (+)= src columns in the padded layout (fp32).
__global__ __launch_bounds__(PAD_THREADS) void unpad_cols_kernel(const float* __restrict__ src, float* __restrict__ dst,
                                                                int rows, int heads, int d, int dp, int accumulate) {
  const int wd = heads * d, ws = heads * dp;
  const int64_t n4 = (int64_t)rows * wd / 4;
  for (int64_t i = (int64_t)blockIdx.x * PAD_THREADS + threadIdx.x; i < n4; i += (int64_t)gridDim.x * PAD_THREADS) {
    const int64_t e = 4 * i;
    const int64_t r = e / wd;
    const int c = (int)(e - r * wd);
    const int h = c / d, s = c % d;
    f32x4 v = *(const f32x4*)(src + r * ws + (int64_t)h * dp + slot_of(s, d, dp));
    if (accumulate) v += *(const f32x4*)(dst + e);
    *(f32x4*)(dst + e) = v;
  }
}

unsigned grid_for(int64_t n4) {
  const int64_t b = (n4 + PAD_THREADS - 1) / PAD_THREADS;
  return (unsigned)(b < 1 ? 1 : (b > 256 * 32 ? 256 * 32 : b));
}

}  // namespace

hipError_t pad_head_rows(const bf16_t* src, bf16_t* dst, int heads, int d, int dp, int cols, hipStream_t s) {
  pad_rows_kernel<<<grid_for((int64_t)heads * dp * cols / 4), PAD_THREADS, 0, s>>>(src, dst, heads, d, dp, cols);
  return hipGetLastError();
}

hipError_t pad_head_cols(const bf16_t* src, bf16_t* dst, int rows, int heads, int d, int dp, hipStream_t s) {
  pad_cols_kernel<<<grid_for((int64_t)rows * heads * dp / 4), PAD_THREADS, 0, s>>>(src, dst, rows, heads, d, dp);
  return hipGetLastError();
}

hipError_t unpad_head_rows(const float* src, float* dst, int heads, int d, int dp, int cols, int accumulate,
                           hipStream_t s) {
  unpad_rows_kernel<<<grid_for((int64_t)heads * d * cols / 4), PAD_THREADS, 0, s>>>(src, dst, heads, d, dp, cols,
                                                                                    accumulate);
  return hipGetLastError();
}

hipError_t unpad_head_cols(const float* src, float* dst, int rows, int heads, int d, int dp, int accumulate,
                           hipStream_t s) {
  unpad_cols_kernel<<<grid_for((int64_t)rows * heads * d / 4), PAD_THREADS, 0, s>>>(src, dst, rows, heads, d, dp,
                                                                                    accumulate);
  return hipGetLastError();
}

}  // namespace ls
