// bf16 matrix products on gfx950 matrix cores (v_mfma_f32_32x32x16_bf16) with
// fp32 accumulation and fused epilogues for the decoder block.
//
// One workgroup computes a BM x BN tile of C; its waves split the tile into
// WM x WN wave tiles of 32x32 MFMA blocks.  Operand tiles of 64 k-values are
// staged global -> registers -> LDS, double-buffered in LDS, so the global
// loads of tile k+1 are in flight while the matrix cores work on tile k.
// LDS always holds both operands k-contiguous ([row][k], rows padded by 8
// elements so the 16-byte fragment reads of 32 consecutive rows hit distinct
// banks).  An operand that is k-strided in memory (the weight-gradient and
// input-gradient products) is loaded as 8x8 blocks with coalesced 16-byte
// row loads and transposed in registers before its LDS store, so the matrix
// core loop is identical for every layout.
//
// Each MFMA takes the B fragment as its first operand and the A fragment as
// its second, so that a lane ends up holding four consecutive output columns
// of one row: 8-byte bf16 / 16-byte fp32 stores, and the RoPE and SwiGLU
// partners of a column sit in the same lane.
#include "common.h"
#include "kernels.h"

namespace ls {

namespace {

constexpr int KT = 64;           // k extent of a staged tile
constexpr int PITCH = KT + 8;    // LDS row pitch in bf16 elements (144 bytes)
constexpr int GROUP_M = 8;       // tile rows per group in the launch order
constexpr int EPI_ROPE64 = 100;  // EPI_ROPE for 64-wide heads

// Launch order: workgroups are handed to the 8 XCDs round-robin, so first
// renumber them so that each XCD receives a contiguous range of logical tiles,
// then walk the tiles in groups of GROUP_M tile rows so that the tiles an XCD
// works on at once share A rows and B columns in its L2.
LS_DEV void map_tile(int wg, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int nwg = tiles_m * tiles_n;
  const int q = nwg >> 3, r = nwg & 7, xcd = wg & 7, idx = wg >> 3;
  const int logical = (xcd < r ? xcd * (q + 1) : r * (q + 1) + (xcd - r) * q) + idx;
  const int group = GROUP_M * tiles_n;
  const int g = logical / group;
  const int first_m = g * GROUP_M;
  const int gm = min(tiles_m - first_m, GROUP_M);
  const int in_g = logical - g * group;
  tm = first_m + in_g % gm;
  tn = in_g / gm;
}

LS_DEV const bf16_t* seg_row(const GemmArgs& p, int row) {
  const int s = row >= p.b_start[2] ? 2 : (row >= p.b_start[1] ? 1 : 0);
  return p.B[s] + (int64_t)(row - p.b_start[s]) * p.ldb;
}

LS_DEV float silu_f(float g) { return g / (1.0f + __expf(-g)); }

template <int BM, int BN, int WGM, int WGN, bool AK, bool BKC, int EPI>
__global__ __launch_bounds__(64 * WGM * WGN, 1) void gemm_kernel(GemmArgs p) {
  constexpr int NT = 64 * WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int TM = WM / 32, TN = WN / 32;
  // per-thread staged 16-byte pieces of each operand tile
  constexpr int A_PIECES = BM * KT / 8 / NT;
  constexpr int B_PIECES = BN * KT / 8 / NT;
  static_assert(A_PIECES * NT * 8 == BM * KT && B_PIECES * NT * 8 == BN * KT, "tile/threads");
  static_assert(AK || A_PIECES % 8 == 0, "transposed loads move 8x8 blocks");
  static_assert(BKC || B_PIECES % 8 == 0, "transposed loads move 8x8 blocks");

  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * PITCH];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN * PITCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  int tm, tn;
  map_tile(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int K = p.K;
  const int nk = (K + KT - 1) / KT;

  // ---- operand sources (fixed for the whole k loop) ------------------------
  // k-contiguous operand: piece c covers row c/8, k-chunk c%8 of the tile.
  // k-strided operand: thread owns 8x8 blocks; block b covers k-rows
  // 8*(b / (R/8)) .. +7 and columns 8*(b % (R/8)) .. +7 of the tile.
  const bf16_t* a_src[AK ? A_PIECES : A_PIECES / 8];
  const bf16_t* b_src[BKC ? B_PIECES : 1];
  if constexpr (AK) {
#pragma unroll
    for (int i = 0; i < A_PIECES; ++i) {
      const int c = tid + i * NT, row = m0 + (c >> 3);
      a_src[i] = row < p.M ? p.A + (int64_t)row * p.lda + (c & 7) * 8 : nullptr;
    }
  } else {
#pragma unroll
    for (int i = 0; i < A_PIECES / 8; ++i) {
      const int b = tid + i * NT, col = m0 + (b % (BM / 8)) * 8;
      a_src[i] = col < p.M ? p.A + col : nullptr;
    }
  }
  if constexpr (BKC) {
#pragma unroll
    for (int i = 0; i < B_PIECES; ++i) {
      const int c = tid + i * NT, n = n0 + (c >> 3);
      const bf16_t* src = nullptr;
      if (p.glu) {
        const int blk = n >> 6, row = (blk >> 1) * 64 + (n & 63);
        if (row < p.glu_rows) src = p.B[blk & 1] + (int64_t)row * p.ldb;
      } else if (n < p.N) {
        src = seg_row(p, n);
      }
      b_src[i] = src ? src + (c & 7) * 8 : nullptr;
    }
  }

  u32x4 ra[A_PIECES], rb[B_PIECES];
  const u32x4 zero4 = {0u, 0u, 0u, 0u};

  auto load_tiles = [&](int kt) {
    const int k0 = kt * KT;
    if constexpr (AK) {
#pragma unroll
      for (int i = 0; i < A_PIECES; ++i) {
        const int c = tid + i * NT, k = k0 + (c & 7) * 8;
        ra[i] = (a_src[i] && k < K) ? *(const u32x4*)(a_src[i] + k0) : zero4;
      }
    } else {
#pragma unroll
      for (int i = 0; i < A_PIECES / 8; ++i) {
        const int b = tid + i * NT, kr = k0 + (b / (BM / 8)) * 8;
#pragma unroll
        for (int j = 0; j < 8; ++j)
          ra[i * 8 + j] = (a_src[i] && kr + j < K) ? *(const u32x4*)(a_src[i] + (int64_t)(kr + j) * p.lda) : zero4;
      }
    }
    if constexpr (BKC) {
#pragma unroll
      for (int i = 0; i < B_PIECES; ++i) {
        const int c = tid + i * NT, k = k0 + (c & 7) * 8;
        rb[i] = (b_src[i] && k < K) ? *(const u32x4*)(b_src[i] + k0) : zero4;
      }
    } else {
#pragma unroll
      for (int i = 0; i < B_PIECES / 8; ++i) {
        const int b = tid + i * NT, kr = k0 + (b / (BN / 8)) * 8, col = n0 + (b % (BN / 8)) * 8;
#pragma unroll
        for (int j = 0; j < 8; ++j)
          rb[i * 8 + j] = (col < p.N && kr + j < K) ? *(const u32x4*)(seg_row(p, kr + j) + col) : zero4;
      }
    }
  };

  auto store_tiles = [&](int buf) {
    if constexpr (AK) {
#pragma unroll
      for (int i = 0; i < A_PIECES; ++i) {
        const int c = tid + i * NT;
        *(u32x4*)&As[buf][(c >> 3) * PITCH + (c & 7) * 8] = ra[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < A_PIECES / 8; ++i) {
        const int b = tid + i * NT, kb = b / (BM / 8), mb = b % (BM / 8);
        u32x4 t[8];
        transpose8x8(&ra[i * 8], t);
#pragma unroll
        for (int c = 0; c < 8; ++c) *(u32x4*)&As[buf][(mb * 8 + c) * PITCH + kb * 8] = t[c];
      }
    }
    if constexpr (BKC) {
#pragma unroll
      for (int i = 0; i < B_PIECES; ++i) {
        const int c = tid + i * NT;
        *(u32x4*)&Bs[buf][(c >> 3) * PITCH + (c & 7) * 8] = rb[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < B_PIECES / 8; ++i) {
        const int b = tid + i * NT, kb = b / (BN / 8), nb = b % (BN / 8);
        u32x4 t[8];
        transpose8x8(&rb[i * 8], t);
#pragma unroll
        for (int c = 0; c < 8; ++c) *(u32x4*)&Bs[buf][(nb * 8 + c) * PITCH + kb * 8] = t[c];
      }
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int lr = lane & 31, lh = lane >> 5;
  const int a_row0 = wm * WM + lr, b_row0 = wn * WN + lr;

  load_tiles(0);
  store_tiles(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_tiles(kt + 1);
    const bf16_t* as = As[cur];
    const bf16_t* bs = Bs[cur];
#pragma unroll
    for (int s = 0; s < KT / 16; ++s) {
      u32x4 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = *(const u32x4*)&as[(a_row0 + 32 * i) * PITCH + 16 * s + 8 * lh];
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[j] = *(const u32x4*)&bs[(b_row0 + 32 * j) * PITCH + 16 * s + 8 * lh];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(bfr[j], af[i], acc[i][j]);
    }
    if (kt + 1 < nk) store_tiles(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: lane holds C[m][n .. n+3], m = row of the lane, n = 8q + 4*lh
  const int wn0 = n0 + wn * WN;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = m0 + wm * WM + 32 * i + lr;
    if (m >= p.M) continue;
    if constexpr (EPI == EPI_GLU_FWD) {
      static_assert(WN == 128, "gate/up interleave needs 128-column wave tiles");
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = wn0 / 2 + 32 * j + 8 * q + 4 * lh;
          if (col >= p.glu_I) continue;
          float g[4], u[4];
          uint32_t pg[2], pu[2], pa[2];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            g[e] = acc[i][j][4 * q + e];
            u[e] = acc[i][j + 2][4 * q + e];
          }
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            pg[e] = pack_bf2(g[2 * e], g[2 * e + 1]);
            pu[e] = pack_bf2(u[2 * e], u[2 * e + 1]);
            pa[e] = pack_bf2(silu_f(g[2 * e]) * u[2 * e], silu_f(g[2 * e + 1]) * u[2 * e + 1]);
          }
          bf16_t* row = p.C + (int64_t)m * p.ldc;
          *(u32x2*)(row + col) = u32x2{pg[0], pg[1]};
          *(u32x2*)(row + p.glu_I + col) = u32x2{pu[0], pu[1]};
          *(u32x2*)(p.act + (int64_t)m * p.glu_I + col) = u32x2{pa[0], pa[1]};
        }
    } else if constexpr (EPI == EPI_ROPE || EPI == EPI_ROPE64) {
      constexpr int HD = EPI == EPI_ROPE ? 128 : 64, HALF = HD / 2, JP = HALF / 32;
      static_assert(WN % HD == 0, "wave tiles hold whole heads");
      const int pos = m % p.seq;
      const float* cs = p.rope_cs + (int64_t)pos * HALF;
      const float* sn = p.rope_cs + (int64_t)p.seq * HALF + (int64_t)pos * HALF;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int nb = wn0 + 32 * j;
        if (nb >= p.N) continue;
        const bool rot = nb < p.rope_cols;
        const int dcol = (32 * j) % HD;  // wave tiles start on a head boundary
        if (rot && dcol >= HALF) continue;  // written together with its partner
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int n = nb + 8 * q + 4 * lh;
          bf16_t* out = p.C + (int64_t)m * p.ldc + n;
          if (!rot || j + JP >= TN) {
            *(u32x2*)out = u32x2{pack_bf2(acc[i][j][4 * q], acc[i][j][4 * q + 1]),
                                 pack_bf2(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3])};
            continue;
          }
          float lo[4], hi[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int dc = dcol + 8 * q + 4 * lh + e;
            const float c = cs[dc], s = sn[dc];
            const float x1 = acc[i][j][4 * q + e], x2 = acc[i][(j + JP) % TN][4 * q + e];
            lo[e] = x1 * c - x2 * s;
            hi[e] = x2 * c + x1 * s;
          }
          *(u32x2*)out = u32x2{pack_bf2(lo[0], lo[1]), pack_bf2(lo[2], lo[3])};
          *(u32x2*)(out + HALF) = u32x2{pack_bf2(hi[0], hi[1]), pack_bf2(hi[2], hi[3])};
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int n = wn0 + 32 * j + 8 * q + 4 * lh;
          if (n >= p.N) continue;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * q + e];
          if constexpr (EPI == EPI_F32) {
            const int s = m >= p.f_start[2] ? 2 : (m >= p.f_start[1] ? 1 : 0);
            float* dst = p.F[s] + (int64_t)(m - p.f_start[s]) * p.ldf + n;
            f32x4 o = {v[0], v[1], v[2], v[3]};
            if (p.accumulate) o += *(const f32x4*)dst;
            *(f32x4*)dst = o;
          } else if constexpr (EPI == EPI_GLU_BWD) {
            const bf16_t* gsrc = p.gu_in + (int64_t)m * 2 * p.glu_I + n;
            const u32x2 gw = *(const u32x2*)gsrc;
            const u32x2 uw = *(const u32x2*)(gsrc + p.glu_I);
            const float g[4] = {bf_lo(gw[0]), bf_hi(gw[0]), bf_lo(gw[1]), bf_hi(gw[1])};
            const float u[4] = {bf_lo(uw[0]), bf_hi(uw[0]), bf_lo(uw[1]), bf_hi(uw[1])};
            float dg[4], du[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float sg = 1.0f / (1.0f + __expf(-g[e]));
              du[e] = v[e] * g[e] * sg;
              dg[e] = v[e] * u[e] * sg * (1.0f + g[e] * (1.0f - sg));
            }
            bf16_t* out = p.C + (int64_t)m * p.ldc + n;
            *(u32x2*)out = u32x2{pack_bf2(dg[0], dg[1]), pack_bf2(dg[2], dg[3])};
            *(u32x2*)(out + p.glu_I) = u32x2{pack_bf2(du[0], du[1]), pack_bf2(du[2], du[3])};
          } else {
            bf16_t* out = p.C + (int64_t)m * p.ldc + n;
            if constexpr (EPI == EPI_RESID) {
              const u32x2 rw = *(const u32x2*)(p.R + (int64_t)m * p.ldc + n);
              v[0] += bf_lo(rw[0]);
              v[1] += bf_hi(rw[0]);
              v[2] += bf_lo(rw[1]);
              v[3] += bf_hi(rw[1]);
            }
            *(u32x2*)out = u32x2{pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3])};
          }
        }
    }
  }
}

// Tile configuration: 256x256 tiles, 4 waves in a 2 x 2 grid (128x128 wave
// tiles; the gate/up pairing and the RoPE partner columns rely on 128-column
// wave tiles).
template <bool AK, bool BKC, int EPI>
hipError_t launch(const GemmArgs& a, hipStream_t s) {
  constexpr int BM = 256, BN = 256, WGM = 2, WGN = 2;
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_kernel<BM, BN, WGM, WGN, AK, BKC, EPI>), dim3(tiles), dim3(64 * WGM * WGN), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm(const GemmArgs& a, hipStream_t s) {
  if (a.a_kcontig && a.b_kcontig) {
    switch (a.epi) {
      case EPI_BF16: return launch<true, true, EPI_BF16>(a, s);
      case EPI_RESID: return launch<true, true, EPI_RESID>(a, s);
      case EPI_ROPE:
        return a.head_dim == 64 ? launch<true, true, EPI_ROPE64>(a, s) : launch<true, true, EPI_ROPE>(a, s);
      case EPI_GLU_FWD: return launch<true, true, EPI_GLU_FWD>(a, s);
      default: break;
    }
  } else if (a.a_kcontig && !a.b_kcontig) {
    switch (a.epi) {
      case EPI_BF16: return launch<true, false, EPI_BF16>(a, s);
      case EPI_GLU_BWD: return launch<true, false, EPI_GLU_BWD>(a, s);
      default: break;
    }
  } else if (!a.a_kcontig && !a.b_kcontig) {
    if (a.epi == EPI_F32) return launch<false, false, EPI_F32>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace ls
