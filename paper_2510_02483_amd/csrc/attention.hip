// Causal grouped-query attention on gfx950 matrix cores: forward with an
// online softmax over key tiles (log-sum-exp saved), backward that recomputes
// the probabilities from the log-sum-exp.
//
// Layouts: qkv is [batch*seq, (nq + 2*nkv)*d] bf16 (q heads, then k heads, then
// v heads of one token in one row), o and dout are [batch*seq, nq*d], lse and
// D are [batch, nq, seq] fp32.  Query head h reads kv head h / (nq/nkv).
//
// Every streamed operand (K and V tiles in the forward and dQ kernels, Q and
// dO tiles in the dK/dV kernel) goes from global memory to LDS with buffer
// loads that write LDS directly, double-buffered: the loads of tile t+1 are in
// flight while the matrix cores work on tile t, with one barrier per tile.
// Tiles stay row-major in LDS ([row][d], 16-byte chunks XOR-swizzled by the
// row).  An operand is read either along d (a 16-byte read per lane: keys or
// queries as MFMA rows) or transposed (two ds_read_b64_tr_b16 per lane: d as
// MFMA rows, 4 consecutive keys/queries per read), and the swizzle keeps both
// kinds of read free of bank conflicts.
//
// The probabilities of a 32x32 MFMA block sit in registers with a lane owning
// one query (forward, dQ) or one key (dK/dV) and holding, for each 16-row
// k-step, the rows 4lh+{0..3} and 8+4lh+{0..3} (lh = lane/32).  Used as the B
// operand of the next product they define a permuted k order, and the
// transposed reads of the A operand fetch their rows in that same order.
//
// Forward (one workgroup = 128 queries of one head, 4 waves x 32): S^T = K Q^T
// per 64-key tile with Q in registers, base-2 online softmax with 1/sqrt(d)
// folded into one multiplier, O^T += V^T P^T.
// Backward, two kernels and no atomics.  dK/dV (one workgroup = 128 keys of
// one kv head, 4 waves x 32 keys, K and V in registers) loops over the query
// heads of its group and over 64-query tiles from the diagonal on: S = Q K^T,
// dP = dO V^T, P and dS = P (dP - D) in registers, dV^T += dO^T P and
// dK^T += Q^T dS (the sum over the group's heads happens in the same
// registers).  dQ (one workgroup = 128 queries of one head) loops over key
// tiles like the forward: S^T, dP^T, dQ^T += K^T dS^T.  Both write their
// gradient already scaled and un-rotated (inverse RoPE) in bf16.
//
// Workgroups are numbered so that the longest (most causal tiles) start
// first, which balances the triangular work over the compute units.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace ls {

namespace {

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

constexpr int BQ = 128;       // queries per workgroup (forward, dQ)
constexpr int BKV = 64;       // keys per tile (forward, dQ)
constexpr int BWD_BKV = 128;  // keys per workgroup (dK/dV)
constexpr int BWD_BQ = 64;    // queries per tile (dK/dV)

LS_DEV u32x4 load16(const bf16_t* p) { return *(const u32x4*)p; }
LS_DEV u32x4 pack_frag(const f32x16& v, int r0) {
  return u32x4{pack_bf2(v[r0], v[r0 + 1]), pack_bf2(v[r0 + 2], v[r0 + 3]), pack_bf2(v[r0 + 4], v[r0 + 5]),
               pack_bf2(v[r0 + 6], v[r0 + 7])};
}
LS_DEV float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

// Row-major LDS tile [rows][D]: 16-byte chunk c of row r sits at slot
// c ^ tile_swz(r).  The LDS serves 16 lanes of a 16-byte read and 32 lanes of
// an 8-byte read per clock over 64 banks (a 256-byte window):
//  - a 16-byte read along d covers 16 consecutive rows at one chunk: the swizzle
//    is a bijection of r % 16 (D = 128, one row per window) or of (r/2) % 8 for
//    each parity of r (D = 64, two rows per window);
//  - a transposing read covers 4 consecutive rows (4-aligned) x 4 consecutive
//    chunks (4-aligned): the swizzle moves the rows' chunk groups apart
//    (bits 2..3 of the slot for D = 128, bit 2 plus the window half for D = 64)
//    while its low two bits only depend on r / 4.
template <int D>
LS_DEV int tile_swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

// Loads of tiles: rows row0 .. row0+ROWS-1, columns col0 .. col0+D-1 of a
// row-major bf16 matrix (leading dimension ld elements, `rows` rows) into an
// LDS tile in the swizzled layout above; rows at or past `rows` read as zero.
// Each load fills 1 KB of the tile (64/(D/8) rows); wave w fills the
// consecutive blocks w*PER .. w*PER+PER-1 with one M0 write.  The per-lane
// byte offsets of the wave's share are computed once, for every tile of a
// loop; a tile only moves the scalar resource, whose base is the tile's first
// element and whose end is row `rows` (the tile's columns lie within a row:
// col0 + D <= ld).
template <int D, int ROWS>
struct TileLoader {
  static constexpr int CPR = D / 8, RPI = 64 / CPR, PER = ROWS / RPI / 4;
  static_assert(PER == 2 || PER == 4, "loads split evenly over 4 waves in groups of 2 or 4");
  uint32_t off[PER];
  LS_DEV TileLoader(int64_t ld, int wave, int lane) {
#pragma unroll
    for (int jj = 0; jj < PER; ++jj) {
      const int rr = (wave * PER + jj) * RPI + lane / CPR;
      const int c = (lane % CPR) ^ tile_swz<D>(rr);
      off[jj] = ((uint32_t)rr * (uint32_t)ld + (uint32_t)(8 * c)) * 2u;
    }
  }
  LS_DEV void operator()(const bf16_t* m, int64_t ld, int row0, int rows, int col0, bf16_t* t, int wave) const {
    const i32x4 r = rsrc(m + (int64_t)row0 * ld + col0, clamp_bytes((int64_t)(rows - row0) * ld * 2 - (int64_t)col0 * 2));
    DmaLoad l[PER];
#pragma unroll
    for (int jj = 0; jj < PER; ++jj) l[jj] = DmaLoad{r, off[jj]};
    dma16_group<PER>(l, t + wave * PER * 512);
  }
};

// 64 floats v[i0 .. i0+63] of a buffer of `n` floats (resource r; entries at or
// past n read as zero) into t[0..63]; t must hold 256 floats (lanes 16..63 of
// the instruction write zeros to t[64..255]).
LS_DEV void load_vec64(i32x4 r, int i0, int n, float* t, int lane) {
  const int i = i0 + 4 * lane;
  dma16(r, (lane < 16 && i < n) ? (uint32_t)(i * 4) : LS_OOB, t);
}

// MFMA operand from a tile, read along d: lane gets row `row`, d = 16s + 8lh .. +7.
template <int D>
LS_DEV u32x4 row_frag(const bf16_t* t, int row, int s, int lh) {
  return *(const u32x4*)(t + row * D + 8 * ((2 * s + lh) ^ tile_swz<D>(row)));
}

// MFMA A operand of the transposed tile: lane gets column (d) c32 + lane%32 and
// the 8 rows 16s + 4lh + {0..3} and 16s + 8 + 4lh + {0..3} (the permuted k
// order of probabilities held in registers), via two transposing reads.
template <int D>
LS_DEV u32x4 colt_frag(const bf16_t* t, int c32, int s, int lane) {
  const int g = lane >> 4, q = lane & 15;
  const int col = c32 + 16 * (g & 1) + 4 * (q & 3);
  u32x4 out;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int kk = 16 * s + 4 * (g >> 1) + 8 * hh + (q >> 2);
    const bf16_t* p = t + kk * D + 8 * ((col >> 3) ^ tile_swz<D>(kk)) + (col & 7);
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4*)p);
    const u32x2 w = __builtin_bit_cast(u32x2, v);
    out[2 * hh] = w[0];
    out[2 * hh + 1] = w[1];
  }
  return out;
}

// The same two kinds of operand reads by LDS byte address: this lane's
// addresses relative to a tile at `base` take only D/16 values for row reads
// (row lr, d step s; the 32-row block adds a constant) and 2·D/32 for
// transposing reads (d block i, row group hh; the 16-row step adds a
// constant), so they are computed once and held in registers the compiler
// cannot rematerialise.  With the other tiles in the same layout at constant
// distances (stages, arrays), every read is then one LDS instruction with an
// immediate offset.
template <int D>
struct FragAddr {
  uint32_t row[D / 16], col[D / 32][2];
  LS_DEV FragAddr(uint32_t base, int lane) {
    const int lr = lane & 31, lh = lane >> 5, g = lane >> 4, q = lane & 15;
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
      row[s] = base + 2u * (uint32_t)(lr * D + 8 * ((2 * s + lh) ^ tile_swz<D>(lr)));
      asm volatile("" : "+v"(row[s]));
    }
#pragma unroll
    for (int i = 0; i < D / 32; ++i)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int kk = 4 * (g >> 1) + 8 * hh + (q >> 2), c = 32 * i + 16 * (g & 1) + 4 * (q & 3);
        col[i][hh] = base + 2u * (uint32_t)(kk * D + 8 * ((c >> 3) ^ tile_swz<D>(kk)) + (c & 7));
        asm volatile("" : "+v"(col[i][hh]));
      }
  }
  // row_frag(tile at base + off, 32-row block, s, lh) for off = block * 32 * D * 2 + ...
  LS_DEV u32x4 rows(int s, uint32_t off) const { return *(const LDS_AS u32x4*)(size_t)(row[s] + off); }
  // colt_frag(tile at base + off, 32 i, step, lane) for off = step * 16 * D * 2 + ...
  LS_DEV u32x4 cols(int i, uint32_t off) const {
    u32x4 out;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const u32x2 w = __builtin_bit_cast(
          u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4*)(size_t)(col[i][hh] + off)));
      out[2 * hh] = w[0];
      out[2 * hh + 1] = w[1];
    }
    return out;
  }
};

// Query-tile workgroups (forward, dQ): the 1-D grid runs the longest tiles
// (highest query index, most keys) first.
struct QTile {
  int qt, h, b;
};
LS_DEV QTile q_tile(const AttnShape& sh) {
  const int nqt = (sh.seq + BQ - 1) / BQ, per = sh.nq * sh.batch;
  const int x = (int)blockIdx.x;
  return QTile{nqt - 1 - x / per, (x % per) % sh.nq, (x % per) / sh.nq};
}

// The two halves of a wave (lanes 0-31 and 32-63) hold the same 32 queries
// at different keys: combine a per-lane value with the other half's, through a
// lane swap on the vector unit rather than an LDS permute (which would also
// wait for every LDS read in flight).
LS_DEV float halves_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
LS_DEV float halves_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Online softmax with a lagging reference maximum: the running reference m
// moves only when some query's scores exceed it by more than 2^LAG (base 2), so
// that most tiles skip the rescale of O and l.  P = 2^(s - m) then lies in
// (0, 2^LAG]: bf16 keeps its relative precision at any such magnitude, and O,
// l in fp32 stay far from overflow.  The result, O = sum P V / sum P and the
// log-sum-exp m + log2 l, does not depend on the reference point.
constexpr float LAG = 8.0f;

template <int D>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(AttnShape sh, const bf16_t* __restrict__ qkv,
                                                           bf16_t* __restrict__ o, float* __restrict__ lse,
                                                           float sl2) {
  __shared__ __attribute__((aligned(1024))) bf16_t Ks[2][BKV * D];
  __shared__ __attribute__((aligned(1024))) bf16_t Vs[2][BKV * D];
  // the scale in a register before the loop: a scalar load still in flight
  // at the loop entry makes the first LDS wait of every tile a full wait
  asm volatile("" : "+s"(sl2));

  const int S = sh.seq, nq = sh.nq, nkv = sh.nkv;
  const QTile qtile = q_tile(sh);
  const int h = qtile.h, b = qtile.b, kvh = h / (nq / nkv);
  const int64_t ld = (int64_t)(nq + 2 * nkv) * D;
  const bf16_t* base = qkv + (int64_t)b * S * ld;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lr = lane & 31, lh = lane >> 5;
  const int q0 = qtile.qt * BQ;
  const int qrow = q0 + 32 * wave + lr;
  const int wave_qmin = q0 + 32 * wave, wave_qmax = wave_qmin + 31;
  const int kcol = (nq + kvh) * D, vcol = (nq + nkv + kvh) * D;

  const int kv_end = min(S, q0 + BQ);
  const int nkt = (kv_end + BKV - 1) / BKV;

  const TileLoader<D, BKV> tl(ld, wave, lane);
  auto load_kv = [&](int kv0, bf16_t* kt, bf16_t* vt) {
    tl(base, ld, kv0, S, kcol, kt, wave);
    tl(base, ld, kv0, S, vcol, vt, wave);
  };
  load_kv(0, Ks[0], Vs[0]);

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

  // operand reads by per-lane LDS address (K rows, V^T columns); the stage,
  // the array, the 32-key block and the 16-key step add constants
  const FragAddr<D> fa(lds_offset(&Ks[0][0]), lane);
  constexpr uint32_t STAGE = BKV * D * 2;
  const uint32_t v_minus_k = lds_offset(&Vs[0][0]) - lds_offset(&Ks[0][0]);

  sync_lds();
  // one 64-key tile in stage CUR (a constant: the loop below runs two per pass)
  auto step = [&](auto cur_c, int kt) {
    constexpr int cur = decltype(cur_c)::value;
    const int kv0 = kt * BKV;
    if (kt + 1 < nkt) load_kv(kv0 + BKV, Ks[cur ^ 1], Vs[cur ^ 1]);
    if (kv0 <= wave_qmax) {  // else every key of the tile is in this wave's future
      f32x16 sacc[BKV / 32];
#pragma unroll
      for (int bb = 0; bb < BKV / 32; ++bb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[bb][r] = 0.f;
#pragma unroll
      for (int s = 0; s < D / 16; ++s)
#pragma unroll
        for (int bb = 0; bb < BKV / 32; ++bb)
          sacc[bb] = mfma32(fa.rows(s, cur * STAGE + bb * 32 * D * 2), qf[s], sacc[bb]);
      // lane holds query qrow, keys kv0 + 32bb + 8(r/4) + 4lh + r%4
      if (kv0 + BKV - 1 > wave_qmin) {
#pragma unroll
        for (int bb = 0; bb < BKV / 32; ++bb)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (kv0 + 32 * bb + 8 * (r >> 2) + 4 * lh + (r & 3) > qrow) sacc[bb][r] = -INFINITY;
      }
      float mx = -INFINITY;
#pragma unroll
      for (int bb = 0; bb < BKV / 32; ++bb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[bb][r]);
      // key 0 is visible to every query: finite from the first tile on
      const float mc = fmaxf(m, halves_max(mx) * sl2);
      if (__builtin_amdgcn_ballot_w64(mc > m + LAG)) {
        const float alpha = ex2(m - mc);
        m = mc;
        l *= alpha;
#pragma unroll
        for (int i = 0; i < D / 32; ++i) oacc[i] *= alpha;
      }
      float ls = 0.f;
#pragma unroll
      for (int bb = 0; bb < BKV / 32; ++bb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = ex2(fmaf(sacc[bb][r], sl2, -m));
          sacc[bb][r] = p;
          ls += p;
        }
      l += halves_sum(ls);
#pragma unroll
      for (int s = 0; s < BKV / 16; ++s) {
        const u32x4 pf = pack_frag(sacc[s >> 1], 8 * (s & 1));
#pragma unroll
        for (int i = 0; i < D / 32; ++i)
          oacc[i] = mfma32(fa.cols(i, v_minus_k + cur * STAGE + s * 16 * D * 2), pf, oacc[i]);
      }
    }
    sync_lds();
  };
  for (int kt = 0; kt < nkt; kt += 2) {
    step(std::integral_constant<int, 0>{}, kt);
    if (kt + 1 < nkt) step(std::integral_constant<int, 1>{}, kt + 1);
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

// D[b,h,s] = <dO, O> over the head's d columns (fp32), and the log-sum-exp in
// base 2 (lse * log2(e)), the form the backward kernels subtract.
template <int D>
__global__ __launch_bounds__(256) void attn_bwd_pre_kernel(AttnShape sh, const bf16_t* __restrict__ o,
                                                           const bf16_t* __restrict__ dout,
                                                           const float* __restrict__ lse, float* __restrict__ Dv,
                                                           float* __restrict__ lse2) {
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
    if (c < chunks && (c % CPH) == 0) {
      const int64_t i = ((int64_t)b * sh.nq + c / CPH) * sh.seq + s;
      Dv[i] = acc;
      lse2[i] = lse[i] * LOG2E;
    }
  }
}

// Inverse rotation of a gradient held in MFMA layout: lane holds columns
// 32i + 8(r/4) + 4lh + r%4 of one row at position `pos`; the pair partner of
// column d < D/2 is d + D/2, in register block i + D/64 of the same lane.
template <int D>
LS_DEV void unrotate_store(const f32x16 (&acc)[D / 32], float scale, const float* rope_cs, int seq, int pos, int lh,
                           bf16_t* row) {
  constexpr int HALF = D / 2, IP = HALF / 32;
  if (rope_cs == nullptr) {
#pragma unroll
    for (int i = 0; i < D / 32; ++i)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int d = 32 * i + 8 * rq + 4 * lh;
        *(u32x2*)(row + d) = u32x2{pack_bf2(acc[i][4 * rq] * scale, acc[i][4 * rq + 1] * scale),
                                   pack_bf2(acc[i][4 * rq + 2] * scale, acc[i][4 * rq + 3] * scale)};
      }
    return;
  }
  // cos and sin of the lane's angle indices (4 consecutive ones per 8-column
  // group, 16-byte loads), all in flight before the rotations use them; the
  // second half of the head uses the angles of the first
  const float* cb = rope_cs + (int64_t)pos * HALF;
  const float* sb = rope_cs + (int64_t)seq * HALF + (int64_t)pos * HALF;
  f32x4 c4[IP][4], s4[IP][4];
#pragma unroll
  for (int i = 0; i < IP; ++i)
#pragma unroll
    for (int rq = 0; rq < 4; ++rq) {
      const int d = 32 * i + 8 * rq + 4 * lh;
      c4[i][rq] = *(const f32x4*)(cb + d);
      s4[i][rq] = *(const f32x4*)(sb + d);
    }
#pragma unroll
  for (int i = 0; i < D / 32; ++i)
#pragma unroll
    for (int rq = 0; rq < 4; ++rq) {
      const int d = 32 * i + 8 * rq + 4 * lh;
      float out[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = acc[i][4 * rq + e] * scale;
        if (i < IP) {  // first half: x1' = x1 cos + x2 sin
          const float x2 = acc[i + IP][4 * rq + e] * scale;
          out[e] = x * c4[i][rq][e] + x2 * s4[i][rq][e];
        } else {  // second half: x2' = x2 cos - x1 sin
          const float x1 = acc[i - IP][4 * rq + e] * scale;
          out[e] = x * c4[i - IP][rq][e] - x1 * s4[i - IP][rq][e];
        }
      }
      *(u32x2*)(row + d) = u32x2{pack_bf2(out[0], out[1]), pack_bf2(out[2], out[3])};
    }
}

// dK and dV for 128 keys of one kv head (4 waves x 32 keys), summed over the
// query heads of the group, no atomics.  The 1-D grid runs the key tiles with
// the most queries after them (lowest key index) first.  With few kv heads
// (and so few workgroups) the group's query heads are split over `hsplit`
// workgroups, each of which writes its fp32 partial sums to `part`
// ([hsplit][batch*seq][nkv][dK | dV]); attn_bwd_dkdv_reduce then adds the
// partials in a fixed order and stores dK and dV.
//
// A wave issues one MFMA per slot.  Each 32-query block of a 64-query tile
// takes four phases: S = Q K^T, dP = dO V^T, dV^T += dO^T P, dK^T += Q^T dS.
// The softmax work is spread between the MFMAs: P = exp2(S - LSE) (and its
// bf16 operands) during the dP phase, dS = P (dP - D) during the dV phase, so
// the vector ALU works while the matrix core does.  Every MFMA operand read
// from LDS is issued RA slots ahead into a ring of registers (across tile
// boundaries too), so no MFMA waits on an LDS read.  Three LDS stages: RA
// slots before the end of tile t each wave waits for its loads of tile t+1
// and for the other waves (whose reads of tile t-1 are then done), and the
// loads of tile t+2 go into tile t-1's stage.
template <int D, bool SPLIT>
__global__ __launch_bounds__(256, 1) void attn_bwd_dkdv_kernel(AttnShape sh, const bf16_t* __restrict__ qkv,
                                                                const bf16_t* __restrict__ dout,
                                                                const float* __restrict__ lse2,
                                                                const float* __restrict__ Dv, bf16_t* __restrict__ dqkv,
                                                                const float* __restrict__ rope_cs, float scale,
                                                                float sl2, int hsplit_arg, float* __restrict__ part) {
  constexpr int NST = 3;                    // LDS stages
  constexpr int NSD = D / 16, NI = D / 32;  // 16-wide d steps; 32-row d blocks
  constexpr int P1 = NSD, P2 = NSD, P3 = 2 * NI, P4 = 2 * NI;  // slots per phase
  constexpr int NB = P1 + P2 + P3 + P4;     // slots of a 32-query block
  constexpr int NSLOT = 2 * NB;
  constexpr int RING = 8, RA = RING - 1;    // operand ring; read-ahead in slots
  static_assert(NSLOT % RING == 0, "ring positions repeat every tile");
  static_assert(P1 >= 4 && P2 >= 4 && 16 % P2 == 0 && 16 % P3 == 0, "phase sizes");
  constexpr int BAR = NSLOT - RA;           // slot of the barrier
  // one stage: Q tile, dO tile, log-sum-exp (base 2) and D of its queries
  // (every operand of a stage within the reach of an LDS instruction's offset)
  struct Stage {
    bf16_t q[BWD_BQ * D];
    bf16_t o[BWD_BQ * D];
    float l[256];
    float d[256];
  };
  __shared__ __attribute__((aligned(1024))) Stage stg[NST];

  const int hsplit = SPLIT ? hsplit_arg : 1;  // the unsplit instance folds every split term away
  const int S = sh.seq, nq = sh.nq, nkv = sh.nkv, G = nq / nkv, Gs = SPLIT ? G / hsplit : G;
  const int per = nkv * sh.batch * hsplit, x = (int)blockIdx.x;
  const int kvt = x / per, hs = (x % per) % hsplit, kvh = ((x % per) / hsplit) % nkv,
            b = ((x % per) / hsplit) / nkv;
  const int64_t ld = (int64_t)(nq + 2 * nkv) * D;
  const int64_t ldo = (int64_t)nq * D;
  const bf16_t* base = qkv + (int64_t)b * S * ld;
  const bf16_t* dbase = dout + (int64_t)b * S * ldo;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 31, lh = lane >> 5;
  const int kv0 = kvt * BWD_BKV;
  const int kvrow = kv0 + 32 * wave + lr;

  // tiles t = 0 .. Gs*nqt-1: query head kvh*G + hs*Gs + t/nqt, queries q_begin + (t%nqt)*BWD_BQ ..
  const int q_begin = kv0;  // earlier queries see none of these keys
  const int nqt = (S - q_begin + BWD_BQ - 1) / BWD_BQ;
  const int ntiles = Gs * nqt;
  const TileLoader<D, BWD_BQ> tlq(ld, wave, lane), tlo(ldo, wave, lane);
  auto issue = [&](int t, int st) {
    const int h = kvh * G + hs * Gs + t / nqt, q0 = q_begin + (t % nqt) * BWD_BQ;
    tlq(base, ld, q0, S, h * D, stg[st].q, wave);
    tlo(dbase, ldo, q0, S, h * D, stg[st].o, wave);
    if (wave == 0) load_vec64(rsrc(lse2 + ((int64_t)b * nq + h) * S, (uint32_t)S * 4), q0, S, stg[st].l, lane);
    if (wave == 1) load_vec64(rsrc(Dv + ((int64_t)b * nq + h) * S, (uint32_t)S * 4), q0, S, stg[st].d, lane);
  };
  issue(0, 0);
  if (ntiles > 1) issue(1, 1);

  u32x4 kf[NSD], vf[NSD];
#pragma unroll
  for (int s = 0; s < NSD; ++s) {
    const bool ok = kvrow < S;
    kf[s] = ok ? load16(base + (int64_t)kvrow * ld + (nq + kvh) * D + 16 * s + 8 * lh) : u32x4{0u, 0u, 0u, 0u};
    vf[s] = ok ? load16(base + (int64_t)kvrow * ld + (nq + nkv + kvh) * D + 16 * s + 8 * lh) : u32x4{0u, 0u, 0u, 0u};
  }

  f32x16 dk[NI], dv[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[i][r] = dv[i][r] = 0.f;

  // MFMA A operand of slot j of the tile in stage st.
  auto operand = [&](auto j_c, int st) -> u32x4 {
    constexpr int j = decltype(j_c)::value;
    constexpr int qb = j / NB, k = j % NB;
    if constexpr (k < P1) return row_frag<D>(stg[st].q, 32 * qb + lr, k, lh);
    else if constexpr (k < P1 + P2) return row_frag<D>(stg[st].o, 32 * qb + lr, k - P1, lh);
    else if constexpr (k < P1 + P2 + P3) {
      constexpr int c = k - P1 - P2;
      return colt_frag<D>(stg[st].o, 32 * (c % NI), 2 * qb + c / NI, lane);
    } else {
      constexpr int c = k - P1 - P2 - P3;
      return colt_frag<D>(stg[st].q, 32 * (c % NI), 2 * qb + c / NI, lane);
    }
  };

  u32x4 ring[RING];
  f32x16 sacc, pacc;
  f32x4 Lq[2], Dq[2];  // base-2 log-sum-exp and D of the block's queries 8rq + 4lh + {0..3}, rq even / odd
  u32x4 pf[2], sf[2];

  // One tile in stage st; st1 and st2 are the stages of the next two tiles
  // (the three rotate from tile to tile).
  auto tile = [&](int t, int st, int st1, int st2) {
    const int q0 = q_begin + (t % nqt) * BWD_BQ;
    // causal mask, on the tiles at the diagonal only (some query of the tile
    // precedes some key of the wave): element r of block qb is query
    // q0 + 4lh + c with c = 32qb + 8(r/4) + r%4, kept when c >= lo, i.e.
    // q >= kvrow; a masked score becomes -inf, so its probability is
    // exp2(-inf) = 0.  Queries past the end of the sequence need no mask: their
    // Q, dO, LSE and D read as zero, so they add nothing to dK or dV.
    const int lo = kvrow - q0 - 4 * lh;
    const bool diag = q0 < kv0 + 32 * wave + 31;
    static_for<NSLOT>([&](auto j_c) {
      constexpr int j = decltype(j_c)::value;
      constexpr int qb = j / NB, k = j % NB;
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (j == BAR) {
        LS_WAIT_VMCNT(0);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        if (t + 2 < ntiles) issue(t + 2, st2);
      }
      const u32x4 a = ring[j % RING];
      if constexpr (k < P1) {  // S = Q K^T; read the block's log-sum-exp
        sacc = mfma32(a, kf[k], k == 0 ? f32x16{} : sacc);
        if constexpr (k == P1 - 1) Lq[0] = *(const f32x4*)&stg[st].l[32 * qb + 4 * lh];
      } else if constexpr (k < P1 + P2) {  // dP = dO V^T, meanwhile P = exp2(S sl2 - LSE2)
        constexpr int c = k - P1, PER = 16 / P2;
        pacc = mfma32(a, vf[c], c == 0 ? f32x16{} : pacc);
        if constexpr (c == 0) {
          if (diag) {
            asm volatile("");  // keeps the block a branch rather than selects on every tile
#pragma unroll
            for (int r = 0; r < 16; ++r)
              if (32 * qb + 8 * (r >> 2) + (r & 3) < lo) sacc[r] = -INFINITY;
          }
        }
        static_for<PER>([&](auto u_c) {
          constexpr int r = c * PER + decltype(u_c)::value, rq = r >> 2, e = r & 3;
          // the next group's log-sum-exp, one group ahead
          if constexpr (e == 0 && rq < 3) Lq[(rq + 1) & 1] = *(const f32x4*)&stg[st].l[32 * qb + 8 * (rq + 1) + 4 * lh];
          if constexpr (r == 12) Dq[0] = *(const f32x4*)&stg[st].d[32 * qb + 4 * lh];
          sacc[r] = ex2(fmaf(sacc[r], sl2, -Lq[rq & 1][e]));
          if constexpr ((r & 7) == 7) pf[r >> 3] = pack_frag(sacc, r - 7);
        });
      } else if constexpr (k < P1 + P2 + P3) {  // dV^T += dO^T P, meanwhile dS = P (dP - D)
        constexpr int c = k - P1 - P2, PER = 16 / P3;
        dv[c % NI] = mfma32(a, pf[c / NI], dv[c % NI]);
        static_for<PER>([&](auto u_c) {
          constexpr int r = c * PER + decltype(u_c)::value, rq = r >> 2, e = r & 3;
          if constexpr (e == 0 && rq < 3) Dq[(rq + 1) & 1] = *(const f32x4*)&stg[st].d[32 * qb + 8 * (rq + 1) + 4 * lh];
          pacc[r] = sacc[r] * (pacc[r] - Dq[rq & 1][e]);
          if constexpr ((r & 7) == 7) sf[r >> 3] = pack_frag(pacc, r - 7);
        });
      } else {  // dK^T += Q^T dS
        constexpr int c = k - P1 - P2 - P3;
        dk[c % NI] = mfma32(a, sf[c / NI], dk[c % NI]);
      }
      // operand of slot j + RA (of this tile or, past its end, of the next)
      if constexpr (j + RA < NSLOT) ring[(j + RA) % RING] = operand(std::integral_constant<int, j + RA>{}, st);
      else ring[(j + RA) % RING] = operand(std::integral_constant<int, j + RA - NSLOT>{}, st1);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  LS_WAIT_VMCNT(0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  static_for<RA>([&](auto j_c) { ring[decltype(j_c)::value] = operand(j_c, 0); });
  int st = 0, st1 = 1, st2 = 2;
  for (int t = 0; t < ntiles; ++t) {
    tile(t, st, st1, st2);
    const int tmp = st;
    st = st1;
    st1 = st2;
    st2 = tmp;
  }

  // dK = scale * dS^T Q (un-rotated), dV = P^T dO.  Lane holds key kvrow.
  if (kvrow >= S) return;
  if constexpr (SPLIT) {  // partial sums of this workgroup's heads; lane holds columns 32i + 8(r/4) + 4lh + r%4
    float* row = part + (((int64_t)hs * sh.batch * S + (int64_t)b * S + kvrow) * nkv + kvh) * (2 * D);
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int c = 32 * i + 8 * rq + 4 * lh;
        *(f32x4*)(row + c) = f32x4{dk[i][4 * rq], dk[i][4 * rq + 1], dk[i][4 * rq + 2], dk[i][4 * rq + 3]};
        *(f32x4*)(row + D + c) = f32x4{dv[i][4 * rq], dv[i][4 * rq + 1], dv[i][4 * rq + 2], dv[i][4 * rq + 3]};
      }
  } else {
    unrotate_store<D>(dk, scale, rope_cs, S, kvrow, lh, dqkv + ((int64_t)b * S + kvrow) * ld + (nq + kvh) * D);
    unrotate_store<D>(dv, 1.0f, nullptr, S, kvrow, lh, dqkv + ((int64_t)b * S + kvrow) * ld + (nq + nkv + kvh) * D);
  }
}

// Sum of the hsplit partial dK / dV rows of attn_bwd_dkdv_kernel, in split
// order, then scale and inverse RoPE for dK, bf16 stores into dqkv.  One wave
// per (token, kv head): lane l holds columns 4l .. 4l+3 of [dK | dV] (D = 128)
// or 2l .. 2l+1 (D = 64); the RoPE partner of dK column c < D/2 is c + D/2.
template <int D>
__global__ __launch_bounds__(256) void attn_bwd_dkdv_reduce(AttnShape sh, int hsplit, const float* __restrict__ part,
                                                            bf16_t* __restrict__ dqkv, const float* __restrict__ rope_cs,
                                                            float scale) {
  constexpr int E = 2 * D / 64;  // columns per lane
  constexpr int HALF = D / 2;
  const int lane = threadIdx.x & 63;
  const int64_t T = (int64_t)sh.batch * sh.seq;
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (token, kv head)
  if (w >= T * sh.nkv) return;
  const int64_t t = w / sh.nkv;
  const int kvh = (int)(w % sh.nkv), pos = (int)(t % sh.seq);
  const int c0 = E * lane;  // first of this lane's columns in [dK | dV]
  float v[E];
#pragma unroll
  for (int e = 0; e < E; ++e) v[e] = 0.f;
  for (int hs = 0; hs < hsplit; ++hs) {
    const float* src = part + ((int64_t)hs * T * sh.nkv + w) * (2 * D) + c0;
    if constexpr (E == 4) {
      const f32x4 a = *(const f32x4*)src;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += a[e];
    } else {
      const float2 a = *(const float2*)src;
      v[0] += a.x;
      v[1] += a.y;
    }
  }
  const bool is_k = c0 < D;
  // partner columns of dK (c0 +- D/2): lanes HALF/E apart
  float pv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) pv[e] = __shfl_xor(v[e], HALF / E);
  const int64_t ld = (int64_t)(sh.nq + 2 * sh.nkv) * D;
  bf16_t* row = dqkv + t * ld + (int64_t)(sh.nq + (is_k ? 0 : sh.nkv) + kvh) * D;
  const int d0 = is_k ? c0 : c0 - D;
  float out[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    if (!is_k) {
      out[e] = v[e];
    } else if (!rope_cs) {
      out[e] = v[e] * scale;
    } else {
      const int d = d0 + e, i = d % HALF;
      const float cs = rope_cs[(int64_t)pos * HALF + i];
      const float sn = rope_cs[(int64_t)sh.seq * HALF + (int64_t)pos * HALF + i];
      // inverse rotation: x1' = x1 cos + x2 sin, x2' = x2 cos - x1 sin
      out[e] = d < HALF ? (v[e] * cs + pv[e] * sn) * scale : (v[e] * cs - pv[e] * sn) * scale;
    }
  }
  if constexpr (E == 4) *(u32x2*)(row + d0) = u32x2{pack_bf2(out[0], out[1]), pack_bf2(out[2], out[3])};
  else *(uint32_t*)(row + d0) = pack_bf2(out[0], out[1]);
}

// dQ for 128 queries of one head (4 waves x 32 queries): loops over the key
// tiles up to the diagonal, recomputes S^T and dP^T with keys as MFMA rows (a
// lane owns one query, as in the forward), forms dS^T in registers and
// accumulates dQ^T += K^T dS^T.
//
// Per 64-key tile a wave issues one MFMA per slot: S^T and dP^T of key block 0,
// then of key block 1, then dQ^T for block 0 and for block 1.  The softmax work
// of block 0 (P = exp2(S - LSE), dS = P (dP - D), bf16 operands) runs between
// the MFMAs of block 1's S^T and dP^T, that of block 1 between the MFMAs of
// block 0's dQ^T.  MFMA operands from LDS are read RA slots ahead into a ring
// of registers within the tile; two workgroups per compute unit keep the
// matrix cores busy across tile boundaries and while one wave waits.
template <int D>
__global__ __launch_bounds__(256, 2) void attn_bwd_dq_kernel(AttnShape sh, const bf16_t* __restrict__ qkv,
                                                              const bf16_t* __restrict__ dout,
                                                              const float* __restrict__ lse2,
                                                              const float* __restrict__ Dv, bf16_t* __restrict__ dqkv,
                                                              const float* __restrict__ rope_cs, float scale,
                                                              float sl2) {
  constexpr int NSD = D / 16, NI = D / 32;
  constexpr int PS = 2 * NSD;                // slots of one block's S^T and dP^T (interleaved)
  constexpr int PQ = 2 * NI;                 // slots of one block's dQ^T
  constexpr int NSLOT = 2 * PS + 2 * PQ;
  constexpr int RING = 2, RA = RING - 1;
  static_assert(NSLOT % RING == 0 && 16 % PS == 0 && 16 % PQ == 0, "slot counts");
  __shared__ __attribute__((aligned(1024))) bf16_t Ks[2][BKV * D];
  __shared__ __attribute__((aligned(1024))) bf16_t Vs[2][BKV * D];

  const int S = sh.seq, nq = sh.nq, nkv = sh.nkv;
  const QTile qtile = q_tile(sh);
  const int h = qtile.h, b = qtile.b, kvh = h / (nq / nkv);
  const int64_t ld = (int64_t)(nq + 2 * nkv) * D;
  const int64_t ldo = (int64_t)nq * D;
  const bf16_t* base = qkv + (int64_t)b * S * ld;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 31, lh = lane >> 5;
  const int q0 = qtile.qt * BQ;
  const int qrow = q0 + 32 * wave + lr;
  const bool qok = qrow < S;
  const int kcol = (nq + kvh) * D, vcol = (nq + nkv + kvh) * D;

  const int kv_end = min(S, q0 + BQ);
  const int nkt = (kv_end + BKV - 1) / BKV;
  const TileLoader<D, BKV> tl(ld, wave, lane);
  tl(base, ld, 0, S, kcol, Ks[0], wave);
  tl(base, ld, 0, S, vcol, Vs[0], wave);

  u32x4 qf[NSD], df[NSD];
#pragma unroll
  for (int s = 0; s < NSD; ++s) {
    qf[s] = qok ? load16(base + (int64_t)qrow * ld + h * D + 16 * s + 8 * lh) : u32x4{0u, 0u, 0u, 0u};
    df[s] = qok ? load16(dout + ((int64_t)b * S + qrow) * ldo + h * D + 16 * s + 8 * lh) : u32x4{0u, 0u, 0u, 0u};
  }
  const float L2 = qok ? lse2[((int64_t)b * nq + h) * S + qrow] : 0.f;
  const float Dq = qok ? Dv[((int64_t)b * nq + h) * S + qrow] : 0.f;

  f32x16 dq[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dq[i][r] = 0.f;

  // operand reads by per-lane LDS address (K and V rows, K^T columns); the
  // stage, the array, the 32-key block and the 16-key step add constants
  const FragAddr<D> fa(lds_offset(&Ks[0][0]), lane);
  constexpr uint32_t STAGE = BKV * D * 2;
  const uint32_t v_minus_k = lds_offset(&Vs[0][0]) - lds_offset(&Ks[0][0]);

  // MFMA A operand of slot j of the tile in stage ST.
  auto operand = [&](auto j_c, auto st_c) -> u32x4 {
    constexpr int j = decltype(j_c)::value, st = decltype(st_c)::value;
    if constexpr (j < 2 * PS) {  // rows of K (k even) or V (k odd)
      constexpr int bb = j / PS, k = j % PS;
      return fa.rows(k >> 1, st * STAGE + bb * 32 * D * 2 + ((k & 1) ? v_minus_k : 0u));
    } else {  // K^T columns
      constexpr int bb = (j - 2 * PS) / PQ, c = (j - 2 * PS) % PQ;
      return fa.cols(c % NI, st * STAGE + (2 * bb + c / NI) * 16 * D * 2);
    }
  };

  u32x4 ring[RING];
  f32x16 sacc[2], pacc[2];
  u32x4 sf[2][2];
  // causal mask: element r of key block bb is key kv0 + 4lh + c with
  // c = 32bb + 8(r/4) + r%4, kept when c <= hi, i.e. key <= qrow.  Keys past the
  // end of the sequence need no mask beyond that: their K and V read as zero.
  auto soft = [&](auto bb_c, auto r_c, int hi) {
    constexpr int bb = decltype(bb_c)::value, r = decltype(r_c)::value;
    constexpr int c = 32 * bb + 8 * (r >> 2) + (r & 3);
    float p = ex2(fmaf(sacc[bb][r], sl2, -L2));
    if (c > hi) p = 0.f;
    pacc[bb][r] = p * (pacc[bb][r] - Dq);
    if constexpr ((r & 7) == 7) sf[bb][r >> 3] = pack_frag(pacc[bb], r - 7);
  };

  sync_lds();
  // one 64-key tile in stage CUR (a constant: the loop below runs two per pass)
  auto step = [&](auto cur_c, int kt) {
    constexpr int cur = decltype(cur_c)::value;
    const int kv0 = kt * BKV;
    if (kt + 1 < nkt) {
      tl(base, ld, kv0 + BKV, S, kcol, Ks[cur ^ 1], wave);
      tl(base, ld, kv0 + BKV, S, vcol, Vs[cur ^ 1], wave);
    }
    const int hi = qrow - kv0 - 4 * lh;
    static_for<RA>([&](auto j_c) { ring[decltype(j_c)::value] = operand(j_c, cur_c); });
    static_for<NSLOT>([&](auto j_c) {
      constexpr int j = decltype(j_c)::value;
      __builtin_amdgcn_sched_barrier(0);
      const u32x4 a = ring[j % RING];
      if constexpr (j < 2 * PS) {
        constexpr int bb = j / PS, k = j % PS, s = k >> 1;
        if constexpr (k & 1) pacc[bb] = mfma32(a, df[s], s == 0 ? f32x16{} : pacc[bb]);
        else sacc[bb] = mfma32(a, qf[s], s == 0 ? f32x16{} : sacc[bb]);
        if constexpr (bb == 1) {  // softmax of block 0
          constexpr int PER = 16 / PS;
          static_for<PER>([&](auto u) {
            soft(std::integral_constant<int, 0>{}, std::integral_constant<int, k * PER + decltype(u)::value>{}, hi);
          });
        }
      } else {
        constexpr int bb = (j - 2 * PS) / PQ, c = (j - 2 * PS) % PQ;
        dq[c % NI] = mfma32(a, sf[bb][c / NI], dq[c % NI]);
        if constexpr (bb == 0) {  // softmax of block 1
          constexpr int PER = 16 / PQ;
          static_for<PER>([&](auto u) {
            soft(std::integral_constant<int, 1>{}, std::integral_constant<int, c * PER + decltype(u)::value>{}, hi);
          });
        }
      }
      if constexpr (j + RA < NSLOT) ring[(j + RA) % RING] = operand(std::integral_constant<int, j + RA>{}, cur_c);
      __builtin_amdgcn_sched_barrier(0);
    });
    sync_lds();
  };
  for (int kt = 0; kt < nkt; kt += 2) {
    step(std::integral_constant<int, 0>{}, kt);
    if (kt + 1 < nkt) step(std::integral_constant<int, 1>{}, kt + 1);
  }
  if (!qok) return;
  unrotate_store<D>(dq, scale, rope_cs, S, qrow, lh, dqkv + ((int64_t)b * S + qrow) * ld + h * D);
}

template <int D>
hipError_t attn_fwd_t(const AttnShape& sh, const bf16_t* qkv, bf16_t* o, float* lse, hipStream_t s) {
  const unsigned grid = (unsigned)((sh.seq + BQ - 1) / BQ) * sh.nq * sh.batch;
  const float sl2 = LOG2E / sqrtf((float)(sh.d_scale > 0 ? sh.d_scale : D));
  hipLaunchKernelGGL((attn_fwd_kernel<D>), dim3(grid), dim3(256), 0, s, sh, qkv, o, lse, sl2);
  return hipGetLastError();
}

// Split of each kv head's query-head group over workgroups of the dK/dV
// kernel: the smallest divisor of the group size that gives at least two
// workgroups per compute unit (256 CUs), or the whole group.
int dkdv_split(const AttnShape& sh) {
  const int G = sh.nq / sh.nkv;
  const int64_t g1 = (int64_t)((sh.seq + BWD_BKV - 1) / BWD_BKV) * sh.nkv * sh.batch;
  for (int h = 1; h < G; ++h)
    if (G % h == 0 && g1 * h >= 512) return h;
  return G;
}

// Bytes of the backward workspace before the partial sums: D, then the base-2 log-sum-exp.
int64_t bwd_ws_head(const AttnShape& sh) {
  return 2 * (int64_t)sh.batch * sh.seq * sh.nq * (int64_t)sizeof(float);
}

template <int D>
hipError_t attn_bwd_t(const AttnShape& sh, const bf16_t* qkv, const bf16_t* o, const float* lse, const bf16_t* dout,
                      bf16_t* dqkv, const float* rope_cs, void* ws, hipStream_t s) {
  const int64_t T = (int64_t)sh.batch * sh.seq;
  float* Dv = (float*)ws;
  float* lse2 = Dv + T * sh.nq;
  hipLaunchKernelGGL((attn_bwd_pre_kernel<D>), dim3((unsigned)((T + 3) / 4)), dim3(256), 0, s, sh, o, dout, lse, Dv,
                     lse2);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const float scale = 1.0f / sqrtf((float)(sh.d_scale > 0 ? sh.d_scale : D));
  const int hsplit = dkdv_split(sh);
  float* part = hsplit > 1 ? (float*)((char*)ws + bwd_ws_head(sh)) : nullptr;
  const unsigned gkv = (unsigned)((sh.seq + BWD_BKV - 1) / BWD_BKV) * sh.nkv * sh.batch * hsplit;
  if (part)
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, true>), dim3(gkv), dim3(256), 0, s, sh, qkv, dout, (const float*)lse2,
                       (const float*)Dv, dqkv, rope_cs, scale, scale * LOG2E, hsplit, part);
  else
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, false>), dim3(gkv), dim3(256), 0, s, sh, qkv, dout,
                       (const float*)lse2, (const float*)Dv, dqkv, rope_cs, scale, scale * LOG2E, 1, nullptr);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (part) {
    const int64_t rows = T * sh.nkv;  // one wave each, four per workgroup
    hipLaunchKernelGGL((attn_bwd_dkdv_reduce<D>), dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, sh, hsplit,
                       (const float*)part, dqkv, rope_cs, scale);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const unsigned gq = (unsigned)((sh.seq + BQ - 1) / BQ) * sh.nq * sh.batch;
  hipLaunchKernelGGL((attn_bwd_dq_kernel<D>), dim3(gq), dim3(256), 0, s, sh, qkv, dout, (const float*)lse2,
                     (const float*)Dv, dqkv, rope_cs, scale, scale * LOG2E);
  return hipGetLastError();
}

}  // namespace

hipError_t attn_fwd(const AttnShape& sh, const bf16_t* qkv, bf16_t* o, float* lse, hipStream_t s) {
  if (sh.d == 128) return attn_fwd_t<128>(sh, qkv, o, lse, s);
  if (sh.d == 64) return attn_fwd_t<64>(sh, qkv, o, lse, s);
  return hipErrorInvalidValue;
}

size_t attn_bwd_workspace(const AttnShape& sh) {
  // D and the base-2 log-sum-exp of every query, then (when the dK/dV group
  // is split) the fp32 partial dK | dV rows of every split
  const int hsplit = dkdv_split(sh);
  const int64_t part = hsplit > 1 ? (int64_t)hsplit * sh.batch * sh.seq * sh.nkv * 2 * sh.d * (int64_t)sizeof(float) : 0;
  return (size_t)(bwd_ws_head(sh) + part);
}

hipError_t attn_bwd(const AttnShape& sh, const bf16_t* qkv, const bf16_t* o, const float* lse, const bf16_t* dout,
                    bf16_t* dqkv, const float* rope_cs, void* ws, hipStream_t s) {
  if (sh.d == 128) return attn_bwd_t<128>(sh, qkv, o, lse, dout, dqkv, rope_cs, ws, s);
  if (sh.d == 64) return attn_bwd_t<64>(sh, qkv, o, lse, dout, dqkv, rope_cs, ws, s);
  return hipErrorInvalidValue;
}

}  // namespace ls
