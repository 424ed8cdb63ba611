// bf16 matrix products on gfx950 matrix cores (v_mfma_f32_32x32x16_bf16) with
// fp32 accumulation and fused epilogues for the decoder block.
//
// One workgroup of 4 waves (one per SIMD, 2 x 2 wave tiles) or 8 waves (two
// per SIMD, 4 x 2) computes a BM x BN tile of C (256 or 192 on each side);
// each wave owns up to 16 MFMA blocks of 32x32 with their accumulators in
// registers.  Operand tiles of 64 k-values move global -> LDS with buffer
// loads that write LDS directly (16 bytes per lane, no staging registers)
// and return zero outside the operand, so ragged edges need no branches.  Two
// LDS stages of about 64 KB: tile k+1 is in flight while the matrix cores
// consume tile k.
//
// The tile shape is picked per launch: on 256 compute units an 8192 x 3072
// output is 384 tiles of 256 x 256 (one and a half waves of workgroups) but
// exactly 512 tiles of 256 x 192, so the launcher estimates waves x tile area
// for each shape the epilogue allows and takes the smallest.
//
// The tile depth is set by the load path: a k-contiguous operand row
// contributes KT*2 bytes per tile, and the buffer->LDS path moves 128-byte row
// pieces at well over one and a half times the rate of 64-byte ones (each
// piece is one L1->L2 request and the number of requests in flight is capped).
//
// LDS layouts (the fragment reads are free of bank conflicts):
//   k-contiguous operand  1 KB blocks of 8 rows x 64 k, KC_PITCH = 1040 bytes
//                         apart (16 bytes of padding): block (r % 8) + 8 (r / 64)
//                         holds the rows of one 64-row segment that are equal
//                         mod 8, row r at 128-byte position (r / 8) % 8.  A
//                         block's load reads each row's 128 bytes with 8
//                         consecutive lanes in order; the 16 consecutive rows
//                         a 16-lane group reads at one k step fall on 16
//                         distinct 16-byte bank groups (padding and the mod-8
//                         interleave); fragments are 16-byte reads at a
//                         per-lane base plus constant offsets.
//   k-strided operand     [64 k][W cols]: for W = 256, k-rows 2j and 2j+1 fill
//                         the 1 KB block j (at bytes 0 and 512); for W = 192,
//                         block 8g + b holds k-rows 8b .. 8b+7 of the 64-column
//                         group g (128 bytes each), so no block carries padding.
//                         Chunk c of row k sits at slot c ^ ks_swz(k);
//                         fragments are two transposing 8-byte reads
//                         (ds_read_b64_tr_b16), which hand each lane 4
//                         consecutive k of one column.
// So every layout (forward, input-gradient and weight-gradient products)
// runs the same matrix-core loop without any explicit transpose.
//
// Each MFMA takes the B fragment as its first operand and the A fragment as
// its second, so that a lane ends up holding four consecutive output columns
// of one row: 8-byte bf16 / 16-byte fp32 stores, and the RoPE and SwiGLU
// partners of a column sit in the same lane.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "common.h"
#include "kernels.h"


namespace ls {

namespace {

constexpr int KT = 64;                      // tile depth
constexpr int KSTEPS = KT / 16;             // MFMA k-steps per tile
constexpr int TILE_ELEMS = 256 * KT;        // LDS region of one k-strided operand tile (32 KB)
constexpr int KC_PITCH = 1040;              // bytes per 1 KB block of a k-contiguous tile (16 B of padding)
constexpr int EPI_ROPE64 = 100;             // EPI_ROPE for 64-wide heads
constexpr uint32_t OOB = LS_OOB;
#ifndef GEMM_LOAD_SPAN_PCT
#define GEMM_LOAD_SPAN_PCT 60  // share of a tile's MFMA slots over which its loads are spread
#endif
#ifndef GEMM_LOAD_SPAN_NT
#define GEMM_LOAD_SPAN_NT 45  // the same for the forward (NT) products, whose loop has no transposing reads
#endif
#ifndef GEMM_READ_AHEAD
#define GEMM_READ_AHEAD 2  // k-steps between a fragment read and its MFMAs
#endif


// Launch order: workgroups are handed to the 8 XCDs round-robin, so first
// renumber them so that each XCD receives a contiguous range of logical tiles,
// then walk the tiles in groups of group_m tile rows so that the tiles an XCD
// works on at once share A rows and B columns in its L2.
// (Also run on the host, to pick group_m.)
__host__ __device__ inline void map_tile(int wg, int tiles_m, int tiles_n, int group_m, int& tm, int& tn) {
  const int nwg = tiles_m * tiles_n;
  const int q = nwg >> 3, r = nwg & 7, xcd = wg & 7, idx = wg >> 3;
  const int logical = (xcd < r ? xcd * (q + 1) : r * (q + 1) + (xcd - r) * q) + idx;
  const int group = group_m * tiles_n;
  const int g = logical / group;
  const int first_m = g * group_m;
  const int gm = tiles_m - first_m < group_m ? tiles_m - first_m : group_m;
  const int in_g = logical - g * group;
  tm = first_m + in_g % gm;
  tn = in_g / gm;
}

int group_rows(int M, int N, int K, int bm, int bn);

// LDS swizzles (XOR on the 16-byte chunk index).  The LDS serves 16 lanes of a
// 16-byte read (32 lanes of an 8-byte read) per clock across 64 banks, so:
//  - k-contiguous tiles (128-byte rows, 8 chunks): the 16 rows a 16-lane group
//    reads at one logical chunk must land on 16 distinct 16-byte bank groups of
//    a 256-byte window; r % 2 picks the row's half of the window, (r/2) % 8
//    the slot.
//  - k-strided tiles: a 32-lane transposing read covers 4 consecutive k-rows
//    (4-aligned) x 64 bytes.  With W = 256 the rows are 512 bytes apart, all at
//    the same offset of a 256-byte window, and XOR with 4 * (k % 4) puts their
//    64-byte runs on distinct quarters.  With W = 192 the rows of a block are
//    128 bytes apart (window offsets 0, 128, 0, 128), and XOR with
//    4 * ((k/2) % 2) moves the second pair by 64 bytes.
// Byte offset of tile row r in a k-contiguous tile: block (r % 8) + 8 (r / 64)
// of KC_PITCH bytes holds the 8 rows of one 64-row segment that are equal
// mod 8, at 128-byte positions (r / 8) % 8.
LS_DEV constexpr int kc_row_off(int r) { return ((r & 7) | ((r >> 6) << 3)) * KC_PITCH + ((r >> 3) & 7) * 128; }
template <int W>
LS_DEV int ks_swz(int k) {
  return W == 256 ? 4 * (k & 3) : 4 * ((k >> 1) & 1);
}
// Element offset of (k-row kk, column col) in a k-strided tile of width W.
template <int W>
LS_DEV int ks_off(int kk, int col) {
  if constexpr (W == 256) return (kk >> 1) * 512 + (kk & 1) * W + 8 * ((col >> 3) ^ ks_swz<W>(kk)) + (col & 7);
  else return ((col >> 6) * 8 + (kk >> 3)) * 512 + (kk & 7) * 64 + 8 * (((col & 63) >> 3) ^ ks_swz<W>(kk)) + (col & 7);
}
// 1 KB blocks (one load instruction each) of a k-strided tile of width W, and
// the first k-row of block j.
template <int W>
constexpr int ks_blocks() {
  return W == 256 ? 32 : 24;
}
template <int W>
LS_DEV int ks_row0(int j) {
  return W == 256 ? 2 * j : 8 * (j & 7);
}

LS_DEV float silu_f(float g) { return g * __frcp_rn(1.0f + __expf(-g)); }

// ---- operand loads ------------------------------------------------------------
// Each wave fills NL consecutive 1 KB blocks of an operand tile per k-tile
// (blocks wave*NL ..).  What does not change along k is computed once before
// the k loop: the per-lane byte offset of every load for a tile at k = 0
// (LS_OOB where the lane's row or column lies outside the operand) and the
// buffer resources.  Per k-tile only a scalar offset moves, and in a tile cut
// short by the end of K (or of a k segment of B) the lanes past the end read
// zeros.
//
// k-contiguous operand (rows m or n, 128-byte pieces of k): block j holds
// tile rows 8j .. 8j+7; lane l writes slot l%8 of row 8j + l/8 with that row's
// logical chunk c = (l%8) ^ kc_swz(row), i.e. k = k0 + 8c.  The chunk only
// depends on the parity of j.
// k-strided operand (rows k, columns m or n), W = 256: block j holds k-rows 2j
// and 2j+1 of the tile (32 chunks each); lane l writes slot l % 32 of k-row
// 2j + l / 32 with logical chunk slot ^ ks_swz(k-row).  W = 192: block 8g + b
// holds k-rows 8b .. 8b+7 of columns 64g .. 64g+63; lane l writes slot l % 8 of
// k-row 8b + l / 8.
template <int NL>
struct OpLoads {
  i32x4 r;            // resource of the operand (or of B's current k segment)
  uint32_t voff[NL];  // per-lane byte offsets of the loads for the tile at k = 0
  uint32_t kpos[2];   // k-contiguous: 8c for even / odd blocks; k-strided: the lane's k-row in its block
};

// k-contiguous operand.  Block j of the tile holds rows 64 (j / 8) + j % 8 +
// 8 i (i = 0..7): lane l of its load reads 16 bytes (k = k0 + 8 (l % 8) ..)
// of row i = l / 8 and writes them at 16 l of the block, so the lanes of a
// row read its 128 bytes in order.  The wave's blocks jb .. jb+NL-1 start at
// row res_row0 of a resource of `lrows` rows at `base` (leading dimension ld
// elements); when they span two 64-row segments the resource is one buffer.
template <int NL>
LS_DEV void kc_setup(OpLoads<NL>& o, const void* base, int res_row0, int lrows, int64_t ld, int lane, int jb) {
  o.r = rsrc(base, clamp_bytes((int64_t)lrows * ld * 2));
#pragma unroll
  for (int l = 0; l < NL; ++l) {
    const int j = jb + l;
    const int lr = res_row0 + 64 * ((j >> 3) - (jb >> 3)) + (j & 7) + 8 * (lane >> 3);
    o.voff[l] = lr < lrows ? (uint32_t)((int64_t)lr * ld * 2 + 16 * (lane & 7)) : OOB;
  }
  o.kpos[0] = 8 * (lane & 7);
  o.kpos[1] = 8 * (lane & 7);
}

// k-strided operand: columns col0 .. col0 + W - 1 of `cols`; the k rows are
// placed by the scalar offset (and the resource) of each tile.
template <int NL, int W, int NW>
LS_DEV void ks_setup(OpLoads<NL>& o, int col0, int cols, int64_t ld, int wave, int lane) {
  static_assert(NL * NW == ks_blocks<W>(), "one load per 1 KB block");
  constexpr int CPR = W == 256 ? 32 : 8;  // lanes per k-row
  const int sub = lane / CPR;              // the lane's k-row within its block
#pragma unroll
  for (int l = 0; l < NL; ++l) {
    const int j = wave * NL + l;
    const int kr = ks_row0<W>(j) + sub;
    const int col = col0 + (W == 256 ? 0 : 64 * (j >> 3)) + 8 * ((lane % CPR) ^ ks_swz<W>(kr));
    o.voff[l] = col < cols ? (uint32_t)((int64_t)kr * ld * 2 + col * 2) : OOB;
  }
  o.kpos[0] = sub;
  o.kpos[1] = sub;
}

// Offset of load l of a tile with `kvalid` valid k values (64 for a whole tile);
// W: the width of a k-strided tile (unused for k-contiguous ones).  FULL: the
// caller knows the tile is whole, so no lane is masked.
template <bool KC, int NL, int W, bool FULL>
LS_DEV uint32_t load_off(const OpLoads<NL>& o, int l, int kvalid, int wave) {
  if constexpr (FULL) return o.voff[l];
  bool ok;
  if constexpr (KC) ok = (int)o.kpos[l & 1] < kvalid;
  else ok = (int)o.kpos[0] < kvalid - ks_row0<W>(wave * NL + l);
  return ok ? o.voff[l] : OOB;
}

// Load l of an operand tile into the LDS block at byte address m0 + l KB
// (m0: the wave's first block of the stage).
template <bool KC, int NL, int W, bool FULL>
LS_DEV void load_one(const OpLoads<NL>& o, int l, uint32_t soff, int kvalid, uint32_t m0, int wave) {
  dma1(o.r, load_off<KC, NL, W, FULL>(o, l, kvalid, wave), soff, m0 + (KC ? (uint32_t)KC_PITCH : 1024u) * l);
}

// Fragment of a k-contiguous tile (at byte address t): lane gets row `r`
// (tile-local), k = 16s + 8*(lane/32) .. +7.  The 16 rows a 16-lane group
// reads at one k step sit in 16 distinct 16-byte bank groups.
LS_DEV u32x4 frag_kc(const char* t, int r, int s, int lh) {
  return *(const u32x4*)(t + kc_row_off(r) + 16 * (2 * s + lh));
}

// Fragment of a k-strided tile (width W) for the 32 columns starting at c32
// (tile-local): lane gets column c32 + lane%32, k = 16s + 8*(lane/32) .. +7,
// via two transposing reads.
template <int W>
LS_DEV u32x4 frag_ks(const bf16_t* lds, int c32, int s, int lane) {
  const int g = lane >> 4, q = lane & 15;
  const int col = c32 + 16 * (g & 1) + 4 * (q & 3);
  u32x4 out;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int kk = 16 * s + 8 * (g >> 1) + 4 * t + (q >> 2);
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS s16x4*)(lds + ks_off<W>(kk, col)));
    const u32x2 w = __builtin_bit_cast(u32x2, v);
    out[2 * t] = w[0];
    out[2 * t + 1] = w[1];
  }
  return out;
}

// 16 bytes (8 consecutive bf16) of row lr per lane from the MFMA layout: the
// lane holds columns 8q + 4lh .. +3 of one row for q = 2pp, 2pp+1 (packed in
// w0 and w1); lanes lr and lr + 32 swap halves (v_permlane32_swap: lanes 32..63
// of the first operand trade places with lanes 0..31 of the second), after
// which the lane holds columns 16pp + 8lh .. +7.
LS_DEV u32x4 swap_pack(u32x2 w0, u32x2 w1) {
  const auto x = __builtin_amdgcn_permlane32_swap(w0[0], w1[0], false, false);
  const auto y = __builtin_amdgcn_permlane32_swap(w0[1], w1[1], false, false);
  return u32x4{x[0], y[0], x[1], y[1]};
}
// The same for fp32 values: v0, v1 hold columns 8q + 4lh .. +3 (q = 2pp,
// 2pp+1); afterwards lo and hi hold columns 16pp + 8lh + 0..3 and + 4..7.
LS_DEV void swap_f32(f32x4 v0, f32x4 v1, f32x4& lo, f32x4& hi) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const auto t = __builtin_amdgcn_permlane32_swap(__float_as_uint(v0[e]), __float_as_uint(v1[e]), false, false);
    lo[e] = __uint_as_float(t[0]);
    hi[e] = __uint_as_float(t[1]);
  }
}
LS_DEV u32x2 pack4(float a, float b, float c, float d) { return u32x2{pack_bf2(a, b), pack_bf2(c, d)}; }

template <bool AK, bool BKC, int EPI, int BM, int BN, int NW>
__global__ __launch_bounds__(NW * 64, 1) void gemm_kernel(GemmArgs p) {
  // NW waves: 4 (one per SIMD, 2 x 2 wave tiles) or 8 (two per SIMD, 4 x 2)
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");
  constexpr int WM = BM / (NW / 2), WN = BN / 2;  // wave tile
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tiles of whole 32 x 32 blocks");
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int NA = AK ? BM / (8 * NW) : ks_blocks<BM>() / NW;  // loads per wave and tile
  constexpr int NB = BKC ? BN / (8 * NW) : ks_blocks<BN>() / NW;
  constexpr int NL = NA + NB;                                    // loads per wave and tile
  constexpr int NMF = TM * TN;                                   // MFMAs per k-step
  constexpr int NRU = TM + TN;                                   // fragments per k-step
  // The last k-step of a tile runs BAR_AT MFMAs, then waits for the next
  // tile's loads and for the other waves, then reads the next tile's first
  // fragments between its remaining MFMAs.  From the same point on, the
  // loads of the tile after next go into the stage this tile has just
  // released, spread evenly over the next LSPAN MFMA slots (into the next
  // tile): issued back to back, the four waves' loads outrun the rate at which
  // the texture units take buffer->LDS loads, and a wave whose load does not
  // fit into the full address queue stalls its matrix core.  The rest of the
  // period is left for the last loads to arrive.
  constexpr int BAR_AT = NMF >= 16 ? 2 : 1;
  static_assert(BAR_AT + NRU <= NMF, "the next tile's first fragments are read within one k-step");
  constexpr int LSPAN = (KSTEPS * NMF * (AK && BKC ? GEMM_LOAD_SPAN_NT : GEMM_LOAD_SPAN_PCT)) / 100;
  static_assert(BAR_AT + LSPAN < KSTEPS * NMF, "every load is issued before the next barrier");
  // Fragments are read RA k-steps ahead of the MFMAs that use them (RA + 1
  // register buffers; with RA = 2 four, one per k-step of a tile), so that a
  // read delayed by the buffer->LDS writes does not hold up the matrix core.
  // Measured: two steps with one wave per SIMD, one with two waves per SIMD.
  constexpr int RA = NW == 8 ? 1 : GEMM_READ_AHEAD;
  static_assert(RA == 1 || RA == 2, "read-ahead of one or two k-steps");
  constexpr int NBUF = RA == 1 ? 2 : 4;
  constexpr int BS = KSTEPS - RA;  // the k-step of a tile that holds the barrier
  constexpr bool KSEG = !BKC;  // a k-strided B may come from up to three buffers along k
  constexpr bool GLU = EPI == EPI_GLU_FWD;
  constexpr uint32_t A_BYTES = AK ? (BM / 8) * KC_PITCH : TILE_ELEMS * 2;
  constexpr uint32_t B_BYTES = BKC ? (BN / 8) * KC_PITCH : TILE_ELEMS * 2;
  constexpr uint32_t STAGE_BYTES = A_BYTES + B_BYTES;
  // the epilogue stages results in the first 128 KB
  constexpr uint32_t LDS_BYTES = 2 * STAGE_BYTES > 4 * TILE_ELEMS * 2 ? 2 * STAGE_BYTES : 4 * TILE_ELEMS * 2;
  // Two LDS stages of [A tile | B tile].  The buffer->LDS loads are inline
  // assembly the compiler does not see, so the stage can be picked at run time.
  constexpr uint32_t PF_LDS = EPI == EPI_GLU_BWD ? 1024 : 0;
  __shared__ __attribute__((aligned(1024))) char lds[LDS_BYTES + PF_LDS];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / 2, wn = wave % 2;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  // fp32 weight gradients may split K: workgroup x runs slice x / tiles of tile x % tiles
  const int ks = EPI == EPI_F32 ? p.ksplit : 1;
  const int slice = ks > 1 ? (int)blockIdx.x / (tiles_m * tiles_n) : 0;
  int tm, tn;
  map_tile((int)blockIdx.x - slice * tiles_m * tiles_n, tiles_m, tiles_n, p.group_m, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int K = p.K;

  // k segments of B: [0, S1), [S1, S2), [S2, K) (one segment unless a
  // k-strided B is split over buffers).  The tiles of a segment start at its
  // first k; the last one may be cut short.
  int S1 = K, S2 = K;
  if constexpr (KSEG) {
    S1 = min(p.b_start[1], K);
    S2 = max(S1, min(p.b_start[2], K));
  }
  int kbeg = 0, kend = K;  // k range of this workgroup (a slice of the k tiles when K is split)
  auto seg_end = [&](int k) { return min(kend, k < S1 ? S1 : (k < S2 ? S2 : K)); };
  int nk = (S1 + KT - 1) / KT + (S2 - S1 + KT - 1) / KT + (K - S2 + KT - 1) / KT;
  if (ks > 1) {  // slice j: k tiles [j nk / ks, (j+1) nk / ks) of the whole sequence
    const int n0t = (S1 + KT - 1) / KT, n1t = (S2 - S1 + KT - 1) / KT;
    auto k_of = [&](int t) { return t < n0t ? t * KT : (t < n0t + n1t ? S1 + (t - n0t) * KT : S2 + (t - n0t - n1t) * KT); };
    const int t0 = (int)((int64_t)slice * nk / ks), t1 = (int)((int64_t)(slice + 1) * nk / ks);
    kbeg = k_of(t0);
    kend = t1 == nk ? K : k_of(t1);
    nk = t1 - t0;
  }

  OpLoads<NA> la;
  OpLoads<NB> lb;
  if constexpr (AK) {
    kc_setup(la, p.A, m0 + 64 * (wave * NA >> 3), p.M, p.lda, lane, wave * NA);
  } else {
    ks_setup<NA, BM, NW>(la, m0, p.M, p.lda, wave, lane);
    la.r = rsrc(p.A, clamp_bytes((int64_t)K * p.lda * 2));
  }
  if constexpr (BKC) {
    const int rb = n0 + 64 * (wave * NB >> 3);  // first row of the wave's 64-row segment (uniform)
    if constexpr (GLU) {
      // gate and up rows interleaved in blocks of 64: a wave's blocks lie in one segment
      static_assert(BN == 256, "a wave's blocks in one 64-row segment");
      kc_setup(lb, (rb >> 6) & 1 ? p.B[1] : p.B[0], (rb >> 7) * 64, p.glu_rows, p.ldb, lane, wave * NB);
    } else {
      // row segments start at multiples of 64; a wave's blocks lie in one of them
      // when B is split (256-wide tiles), or span two of a single buffer
      const int sg = rb >= p.b_start[2] ? 2 : (rb >= p.b_start[1] ? 1 : 0);
      const int st = sg == 2 ? p.b_start[2] : (sg == 1 ? p.b_start[1] : 0);
      const int en = min(p.N, sg == 2 ? p.N : (sg == 1 ? p.b_start[2] : p.b_start[1]));
      kc_setup(lb, p.B[sg], rb - st, en - st, p.ldb, lane, wave * NB);
    }
  } else {
    ks_setup<NB, BN, NW>(lb, n0, p.N, p.ldb, wave, lane);
    if constexpr (!KSEG) lb.r = rsrc(p.B[0], clamp_bytes((int64_t)K * p.ldb * 2));
  }

  // The load cursor: first k of the next tile to load, its valid k count and
  // the scalar offsets of both operands (B's resource follows its segment).
  int ck = 0, kval = 0;
  uint32_t soa = 0, sob = 0;
  auto set_cursor = [&](int k0) {
    ck = k0;
    const int se = seg_end(k0);
    kval = min(KT, se - k0);
    soa = AK ? (uint32_t)(k0 * 2) : (uint32_t)((int64_t)k0 * p.lda * 2);
    if constexpr (KSEG) {
      const int sg = k0 >= S2 ? 2 : (k0 >= S1 ? 1 : 0);
      const int st = sg == 2 ? S2 : (sg == 1 ? S1 : 0);
      const bf16_t* bp = p.B[sg] ? p.B[sg] : p.B[0];
      lb.r = rsrc(bp, clamp_bytes((int64_t)(se - st) * p.ldb * 2));
      sob = (uint32_t)((int64_t)(k0 - st) * p.ldb * 2);
    } else {
      sob = BKC ? (uint32_t)(k0 * 2) : (uint32_t)((int64_t)k0 * p.ldb * 2);
    }
  };
  // The next tile's cursor.
  auto advance = [&]() { set_cursor(ck + kval); };
  const uint32_t lds0 = lds_offset(&lds[0]);
  const uint32_t ma = lds0 + wave * NA * (AK ? KC_PITCH : 1024), mb = lds0 + A_BYTES + wave * NB * (BKC ? KC_PITCH : 1024);
  // Load q of the tile at the cursor (A loads first) into the stage at byte
  // offset stage_off; full_c: std::true_type where that tile is known to be whole.
  auto issue = [&](auto full_c, int q, uint32_t stage_off) {
    constexpr bool FULL = decltype(full_c)::value;
    if (q < NA) load_one<AK, NA, BM, FULL>(la, q, soa, kval, ma + stage_off, wave);
    else load_one<BKC, NB, BN, FULL>(lb, q - NA, sob, kval, mb + stage_off, wave);
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int lr = lane & 31, lh = lane >> 5;
  u32x4 af[NBUF][TM], bfr[NBUF][TN];
  // Fragment u of a k-step: A fragments 0 .. TM-1, then B fragments.
  auto read_unit = [&](int stage, int s, int buf, int u) {
    const char* as = lds + stage * STAGE_BYTES;
    const char* bs = as + A_BYTES;
    if (u < TM) {
      af[buf][u] = AK ? frag_kc(as, wm * WM + 32 * u + lr, s, lh) : frag_ks<BM>((const bf16_t*)as, wm * WM + 32 * u, s, lane);
    } else {
      const int v = u - TM;
      bfr[buf][v] = BKC ? frag_kc(bs, wn * WN + 32 * v + lr, s, lh) : frag_ks<BN>((const bf16_t*)bs, wn * WN + 32 * v, s, lane);
    }
  };

  // MFMA slot (counted from the start of the barrier's k-step) of load q of
  // the tile after next.
  constexpr auto slot_of = [](int q) { return BAR_AT + (q * LSPAN) / NL; };
  constexpr auto bufi = [](int s) { return NBUF == 4 ? s : s & 1; };

  // One 64-k tile in stage `cur` (NX: how many of the next two tiles exist).
  // The k loop is one continuous stream of 16-k steps: the fragments of step
  // s+RA are read between the MFMAs of step s, across tile boundaries too.  In
  // k-step BS each wave waits for its loads of the next tile (vmcnt) and for
  // the other waves (barrier): then the next tile is in LDS and every wave is
  // done reading this stage (its last fragments were read one step earlier),
  // so the loads of the tile after next can go into it while the MFMAs run.
  // Every instruction is pinned in place with scheduling barriers.
  //
  // SwiGLU backward: the saved gate/up rows of this tile (256 rows x 2 x 512
  // bytes, 2048 lines of 128 bytes) are touched during the last 36 k-tiles of
  // the main loop but 4, one 64-line gather per k-tile (lane l: row l / 8,
  // gate or up, 64-element segment l % 4) into a 1 KB LDS scratch block, so
  // that the epilogue finds them in the last-level cache instead of HBM.  The
  // gather follows the barrier, so it has a whole k-tile to arrive before the
  // next barrier waits for the wave's loads.  Measured: dact 437-441 -> 424-425
  // us at the 3B shape.
  int kt = 0;
  i32x4 pf_r = {0, 0, 0, 0};
  uint32_t pf_voff = 0;
  if constexpr (EPI == EPI_GLU_BWD) {
    const int64_t ld2 = 2 * (int64_t)p.glu_I;
    pf_r = rsrc(p.gu_in + (int64_t)m0 * ld2, clamp_bytes((int64_t)(p.M - m0) * ld2 * 2));
    const int part = lane & 7, arr = part >> 2, seg = part & 3;
    pf_voff = (uint32_t)(((int64_t)(lane >> 3) * ld2 + arr * p.glu_I + n0 + seg * 64) * 2);
  }
  const int pf_first = nk - 36;
  // cur_c: the stage, a compile-time constant in the unrolled loop over whole
  // tiles (every LDS address is then a register plus an immediate) or an int;
  // full_c: every tile this one loads is whole (no lane masking).
  auto tile = [&](auto nx_c, auto cur_c, auto full_c) {
    constexpr int NX = decltype(nx_c)::value;
    const int cur = cur_c;
    const uint32_t here = (uint32_t)cur * STAGE_BYTES, there = (uint32_t)(cur ^ 1) * STAGE_BYTES;
    static_for<KSTEPS>([&](auto s_c) {
      constexpr int s = s_c;
      constexpr int buf = bufi(s);
      constexpr int t = s + RA;  // step whose fragments are read now (>= KSTEPS: the next tile's)
      static_for<NMF>([&](auto i_c) {
        constexpr int i = i_c;
        if constexpr (NX >= 1 && s == BS && i == BAR_AT) {
          sync_lds();
          if constexpr (EPI == EPI_GLU_BWD) {
            const int j = kt - pf_first;
            if (j >= 0 && j < 32 && (j & (NW - 1)) == wave)
              dma1(pf_r, pf_voff, (uint32_t)((int64_t)j * 8 * 2 * p.glu_I * 2), lds0 + LDS_BYTES);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        acc[i / TN][i % TN] = mfma32(bfr[buf][i % TN], af[buf][i / TN], acc[i / TN][i % TN]);
        if constexpr (t < KSTEPS) {
          if constexpr (i < NRU) read_unit(cur, t, bufi(t), i);
        } else if constexpr (NX >= 1) {
          constexpr int u = s == BS ? i - BAR_AT : i;
          if constexpr (u >= 0 && u < NRU) read_unit(cur ^ 1, t - KSTEPS, bufi(t - KSTEPS), u);
        }
        static_for<NL>([&](auto q_c) {
          constexpr int q = q_c;
          constexpr int at = slot_of(q) + BS * NMF;  // tile-relative slot of load q (may be in the next tile)
          // the later loads of the next tile (its first ones went out in the previous tile)
          if constexpr (NX >= 1 && at >= KSTEPS * NMF && at - KSTEPS * NMF == s * NMF + i) {
            issue(full_c, q, there);
            if constexpr (q == NL - 1) advance();
          }
          // the first loads of the tile after next, into this stage
          if constexpr (NX >= 2 && at < KSTEPS * NMF && at == s * NMF + i) {
            issue(full_c, q, here);
            if constexpr (q == NL - 1) advance();
          }
        });
        __builtin_amdgcn_sched_barrier(0);
      });
    });
  };

  // Prologue: tile 0 whole, then the loads of tile 1 that the previous tile
  // would have issued in its last k-step; wait for tile 0.
  constexpr int FIRST = [] {
    int n = 0;
    for (int q = 0; q < NL; ++q) n += BAR_AT + (q * LSPAN) / NL + BS * NMF < KSTEPS * NMF;
    return n;
  }();
  set_cursor(kbeg);
#pragma unroll
  for (int q = 0; q < NL; ++q) issue(std::false_type{}, q, 0);
  advance();
  if (nk > 1) {
#pragma unroll
    for (int q = 0; q < FIRST; ++q) issue(std::false_type{}, q, STAGE_BYTES);
    if (FIRST == NL) advance();
    LS_WAIT_VMCNT(FIRST);
  } else {
    LS_WAIT_VMCNT(0);
  }
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
#pragma unroll
  for (int t = 0; t < RA; ++t)
#pragma unroll
    for (int u = 0; u < NRU; ++u) read_unit(0, t, bufi(t), u);
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  // Every tile of every k segment whole (k lengths multiples of the tile
  // depth): no load masks, and with one wave per SIMD two tiles per pass, one
  // per stage, so every fragment address is a register plus an immediate (with
  // two waves per SIMD that copy of the loop needs more registers than a wave
  // has and spills).
  const bool whole = S1 % KT == 0 && (S2 - S1) % KT == 0 && (K - S2) % KT == 0;
  if (whole) {
    if constexpr (NW == 4) {
      for (; kt + 3 < nk; kt += 2) {
        tile(I2{}, I0{}, std::true_type{});
        tile(I2{}, I1{}, std::true_type{});
      }
    } else {
      for (; kt + 2 < nk; ++kt) tile(I2{}, kt & 1, std::true_type{});
    }
  }
  for (; kt + 2 < nk; ++kt) tile(I2{}, kt & 1, std::false_type{});
  if (kt + 1 < nk) tile(I1{}, kt++ & 1, std::false_type{});
  tile(I0{}, kt & 1, std::false_type{});
  auto sync_tile = []() { sync_lds(); };
  sync_tile();  // every wave is done with both stages before they become staging space

  // ---- epilogue ---------------------------------------------------------------
  // Lane holds C[32i + lr][32j + 8q + 4lh .. +3] of its wave tile (acc[i][j][4q..]).
  // Results go through a 32 KB LDS region per wave so that global loads and
  // stores move whole row segments (16 bytes per lane).  Staging rows have a
  // fixed pitch (bf16: 128 columns = 256 B, up to 128 rows; fp32: 128 columns =
  // 512 B, 32 rows) with the 16-byte chunk index XOR-swizzled by the row, so the
  // column-wise writes from the MFMA layout and the row-wise reads both avoid
  // bank conflicts; a 96-wide wave tile uses 12 of the 16 (24 of the 32) chunks.
  bf16_t* stg = (bf16_t*)lds + wave * (4 * TILE_ELEMS / NW);  // 128 KB / NW per wave
  float* stgf = (float*)stg;
  auto sb = [](int r, int col) { return r * 128 + ((((col >> 3) ^ (r & 15)) << 3) | (col & 7)); };
  auto sf = [](int r, int col) { return r * 128 + ((((col >> 2) ^ (r & 31)) << 2) | (col & 3)); };
  const int mw = m0 + wm * WM, nw = n0 + wn * WN;

  // bf16 staging: WM rows x WN columns -> rows of `dst` (row-major, ld) from column col0
  auto put4 = [&](int r, int c, const float v[4]) {
    *(u32x2*)&stg[sb(r, c)] = u32x2{pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3])};
  };
  auto flush_bf16 = [&](bf16_t* dst, int64_t ldd, int col0, int ncols_valid) {
#pragma unroll 4
    for (int t = 0; t < WM / 4; ++t) {
      const int c = lane + 64 * t, r = c >> 4, cc = c & 15;
      const u32x4 v = *(const u32x4*)&stg[sb(r, cc * 8)];
      if (cc < WN / 8 && mw + r < p.M && cc * 8 < ncols_valid)
        *(u32x4*)(dst + (int64_t)(mw + r) * ldd + col0 + cc * 8) = v;
    }
  };

  if constexpr (EPI == EPI_F32) {
    // fp32 weight gradients straight from the registers: a lane's 4 columns are
    // 16 contiguous bytes (read-modify-write with accumulate).  Slices 1.. of a
    // split K store plain partial sums ([M][N] each) for kpart_reduce_kernel.
    float* kp = slice > 0 ? p.kpart + (int64_t)(slice - 1) * p.M * p.N : nullptr;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = mw + 32 * i + lr;
      const int sg = m >= p.f_start[2] ? 2 : (m >= p.f_start[1] ? 1 : 0);
      float* base = sg == 2 ? p.F[2] : (sg == 1 ? p.F[1] : p.F[0]);
      const int fs = sg == 2 ? p.f_start[2] : (sg == 1 ? p.f_start[1] : 0);
      float* row = kp ? kp + (int64_t)m * p.N : base + (int64_t)(m - fs) * p.ldf;
      // the accumulated values of the row block, all loads in flight at once
      // (one at a time, each load and store waited for the one before)
      f32x4 old[TN][4];
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int n = nw + 32 * j + 8 * q + 4 * lh;
          old[j][q] = f32x4{0.f, 0.f, 0.f, 0.f};
          if (p.accumulate && !kp && m < p.M && n < p.N) old[j][q] = *(const f32x4*)(row + n);
        }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < TN; ++j) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int n = nw + 32 * j + 8 * q + 4 * lh;
          const f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
          if (m < p.M && n < p.N) *(f32x4*)(row + n) = v + old[j][q];
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  } else if constexpr (EPI == EPI_RESID) {
    // Straight from the registers: the fp32 results are moved into 16-byte
    // row pieces (8 columns per lane), added to the residual (one 16-byte
    // load each, a row block's loads issued together) and rounded once.
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = mw + 32 * i + lr;
      // the residual pieces of the row block, all loads in flight at once
      u32x4 res[TN][2];
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
          const int n = nw + 32 * j + 16 * pp + 8 * lh;
          res[j][pp] = m < p.M && n < p.N ? *(const u32x4*)(p.R + (int64_t)m * p.ldc + n) : u32x4{0u, 0u, 0u, 0u};
        }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
          const int n = nw + 32 * j + 16 * pp + 8 * lh;
          f32x4 lo, hi;
          swap_f32(f32x4{acc[i][j][8 * pp], acc[i][j][8 * pp + 1], acc[i][j][8 * pp + 2], acc[i][j][8 * pp + 3]},
                   f32x4{acc[i][j][8 * pp + 4], acc[i][j][8 * pp + 5], acc[i][j][8 * pp + 6], acc[i][j][8 * pp + 7]},
                   lo, hi);
          if (m < p.M && n < p.N) {
            const u32x4 rw = res[j][pp];
            *(u32x4*)(p.C + (int64_t)m * p.ldc + n) =
                u32x4{pack_bf2(lo[0] + bf_lo(rw[0]), lo[1] + bf_hi(rw[0])), pack_bf2(lo[2] + bf_lo(rw[1]), lo[3] + bf_hi(rw[1])),
                      pack_bf2(hi[0] + bf_lo(rw[2]), hi[1] + bf_hi(rw[2])), pack_bf2(hi[2] + bf_lo(rw[3]), hi[3] + bf_hi(rw[3]))};
          }
          __builtin_amdgcn_sched_barrier(0);
        }
    }
  } else if constexpr (EPI == EPI_GLU_FWD) {
    static_assert(WN == 128, "gate/up interleave needs 128-column wave tiles");
    // subtiles j = 0, 1 hold gate columns, j = 2, 3 the up columns of the same 64 features
    const int col0 = nw / 2;  // first feature of the wave tile
    const int nvalid = p.glu_I - col0;
    // One 32-row block at a time: its gate and up values (rows 0..31 of the
    // staging region, [g(64) | u(64)]) and its act values (rows 32..63, 64
    // columns) are staged, then stored while the next block is computed; each
    // block's accumulators are done with after it (fewer live registers than
    // staging all gate/up rows first and computing act from them afterwards).
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float g[4], u[4], a[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            g[e] = acc[i][j][4 * q + e];
            u[e] = acc[i][j + 2][4 * q + e];
            a[e] = silu_f(g[e]) * u[e];
          }
          if (p.C) {
            put4(lr, 32 * j + 8 * q + 4 * lh, g);
            put4(lr, 64 + 32 * j + 8 * q + 4 * lh, u);
          }
          put4(32 + lr, 32 * j + 8 * q + 4 * lh, a);
        }
      const int mb = mw + 32 * i;
      if (p.C) {
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int c = lane + 64 * t, r = c >> 4, cc = c & 15;
          const u32x4 v = *(const u32x4*)&stg[sb(r, cc * 8)];
          const int f = (cc & 7) * 8;  // feature offset within the 64
          if (mb + r < p.M && f < nvalid)
            *(u32x4*)(p.C + (int64_t)(mb + r) * p.ldc + (cc < 8 ? 0 : p.glu_I) + col0 + f) = v;
        }
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int c = lane + 64 * t, r = c >> 3, cc = c & 7;
        const u32x4 v = *(const u32x4*)&stg[sb(32 + r, cc * 8)];
        if (mb + r < p.M && cc * 8 < nvalid) *(u32x4*)(p.act + (int64_t)(mb + r) * p.glu_I + col0 + cc * 8) = v;
      }
    }
  } else if constexpr (EPI == EPI_GLU_BWD) {
    static_assert(WN == 128, "the gate/up staging covers 128-column wave tiles");
    // acc = dact.  Per 32-row block: the saved gate and up values are read
    // coalesced into LDS, dg = dact u silu'(g) and du = dact silu(g) replace
    // them in place, and both go out coalesced.  The reads run two blocks
    // ahead (in registers the main loop no longer needs), so each block's
    // values have arrived when it is processed.
    bf16_t* sg_ = stg;             // gate / dg rows (32 x 128)
    bf16_t* su_ = stg + 32 * 128;  // up / du rows
    // (two blocks in flight with one wave per SIMD; one with two, whose
    // registers are half as many)
    constexpr int PF = NW == 8 ? 1 : 2;
    u32x4 gpre[PF][8], upre[PF][8];
    auto fetch = [&](int i, int b) {
      const int mb = mw + 32 * i;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int c = lane + 64 * t, r = c >> 4, cc = c & 15;
        u32x4 gv = {0u, 0u, 0u, 0u}, uv = {0u, 0u, 0u, 0u};
        if (mb + r < p.M && nw + cc * 8 < p.N) {
          const bf16_t* src = p.gu_in + (int64_t)(mb + r) * 2 * p.glu_I + nw + cc * 8;
          gv = *(const u32x4*)src;
          uv = *(const u32x4*)(src + p.glu_I);
        }
        gpre[b][t] = gv;
        upre[b][t] = uv;
      }
    };
    fetch(0, 0);
    if constexpr (TM > 1 && PF > 1) fetch(1, 1);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int mb = mw + 32 * i;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int c = lane + 64 * t, r = c >> 4, cc = c & 15;
        *(u32x4*)&sg_[sb(r, cc * 8)] = gpre[i % PF][t];
        *(u32x4*)&su_[sb(r, cc * 8)] = upre[i % PF][t];
      }
      if (i + PF < TM) fetch(i + PF, i % PF);
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int off = sb(lr, 32 * j + 8 * q + 4 * lh);
          const u32x2 gw = *(const u32x2*)&sg_[off], uw = *(const u32x2*)&su_[off];
          const float g[4] = {bf_lo(gw[0]), bf_hi(gw[0]), bf_lo(gw[1]), bf_hi(gw[1])};
          const float u[4] = {bf_lo(uw[0]), bf_hi(uw[0]), bf_lo(uw[1]), bf_hi(uw[1])};
          float dg[4], du[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float da = acc[i][j][4 * q + e];
            const float sgm = __frcp_rn(1.0f + __expf(-g[e]));
            dg[e] = da * u[e] * sgm * (1.0f + g[e] * (1.0f - sgm));
            du[e] = da * g[e] * sgm;
          }
          *(u32x2*)&sg_[off] = u32x2{pack_bf2(dg[0], dg[1]), pack_bf2(dg[2], dg[3])};
          *(u32x2*)&su_[off] = u32x2{pack_bf2(du[0], du[1]), pack_bf2(du[2], du[3])};
        }
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int c = lane + 64 * t, r = c >> 4, cc = c & 15;
        if (mb + r < p.M && nw + cc * 8 < p.N) {
          bf16_t* dst = p.C + (int64_t)(mb + r) * p.ldc + nw + cc * 8;
          *(u32x4*)dst = *(const u32x4*)&sg_[sb(r, cc * 8)];
          *(u32x4*)(dst + p.glu_I) = *(const u32x4*)&su_[sb(r, cc * 8)];
        }
      }
    }
  } else {
    // EPI_BF16, EPI_ROPE, EPI_ROPE64
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = mw + 32 * i + lr;
      if constexpr (EPI == EPI_ROPE || EPI == EPI_ROPE64) {
        constexpr int HD = EPI == EPI_ROPE ? 128 : 64, HALF = HD / 2, JP = HALF / 32;
        static_assert(WN % HD == 0, "wave tiles hold whole heads");
        const int pos = (m < p.M ? m : 0) % p.seq;
        const float* cs = p.rope_cs + (int64_t)pos * HALF;
        const float* sn = p.rope_cs + (int64_t)p.seq * HALF + (int64_t)pos * HALF;
        // cos and sin of the lane's 4 consecutive angle indices at each 32-column
        // offset of the first half of a head (16-byte loads), all in flight at
        // once before the rotations that use them
        f32x4 cpre[JP][4], spre[JP][4];
#pragma unroll
        for (int d = 0; d < JP; ++d)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            cpre[d][q] = f32x4{1.f, 1.f, 1.f, 1.f};
            spre[d][q] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (nw < p.rope_cols) {
              cpre[d][q] = *(const f32x4*)(cs + 32 * d + 8 * q + 4 * lh);
              spre[d][q] = *(const f32x4*)(sn + 32 * d + 8 * q + 4 * lh);
            }
          }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const bool rot = nw + 32 * j < p.rope_cols;
          const int dcol = (32 * j) % HD;  // wave tiles start on a head boundary
          if (rot && dcol >= HALF) continue;  // written together with its partner
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float lo[4], hi[4];
            const f32x4 c4 = cpre[(dcol / 32) % JP][q], s4 = spre[(dcol / 32) % JP][q];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float x1 = acc[i][j][4 * q + e];
              if (rot && j + JP < TN) {
                const float c = c4[e], sv = s4[e];
                const float x2 = acc[i][(j + JP) % TN][4 * q + e];
                lo[e] = x1 * c - x2 * sv;
                hi[e] = x2 * c + x1 * sv;
              } else {
                lo[e] = x1;
              }
            }
            put4(32 * i + lr, 32 * j + 8 * q + 4 * lh, lo);
            if (rot && j + JP < TN) put4(32 * i + lr, 32 * (j + JP) + 8 * q + 4 * lh, hi);
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * q + e];
            put4(32 * i + lr, 32 * j + 8 * q + 4 * lh, v);
          }
      }
    }
    flush_bf16(p.C, p.ldc, nw, p.N - nw);
  }
}

// Waves per workgroup, chosen by measurement on the block's products: two per
// SIMD (8) for the weight-gradient (TN) products and the input-gradient (NN)
// product with the SwiGLU backward epilogue (which then prefetches one 32-row
// block of the saved gate/up values instead of two); one per SIMD (4) for the
// forward (NT) products and the plain input-gradient ones (whose main loop,
// with the registers of one wave per SIMD, runs two tiles per pass).  BM = 192
// tiles keep 4 (a wave tile of 48 rows is not whole 32-row blocks).
template <bool AK, bool BKC, int EPI, int BM>
constexpr int waves_of() {
  return BM == 256 && (!AK || (!BKC && EPI == EPI_GLU_BWD)) ? 8 : 4;
}
template <bool AK, bool BKC, int EPI, int BM, int BN, int NW = waves_of<AK, BKC, EPI, BM>()>
hipError_t launch(const GemmArgs& args, hipStream_t s) {
  GemmArgs a = args;
  a.group_m = group_rows(a.M, a.N, a.K, BM, BN);
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_kernel<AK, BKC, EPI, BM, BN, NW>), dim3(tiles * a.ksplit), dim3(NW * 64), 0, s, a);
  return hipGetLastError();
}

// F (already holding slice 0's result, with the accumulate read) += the
// partial sums of slices 1 .. ksplit-1, added in slice order.  N % 4 == 0.
__global__ __launch_bounds__(256) void kpart_reduce_kernel(GemmArgs p) {
  const int64_t per = (int64_t)p.M * p.N, n4 = per / 4;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    const int64_t e = 4 * i;
    const int m = (int)(e / p.N), n = (int)(e - (int64_t)m * p.N);
    const int sg = m >= p.f_start[2] ? 2 : (m >= p.f_start[1] ? 1 : 0);
    float* base = sg == 2 ? p.F[2] : (sg == 1 ? p.F[1] : p.F[0]);
    const int fs = sg == 2 ? p.f_start[2] : (sg == 1 ? p.f_start[1] : 0);
    float* dst = base + (int64_t)(m - fs) * p.ldf + n;
    f32x4 v = *(const f32x4*)dst;
    for (int j = 0; j < p.ksplit - 1; ++j) v += *(const f32x4*)(p.kpart + j * per + e);
    *(f32x4*)dst = v;
  }
}

int compute_units() {
  static const int n = [] {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        v <= 0)
      v = 256;
    return v;
  }();
  return n;
}

// Tile rows per group of the launch order (map_tile) for an M x N x K product
// in BM x BN tiles.  Two caches decide it.  The workgroups an XCD runs at once
// (one per CU, 32) cover g tile rows x 32/g tile columns and stream g A panels
// of BM rows and 32/g B panels of BN rows along K through its 4 MB L2: fewer
// panel rows, fewer L2 misses (4 for 256 x 192 tiles, 8 for 192 x 256).  And
// the panels the whole chip reads in its first round of workgroups should fit
// the 256 MB last-level cache, or every round fetches them from HBM again:
// for K = 16384 and 368 MB of operands only g = 2 keeps a round within it.
// So: among g = 8, 4, 2 whose first round fits, the fewest panel rows (the
// larger g on a tie); if none fits, the smallest first-round footprint.
int group_rows(int M, int N, int K, int bm, int bn) {
  const int tiles_m = (M + bm - 1) / bm, tiles_n = (N + bn - 1) / bn;
  const int ncu = compute_units(), round = std::min(tiles_m * tiles_n, ncu), per_xcd = std::max(ncu / 8, 1);
  constexpr int64_t LLC_BYTES = (int64_t)256 << 20;
  constexpr int MAX_TILES = 4096;  // per dimension (no allocation in a call): larger grids keep 8
  if (tiles_m > MAX_TILES || tiles_n > MAX_TILES) return 8;
  int best = 8;
  bool best_fits = false;
  int64_t best_rows = 0, best_bytes = 0;
  char used_m[MAX_TILES], used_n[MAX_TILES];
  for (int g : {8, 4, 2}) {
    std::fill(used_m, used_m + tiles_m, 0);
    std::fill(used_n, used_n + tiles_n, 0);
    for (int wg = 0; wg < round; ++wg) {
      int tm, tn;
      map_tile(wg, tiles_m, tiles_n, g, tm, tn);
      used_m[tm] = used_n[tn] = 1;
    }
    const int64_t panels = (int64_t)std::count(used_m, used_m + tiles_m, 1) * bm +
                           (int64_t)std::count(used_n, used_n + tiles_n, 1) * bn;
    const int64_t bytes = panels * K * 2, rows = (int64_t)g * bm + (int64_t)(per_xcd / g) * bn;
    const bool fits = bytes <= LLC_BYTES;
    const bool better = g == 8 || (fits && !best_fits) || (fits == best_fits && (fits ? rows < best_rows : bytes < best_bytes));
    if (better) {
      best = g;
      best_fits = fits;
      best_rows = rows;
      best_bytes = bytes;
    }
  }
  return best;
}

std::atomic<int> g_tile_override{0};  // 0: automatic, else 1000 * BM + BN

// Slices of K for an fp32 weight-gradient product whose 256 x 256 tiles fill
// at most half the compute units: as many as fill them, at most 8, each at
// least 8 k tiles deep.
int ksplit_of(int M, int N, int K) {
  const int64_t tiles = (int64_t)((M + 255) / 256) * ((N + 255) / 256);
  const int ncu = compute_units();
  if (N % 4 != 0 || tiles == 0 || 2 * tiles > ncu) return 1;
  const int64_t s = std::min<int64_t>(std::min<int64_t>(ncu / tiles, ((int64_t)K + KT - 1) / KT / 8), 8);
  return s < 2 ? 1 : (int)s;
}

// Tile shape (1000 * BM + BN) of a launch: among the shapes the kernel variant
// allows, the one with the fewest waves of workgroups times tile area; a
// 192-wide side counts 10% extra for its higher LDS traffic per flop.
int pick_tile(int M, int N, bool m192, bool n192) {
  const int forced = g_tile_override.load(std::memory_order_relaxed);
  if (forced) {
    const int bm = forced / 1000, bn = forced % 1000;
    return (bm == 256 || m192) && (bn == 256 || n192) ? forced : 256256;
  }
  const int ncu = compute_units();
  double best = 0.0;
  int code = 0;
  for (int bm : {256, 192}) {
    if (bm == 192 && !m192) continue;
    for (int bn : {256, 192}) {
      if (bn == 192 && !n192) continue;
      const int64_t tiles = (int64_t)((M + bm - 1) / bm) * ((N + bn - 1) / bn);
      const double cost = (double)((tiles + ncu - 1) / ncu) * bm * bn * (bm == 256 ? 1.0 : 1.1) * (bn == 256 ? 1.0 : 1.1);
      if (code == 0 || cost < best) {
        best = cost;
        code = bm * 1000 + bn;
      }
    }
  }
  return code;
}

}  // namespace

int gemm_tile_override(int bm, int bn) {
  if (bm == 0 && bn == 0) {
    g_tile_override.store(0);
    return 0;
  }
  if ((bm != 256 && bm != 192) || (bn != 256 && bn != 192)) return -1;
  g_tile_override.store(bm * 1000 + bn);
  return 0;
}

int64_t gemm_kpart_floats(int M, int N, int K) {
  const int ks = ksplit_of(M, N, K);
  return ks > 1 ? (int64_t)(ks - 1) * M * N : 0;
}

hipError_t gemm(const GemmArgs& args, hipStream_t s) {
  GemmArgs a = args;
  a.ksplit = 1;
  // A k-contiguous B split over buffers (or gate/up interleaved) is loaded a
  // wave's 64 rows at a time from one buffer: segments start at multiples of 64.
  if (a.b_kcontig && ((a.b_start[1] % 64 && a.b_start[1] < a.N) || (a.b_start[2] % 64 && a.b_start[2] < a.N)))
    return hipErrorInvalidValue;
  if (a.a_kcontig && a.b_kcontig) {
    // 192-wide tiles put a wave's B blocks in two 64-row segments: one buffer only
    const bool n192 = a.b_start[1] >= a.N;
    switch (a.epi) {
      case EPI_BF16:
        return pick_tile(a.M, a.N, false, n192) == 256192 ? launch<true, true, EPI_BF16, 256, 192>(a, s)
                                                          : launch<true, true, EPI_BF16, 256, 256>(a, s);
      case EPI_RESID:
        return pick_tile(a.M, a.N, false, n192) == 256192 ? launch<true, true, EPI_RESID, 256, 192>(a, s)
                                                          : launch<true, true, EPI_RESID, 256, 256>(a, s);
      case EPI_ROPE:
        return a.head_dim == 64 ? launch<true, true, EPI_ROPE64, 256, 256>(a, s)
                                : launch<true, true, EPI_ROPE, 256, 256>(a, s);
      case EPI_GLU_FWD: return launch<true, true, EPI_GLU_FWD, 256, 256>(a, s);
      default: break;
    }
  } else if (a.a_kcontig && !a.b_kcontig) {
    switch (a.epi) {
      case EPI_BF16:
        return pick_tile(a.M, a.N, false, true) == 256192 ? launch<true, false, EPI_BF16, 256, 192>(a, s)
                                                          : launch<true, false, EPI_BF16, 256, 256>(a, s);
      case EPI_GLU_BWD: return launch<true, false, EPI_GLU_BWD, 256, 256>(a, s);
      default: break;
    }
  } else if (!a.a_kcontig && !a.b_kcontig) {
    if (a.epi == EPI_F32) {
      int ks = ksplit_of(a.M, a.N, a.K);
      if (ks > 1)  // as many slices as the workspace holds
        ks = (int)std::min<int64_t>(ks, a.kpart ? a.kpart_floats / ((int64_t)a.M * a.N) + 1 : 1);
      if (ks > 1) {
        a.ksplit = ks;
        hipError_t e = launch<false, false, EPI_F32, 256, 256>(a, s);
        if (e != hipSuccess) return e;
        const int64_t n4 = (int64_t)a.M * a.N / 4;
        const unsigned grid = (unsigned)std::min<int64_t>((n4 + 255) / 256, 256 * 8);
        hipLaunchKernelGGL(kpart_reduce_kernel, dim3(grid), dim3(256), 0, s, a);
        return hipGetLastError();
      }
      switch (pick_tile(a.M, a.N, true, true)) {
        case 192192: return launch<false, false, EPI_F32, 192, 192>(a, s);
        case 192256: return launch<false, false, EPI_F32, 192, 256>(a, s);
        case 256192: return launch<false, false, EPI_F32, 256, 192>(a, s);
        default: return launch<false, false, EPI_F32, 256, 256>(a, s);
      }
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace ls
