// Shared device helpers for the gfx950 kernels: bf16 conversion, vector types
// and the MFMA wrapper.  Host-only code does not include this file.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

typedef uint16_t bf16_t;
typedef __bf16 bf16x8_v __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define LS_DEV __device__ __forceinline__

// f(integral_constant<int, 0>), ..., f(integral_constant<int, N-1>): a loop
// unrolled at compile time, so that indices into register arrays and the
// schedule of every slot are constants whatever the size of the body.
template <class F, int... I>
LS_DEV void static_for_(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
LS_DEV void static_for(F&& f) {
  static_for_(f, std::make_integer_sequence<int, N>{});
}

LS_DEV float bf2f(uint32_t b16) { return __uint_as_float(b16 << 16); }
LS_DEV float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
LS_DEV float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// float -> bf16 bits, round to nearest even (the compiler's conversion, which
// gfx950 executes as a hardware convert).
LS_DEV uint32_t f2bf(float f) { return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f); }
typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
// Two floats -> two bf16 (RNE) in one word, lo in the low half: one packed
// hardware convert.
LS_DEV uint32_t pack_bf2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2_v));
}

// D(32x32, fp32) += A(32x16) * B(16x32), bf16 operands.  Lane l supplies
// A[l%32][8*(l/32) .. +7] in `a` and B[8*(l/32) .. +7][l%32] in `b`; it holds
// D[8*(r/4) + 4*(l/32) + r%4][l%32] in element r of the result.
LS_DEV f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_v, a),
                                                 __builtin_bit_cast(bf16x8_v, b), c, 0, 0, 0);
}

// Transpose an 8x8 block of bf16 held as 8 rows of 16 bytes: out[c] holds
// column c of the input (its 8 row values, row 0 in the low half of word 0).
LS_DEV void transpose8x8(const u32x4 in[8], u32x4 out[8]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      uint32_t a = in[2 * v][c >> 1], b = in[2 * v + 1][c >> 1];
      out[c][v] = (c & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
    }
  }
}

// ---- buffer loads -----------------------------------------------------------
#define LDS_AS __attribute__((address_space(3)))
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t LS_OOB = 0x80000000u;  // a buffer offset past any operand: loads zero

// Buffer resource over [base, base + bytes) (raw buffer, stride 0).  Every
// caller passes wave-uniform values; reading them through readfirstlane keeps
// the resource in scalar registers.
LS_DEV i32x4 rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)base;
  return i32x4{(int32_t)__builtin_amdgcn_readfirstlane((uint32_t)a),
               (int32_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32) & 0xffffu),
               (int32_t)__builtin_amdgcn_readfirstlane(bytes), 0x00020000};
}

// Buffer sizes are clamped below 2^31 - 1 MB, so that LS_OOB plus any
// instruction offset stays outside every (possibly shifted, see dma16_group)
// resource.  The C ABI rejects buffers of 2 GiB and more.
LS_DEV uint32_t clamp_bytes(int64_t b) { return b <= 0 ? 0u : (b >= 0x7ff00000 ? 0x7ff00000u : (uint32_t)b); }

// One 16-byte-per-lane buffer->LDS load: resource and per-lane byte offset.
struct DmaLoad {
  i32x4 r;
  uint32_t voff;
};

// LDS byte address of a generic pointer into LDS: a generic LDS address is the
// LDS aperture in the high 32 bits and the LDS address in the low 32 bits.
// (Taken from the bits rather than through an address-space cast, whose null
// check the compiler folds into an invalid instruction in some kernels.)
LS_DEV uint32_t lds_offset(const void* p) { return (uint32_t)(uintptr_t)p; }

// 16 bytes per lane from a buffer (zero outside it) straight into LDS: lane l's
// bytes land at lds + 16 l (the address is uniform over the wave).  Issued as
// inline assembly so that the compiler does not see the LDS write: it would
// otherwise make every later LDS read wait for all loads in flight.  The
// caller orders the LDS reads with explicit vmcnt waits and barriers.
LS_DEV void dma16(i32x4 r, uint32_t voff, const void* lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds_offset(lds));
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(m0), "v"(voff), "s"(r)
               : "memory", "m0");
}

// N (1..4) buffer->LDS loads into the consecutive 1 KB LDS blocks lds,
// lds + 1 KB, ... with a single M0 write: each M0 write waits for the loads
// before it to leave the issue stage, so writing it once per load serialises
// the wave.  Load i carries the instruction offset i KB, which the hardware
// adds to both its LDS and its memory address, so its resource is moved back
// by i KB (base - i KB, size + i KB) to read the same bytes.
template <int N>
LS_DEV void dma16_group(DmaLoad (&l)[N], const void* lds) {
#pragma unroll
  for (int i = 1; i < N; ++i) {
    const uint64_t base = ((uint64_t)(uint32_t)l[i].r[1] << 32 | (uint32_t)l[i].r[0]) - 1024u * i;
    l[i].r[0] = (int32_t)(uint32_t)base;
    l[i].r[1] = (int32_t)((uint32_t)(base >> 32) & 0xffffu);
    l[i].r[2] = (int32_t)((uint32_t)l[i].r[2] + 1024u * i);
  }
  const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds_offset(lds));
  if constexpr (N == 4) {
    asm volatile(
        "s_mov_b32 m0, %0\n\ts_nop 0\n\t"
        "buffer_load_dwordx4 %1, %5, 0 offen lds\n\t"
        "buffer_load_dwordx4 %2, %6, 0 offen offset:1024 lds\n\t"
        "buffer_load_dwordx4 %3, %7, 0 offen offset:2048 lds\n\t"
        "buffer_load_dwordx4 %4, %8, 0 offen offset:3072 lds"
        :
        : "s"(m0), "v"(l[0].voff), "v"(l[1].voff), "v"(l[2].voff), "v"(l[3].voff), "s"(l[0].r), "s"(l[1].r),
          "s"(l[2].r), "s"(l[3].r)
        : "memory", "m0");
  } else if constexpr (N == 2) {
    asm volatile(
        "s_mov_b32 m0, %0\n\ts_nop 0\n\t"
        "buffer_load_dwordx4 %1, %3, 0 offen lds\n\t"
        "buffer_load_dwordx4 %2, %4, 0 offen offset:1024 lds"
        :
        : "s"(m0), "v"(l[0].voff), "v"(l[1].voff), "s"(l[0].r), "s"(l[1].r)
        : "memory", "m0");
  } else {
    static_assert(N == 1, "groups of 1, 2 or 4 loads");
    dma16(l[0].r, l[0].voff, lds);
  }
}

// One buffer->LDS load with a scalar offset: 16 bytes per lane from offset
// soff + voff of the buffer (zero outside it) into LDS at m0 + 16 lane.  The
// scalar offset moves every load of a tile along k; voff = LS_OOB reads zeros.
// The M0 write waits until the wave's earlier loads have left the issue
// stage, so callers keep other instructions between consecutive loads.
LS_DEV void dma1(i32x4 r, uint32_t voff, uint32_t soff, uint32_t m0) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(m0), "v"(voff), "s"(r), "s"(soff)
               : "memory", "m0");
}

// s_waitcnt for at most n (0..63) outstanding vector-memory operations.
#define LS_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | 0x0f70)

// Wait for every buffer->LDS load of this wave and every LDS access, then for
// the whole workgroup.  A plain s_barrier: __syncthreads() does not know about
// the inline-assembly loads; the empty asm statements keep the compiler from
// moving LDS accesses across it.
LS_DEV void sync_lds() {
  __builtin_amdgcn_s_waitcnt(0x0070);  // vmcnt(0) lgkmcnt(0)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

LS_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
LS_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
