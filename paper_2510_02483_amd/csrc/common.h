// Shared device helpers for the gfx950 kernels: bf16 conversion, vector types
// and the MFMA wrapper.  Host-only code does not include this file.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;
typedef __bf16 bf16x8_v __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define LS_DEV __device__ __forceinline__

LS_DEV float bf2f(uint32_t b16) { return __uint_as_float(b16 << 16); }
LS_DEV float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
LS_DEV float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// float -> bf16 bits, round to nearest even (the compiler's conversion, which
// gfx950 executes as a hardware convert).
LS_DEV uint32_t f2bf(float f) { return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f); }
LS_DEV uint32_t pack_bf2(float lo, float hi) { return f2bf(lo) | (f2bf(hi) << 16); }

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

LS_DEV uint32_t clamp_bytes(int64_t b) { return b <= 0 ? 0u : (b >= 0x7fffffff ? 0x7fffffffu : (uint32_t)b); }

// 16 bytes per lane from a buffer (zero outside it) straight into LDS: lane l's
// bytes land at lds + 16 l (the address is uniform over the wave).  Issued as
// inline assembly so that the compiler does not see the LDS write: it would
// otherwise make every later LDS read wait for all loads in flight.  The
// caller orders the LDS reads with explicit vmcnt waits and barriers.
LS_DEV void dma16(i32x4 r, uint32_t voff, const void* lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const LDS_AS void*)lds);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(m0), "v"(voff), "s"(r)
               : "memory", "m0");
}

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
