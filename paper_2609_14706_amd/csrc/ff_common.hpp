// Shared device-side definitions of the FlipFlop engine (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ff {

// Vector types of the matrix-core builtins.
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef uint16_t bf16_t;  // bf16 bit pattern in memory

// Device status block shared by every kernel of one handle.
//   st[0]: 0 = healthy; otherwise the 1-based global iteration at which a
//          factor to be inverted was not positive definite.
//   st[1]: side that failed (1 = A, 2 = B).
//   st[2]: 0-based pivot index of the first failing pivot.
//   st[3]: 0, or the 1-based global iteration after which the relative
//          change of A (x) B fell to the caller's tolerance.
// Every kernel that belongs to the iteration returns at once when st[0] or
// st[3] is set, so that the factors of the last completed iteration stay
// intact.
__device__ __forceinline__ bool ff_halted(const int* st) {
  return st != nullptr && (__builtin_nontemporal_load(st) | __builtin_nontemporal_load(st + 3)) != 0;
}

__device__ __forceinline__ bf16_t f32_to_bf16(float x) {
  __bf16 h = (__bf16)x;  // round to nearest even (v_cvt_pk_bf16_f32)
  return __builtin_bit_cast(bf16_t, h);
}

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __builtin_bit_cast(float, (uint32_t)b << 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ static float from_f32(float x) { return x; }
  __device__ static float to_f32(float x) { return x; }
};
template <> struct Elem<bf16_t> {
  __device__ static bf16_t from_f32(float x) { return f32_to_bf16(x); }
  __device__ static float to_f32(bf16_t x) { return bf16_to_f32(x); }
};

// Workgroups of one launch are spread round-robin over the 8 XCDs (each with
// its own L2).  Remap the hardware id so that consecutive logical ids run on
// the same XCD; a bijection for any grid size.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t w, uint32_t total) {
  const uint32_t q = total >> 3, r = total & 7u;
  const uint32_t x = w & 7u, local = w >> 3;
  const uint32_t start = x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q;
  return start + local;
}

}  // namespace ff
