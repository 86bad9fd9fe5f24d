// Shared device/host definitions of the gfx950 library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <utility>

namespace atspeed {

typedef uint16_t bf16_t;  // bf16 storage (bit pattern)

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));  // 16-byte chunk

// Compile-time loop: f(std::integral_constant<int, i>) for i = 0..N-1, so that
// register arrays are only ever indexed by constants.
template <class F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// fp32 -> bf16, round to nearest even (finite inputs).
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// Storage-type traits: activations, weights and KV caches are float or bf16.
template <class T> struct St;
template <> struct St<float> {
  static __device__ __forceinline__ float ld(const float* p) { return *p; }
  static __device__ __forceinline__ void st(float* p, float v) { *p = v; }
};
template <> struct St<bf16_t> {
  static __device__ __forceinline__ float ld(const bf16_t* p) { return bf2f(*p); }
  static __device__ __forceinline__ void st(bf16_t* p, float v) { *p = f2bf(v); }
};

// Monotone map float -> uint32 (a < b  <=>  key(a) < key(b)) for finite floats.
__device__ __forceinline__ uint32_t float_order_key(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Row descriptors of one forward: which token runs where, and where its K/V go.
struct Rows {
  int* M;            // [1] number of rows (device)
  int* user;         // [Mmax]
  int* token;        // [Mmax]
  int* pos;          // [Mmax] rotary position
  int* slot;         // [Mmax] tree slot (u*Tmax + s) or -1 for prefix rows
  int* nctx;         // [Mmax] visible prefix-cache keys
  int* anc;          // [Mmax * 4] tree slots of ancestors-or-self, depth order
  int* nanc;         // [Mmax]
  int* user_off;     // [B + 1] first row of each user (rows of a user are contiguous)
};

}  // namespace atspeed
