// Device helpers shared by the ReSA kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace resa {

constexpr int kHeadDim = 128;
constexpr int kWave = 64;
constexpr int kChunk = 16;  // tokens handled per decode step of a wave

// A 16-byte vector: 8 bf16 values (one lane's share of a 256-byte key row).
struct __attribute__((aligned(16))) U4 {
  uint32_t x, y, z, w;
};

__device__ __forceinline__ U4 ld16(const void* p) {
  return *reinterpret_cast<const U4*>(p);
}
__device__ __forceinline__ U4 ld16_stream(const void* p) {
  // Read-once data: non-temporal hint keeps it from displacing reused lines.
  const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
  typedef uint32_t v4u __attribute__((ext_vector_type(4)));
  v4u v = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(q));
  return U4{v[0], v[1], v[2], v[3]};
}
__device__ __forceinline__ void st16(void* p, U4 v) {
  *reinterpret_cast<U4*>(p) = v;
}

// bf16 halves of a packed dword, widened exactly to fp32.
__device__ __forceinline__ float bf_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

// fp32 -> bf16 bits for values known to be bf16-exact (summaries): truncation is exact.
__device__ __forceinline__ uint32_t pack_exact(float lo, float hi) {
  return (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xffff0000u);
}

// Element-wise min / max of two packed bf16 pairs (exact, compared as values).
__device__ __forceinline__ uint32_t bf2_min(uint32_t a, uint32_t b) {
  return pack_exact(fminf(bf_lo(a), bf_lo(b)), fminf(bf_hi(a), bf_hi(b)));
}
__device__ __forceinline__ uint32_t bf2_max(uint32_t a, uint32_t b) {
  return pack_exact(fmaxf(bf_lo(a), bf_lo(b)), fmaxf(bf_hi(a), bf_hi(b)));
}
__device__ __forceinline__ U4 u4_min(U4 a, U4 b) {
  return U4{bf2_min(a.x, b.x), bf2_min(a.y, b.y), bf2_min(a.z, b.z), bf2_min(a.w, b.w)};
}
__device__ __forceinline__ U4 u4_max(U4 a, U4 b) {
  return U4{bf2_max(a.x, b.x), bf2_max(a.y, b.y), bf2_max(a.z, b.z), bf2_max(a.w, b.w)};
}

// Two-term bf16 dot product accumulated in fp32 (v_dot2c_f32_bf16).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

// DPP lane moves inside a row of 16 lanes.
template <int kCtrl>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), kCtrl, 0xf, 0xf, false));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7 - i within each half row
constexpr int kDppMirror = 0x140;     // lane i <-> 15 - i within the row

// Sum over the 16 lanes of a row; every lane of the row receives the total.
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp<kDppXor1>(x);
  x += dpp<kDppXor2>(x);
  x += dpp<kDppHalfMirror>(x);
  x += dpp<kDppMirror>(x);
  return x;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Monotone map of fp32 to uint32 (larger float -> larger key); NaN maps low.
__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (f != f) return 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace resa
