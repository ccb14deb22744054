// Device helpers shared by the ReSA kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace resa {

constexpr int kHeadDim = 128;
constexpr int kWave = 64;
constexpr int kChunk = 16;  // tokens handled per decode step of a wave
constexpr int kMaxGroup = 8;  // query heads per kv head (RESA_MAX_GROUP)
constexpr int kBufWord3 = 0x00020000;  // raw buffer resource word 3: 32-bit data format
constexpr int kSc1 = 16;              // buffer cache policy: agent-scope coherent
constexpr int kPolicyNt = 2;          // buffer cache policy: non-temporal (read-once data)
// s_waitcnt immediate that waits for every outstanding vector memory
// operation (vmcnt 0) and leaves expcnt and lgkmcnt alone (gfx9 encoding).
constexpr int kWaitVmcnt0 = 0x0F70;

// A 16-byte vector: 8 bf16 values (one lane's share of a 256-byte key row).
struct __attribute__((aligned(16))) U4 {
  uint32_t x, y, z, w;
};

// Workgroup barrier that orders LDS accesses only. __syncthreads() also
// waits for every outstanding global load and store of the thread (its fence
// covers global memory), which would drain prefetches issued before the
// barrier; here global loads stay in flight and are waited for where their
// data is used. Not for ordering global memory between threads.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// threadIdx.x through an opaque move. A persistent kernel runs several
// phases in loops; values derived from the thread index (addresses, lane
// roles) are then computed inside each phase instead of being hoisted to the
// kernel entry and held in registers across every phase.
__device__ __forceinline__ int thread_id() {
  int t = threadIdx.x;
  __asm__ volatile("" : "+v"(t));
  return t;
}

// The thread index: opaque in the persistent step kernel (kOpaque, see
// thread_id), plain otherwise (an opaque move would also keep the compiler
// from reading uniform data with scalar loads).
template <bool kOpaque>
__device__ __forceinline__ int tid_of() {
  if constexpr (kOpaque) return thread_id();
  else return (int)threadIdx.x;
}

__device__ __forceinline__ U4 ld16(const void* p) {
  return *reinterpret_cast<const U4*>(p);
}
// A pointer that is the same in every lane of the wave, marked so for the
// compiler (buffer resources built from it then stay in scalar registers).
template <typename T>
__device__ __forceinline__ T* wave_uniform(T* p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return reinterpret_cast<T*>(((uint64_t)hi << 32) | lo);
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

// DPP lane moves inside a row of 16 lanes. Every pattern used here reads a
// lane of the same row, so bound_ctrl (out-of-row reads give 0) never applies
// and the destination needs no initial value.
template <int kCtrl>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), kCtrl, 0xf, 0xf, true));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7 - i within each half row
constexpr int kDppMirror = 0x140;     // lane i <-> 15 - i within the row
constexpr int kDppXor3 = 0x1B;        // quad_perm [3,2,1,0]
constexpr int kDppRor4 = 0x124;       // rotate the row by 4 lanes
constexpr int kDppRor8 = 0x128;       // rotate the row by 8 lanes
constexpr int kDppBcast0 = 0x150;     // + k: every lane of the row reads lane k

// Inclusive prefix sum over the 64 lanes of a wave: Hillis-Steele steps
// within each 16-lane row (DPP row_shr 1, 2, 4, 8; lanes shifted in from
// outside the row read 0), then every row adds the totals of the rows below
// it, read from lanes 15, 31 and 47.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true);
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)x, 15);
  const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 31);
  const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)x, 47);
  const int row = (threadIdx.x & 63) >> 4;
  return x + (row >= 1 ? r0 : 0u) + (row >= 2 ? r1 : 0u) + (row >= 3 ? r2 : 0u);
}

// Lane pairs (l, l ^ 16) and (l, l ^ 32) through gfx950's VALU lane swaps:
// with both operands x, permlane16_swap leaves x and x[l ^ 16] in the two
// results (in an order that depends on the row), so a sum or max of the two
// equals x op x[l ^ 16] exactly; permlane32_swap does the same for l ^ 32.
// Every lane must be active.
__device__ __forceinline__ float sum_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Bitwise OR over the 64 lanes of a wave, which must all be active: each row
// ORs its 16 lanes by DPP (quad swaps, then the half-row and row mirrors),
// then the four rows' results are combined. The result is wave-uniform.
__device__ __forceinline__ uint32_t wave_or(uint32_t x) {
  x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppXor1, 0xf, 0xf, true);
  x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppXor2, 0xf, 0xf, true);
  x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppHalfMirror, 0xf, 0xf, true);
  x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppMirror, 0xf, 0xf, true);
  return (uint32_t)(__builtin_amdgcn_readlane((int)x, 0) | __builtin_amdgcn_readlane((int)x, 16) |
                    __builtin_amdgcn_readlane((int)x, 32) | __builtin_amdgcn_readlane((int)x, 48));
}

// Transpose-reduce of 16 values across the 16 lanes of a row. Lane c enters
// with v[s] holding the lane's partial of value n = s ^ c; it leaves with
// v[0] = the full 16-lane sum of value n = c. Each step pairs lanes that
// differ in one more bit of c (partners c ^ 15, c ^ 7, c ^ 3, c ^ 1), keeps
// the half of its values whose bit matches its own, and receives the
// partner's partial of that half: 8 + 4 + 2 + 1 adds instead of 4 * 16.
__device__ __forceinline__ void transpose_reduce16(float* v) {
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] += dpp<kDppMirror>(v[15 - j]);
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] += dpp<kDppHalfMirror>(v[7 - j]);
#pragma unroll
  for (int j = 0; j < 2; ++j) v[j] += dpp<kDppXor3>(v[3 - j]);
  v[0] += dpp<kDppXor1>(v[1]);
}

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

typedef float f4_t __attribute__((ext_vector_type(4)));
typedef float f2_t __attribute__((ext_vector_type(2)));

// Log-sum-exp merge of split partials (Alg. 2, "Combine"), for one workgroup.
//
// Split s holds `rows` normalised rows of 128 floats at po + s * o_stride +
// row * 128 and their log2-domain lse at pl + s * l_stride + row. Row r of the
// result is written to out_row(r) (128 floats) and its natural-log lse is
// passed to lse_out(r, value). LDS: `w` holds S * rows floats, `red` blockDim.x
// float4. Every float4 column of the output gets blockDim.x / (32 * rows)
// threads, each summing a strided subset of the splits, so the partial reads
// are spread over the whole workgroup instead of one dependent chain per
// output.
typedef float f4_t __attribute__((ext_vector_type(4)));

// Loads of partials written by other workgroups of the same kernel use agent
// scope (coherent across the chip's L2 slices); plain loads otherwise.
template <bool kCoherent>
__device__ __forceinline__ float ld_part(const float* p) {
  if constexpr (kCoherent) return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else return *p;
}
template <bool kCoherent>
__device__ __forceinline__ f4_t ld_part4(const float* p) {
  if constexpr (kCoherent) {
    return f4_t{ld_part<true>(p), ld_part<true>(p + 1), ld_part<true>(p + 2), ld_part<true>(p + 3)};
  } else {
    return *reinterpret_cast<const f4_t*>(p);
  }
}

template <bool kCoherent, typename OutRow, typename LseOut>
__device__ void merge_splits(const float* po, size_t o_stride, const float* pl, size_t l_stride,
                             int S, int rows, float* w, f4_t* red, OutRow out_row, LseOut lse_out) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const float ninf = -__builtin_inff();
  for (int i = tid; i < S * rows; i += nt) w[i] = ld_part<kCoherent>(pl + (size_t)(i / rows) * l_stride + i % rows);
  lds_sync();
  for (int r = tid; r < rows; r += nt) {
    float mx = ninf;
    for (int s = 0; s < S; ++s) mx = fmaxf(mx, w[s * rows + r]);
    float sum = 0.f;
    for (int s = 0; s < S; ++s) {
      const float l = w[s * rows + r];
      const float e = (l == ninf) ? 0.f : fast_exp2(l - mx);
      w[s * rows + r] = e;
      sum += e;
    }
    const float inv = sum > 0.f ? 1.f / sum : 0.f;
    for (int s = 0; s < S; ++s) w[s * rows + r] *= inv;
    lse_out(r, sum > 0.f ? (mx + fast_log2(sum)) * kLn2 : ninf);
  }
  lds_sync();
  const int U = rows * (kHeadDim / 4);          // float4 columns
  const int T = U >= nt ? 1 : nt / U;           // threads per column
  for (int base = 0; base < U; base += nt) {
    const int u = base + (tid % (U < nt ? U : nt));
    const int phase = U < nt ? tid / U : 0;
    const bool active = phase < T && u < U;
    const int r = active ? u / (kHeadDim / 4) : 0;
    const int c4 = active ? u % (kHeadDim / 4) : 0;
    f4_t acc = {0.f, 0.f, 0.f, 0.f};
    if (active) {
      const float* src = po + (size_t)r * kHeadDim + 4 * c4;
#pragma unroll 8
      for (int s = phase; s < S; s += T)
        acc += w[s * rows + r] * ld_part4<kCoherent>(src + (size_t)s * o_stride);
    }
    if (T > 1) {
      red[tid] = acc;
      lds_sync();
      if (active && phase == 0) {
        for (int k = 1; k < T; ++k) acc += red[tid + k * U];
      }
      lds_sync();
    }
    if (active && phase == 0) *reinterpret_cast<f4_t*>(out_row(r) + 4 * c4) = acc;
  }
}

}  // namespace resa
