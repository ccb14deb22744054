// Dense rectification (Sec. 2.2; Alg. 1 "DenseForward" every f steps) on
// gfx950 matrix cores.
//
// The f re-encoded query rows of a (sequence, kv head) group, times its g
// heads, are R = g * f rows (row rho = r * g + h sits at position L - f + r).
// Against the whole cache they form a dense contraction, so this is the one
// place the library uses MFMA (v_mfma_f32_16x16x32_bf16).
//
// Grid (num_splits, ceil(R / 128), batch * kv_heads); 4 waves per workgroup,
// each owning 32 query rows (two 16-row tiles). A workgroup walks its key
// range in tiles of 32 keys staged through LDS (K row-major, V transposed).
// Per tile and wave:
//   S^T = K . Q^T        (keys x queries; lane l holds query l % 16 and keys
//                          16 kt + 4 (l / 16) + i)
//   online softmax per query row in the log2 domain; P is split into a bf16
//   high part and a bf16 low part (p - hi) so the product keeps ~16 bits
//   O^T += V^T . P^T     (dims x queries; the contraction index is ordered so
//                          that P^T is already in the B-operand layout)
// A second kernel merges the splits by log-sum-exp (Alg. 2, "Combine"),
// spread over many workgroups.
#include "resa_device.h"
#include "resa_internal.h"

namespace resa {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kRowsPerWave = 32;
constexpr int kRowsPerWg = 128;
constexpr int kKeyTile = 32;
constexpr int kKStride = kHeadDim + 8;  // bf16 per K row in LDS (272 B, 16-B aligned)
constexpr int kVStride = kKeyTile + 4;  // bf16 per transposed V row in LDS (72 B)
constexpr int kMaxRectSplits = 1024;     // splits per group (bounded by the host)

__device__ __forceinline__ f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Writes the re-encoded rows k_f, v_f over cache rows [L - f, L).
__global__ __launch_bounds__(256) void k_rectify_rows(RectifyArgs a) {
  const int grp = blockIdx.x;
  const int bb = grp / a.c.kv_heads;
  const int L = a.seq_lens[bb];
  if (L < a.f || L > a.c.capacity) return;
  uint16_t* k = const_cast<uint16_t*>(a.c.k);
  uint16_t* v = const_cast<uint16_t*>(a.c.v);
  for (int s = threadIdx.x; s < a.f * 16; s += 256) {
    const int row = s >> 4, part = s & 15;
    const size_t src = ((size_t)grp * a.f + row) * kHeadDim + part * 8;
    const size_t dst = ((size_t)grp * a.c.capacity + (L - a.f + row)) * kHeadDim + part * 8;
    st16(k + dst, ld16(a.k_f + src));
    st16(v + dst, ld16(a.v_f + src));
  }
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_rectify_attn(RectifyArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sK[kKeyTile * kKStride];
  __shared__ __attribute__((aligned(16))) uint16_t sV[kHeadDim * kVStride];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int split = blockIdx.x, qblk = blockIdx.y, grp = blockIdx.z;
  const int bb = grp / a.c.kv_heads, hk = grp % a.c.kv_heads;
  const int G = a.group, f = a.f, R = G * f;
  const int S = a.num_splits;
  const int L = a.seq_lens[bb];
  const bool seq_ok = L >= f && L <= a.c.capacity;
  const int k0 = split * a.chunk;
  const int k1 = seq_ok ? min(k0 + a.chunk, L) : k0;
  const int j = lane >> 4, lq = lane & 15;
  const int row_base = qblk * kRowsPerWg + wave * kRowsPerWave;
  const float ninf = -__builtin_inff();

  // Q^T operand (B of the S^T product): lane holds query row lq of each tile,
  // dims 32 s + 8 j .. + 8 for k-step s.
  bf16x8_t qb[2][4];
  int lim[2];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int rho = row_base + 16 * qt + lq;
    if (rho < R && seq_ok) {
      const int h = rho % G, r = rho / G;
      lim[qt] = L - f + r;
      const uint16_t* qp = a.q_f + (((size_t)bb * a.q_heads + (size_t)hk * G + h) * f + r) * kHeadDim;
#pragma unroll
      for (int s = 0; s < 4; ++s) qb[qt][s] = __builtin_bit_cast(bf16x8_t, ld16(qp + 32 * s + 8 * j));
    } else {
      lim[qt] = -1;
#pragma unroll
      for (int s = 0; s < 4; ++s) qb[qt][s] = __builtin_bit_cast(bf16x8_t, U4{0, 0, 0, 0});
    }
  }

  f32x4_t o[8][2];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) o[dt][qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m[2] = {ninf, ninf}, l[2] = {0.f, 0.f};

  const size_t gbase = (size_t)grp * a.c.capacity * kHeadDim;
  U4 rk[2], rv[2];
  auto gload = [&](int t0) {
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int seg = tid + 256 * e, key = seg >> 4, part = seg & 15;
      const int kk = t0 + key;
      if (kk < k1) {
        rk[e] = ld16_stream(a.c.k + gbase + (size_t)kk * kHeadDim + part * 8);
        rv[e] = ld16_stream(a.c.v + gbase + (size_t)kk * kHeadDim + part * 8);
      } else {
        rk[e] = U4{0, 0, 0, 0};
        rv[e] = U4{0, 0, 0, 0};
      }
    }
  };
  auto lstore = [&]() {
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int seg = tid + 256 * e, key = seg >> 4, part = seg & 15;
      st16(&sK[key * kKStride + part * 8], rk[e]);
      const uint32_t w[4] = {rv[e].x, rv[e].y, rv[e].z, rv[e].w};
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        sV[(part * 8 + 2 * d) * kVStride + key] = (uint16_t)(w[d] & 0xffffu);
        sV[(part * 8 + 2 * d + 1) * kVStride + key] = (uint16_t)(w[d] >> 16);
      }
    }
  };

  if (k0 < k1) gload(k0);
  for (int t0 = k0; t0 < k1; t0 += kKeyTile) {
    __syncthreads();
    lstore();
    __syncthreads();
    if (t0 + kKeyTile < k1) gload(t0 + kKeyTile);

    f32x4_t sacc[2][2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) sacc[kt][qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const bf16x8_t ka = *reinterpret_cast<const bf16x8_t*>(&sK[(16 * kt + lq) * kKStride + 32 * s + 8 * j]);
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) sacc[kt][qt] = mfma16(ka, qb[qt][s], sacc[kt][qt]);
      }
    }

    bf16x8_t phi[2], plo[2];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      float x[8];
      float tmax = ninf;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = t0 + 16 * kt + 4 * j + i;
          float y = sacc[kt][qt][i] * a.scale_log2;
          y = (key > lim[qt] || key >= k1) ? ninf : y;
          x[4 * kt + i] = y;
          tmax = fmaxf(tmax, y);
        }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
      const float mn = fmaxf(m[qt], tmax);
      const float mref = mn == ninf ? 0.f : mn;
      const float alpha = fast_exp2(m[qt] - mref);
      m[qt] = mn;
      float ps = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = fast_exp2(x[e] - mref);
        ps += p;
        const __bf16 hi = (__bf16)p;
        phi[qt][e] = hi;
        plo[qt][e] = (__bf16)(p - (float)hi);
      }
      l[qt] = fmaf(l[qt], alpha, ps);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) o[dt][qt] *= alpha;
    }

#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const uint16_t* vr = &sV[(16 * dt + lq) * kVStride];
      const bf16x4_t v0 = *reinterpret_cast<const bf16x4_t*>(vr + 4 * j);
      const bf16x4_t v1 = *reinterpret_cast<const bf16x4_t*>(vr + 16 + 4 * j);
      const bf16x8_t va = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        o[dt][qt] = mfma16(va, phi[qt], o[dt][qt]);
        o[dt][qt] = mfma16(va, plo[qt], o[dt][qt]);
      }
    }
  }

  // This split's normalised partial rows and their lse (log2 domain).
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    float lt = l[qt];
    lt += __shfl_xor(lt, 16);
    lt += __shfl_xor(lt, 32);
    const int rho = row_base + 16 * qt + lq;
    if (rho < R) {
      const float inv = lt > 0.f ? 1.f / lt : 0.f;
      float* po = a.part_o + (((size_t)grp * S + split) * R + rho) * kHeadDim;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        const f32x4_t y = o[dt][qt] * inv;
        *reinterpret_cast<f32x4_t*>(po + 16 * dt + 4 * j) = y;
      }
      if (j == 0) a.part_lse[((size_t)grp * S + split) * R + rho] = lt > 0.f ? m[qt] + fast_log2(lt) : ninf;
    }
  }

}

// Log-sum-exp merge of the splits (Alg. 2, "Combine") spread over many
// workgroups: each takes kCombineRows query rows of one group.
constexpr int kCombineRows = 2;

__global__ __launch_bounds__(256) void k_rectify_combine(RectifyArgs a) {
  __shared__ float s_w[kMaxRectSplits * kCombineRows];
  __shared__ f4_t s_red[256];
  const int grp = blockIdx.y;
  const int bb = grp / a.c.kv_heads, hk = grp % a.c.kv_heads;
  const int G = a.group, f = a.f, R = G * f, S = a.num_splits;
  const int rho0 = blockIdx.x * kCombineRows;
  const int rows = min(kCombineRows, R - rho0);
  if (rows <= 0) return;
  auto out_index = [&](int r) {
    const int rho = rho0 + r;
    return ((size_t)bb * a.q_heads + (size_t)hk * G + rho % G) * f + rho / G;
  };
  merge_splits<false>(a.part_o + ((size_t)grp * S * R + rho0) * kHeadDim, (size_t)R * kHeadDim,
               a.part_lse + (size_t)grp * S * R + rho0, (size_t)R, S, rows, s_w, s_red,
               [&](int r) { return a.out + out_index(r) * kHeadDim; },
               [&](int r, float v) { if (a.lse) a.lse[out_index(r)] = v; });
}

}  // namespace

int32_t rectify_num_qblocks(int32_t group, int32_t f) {
  return (group * f + kRowsPerWg - 1) / kRowsPerWg;
}

int32_t rectify_chunk(int32_t batch, int32_t kv_heads, int32_t nqblk, int32_t max_seq_len) {
  const int64_t wgs = (int64_t)batch * kv_heads * nqblk;
  int64_t target = (512 + wgs - 1) / wgs;
  if (target < 1) target = 1;
  int64_t chunk = (max_seq_len + target - 1) / target;
  chunk = (chunk + kKeyTile - 1) / kKeyTile * kKeyTile;
  if (chunk < 512) chunk = 512;
  // At most kMaxRectSplits splits, so the combine's weights fit in LDS.
  const int64_t least = ((int64_t)max_seq_len + kMaxRectSplits - 1) / kMaxRectSplits;
  if (chunk < least) chunk = (least + kKeyTile - 1) / kKeyTile * kKeyTile;
  return (int32_t)chunk;
}

hipError_t launch_rectify(const RectifyArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(k_rectify_rows, dim3(a.c.batch * a.c.kv_heads), dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.refresh) {
    e = launch_summarize_tail(a.c, a.seq_lens, a.f, stream);
    if (e != hipSuccess) return e;
  }
  const int32_t nq = rectify_num_qblocks(a.group, a.f);
  hipLaunchKernelGGL(k_rectify_attn, dim3(a.num_splits, nq, a.c.batch * a.c.kv_heads), dim3(256), 0,
                     stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int32_t rows = a.group * a.f;
  hipLaunchKernelGGL(k_rectify_combine, dim3((rows + kCombineRows - 1) / kCombineRows,
                     a.c.batch * a.c.kv_heads), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace resa
