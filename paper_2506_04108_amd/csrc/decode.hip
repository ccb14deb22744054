// Group block-sparse flash-decoding (Eq. 2; App. A, Alg. 2) for gfx950.
//
// Grid (num_splits, kv_heads, batch); 4 waves per workgroup. The selected
// blocks of a (sequence, kv head) group are cut into 16-token chunks and the
// chunks into num_splits contiguous ranges; wave w of split s takes chunks
// c0 + w, c0 + w + 4, ... of its range.
//
// Lane layout inside a wave: lane = 16 * r + c. Lane (r, c) owns dims
// [8c, 8c + 8) of the chunk's rows r, r + 4, r + 8, r + 12, for K and for V,
// so every wave-wide 16-byte load covers four consecutive 256-byte rows
// (1 KiB contiguous) and one chunk is 4 K loads + 4 V loads per lane.
// q.k partial sums use v_dot2 on bf16 pairs, then a 16-lane DPP reduction.
// Each row group r keeps its own online-softmax state (running max m, sum l,
// accumulator over its 8 dims) for the g query heads of the group, in the
// log2 domain; the four row groups, then the four waves, then the splits are
// merged by log-sum-exp. The workgroup that finishes a group last (atomic
// ticket) merges that group's splits, so no second launch is needed.
#include "resa_device.h"
#include "resa_internal.h"

namespace resa {
namespace {

constexpr int kDecodeWaves = 4;

template <int G>
struct QRegs {
  uint32_t w[G][4];
};

template <int G, int BS>
__global__ __launch_bounds__(256) void k_decode(DecodeArgs a) {
  __shared__ float sm_acc[kDecodeWaves][G][kHeadDim];
  __shared__ float sm_m[kDecodeWaves][G], sm_l[kDecodeWaves][G];
  __shared__ uint32_t s_ticket;

  constexpr int CPB = BS / kChunk;  // chunks per block
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int split = blockIdx.x, hk = blockIdx.y, bb = blockIdx.z;
  const int S = a.num_splits;
  const size_t grp = (size_t)bb * a.c.kv_heads + hk;
  const int L = a.seq_lens[bb];
  const int M = min((L + BS - 1) / BS, a.c.max_blocks);
  const int n = max(0, min(a.num_sel[grp], a.n_cap));
  const int C = n * CPB;
  const int c0 = (int)((int64_t)split * C / S);
  const int c1 = (int)((int64_t)(split + 1) * C / S);
  const int r = lane >> 4, col = (lane & 15) * 8;
  const int32_t* idx = a.block_idx + grp * a.n_cap;

  QRegs<G> q;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const U4 t = ld16(a.q + ((size_t)bb * a.q_heads + (size_t)hk * G + h) * kHeadDim + col);
    q.w[h][0] = t.x;
    q.w[h][1] = t.y;
    q.w[h][2] = t.z;
    q.w[h][3] = t.w;
  }
  const size_t gbase = grp * (size_t)a.c.capacity * kHeadDim + (size_t)r * kHeadDim + col;
  const uint16_t* kp = a.c.k + gbase;
  const uint16_t* vp = a.c.v + gbase;
  const float scale = a.scale_log2;
  const float ninf = -__builtin_inff();

  float m_[G], l_[G], acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m_[h] = ninf;
    l_[h] = 0.f;
#pragma unroll
    for (int d = 0; d < 8; ++d) acc[h][d] = 0.f;
  }

  // First token of chunk c, or -1 when its block id is out of range.
  auto tok0_of = [&](int c) -> int {
    const int blk = idx[c / CPB];
    if (blk < 0 || blk >= M) return -1;
    return blk * BS + (c % CPB) * kChunk;
  };

  int c = c0 + wave;
  int t0 = c < c1 ? tok0_of(c) : -1;
  U4 kc[4], vc[4];
  if (t0 >= 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      kc[i] = ld16_stream(kp + (size_t)(t0 + 4 * i) * kHeadDim);
      vc[i] = ld16_stream(vp + (size_t)(t0 + 4 * i) * kHeadDim);
    }
  }
  while (c < c1) {
    const int cn = c + kDecodeWaves;
    const int tn = cn < c1 ? tok0_of(cn) : -1;
    U4 kn[4], vn[4];
    if (tn >= 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        kn[i] = ld16_stream(kp + (size_t)(tn + 4 * i) * kHeadDim);
        vn[i] = ld16_stream(vp + (size_t)(tn + 4 * i) * kHeadDim);
      }
    }
    if (t0 >= 0) {
      // Scores of rows r + 4i for every head, log2 domain; rows >= L excluded.
      float s[4][G];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool valid = t0 + r + 4 * i < L;
#pragma unroll
        for (int h = 0; h < G; ++h) {
          float d = dot2_bf16(q.w[h][0], kc[i].x, 0.f);
          d = dot2_bf16(q.w[h][1], kc[i].y, d);
          d = dot2_bf16(q.w[h][2], kc[i].z, d);
          d = dot2_bf16(q.w[h][3], kc[i].w, d);
          d = row16_sum(d);
          s[i][h] = valid ? d * scale : ninf;
        }
      }
      float v[4][8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[i][0] = bf_lo(vc[i].x); v[i][1] = bf_hi(vc[i].x);
        v[i][2] = bf_lo(vc[i].y); v[i][3] = bf_hi(vc[i].y);
        v[i][4] = bf_lo(vc[i].z); v[i][5] = bf_hi(vc[i].z);
        v[i][6] = bf_lo(vc[i].w); v[i][7] = bf_hi(vc[i].w);
      }
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float cm = fmaxf(fmaxf(s[0][h], s[1][h]), fmaxf(s[2][h], s[3][h]));
        const float mn = fmaxf(m_[h], cm);
        const float mref = mn == ninf ? 0.f : mn;
        const float alpha = fast_exp2(m_[h] - mref);
        float p[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) p[i] = fast_exp2(s[i][h] - mref);
        l_[h] = fmaf(l_[h], alpha, (p[0] + p[1]) + (p[2] + p[3]));
        m_[h] = mn;
#pragma unroll
        for (int d = 0; d < 8; ++d) {
          float x = acc[h][d] * alpha;
          x = fmaf(p[0], v[0][d], x);
          x = fmaf(p[1], v[1][d], x);
          x = fmaf(p[2], v[2][d], x);
          x = fmaf(p[3], v[3][d], x);
          acc[h][d] = x;
        }
      }
    }
    c = cn;
    t0 = tn;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      kc[i] = kn[i];
      vc[i] = vn[i];
    }
  }

  // Merge the four row groups of the wave (lanes c, c+16, c+32, c+48).
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float mx = fmaxf(m_[h], __shfl_xor(m_[h], 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float w = (m_[h] == ninf) ? 0.f : fast_exp2(m_[h] - mx);
    float l = l_[h] * w;
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    m_[h] = mx;
    l_[h] = l;
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      float x = acc[h][d] * w;
      x += __shfl_xor(x, 16);
      x += __shfl_xor(x, 32);
      acc[h][d] = x;
    }
  }
  if (r == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
#pragma unroll
      for (int d = 0; d < 8; ++d) sm_acc[wave][h][col + d] = acc[h][d];
      if (lane == 0) {
        sm_m[wave][h] = m_[h];
        sm_l[wave][h] = l_[h];
      }
    }
  }
  __syncthreads();

  // Merge the waves and store this split's normalised partial and its lse (log2).
  float* po = a.part_o + (grp * S + split) * (size_t)(G * kHeadDim);
  float* pl = a.part_lse + (grp * S + split) * (size_t)G;
  for (int o = threadIdx.x; o < G * kHeadDim; o += 256) {
    const int h = o / kHeadDim, d = o % kHeadDim;
    float mx = ninf;
#pragma unroll
    for (int w = 0; w < kDecodeWaves; ++w) mx = fmaxf(mx, sm_m[w][h]);
    float lsum = 0.f, x = 0.f;
#pragma unroll
    for (int w = 0; w < kDecodeWaves; ++w) {
      const float f = sm_m[w][h] == ninf ? 0.f : fast_exp2(sm_m[w][h] - mx);
      lsum = fmaf(sm_l[w][h], f, lsum);
      x = fmaf(sm_acc[w][h][d], f, x);
    }
    const bool any = lsum > 0.f;
    po[o] = any ? x / lsum : 0.f;
    if (d == 0) pl[h] = any ? mx + fast_log2(lsum) : ninf;
  }

  // Last workgroup of the group merges all splits (Alg. 2, "Combine").
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) s_ticket = atomicAdd(&a.counters[grp], 1u);
  __syncthreads();
  if (s_ticket != (uint32_t)(S - 1)) return;
  __threadfence();
  const float* go = a.part_o + grp * S * (size_t)(G * kHeadDim);
  const float* gl = a.part_lse + grp * S * (size_t)G;
  for (int o = threadIdx.x; o < G * kHeadDim; o += 256) {
    const int h = o / kHeadDim, d = o % kHeadDim;
    float mx = ninf;
    for (int s = 0; s < S; ++s) mx = fmaxf(mx, gl[s * G + h]);
    float wsum = 0.f, x = 0.f;
    if (mx != ninf) {
      for (int s = 0; s < S; ++s) {
        const float ls = gl[s * G + h];
        const float f = ls == ninf ? 0.f : fast_exp2(ls - mx);
        wsum += f;
        x = fmaf(f, go[(size_t)s * G * kHeadDim + o], x);
      }
    }
    const size_t oh = (size_t)bb * a.q_heads + (size_t)hk * G + h;
    a.out[oh * kHeadDim + d] = wsum > 0.f ? x / wsum : 0.f;
    if (d == 0 && a.lse) a.lse[oh] = wsum > 0.f ? (mx + fast_log2(wsum)) * kLn2 : ninf;
  }
  if (threadIdx.x == 0) a.counters[grp] = 0u;
}

template <int G>
hipError_t launch_g(const DecodeArgs& a, hipStream_t stream) {
  dim3 grid(a.num_splits, a.c.kv_heads, a.c.batch);
  switch (a.c.block_size) {
    case 16: hipLaunchKernelGGL((k_decode<G, 16>), grid, dim3(256), 0, stream, a); break;
    case 32: hipLaunchKernelGGL((k_decode<G, 32>), grid, dim3(256), 0, stream, a); break;
    case 64: hipLaunchKernelGGL((k_decode<G, 64>), grid, dim3(256), 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int32_t decode_auto_splits(int32_t batch, int32_t kv_heads, int32_t n_cap, int32_t block_size) {
  const int64_t groups = (int64_t)batch * kv_heads;
  const int64_t chunks = (int64_t)n_cap * (block_size / kChunk);
  // Aim for >= 1024 workgroups (4 per CU on 256 CUs) but keep >= 2 chunks per wave.
  int64_t s = (1024 + groups - 1) / groups;
  const int64_t most = chunks / (2 * kDecodeWaves);
  if (s > most) s = most;
  if (s > 256) s = 256;
  if (s < 1) s = 1;
  return (int32_t)s;
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  switch (a.group) {
    case 1: return launch_g<1>(a, stream);
    case 2: return launch_g<2>(a, stream);
    case 3: return launch_g<3>(a, stream);
    case 4: return launch_g<4>(a, stream);
    case 5: return launch_g<5>(a, stream);
    case 6: return launch_g<6>(a, stream);
    case 7: return launch_g<7>(a, stream);
    case 8: return launch_g<8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace resa
