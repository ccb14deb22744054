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
// log2 domain; the four row groups, then the four waves are merged by
// log-sum-exp inside the workgroup, and a second small kernel merges the
// splits (a single split writes the output directly).
#include "resa_device.h"
#include "resa_internal.h"

namespace resa {
namespace {

constexpr int kDecodeWaves = 4;

constexpr int kIdxBatch = 1024;  // chunk start tokens staged in LDS per pass
constexpr int kMaxSplits = 256;  // splits per group (bounded by the host)

// One 16-token chunk of K and V for this lane: rows r, r+4, r+8, r+12.
struct Chunk {
  U4 k[4], v[4];
};

__device__ __forceinline__ void load_chunk(Chunk& ch, const uint16_t* kp, const uint16_t* vp, int t0) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ch.k[i] = ld16_stream(kp + (size_t)(t0 + 4 * i) * kHeadDim);
    ch.v[i] = ld16_stream(vp + (size_t)(t0 + 4 * i) * kHeadDim);
  }
}

// Online-softmax update of this lane's row group with one chunk. Rows whose
// token is >= L, and every row of an invalid chunk (t0 < 0), are excluded.
template <int G>
__device__ __forceinline__ void consume_chunk(const Chunk& ch, int t0, int r, int L, float scale,
                                              const uint32_t (&q)[G][4], float (&m_)[G],
                                              float (&l_)[G], float (&acc)[G][8]) {
  const float ninf = -__builtin_inff();
  float s[4][G];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bool valid = t0 >= 0 && t0 + r + 4 * i < L;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float d = dot2_bf16(q[h][0], ch.k[i].x, 0.f);
      d = dot2_bf16(q[h][1], ch.k[i].y, d);
      d = dot2_bf16(q[h][2], ch.k[i].z, d);
      d = dot2_bf16(q[h][3], ch.k[i].w, d);
      d = row16_sum(d);
      s[i][h] = valid ? d * scale : ninf;
    }
  }
  float v[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[i][0] = bf_lo(ch.v[i].x); v[i][1] = bf_hi(ch.v[i].x);
    v[i][2] = bf_lo(ch.v[i].y); v[i][3] = bf_hi(ch.v[i].y);
    v[i][4] = bf_lo(ch.v[i].z); v[i][5] = bf_hi(ch.v[i].z);
    v[i][6] = bf_lo(ch.v[i].w); v[i][7] = bf_hi(ch.v[i].w);
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

template <int G, int BS>
__global__ __launch_bounds__(256) void k_decode(DecodeArgs a) {
  __shared__ float sm_acc[kDecodeWaves][G][kHeadDim];
  __shared__ float sm_m[kDecodeWaves][G], sm_l[kDecodeWaves][G];
  __shared__ int s_tok[kIdxBatch];

  constexpr int CPB = BS / kChunk;  // chunks per block
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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

  uint32_t q[G][4];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const U4 t = ld16(a.q + ((size_t)bb * a.q_heads + (size_t)hk * G + h) * kHeadDim + col);
    q[h][0] = t.x;
    q[h][1] = t.y;
    q[h][2] = t.z;
    q[h][3] = t.w;
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

  for (int cb = c0; cb < c1; cb += kIdxBatch) {
    const int ce = min(c1, cb + kIdxBatch);
    // First token of each chunk of this pass; -1 for ids outside [0, M).
    for (int i = threadIdx.x; i < ce - cb; i += 256) {
      const int c = cb + i;
      const int blk = idx[c / CPB];
      s_tok[i] = (blk < 0 || blk >= M) ? -1 : blk * BS + (c % CPB) * kChunk;
    }
    __syncthreads();
    // Wave w takes chunks cb + w, cb + w + 4, ...; two chunk buffers alternate
    // so the next chunk's loads are in flight while the current one is used.
    // An invalid chunk reads row 0 (in bounds) and is masked out entirely.
    auto tok = [&](int c) -> int { return c < ce ? __builtin_amdgcn_readfirstlane(s_tok[c - cb]) : -1; };
    Chunk A, Bf;
    int c = cb + wave;
    int ta = tok(c);
    load_chunk(A, kp, vp, max(ta, 0));
    // The scheduling barriers keep the prefetch ahead of the compute.
    while (c < ce) {
      const int tb = tok(c + kDecodeWaves);
      load_chunk(Bf, kp, vp, max(tb, 0));
      __builtin_amdgcn_sched_barrier(0);
      consume_chunk<G>(A, ta, r, L, scale, q, m_, l_, acc);
      c += kDecodeWaves;
      if (c >= ce) break;
      ta = tok(c + kDecodeWaves);
      load_chunk(A, kp, vp, max(ta, 0));
      __builtin_amdgcn_sched_barrier(0);
      consume_chunk<G>(Bf, tb, r, L, scale, q, m_, l_, acc);
      c += kDecodeWaves;
    }
    __syncthreads();
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

  // Merge the waves; store this split's normalised partial and its lse (log2
  // domain), or the final output directly when there is a single split.
  const bool single = S == 1;
  const size_t ob = (size_t)bb * a.q_heads + (size_t)hk * G;
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
    const float val = any ? x / lsum : 0.f;
    const float l2 = any ? mx + fast_log2(lsum) : ninf;
    if (single) {
      a.out[(ob + h) * kHeadDim + d] = val;
      if (d == 0 && a.lse) a.lse[ob + h] = any ? l2 * kLn2 : ninf;
    } else {
      po[o] = val;
      if (d == 0) pl[h] = l2;
    }
  }
}

// Alg. 2, "Combine": one workgroup per (query head, group) merges the splits'
// partials by log-sum-exp. Running after the split kernel, it sees their
// partials through the kernel boundary, with no in-kernel fences.
template <int G>
__global__ __launch_bounds__(256) void k_decode_combine(DecodeArgs a) {
  __shared__ float s_w[kMaxSplits];
  __shared__ f4_t s_red[256];
  const int h = blockIdx.x, hk = blockIdx.y, bb = blockIdx.z;
  const int S = a.num_splits;
  const size_t grp = (size_t)bb * a.c.kv_heads + hk;
  const size_t oh = (size_t)bb * a.q_heads + (size_t)hk * G + h;
  merge_splits(a.part_o + grp * S * (size_t)(G * kHeadDim) + (size_t)h * kHeadDim,
               (size_t)(G * kHeadDim), a.part_lse + grp * S * (size_t)G + h, (size_t)G, S, 1, s_w,
               s_red, [&](int) { return a.out + oh * kHeadDim; },
               [&](int, float v) { if (a.lse) a.lse[oh] = v; });
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
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.num_splits == 1) return e;
  hipLaunchKernelGGL((k_decode_combine<G>), dim3(G, a.c.kv_heads, a.c.batch), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

int32_t decode_auto_splits(int32_t batch, int32_t kv_heads, int32_t n_cap, int32_t block_size) {
  const int64_t groups = (int64_t)batch * kv_heads;
  const int64_t chunks = (int64_t)n_cap * (block_size / kChunk);
  // About one workgroup per CU (256 CUs), with at least 4 chunks per wave:
  // measured on MI355X, fewer and longer-running workgroups beat more splits.
  int64_t s = (256 + groups - 1) / groups;
  const int64_t most = chunks / (4 * kDecodeWaves);
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
