// Block selection (Sec. 2.1): average-pooled group query, Quest block score
// (Eq. 4) and the dynamic top-n (Eq. 5) with local forcing.
#include "resa_device.h"
#include "resa_internal.h"

namespace resa {
namespace {

constexpr int kScoreBlocksPerWg = 256;  // 4 waves x 64 blocks
constexpr int kTopnThreads = 1024;

// Scores stream the summaries once: lane (r, c) handles dims [8c, 8c + 8) of
// block base + 4 * it + r, so each wave-wide load is four whole 256-byte
// summary rows. Per dimension the larger of q*kmax and q*kmin is the product
// with kmax when q >= 0 and with kmin otherwise (exactly, as fp32 rounding is
// monotone), so the kernel selects the summary row before multiplying.
template <int BS>
__global__ __launch_bounds__(256) void k_score(SelectArgs a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hk = blockIdx.y, bb = blockIdx.z;
  const int L = a.seq_lens[bb];
  // Lengths beyond max_seq_len are clamped so every access stays in bounds.
  const int M = min(min((L + BS - 1) / BS, a.max_blocks_seq), a.c.max_blocks);
  const int base = blockIdx.x * kScoreBlocksPerWg + wave * 64;
  if (base >= M) return;  // uniform per wave
  const int r = lane >> 4, col = (lane & 15) * 8;

  // Pooled query (Fig. 3: average over the g heads of the group), fp32.
  float qb[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) qb[j] = 0.f;
  for (int h = 0; h < a.group; ++h) {
    const U4 qv = ld16(a.q + ((size_t)bb * a.q_heads + (size_t)hk * a.group + h) * kHeadDim + col);
    const uint32_t w[4] = {qv.x, qv.y, qv.z, qv.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      qb[2 * j] += bf_lo(w[j]);
      qb[2 * j + 1] += bf_hi(w[j]);
    }
  }
  const float inv_g = 1.0f / (float)a.group;
  bool use_max[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    qb[j] *= inv_g;
    use_max[j] = qb[j] >= 0.f;
  }

  const size_t grp = (size_t)bb * a.c.kv_heads + hk;
  const uint16_t* kmin = a.c.kmin + grp * a.c.max_blocks * kHeadDim + col;
  const uint16_t* kmax = a.c.kmax + grp * a.c.max_blocks * kHeadDim + col;
  float* out = a.scores + grp * a.max_blocks_seq;

  constexpr int kUnroll = 4;
  for (int it = 0; it < 16; it += kUnroll) {
    U4 lo[kUnroll], hi[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int m = base + (it + u) * 4 + r;
      if (m < M) {
        lo[u] = ld16(kmin + (size_t)m * kHeadDim);
        hi[u] = ld16(kmax + (size_t)m * kHeadDim);
      } else {
        lo[u] = U4{0, 0, 0, 0};
        hi[u] = U4{0, 0, 0, 0};
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t wl[4] = {lo[u].x, lo[u].y, lo[u].z, lo[u].w};
      const uint32_t wh[4] = {hi[u].x, hi[u].y, hi[u].z, hi[u].w};
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float a0 = use_max[2 * j] ? bf_lo(wh[j]) : bf_lo(wl[j]);
        const float a1 = use_max[2 * j + 1] ? bf_hi(wh[j]) : bf_hi(wl[j]);
        s = fmaf(qb[2 * j], a0, s);
        s = fmaf(qb[2 * j + 1], a1, s);
      }
      s = row16_sum(s);
      const int m = base + (it + u) * 4 + r;
      if ((lane & 15) == 0 && m < M) out[m] = s;
    }
  }
}

// Exclusive prefix sum over the 1024 threads of the workgroup; returns the
// thread's exclusive prefix and writes the total to *total.
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* lds16, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds16[wave] = x;
  __syncthreads();
  if (wave == 0) {
    uint32_t t = lane < 16 ? lds16[lane] : 0u;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const uint32_t y = __shfl_up(t, o);
      if (lane >= o) t += y;
    }
    if (lane < 16) lds16[16 + lane] = t;  // inclusive wave offsets
  }
  __syncthreads();
  const uint32_t wave_off = wave == 0 ? 0u : lds16[16 + wave - 1];
  *total = lds16[16 + 15];
  const uint32_t r = wave_off + x - v;
  __syncthreads();  // lds16 may be reused by the next scan
  return r;
}

// Exact top-n per (sequence, kv head): an MSD radix select over order-
// preserving 32-bit keys finds the n-th largest key T; every block with a
// larger key is kept, and of the blocks equal to T the lowest ids are kept.
// The kept ids are then written in ascending order.
__global__ __launch_bounds__(kTopnThreads) void k_topn(SelectArgs a) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t scan_lds[32];
  __shared__ uint32_t s_digit, s_k, s_cnt;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hk = blockIdx.x, bb = blockIdx.y;
  const int bs = a.c.block_size;
  const int L = a.seq_lens[bb];
  const int M = max(0, min(min((L + bs - 1) / bs, a.max_blocks_seq), a.c.max_blocks));
  const int n = count_selected(M, a.keep_ppm, a.min_blocks, a.n_local);
  const size_t grp = (size_t)bb * a.c.kv_heads + hk;
  int32_t* out = a.block_idx + grp * a.n_cap;
  if (tid == 0) a.num_sel[grp] = n;
  if (n == 0 || n >= M) {
    for (int i = tid; i < a.n_cap; i += kTopnThreads) out[i] = i < n ? i : -1;
    return;
  }
  const float* sc = a.scores + grp * a.max_blocks_seq;
  const int forced_from = M - a.n_local;
  const int E = (M + kTopnThreads - 1) / kTopnThreads;
  const int lo = min(tid * E, M), hi = min(lo + E, M);
  auto key_of = [&](int m) -> uint32_t {
    return m >= forced_from ? 0xFFFFFFFFu : order_key(sc[m]);
  };

  uint32_t prefix = 0, pmask = 0, k = (uint32_t)n;
  for (int shift = 24; shift >= 0; shift -= 8) {
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    for (int m = lo; m < hi; ++m) {
      const uint32_t key = key_of(m);
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (wave == 0) {
      // Lane i owns digits 255-4i .. 252-4i (descending); find the digit where
      // the count of larger-or-equal keys first reaches k.
      uint32_t c[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = hist[255 - 4 * lane - j];
      const uint32_t tot = c[0] + c[1] + c[2] + c[3];
      uint32_t incl = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
      }
      uint32_t cum = incl - tot;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (cum < k && cum + c[j] >= k) {
          s_digit = 255 - 4 * lane - j;
          s_k = k - cum;
          s_cnt = c[j];
        }
        cum += c[j];
      }
    }
    __syncthreads();
    prefix |= s_digit << shift;
    pmask |= 255u << shift;
    k = s_k;
    const uint32_t cnt = s_cnt;
    __syncthreads();
    if (cnt == k) break;  // the whole bucket is kept: no need to refine further
  }

  // Rank of each threshold-bucket element among the bucket, in id order.
  uint32_t n_eq = 0;
  for (int m = lo; m < hi; ++m) n_eq += ((key_of(m) & pmask) == prefix);
  uint32_t tot;
  uint32_t eq_rank = block_exclusive_scan(n_eq, scan_lds, &tot);
  uint32_t n_sel = 0;
  {
    uint32_t r = eq_rank;
    for (int m = lo; m < hi; ++m) {
      const uint32_t km = key_of(m) & pmask;
      if (km > prefix) {
        ++n_sel;
      } else if (km == prefix) {
        n_sel += (r < k);
        ++r;
      }
    }
  }
  uint32_t pos = block_exclusive_scan(n_sel, scan_lds, &tot);
  {
    uint32_t r = eq_rank;
    for (int m = lo; m < hi; ++m) {
      const uint32_t km = key_of(m) & pmask;
      bool take = false;
      if (km > prefix) {
        take = true;
      } else if (km == prefix) {
        take = r < k;
        ++r;
      }
      if (take) {
        if (pos < (uint32_t)a.n_cap) out[pos] = m;  // never past the row, whatever the scores
        ++pos;
      }
    }
  }
  for (int i = n + tid; i < a.n_cap; i += kTopnThreads) out[i] = -1;
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  dim3 sgrid((a.max_blocks_seq + kScoreBlocksPerWg - 1) / kScoreBlocksPerWg, a.c.kv_heads, a.c.batch);
  if (a.max_blocks_seq > 0) {
    switch (a.c.block_size) {
      case 16: hipLaunchKernelGGL(k_score<16>, sgrid, dim3(256), 0, stream, a); break;
      case 32: hipLaunchKernelGGL(k_score<32>, sgrid, dim3(256), 0, stream, a); break;
      case 64: hipLaunchKernelGGL(k_score<64>, sgrid, dim3(256), 0, stream, a); break;
      default: return hipErrorInvalidValue;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_topn, dim3(a.c.kv_heads, a.c.batch), dim3(kTopnThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace resa
