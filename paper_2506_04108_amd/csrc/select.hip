// Block selection (Sec. 2.1): average-pooled group query, Quest block score
// (Eq. 4) and the dynamic top-n (Eq. 5) with local forcing.
#include "select_impl.h"

namespace resa {
namespace {

constexpr int kSelThreads = 1024;                 // 16 waves (512 for short ranges)
constexpr int kTopnThreads = 1024;

// Exact top-n per (sequence, kv head): an MSD radix select over order-
// preserving 32-bit keys finds the n-th largest key T; every block with a
// larger key is kept, and of the blocks equal to T the lowest ids are kept.
// The kept ids are then written in ascending order.
__device__ void topn_group(const SelectArgs& a, int L) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t scan_lds[32];
  __shared__ uint32_t s_digit, s_k, s_cnt;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hk = blockIdx.x, bb = blockIdx.y;
  const int bs = a.c.block_size;
  const int M = max(0, min(min((L + bs - 1) / bs, a.max_blocks_seq), a.c.max_blocks));
  const int n = count_selected(M, a.keep_ppm, a.min_blocks, a.n_local);
  const size_t grp = (size_t)bb * a.c.kv_heads + hk;
  int32_t* out = a.block_idx + grp * a.n_cap;
  if (tid == 0) a.num_sel[grp] = n;
  if (n == 0 || n >= M) {
    for (int i = tid; i < a.n_cap; i += kTopnThreads) out[i] = i < n ? i : -1;
    return;
  }
  // Keys as the scoring stored them (the n_local most recent blocks hold the
  // largest key).
  const uint32_t* keys = a.keys + grp * a.score_stride;
  const int E = (M + kTopnThreads - 1) / kTopnThreads;
  const int lo = min(tid * E, M), hi = min(lo + E, M);
  auto key_of = [&](int m) -> uint32_t { return keys[m]; };

  uint32_t prefix = 0, pmask = 0, k = (uint32_t)n;
  for (int shift = 24; shift >= 0; shift -= 8) {
    if (tid < 256) hist[tid] = 0;
    lds_sync();
    for (int m = lo; m < hi; ++m) {
      const uint32_t key = key_of(m);
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    lds_sync();
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
    lds_sync();
    prefix |= s_digit << shift;
    pmask |= 255u << shift;
    k = s_k;
    const uint32_t cnt = s_cnt;
    lds_sync();
    if (cnt == k) break;  // the whole bucket is kept: no need to refine further
  }

  // Rank of each threshold-bucket element among the bucket, in id order.
  uint32_t n_eq = 0;
  for (int m = lo; m < hi; ++m) n_eq += ((key_of(m) & pmask) == prefix);
  uint32_t tot;
  uint32_t eq_rank = block_exclusive_scan<kTopnThreads>(n_eq, scan_lds, &tot);
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
  uint32_t pos = block_exclusive_scan<kTopnThreads>(n_sel, scan_lds, &tot);
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

__global__ __launch_bounds__(kTopnThreads) void k_topn(SelectArgs a) {
  const SeqLen sl = seq_len_of(a, blockIdx.y);
  topn_group(a, sl.L);
  if (a.k_new != nullptr && threadIdx.x == 0)
    finish_append(a, blockIdx.y, sl.L,
                  __hip_atomic_fetch_add(a.seq_counters + blockIdx.y, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}


// Pooled query (Fig. 3), Quest scores (Eq. 4) and, when `fused`, the top-n
// (Eq. 5) in one kernel. Grid (ceil(max_blocks_seq / blocks_per_wg), kv
// heads, batch), about one workgroup per CU (16 waves; 8 for short ranges of
// short groups, see launch_select). Each workgroup streams
// the summaries of its block range (score_range): lane (r, c) handles dims [8c, 8c + 8) of
// 8-block tiles, so each wave-wide load is four whole 256-byte summary rows,
// and the next tile's loads are in flight while one is scored. Per dimension
// the larger of q*kmax and q*kmin is the product with kmax when q >= 0 and
// with kmin otherwise (exactly, as fp32 rounding is monotone), so the
// summary row is selected before the multiply. Scores are staged in LDS and
// written out coalesced; with `fused`, the workgroup also counts its keys' 8
// high bits into its own histogram slot, and the last workgroup of the group
// to finish (ticket) sums the slots and runs select_tail. Scores, slots and
// ticket use agent scope (write-through stores, coherent loads, a relaxed
// atomic after the stores are acknowledged), so no cache writeback is needed
// between workgroups.
template <int NJ, int NT = kSelThreads>
__global__ __launch_bounds__(NT) void k_select(SelectArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t s_hist[kBins2];
  __shared__ __attribute__((aligned(16))) float s_score[kMaxBlocksPerWg];
  __shared__ uint32_t s_lds32[32];
  __shared__ uint32_t s_misc[8];
  const int tid = threadIdx.x;
  const int hk = blockIdx.y, bb = blockIdx.z;
  const size_t grp = (size_t)bb * a.c.kv_heads + hk;
  const RangeInfo ri = score_range<NT / 64, 1, false, window_lists(NJ, NT)>(a, bb, hk, blockIdx.x, gridDim.x, s_hist, s_score);
  if (!a.fused) return;
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0)
    s_misc[3] = __hip_atomic_fetch_add(a.counters + grp, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (s_misc[3] != gridDim.x - 1) return;
  select_tail<NJ, NT>(a, grp, ri.M, ri.forced_from, gridDim.x, ri.win, s_hist, s_lds32, s_misc,
                               reinterpret_cast<int32_t*>(s_score), bb, ri.sl.L, nullptr);
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  if (a.max_blocks_seq > 0) {
    dim3 grid((a.max_blocks_seq + a.blocks_per_wg - 1) / a.blocks_per_wg, a.c.kv_heads, a.c.batch);
    // Keys per thread of the fused top-n: the smallest instantiation that
    // holds the longest group (every group's M <= max_blocks_seq). Short
    // score ranges (at most 256 blocks, two 8-block tiles per wave at 8
    // waves) of groups up to 4096 blocks run in 512-thread workgroups: there
    // the top-n of the last workgroup dominates, and half the waves share
    // the CU's SIMDs (4K batch 1 selection 9.9 -> 9.35 us, 32K batch 4
    // 14.2 -> 13.9 us; 64K batch 8, with 1024-block ranges, is slower so).
    const int per = (a.max_blocks_seq + kSelThreads - 1) / kSelThreads;
    const int per_half = (a.max_blocks_seq + 511) / 512;
    const bool half = a.blocks_per_wg <= 256 && per_half <= 8;
    if (half && per_half <= 4)
      hipLaunchKernelGGL((k_select<4, 512>), grid, dim3(512), 0, stream, a);
    else if (half && per_half <= 5)
      hipLaunchKernelGGL((k_select<5, 512>), grid, dim3(512), 0, stream, a);
    else if (half && per_half <= 6)
      hipLaunchKernelGGL((k_select<6, 512>), grid, dim3(512), 0, stream, a);
    else if (half)
      hipLaunchKernelGGL((k_select<8, 512>), grid, dim3(512), 0, stream, a);
    else if (per <= 4)
      hipLaunchKernelGGL((k_select<4>), grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 5)
      hipLaunchKernelGGL((k_select<5>), grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 6)
      hipLaunchKernelGGL((k_select<6>), grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 8)
      hipLaunchKernelGGL((k_select<8>), grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 12)
      hipLaunchKernelGGL((k_select<12>), grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 16)
      hipLaunchKernelGGL((k_select<16>), grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 24)
      hipLaunchKernelGGL((k_select<24>), grid, dim3(kSelThreads), 0, stream, a);
    else
      hipLaunchKernelGGL((k_select<32>), grid, dim3(kSelThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.fused) return hipSuccess;
  }
  hipLaunchKernelGGL(k_topn, dim3(a.c.kv_heads, a.c.batch), dim3(kTopnThreads), 0, stream, a);
  return hipGetLastError();
}

int32_t select_fused_max_blocks() { return kMaxSelectBlocks; }

int32_t select_blocks_per_wg(int32_t batch, int32_t kv_heads, int32_t max_blocks_seq) {
  // About one workgroup per CU (256 CUs) in all: a group's blocks are cut
  // into equal ranges of whole 32-block words (so a word of the above-window
  // bits belongs to one range), at least one 8-block scoring tile per wave
  // of a 16-wave workgroup (128 blocks: small groups spread over more
  // workgroups, 4K batch 1 selection 11.2 -> 10.0 us against 256) and at
  // most the LDS staging area.
  const int64_t groups = (int64_t)batch * kv_heads;
  const int64_t per_group = (256 + groups - 1) / groups;
  int64_t bpw = ((int64_t)max_blocks_seq + per_group - 1) / per_group;
  bpw = (bpw + 31) / 32 * 32;
  if (bpw < 128) bpw = 128;
  if (bpw > kMaxBlocksPerWg) bpw = kMaxBlocksPerWg;
  return (int32_t)bpw;
}

int32_t select_hist_words(int32_t batch, int32_t kv_heads, int32_t max_blocks_seq) {
  // A bound on the workgroups per group that never decreases as the length
  // grows (the count itself can, by a few, as the ranges are rounded to
  // tiles), so a workspace sized for a longer length fits every shorter one:
  // at most ceil(M / 128) ranges, and at most max(per_group, ceil(M / 8192)).
  const int64_t groups = (int64_t)batch * kv_heads;
  const int64_t per_group = (256 + groups - 1) / groups;
  const int64_t m = max_blocks_seq > 0 ? max_blocks_seq : 0;
  int64_t wgs = (m + kMaxBlocksPerWg - 1) / kMaxBlocksPerWg;
  if (wgs < per_group) wgs = per_group;
  const int64_t most = (m + 127) / 128;
  if (wgs > most) wgs = most;
  return (int32_t)(wgs * kSlotWords);
}

}  // namespace resa
