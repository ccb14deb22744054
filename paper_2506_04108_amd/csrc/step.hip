// Fused decode step (Alg. 1, one decode token): append of the new token with
// its block-summary update, block selection (Sec. 2.1, Eq. 4-5) and
// block-sparse flash-decoding with the split merge (Eq. 2, Alg. 2), in one
// persistent launch.
//
// One workgroup of 8 waves per CU. Workgroups claim work items from
// counters in the workspace, in this order: first the score ranges of every
// group (group-major, so early groups finish early), then the decode splits
// (group-major). The workgroup that completes a group's last score range
// runs its exact top-n and then publishes the group (ready flag); a decode
// split waits for its group's flag. A workgroup only moves on to decode
// splits once every score range has been claimed, and a claimed score range
// belongs to a running workgroup that waits on nothing, so every flag a
// decode split waits for gets set: the waits end without any assumption on
// how many workgroups run at once. (A bounded spin records an error flag, and
// the split decodes nothing rather than hang or read unpublished ids, as a
// guard; the last workgroup to exit clears every ready flag, so a late flag
// cannot leak into the next call.)
//
// The appended token's K and V rows are taken from k_new / v_new by the
// decode splits (the cache rows written in this launch are not read back),
// ids and counts cross workgroups through agent-scope stores and loads, and
// the sequence lengths are bumped by the last workgroup to finish, after
// every item: no item of the launch sees a new length.
#include "select_impl.h"
#include "decode_impl.h"

namespace resa {
namespace {

constexpr int kStepWaves = 8;
constexpr int kStepThreads = 64 * kStepWaves;
// Chunks in flight per wave in the decode splits: one, as in the decode
// kernel (measured against two: 94.3 – 94.6 against 95.5 – 95.8 us per step
// at 64K, 65.8 – 66.1 against 66.6 us at 256K).
template <int G>
constexpr int kStepDepth = 1;

// The kernel arguments through a pointer the compiler cannot follow from
// one call to the next: each phase loads the fields it uses where it uses
// them, instead of every field being held in scalar registers for the whole
// kernel.
__device__ __forceinline__ const StepArgs& launder() {
  const StepArgs* p = (const StepArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  __asm__ volatile("" : "+s"(p));
  return *p;
}

__device__ __forceinline__ uint32_t claim(uint32_t* ctr) {
  return __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int G, int NJ>
__global__ __launch_bounds__(kStepThreads) void k_step(StepArgs) {
  __shared__ __attribute__((aligned(16))) uint32_t s_hist[kBins2];
  __shared__ __attribute__((aligned(16))) float s_score[kMaxBlocksPerWg];
  __shared__ uint32_t s_lds32[32];
  __shared__ uint32_t s_misc[8];
  __shared__ DecodeLds<G, kStepWaves> dl;
  __shared__ uint32_t s_item, s_skip;
  // Score ranges, then the group's top-n in the workgroup that completes it.
  for (;;) {
    const StepArgs& a = launder();
    const SelectArgs& sa = a.s;
    const int H = sa.c.kv_heads;
    const int tid = thread_id();
    if (tid == 0) s_item = claim(a.queue + 0);
    __syncthreads();
    const int item = (int)s_item;
    __syncthreads();  // every thread has read s_item before thread 0 writes it again
    if (item >= a.score_items) break;
    const int g = item / a.nranges, range = item - g * a.nranges;
    const int bb = g / H, hk = g - bb * H;
    const RangeInfo ri = score_range<kStepWaves, 3, true, window_lists(NJ, kStepThreads)>(sa, bb, hk, range, a.nranges, s_hist, s_score);
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0)
      s_misc[3] = __hip_atomic_fetch_add(sa.counters + g, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (s_misc[3] == (uint32_t)a.nranges - 1)
      select_tail<NJ, kStepThreads>(sa, g, ri.M, ri.forced_from, a.nranges, ri.win, s_hist, s_lds32, s_misc,
                                    reinterpret_cast<int32_t*>(s_score), bb, ri.sl.L, a.ready);
    __syncthreads();  // LDS is reused by the next item
  }

  // Decode splits, each once its group's selection is published.
  for (;;) {
    const StepArgs& a = launder();
    const SelectArgs& sa = a.s;
    const int H = sa.c.kv_heads;
    const int S = a.d.num_splits;
    const int tid = thread_id();
    if (tid == 0) {
      const uint32_t item = claim(a.queue + 1);
      s_item = item;
      s_skip = 0;
      if ((int)item < a.dec_items) {
        const uint32_t* flag = a.ready + item / S;
        uint32_t spins = 0;
        while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u) {
          if (++spins > a.max_spins) {
            // Guard: record it and decode nothing (the ids are not published).
            __hip_atomic_store(a.queue + 3, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_skip = 1;
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
      }
    }
    __syncthreads();
    const int item = (int)s_item;
    const bool skip = s_skip != 0;
    __syncthreads();  // every thread has read s_item before thread 0 writes it again
    if (item >= a.dec_items) break;
    const int g = item / S, split = item - g * S;
    const int bb = g / H, hk = g - bb * H;
    bool last = false;
    switch (sa.c.block_size) {
      case 16: last = decode_split<G, 16, kStepWaves, true, kStepDepth<G>>(a.d, bb, hk, split, sa.seq_lens, true, dl, skip); break;
      case 32: last = decode_split<G, 32, kStepWaves, true, kStepDepth<G>>(a.d, bb, hk, split, sa.seq_lens, true, dl, skip); break;
      default: last = decode_split<G, 64, kStepWaves, true, kStepDepth<G>>(a.d, bb, hk, split, sa.seq_lens, true, dl, skip); break;
    }
    // Every split of the group has passed its wait (the merging workgroup
    // holds the last ticket): the flag returns to zero for the next call.
    if (last && tid == 0) __hip_atomic_store(a.ready + g, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
  }

  // The last workgroup to finish returns the claim counters and every ready
  // flag to zero (a flag set late, after a guard gave up on it, included)
  // and stores the new lengths (every item of the launch read the old ones).
  // Each workgroup's stores are acknowledged before it claims its exit.
  const StepArgs& a = launder();
  const SelectArgs& sa = a.s;
  const int tid = thread_id();
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0) s_item = claim(a.queue + 2);
  __syncthreads();
  if (s_item != gridDim.x - 1) return;
  if (tid < 3) __hip_atomic_store(a.queue + tid, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int groups = sa.c.batch * sa.c.kv_heads;
  for (int g = tid; g < groups; g += kStepThreads)
    __hip_atomic_store(a.ready + g, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (int b = tid; b < sa.c.batch; b += kStepThreads) {
    const int L0 = sa.seq_lens[b];
    if (L0 >= 0 && L0 < sa.c.capacity) sa.lens_out[b] = L0 + 1;
  }
}

template <int G>
hipError_t launch_g(const StepArgs& a, int nj, int grid, hipStream_t stream) {
  switch (nj) {
    case 16: hipLaunchKernelGGL((k_step<G, 16>), dim3(grid), dim3(kStepThreads), 0, stream, a); break;
    case 32: hipLaunchKernelGGL((k_step<G, 32>), dim3(grid), dim3(kStepThreads), 0, stream, a); break;
    case 64: hipLaunchKernelGGL((k_step<G, 64>), dim3(grid), dim3(kStepThreads), 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int32_t step_max_blocks() { return kStepThreads * 64; }

int32_t step_blocks_per_range(int32_t batch, int32_t kv_heads, int32_t max_blocks_seq) {
  // About two score ranges per CU in all (256 CUs), so that groups finish
  // scoring in two rounds and the first round's top-n overlaps the second;
  // whole 32-block words (one word of the above-window bits per range), at
  // least 32 blocks per wave, at most the LDS staging area.
  const int64_t groups = (int64_t)batch * kv_heads;
  const int64_t per_group = (512 + groups - 1) / groups;
  int64_t bpr = ((int64_t)max_blocks_seq + per_group - 1) / per_group;
  bpr = (bpr + 31) / 32 * 32;
  if (bpr < 256) bpr = 256;
  if (bpr > kMaxBlocksPerWg) bpr = kMaxBlocksPerWg;
  return (int32_t)bpr;
}

int32_t step_hist_words(int32_t batch, int32_t kv_heads, int32_t max_blocks_seq) {
  // Ranges per group: never more than ceil(M / 256), nor than
  // max(per_group, ceil(M / 8192)); both bounds grow with M.
  const int64_t groups = (int64_t)batch * kv_heads;
  const int64_t per_group = (512 + groups - 1) / groups;
  const int64_t m = max_blocks_seq > 0 ? max_blocks_seq : 0;
  int64_t r = (m + kMaxBlocksPerWg - 1) / kMaxBlocksPerWg;
  if (r < per_group) r = per_group;
  const int64_t most = (m + 255) / 256;
  if (r > most) r = most;
  return (int32_t)(r * kSlotWords);
}

hipError_t launch_step(const StepArgs& a, hipStream_t stream) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int M = a.s.max_blocks_seq;
  const int nj = M <= kStepThreads * 16 ? 16 : (M <= kStepThreads * 32 ? 32 : 64);
  // One workgroup per CU; never more than there are items.
  int grid = cus > 0 ? cus : 1;
  const int items = a.score_items > a.dec_items ? a.score_items : a.dec_items;
  if (grid > items) grid = items > 0 ? items : 1;
  switch (a.d.group) {
    case 1: return launch_g<1>(a, nj, grid, stream);
    case 2: return launch_g<2>(a, nj, grid, stream);
    case 3: return launch_g<3>(a, nj, grid, stream);
    case 4: return launch_g<4>(a, nj, grid, stream);
    case 5: return launch_g<5>(a, nj, grid, stream);
    case 6: return launch_g<6>(a, nj, grid, stream);
    case 7: return launch_g<7>(a, nj, grid, stream);
    case 8: return launch_g<8>(a, nj, grid, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace resa
