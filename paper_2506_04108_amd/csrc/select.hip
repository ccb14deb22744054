// Block selection (Sec. 2.1): average-pooled group query, Quest block score
// (Eq. 4) and the dynamic top-n (Eq. 5) with local forcing.
#include "resa_device.h"
#include "resa_internal.h"

namespace resa {
namespace {

constexpr int kSelThreads = 1024;                 // 16 waves
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kTopnThreads = 1024;
constexpr int kBins1 = 256;                       // first digit: key bits 31..24
constexpr int kSlotWords = 256;                   // per-workgroup slot: two 256-bin 16-bit histograms
constexpr int kBins2 = 4096;                      // next digits: bits 23..12, then 11..0
constexpr int kKeysPerLane = 32;                  // fused top-n: M <= 1024 threads x 32
constexpr int kMaxBlocksPerWg = 8192;             // scores staged in LDS per workgroup (32 KiB)
constexpr int kBufWord3 = 0x00020000;             // raw buffer resource, 32-bit data format
constexpr int kSc1 = 16;                          // cache policy: agent-scope coherent

__device__ __forceinline__ uint32_t block_key(int m, int forced_from, float s) {
  return m >= forced_from ? 0xFFFFFFFFu : order_key(s);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kBufWord3);
}

// Length of sequence bb seen by the selection. With an append fused in
// front (k_new set), the new token goes to row `pos` = the stored length and
// the selection sees one more token; a full cache is left as it is.
struct SeqLen {
  int L, pos;  // pos = row of the appended token, -1 without one
};

__device__ __forceinline__ SeqLen seq_len_of(const SelectArgs& a, int bb) {
  const int L0 = a.seq_lens[bb];
  if (a.k_new != nullptr && L0 >= 0 && L0 < a.c.capacity) return {L0 + 1, L0};
  return {L0, -1};
}

// Each group takes a ticket on its sequence's counter once every workgroup
// of the group has read the old length (after the group's last ticket); the
// group holding the last ticket (t) stores the new length, which therefore
// no workgroup of this launch can see, and returns the counter to zero.
__device__ __forceinline__ void finish_append(const SelectArgs& a, int bb, int L, uint32_t t) {
  if (t == (uint32_t)a.c.kv_heads - 1) {
    a.lens_out[bb] = L;
    __hip_atomic_store(a.seq_counters + bb, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Exclusive prefix sum over the 1024 threads of the workgroup; returns the
// thread's exclusive prefix and writes the total to *total. Waves scan with
// DPP, publish their totals, and every thread adds the totals of the waves
// before its own.
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* lds16, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t x = wave_incl_scan(v);
  if (lane == 63) lds16[wave] = x;
  lds_sync();
  uint32_t off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    const uint32_t t = lds16[w];
    off += w < wave ? t : 0u;
    tot += t;
  }
  *total = tot;
  lds_sync();  // lds16 may be reused by the next scan
  return off + x - v;
}

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
  const float* sc = a.scores + grp * a.score_stride;
  const int forced_from = M - a.n_local;
  const int E = (M + kTopnThreads - 1) / kTopnThreads;
  const int lo = min(tid * E, M), hi = min(lo + E, M);
  auto key_of = [&](int m) -> uint32_t {
    return m >= forced_from ? 0xFFFFFFFFu : order_key(sc[m]);
  };

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

__global__ __launch_bounds__(kTopnThreads) void k_topn(SelectArgs a) {
  const SeqLen sl = seq_len_of(a, blockIdx.y);
  topn_group(a, sl.L);
  if (a.k_new != nullptr && threadIdx.x == 0)
    finish_append(a, blockIdx.y, sl.L,
                  __hip_atomic_fetch_add(a.seq_counters + blockIdx.y, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}


// Among `nbins` counted digits (a larger digit is a larger key), finds the
// digit holding the k-th largest key, with the 1024 threads of the group:
// thread t owns `per` consecutive digits in descending order, waves scan
// their sums with lane shuffles, and every thread adds the totals of the
// waves before its own (two barriers). Leaves {digit, rank within the digit,
// count of the digit} in misc[0..2].
__device__ void find_digit(const uint32_t* hist, int nbins, uint32_t k, uint32_t* lds32,
                           uint32_t* misc) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int per = nbins >= kSelThreads ? nbins / kSelThreads : 1;
  const int owners = nbins / per;
  uint32_t cnt[kBins2 / kSelThreads];
  uint32_t sum = 0;
#pragma unroll
  for (int j = 0; j < kBins2 / kSelThreads; ++j) {
    cnt[j] = (tid < owners && j < per) ? hist[nbins - 1 - (tid * per + j)] : 0u;
    sum += cnt[j];
  }
  const uint32_t x = wave_incl_scan(sum);
  if (lane == 63) lds32[wave] = x;
  lds_sync();
  uint32_t cum = x - sum;
  for (int w = 0; w < wave; ++w) cum += lds32[w];
#pragma unroll
  for (int j = 0; j < kBins2 / kSelThreads; ++j) {
    if (tid < owners && j < per && cum < k && cum + cnt[j] >= k) {
      misc[0] = nbins - 1 - (tid * per + j);
      misc[1] = k - cum;
      misc[2] = cnt[j];
    }
    cum += cnt[j];
  }
  lds_sync();
}

constexpr uint32_t kMaxCand = 256;  // bucket size resolved by ranking (4 threads per candidate)

// Exact top-n of one group by its last workgroup (M <= 1024 * NJ). Thread t
// holds the keys of ids [t NJ, t NJ + NJ) in registers, so id order is
// thread order. The key loads are issued first; while they are in flight the
// workgroup sums the group's slots into the counts of the keys' 8 high bits
// (or of 8 more bits inside the window hint). A bucket too large to rank is
// narrowed by 12 more bits. Then one pass over the keys marks, per thread,
// the keys above the bucket of the n-th largest key and the keys inside it
// (bit masks); the few keys in the bucket are gathered and ranked among
// themselves (key descending, id ascending), and those ranked before the
// remaining count are kept: every key above the n-th largest key T and the
// lowest ids among the keys equal to T. One scan of the per-thread kept
// counts gives every thread its first output position, and the kept ids are
// written in ascending order by walking the set bits. NJ is the smallest
// instantiation that covers M, so the unrolled per-thread loops do no more
// work than the group needs.
template <int NJ>
__device__ __forceinline__ void select_tail(const SelectArgs& a, size_t grp, int M, int forced_from, int W,
                                            uint32_t win, uint32_t* s_hist, uint32_t* lds32, uint32_t* misc,
                                            int32_t* s_out, int bb, int L) {
  const int tid = threadIdx.x;
  const int n = count_selected(M, a.keep_ppm, a.min_blocks, a.n_local);
  int32_t* out = a.block_idx + grp * a.n_cap;
  if (n == 0 || n >= M) {
    if (tid == 0) {
      a.num_sel[grp] = n;
      __hip_atomic_store(a.counters + grp, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (a.k_new != nullptr)
        finish_append(a, bb, L, __hip_atomic_fetch_add(a.seq_counters + bb, 1u, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT));
    }
    for (int i = tid; i < a.n_cap; i += kSelThreads) out[i] = i < n ? i : -1;
    return;
  }
  const int id0 = tid * NJ;
  // The row is padded to a multiple of 4 scores, so each 16-byte load is
  // wholly inside the row or wholly past it (then it reads 0); ids past M
  // are never used.
  const __amdgpu_buffer_rsrc_t rs = buf_rsrc(a.scores + grp * a.score_stride, (uint32_t)((M + 3) & ~3) * 4);
  // The digit search needs only the group's W slots (word d holds two 16-bit
  // counts): word d gets 4 threads, each summing every 4th slot. The first
  // round of slot loads is issued before the key loads, so the slot sums can
  // be used while the keys are still arriving.
  const uint32_t* slots = a.hist + grp * W * kSlotWords;
  const int sd = tid & (kSlotWords - 1), spart = tid / kSlotWords;
  constexpr int kParts = kSelThreads / kSlotWords;
  uint32_t sv[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int w = spart + j * kParts;
    sv[j] = w < W ? __hip_atomic_load(slots + w * kSlotWords + sd, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
  }
  float raw[NJ];
  if constexpr (NJ % 4 == 0) {
#pragma unroll
    for (int i = 0; i < NJ / 4; ++i) {
      const f4_t v = __builtin_bit_cast(f4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, (id0 + 4 * i) * 4, 0, kSc1));
      raw[4 * i] = v.x;
      raw[4 * i + 1] = v.y;
      raw[4 * i + 2] = v.z;
      raw[4 * i + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < NJ; ++i)
      raw[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, (id0 + i) * 4, 0, kSc1));
  }

  // Stores go out after the loads: a wave's memory counter drains in issue
  // order, so a store issued before a load would make the load's consumer
  // wait for the store's acknowledgement too. Every workgroup of the group
  // has taken its ticket, so the counter can be reset for the next call.
  // Every workgroup of the group has read the old length (all took their
  // tickets), so the sequence's counter is bumped now; its result is only
  // looked at after the selection, so the round trip overlaps the tail.
  uint32_t seq_ticket = 0;
  if (tid == 0) {
    if (a.k_new != nullptr)
      seq_ticket = __hip_atomic_fetch_add(a.seq_counters + bb, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    a.num_sel[grp] = n;
    __hip_atomic_store(a.counters + grp, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  {
    // Bins 0..255 of s_hist get the top-byte counts, 256..511 the window
    // counts.
    if (tid < 2 * kSlotWords) s_hist[tid] = 0;
    if (tid == 0) misc[4] = 0;  // candidate counter of the ranking step (misc[3] holds the ticket)
    lds_sync();
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      lo += sv[j] & 0xFFFFu;
      hi += sv[j] >> 16;
    }
    for (int w0 = spart + 16 * kParts; w0 < W; w0 += 16 * kParts) {
      uint32_t v[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int w = w0 + j * kParts;
        v[j] = w < W ? __hip_atomic_load(slots + w * kSlotWords + sd, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        lo += v[j] & 0xFFFFu;
        hi += v[j] >> 16;
      }
    }
    atomicAdd(&s_hist[2 * sd], lo);
    atomicAdd(&s_hist[2 * sd + 1], hi);
    lds_sync();
  }


  // Window hint: keys whose top 9 bits equal W9 were also counted by bits
  // 22..15. When the n-th largest key falls inside that window, those counts
  // pin 17 bits at once; otherwise the top-byte counts give 8.
  uint32_t prefix, pmask, k = (uint32_t)n;
  int known;
  bool in_win = false;
  if (win >> 31) {
    const uint32_t w9 = win & 0x1FFu, w8 = w9 >> 1;
    // Keys in the window, and keys above it.
    uint32_t inw = 0, above = 0;
    if (tid < 64) {
      uint32_t x = 0, y = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x += s_hist[256 + 4 * tid + j];
        const uint32_t t8 = 4 * tid + j;
        y += t8 > w8 ? s_hist[t8] : 0u;
      }
      x = wave_incl_scan(x);
      y = wave_incl_scan(y);
      inw = (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
      above = (uint32_t)__builtin_amdgcn_readlane((int)y, 63);
      // The other half of the window's top byte lies above it when W9 is even.
      if ((w9 & 1u) == 0) above += s_hist[w8] - inw;
      if (tid == 0) {
        misc[5] = inw;
        misc[6] = above;
      }
    }
    lds_sync();
    inw = misc[5];
    above = misc[6];
    in_win = above < k && k <= above + inw;
    if (in_win) {
      find_digit(s_hist + 256, 256, k - above, lds32, misc);
      prefix = (w9 << 23) | (misc[0] << 15);
      pmask = 0xFFFF8000u;
      known = 17;
    }
  }
  if (!in_win) {
    find_digit(s_hist, kBins1, k, lds32, misc);
    prefix = misc[0] << 24;
    pmask = 0xFFu << 24;
    known = 8;
  }
  k = misc[1];
  uint32_t cnt = misc[2];
  // Keys are first needed here; their loads overlapped the digit search.
  uint32_t key[NJ];
#pragma unroll
  for (int i = 0; i < NJ; ++i) key[i] = block_key(id0 + i, forced_from, raw[i]);
  const int nv = min(max(M - id0, 0), NJ);  // this thread's valid keys: j < nv
  const uint32_t valid = nv >= 32 ? 0xFFFFFFFFu : (1u << nv) - 1u;
  // A bucket too large to rank is narrowed by the next 12 bits (rare once
  // the window hint follows the threshold).
  while (known < 32 && cnt != k && cnt > kMaxCand) {
    const int width = min(12, 32 - known), shift = 32 - known - width;
    const uint32_t dmask = (1u << width) - 1u;
    for (int i = tid; i < (1 << width); i += kSelThreads) s_hist[i] = 0;
    lds_sync();
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (j < nv && (key[j] & pmask) == prefix) atomicAdd(&s_hist[(key[j] >> shift) & dmask], 1u);
    lds_sync();
    find_digit(s_hist, 1 << width, k, lds32, misc);
    prefix |= misc[0] << shift;
    pmask |= dmask << shift;
    known += width;
    k = misc[1];
    cnt = misc[2];
  }

  // One pass over the keys: bit j of `take` marks key j above the bucket of
  // the n-th largest key, bit j of `inb` key j inside it.
  uint32_t take = 0, inb = 0;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const uint32_t km = key[j] & pmask;
    take |= km > prefix ? 1u << j : 0u;
    inb |= km == prefix ? 1u << j : 0u;
  }
  take &= valid;
  inb &= valid;
  uint32_t thr = prefix;  // the threshold key (its known bits), for the next call's window
  // 0: the whole bucket is kept; 1: its candidates were ranked; 2: every key
  // of the bucket equals the threshold and the k lowest ids are kept.
  const int mode = cnt == k ? 0 : (cnt <= kMaxCand ? 1 : 2);
  if (mode == 0) {
    take |= inb;
  } else if (mode == 1) {
    // Rank the bucket's keys among themselves in (key descending, id
    // ascending) order: a candidate is kept iff fewer than k candidates come
    // before it, which keeps every key above the threshold T and the lowest
    // ids among the keys equal to T. A candidate is stored as
    // (key << 32 | ~id), so that order is plain 64-bit descending order; the
    // kept ones set their id's bit in an LDS bitmap (ids < 32768: 1024 words).
    uint64_t* cv = reinterpret_cast<uint64_t*>(s_hist);   // words [0, 2 kMaxCand)
    uint32_t* bits = s_hist + 2048;                       // words [2048, 3072)
    bits[tid] = 0;
    const uint32_t mine = __builtin_popcount(inb);
    const uint32_t incl = wave_incl_scan(mine);
    const uint32_t wave_tot = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
    uint32_t base = 0;
    if ((tid & 63) == 63 && wave_tot != 0) base = atomicAdd(&misc[4], wave_tot);
    uint32_t at = (uint32_t)__builtin_amdgcn_readlane((int)base, 63) + incl - mine;
    if (inb != 0) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        if ((inb >> j) & 1u) {
          cv[at] = ((uint64_t)key[j] << 32) | (uint32_t)~(uint32_t)(id0 + j);
          ++at;
        }
      }
    }
    lds_sync();
    {
      // Four threads per candidate (lanes 4c .. 4c + 3 of one wave), each
      // counting over a quarter of the bucket; the quarters are added with
      // DPP quad swaps.
      const uint32_t cand = (uint32_t)tid >> 2, part = (uint32_t)tid & 3u;
      uint32_t before = 0;
      uint64_t vt = 0;
      if (cand < cnt) {
        vt = cv[cand];
        const uint32_t qlen = (cnt + 3) >> 2;
        const uint32_t j1 = min((part + 1) * qlen, cnt);
        uint32_t j = part * qlen;
        for (; j + 8 <= j1; j += 8) {
          uint64_t v[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) v[u] = cv[j + u];
#pragma unroll
          for (int u = 0; u < 8; ++u) before += v[u] > vt;
        }
        for (; j < j1; ++j) before += cv[j] > vt;
      }
      before += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)before, kDppXor1, 0xf, 0xf, true);
      before += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)before, kDppXor2, 0xf, 0xf, true);
      if (cand < cnt && part == 0 && before < k) {
        const uint32_t id = ~(uint32_t)vt;
        atomicOr(&bits[id >> 5], 1u << (id & 31u));
        if (before == k - 1) misc[0] = (uint32_t)(vt >> 32);  // T
      }
    }
    lds_sync();
    thr = misc[0];
    // This thread's ids [id0, id0 + NJ) span at most two bitmap words.
    const uint32_t w0 = (uint32_t)id0 >> 5, sh = (uint32_t)id0 & 31u;
    uint64_t pair = bits[w0];
    if (sh + NJ > 32) pair |= (uint64_t)bits[w0 + 1] << 32;
    take |= (uint32_t)(pair >> sh) & valid;
  }
  // The next call's window: the top 9 bits of this threshold. The stores
  // here go out before the compaction so their latency overlaps it.
  if (tid == 0) {
    if (a.k_new != nullptr) finish_append(a, bb, L, seq_ticket);
    a.window[grp] = 0x80000000u | (thr >> 23);
  }

  // Output positions: one scan of the packed per-thread counts (kept keys in
  // the high half; in mode 2 also the bucket keys, which are kept in id
  // order up to k, in the low half; totals <= M < 2^16).
  const uint32_t nb = mode == 2 ? (uint32_t)__builtin_popcount(inb) : 0u;
  uint32_t tot;
  const uint32_t before = block_exclusive_scan(((uint32_t)__builtin_popcount(take) << 16) | nb, lds32, &tot);
  uint32_t pos = before >> 16;
  if (mode == 2) {
    // Bucket keys kept by earlier threads, then by this one. Written so that
    // no subtraction can wrap: the form `k > e ? k - e : 0` was compiled into
    // an unguarded k - e.
    const uint32_t eb = min(before & 0xFFFFu, k);
    uint32_t keep = min(k - eb, nb);
    uint32_t m = inb;
    for (; keep > 0; --keep) {
      take |= m & (0u - m);  // lowest remaining bucket id
      m &= m - 1u;
    }
    pos += eb;
  }
  // Kept ids in ascending order. Rows shorter than the workgroup's score
  // staging area (free by now) are assembled there and written out coalesced.
  const bool staged = a.n_cap < kMaxBlocksPerWg;
  for (uint32_t m = take; m != 0; m &= m - 1u) {
    const int32_t id = id0 + __builtin_ctz(m);
    if (pos < (uint32_t)a.n_cap) {  // never past the row, whatever the scores
      if (staged) s_out[pos] = id;
      else out[pos] = id;
    }
    ++pos;
  }
  if (staged) {
    lds_sync();
    for (int i = tid; i < a.n_cap; i += kSelThreads) out[i] = i < n ? s_out[i] : -1;
    return;
  }
  for (int i = n + tid; i < a.n_cap; i += kSelThreads) out[i] = -1;
}

// Pooled query (Fig. 3), Quest scores (Eq. 4) and, when `fused`, the top-n
// (Eq. 5) in one kernel. Grid (ceil(max_blocks_seq / blocks_per_wg), kv
// heads, batch), about one 16-wave workgroup per CU. Each workgroup streams
// the summaries of its block range: lane (r, c) handles dims [8c, 8c + 8) of
// 16-block tiles, so each wave-wide load is four whole 256-byte summary rows,
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
template <int NJ>
__global__ __launch_bounds__(kSelThreads) void k_select(SelectArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t s_hist[kBins2];
  __shared__ __attribute__((aligned(16))) float s_score[kMaxBlocksPerWg];
  __shared__ uint32_t s_lds32[32];
  __shared__ uint32_t s_misc[8];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hk = blockIdx.y, bb = blockIdx.z;
  const size_t grp = (size_t)bb * a.c.kv_heads + hk;
  const SeqLen sl = seq_len_of(a, bb);
  const int L = sl.L;
  // Lengths beyond max_seq_len are clamped so every access stays in bounds.
  const int M = max(0, min(min((L + a.c.block_size - 1) / a.c.block_size, a.max_blocks_seq), a.c.max_blocks));
  const int forced_from = M - a.n_local;
  const int b0 = blockIdx.x * a.blocks_per_wg;
  const int b1 = min(b0 + a.blocks_per_wg, M);
  const int r = lane >> 4, c = lane & 15, col = c * 8;

  // Fused append (Alg. 1): the first workgroup of the group writes the new
  // K and V rows; the workgroup owning block pos / b folds the new key into
  // that block's summary (or starts it) before scoring it, and stores it.
  const int m_new = sl.pos >= 0 ? sl.pos / a.c.block_size : -1;
  const bool opening = sl.pos >= 0 && sl.pos % a.c.block_size == 0;
  U4 knew = U4{0, 0, 0, 0}, vnew = U4{0, 0, 0, 0};
  const bool row_writer = sl.pos >= 0 && blockIdx.x == 0 && tid < 32;
  const int64_t new_row = row_writer ? kv_row(a.c, bb, hk, sl.pos) : -1;
  if (sl.pos >= 0) {
    knew = ld16(a.k_new + grp * kHeadDim + col);
    if (row_writer && tid >= 16) vnew = ld16(a.v_new + grp * kHeadDim + col);
  }

  // Window hint left by the previous call on this workspace (any value is
  // valid: it only chooses which key bits get a second histogram).
  const uint32_t win = a.fused ? a.window[grp] : 0u;
  const bool win_on = (win >> 31) != 0;
  const uint32_t w9 = win & 0x1FFu;
  if (a.fused) {
    for (int i = tid; i < 2 * kSlotWords; i += kSelThreads) s_hist[i] = 0;
    lds_sync();
  }
  // The appended block's updated summary row, held by the lanes that score
  // it and stored after the loop (a store inside it would hold up that
  // wave's next tile: the memory counter drains in issue order).
  U4 new_lo = U4{0, 0, 0, 0}, new_hi = U4{0, 0, 0, 0};
  bool owns_row = false;
  if (b0 < b1) {
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
    const uint16_t* kmin = a.c.kmin + grp * a.c.max_blocks * kHeadDim + col;
    const uint16_t* kmax = a.c.kmax + grp * a.c.max_blocks * kHeadDim + col;
    const int ntiles = (b1 - b0 + 15) / 16;
    // Rows past b1 read the last valid block (in bounds) and are ignored.
    auto load_tile = [&](int t, U4 (&lo4)[4], U4 (&hi4)[4]) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int m = min(b0 + 16 * t + 4 * u + r, b1 - 1);
        lo4[u] = ld16_stream(kmin + (size_t)m * kHeadDim);
        hi4[u] = ld16_stream(kmax + (size_t)m * kHeadDim);
      }
    };
    U4 lo4[4], hi4[4], nlo[4], nhi[4];
    int t = wave;
    load_tile(min(t, ntiles - 1), lo4, hi4);
    while (t < ntiles) {
      load_tile(min(t + kSelWaves, ntiles - 1), nlo, nhi);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int mu = b0 + 16 * t + 4 * u + r;
        if (mu == m_new && mu < b1) {
          lo4[u] = opening ? knew : u4_min(lo4[u], knew);
          hi4[u] = opening ? knew : u4_max(hi4[u], knew);
          new_lo = lo4[u];
          new_hi = hi4[u];
          owns_row = true;
        }
        const uint32_t wl[4] = {lo4[u].x, lo4[u].y, lo4[u].z, lo4[u].w};
        const uint32_t wh[4] = {hi4[u].x, hi4[u].y, hi4[u].z, hi4[u].w};
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float a0 = use_max[2 * j] ? bf_lo(wh[j]) : bf_lo(wl[j]);
          const float a1 = use_max[2 * j + 1] ? bf_hi(wh[j]) : bf_hi(wl[j]);
          s = fmaf(qb[2 * j], a0, s);
          s = fmaf(qb[2 * j + 1], a1, s);
        }
        s = row16_sum(s);
        const int m = b0 + 16 * t + 4 * u + r;
        if (c == 0 && m < b1) {
          s_score[m - b0] = s;
          if (a.fused) {
            const uint32_t key = block_key(m, forced_from, s);
            atomicAdd(&s_hist[key >> 24], 1u);
            if (win_on && (key >> 23) == w9) atomicAdd(&s_hist[256 + ((key >> 15) & 0xFFu)], 1u);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        lo4[u] = nlo[u];
        hi4[u] = nhi[u];
      }
      t += kSelWaves;
    }
  }
  lds_sync();
  if (owns_row) {
    const size_t so = (grp * a.c.max_blocks + m_new) * kHeadDim + col;
    st16(a.c.kmin + so, new_lo);
    st16(a.c.kmax + so, new_hi);
  }
  if (new_row >= 0) {
    // The new K and V rows (stored after the scoring, so the loads above have
    // long arrived).
    const size_t row = (size_t)new_row * kHeadDim + col;
    if (tid < 16)
      st16(const_cast<uint16_t*>(a.c.k) + row, knew);
    else
      st16(const_cast<uint16_t*>(a.c.v) + row, vnew);
  }
  // Coalesced write-out of this range's scores: to the workspace rows (16-byte
  // aligned, write-through at agent scope) and, if asked, to scores_out.
  const int nb = max(b1 - b0, 0);
  if (nb > 0) {
    const __amdgpu_buffer_rsrc_t rs = buf_rsrc(a.scores + grp * a.score_stride + b0, (uint32_t)nb * 4);
    for (int i = 4 * tid; i < nb; i += 4 * kSelThreads) {
      const f4_t v = *reinterpret_cast<const f4_t*>(&s_score[i]);
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(__attribute__((ext_vector_type(4))) unsigned, v),
                                             rs, i * 4, 0, kSc1);
    }
    if (a.scores_out != nullptr) {
      float* so = a.scores_out + grp * a.max_blocks_seq + b0;
      for (int i = tid; i < nb; i += kSelThreads) so[i] = s_score[i];
    }
  }
  if (!a.fused) return;
  // This workgroup's digit counts go to its own slot: no shared counters.
  // Counts fit in 16 bits (at most kMaxBlocksPerWg per workgroup): two per word.
  uint32_t* slot = a.hist + (grp * gridDim.x + blockIdx.x) * kSlotWords;
  for (int i = tid; i < kSlotWords; i += kSelThreads)
    __hip_atomic_store(slot + i, s_hist[2 * i] | (s_hist[2 * i + 1] << 16), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0)
    s_misc[3] = __hip_atomic_fetch_add(a.counters + grp, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (s_misc[3] != gridDim.x - 1) return;
  const int W = gridDim.x;
  select_tail<NJ>(a, grp, M, forced_from, W, win, s_hist, s_lds32, s_misc,
                  reinterpret_cast<int32_t*>(s_score), bb, L);
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  if (a.max_blocks_seq > 0) {
    dim3 grid((a.max_blocks_seq + a.blocks_per_wg - 1) / a.blocks_per_wg, a.c.kv_heads, a.c.batch);
    // Keys per thread of the fused top-n: the smallest instantiation that
    // holds the longest group (every group's M <= max_blocks_seq).
    const int per = (a.max_blocks_seq + kSelThreads - 1) / kSelThreads;
    if (per <= 4)
      hipLaunchKernelGGL(k_select<4>, grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 5)
      hipLaunchKernelGGL(k_select<5>, grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 6)
      hipLaunchKernelGGL(k_select<6>, grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 8)
      hipLaunchKernelGGL(k_select<8>, grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 12)
      hipLaunchKernelGGL(k_select<12>, grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 16)
      hipLaunchKernelGGL(k_select<16>, grid, dim3(kSelThreads), 0, stream, a);
    else if (per <= 24)
      hipLaunchKernelGGL(k_select<24>, grid, dim3(kSelThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(k_select<kKeysPerLane>, grid, dim3(kSelThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.fused) return hipSuccess;
  }
  hipLaunchKernelGGL(k_topn, dim3(a.c.kv_heads, a.c.batch), dim3(kTopnThreads), 0, stream, a);
  return hipGetLastError();
}

int32_t select_fused_max_blocks() { return kSelThreads * kKeysPerLane; }

int32_t select_blocks_per_wg(int32_t batch, int32_t kv_heads, int32_t max_blocks_seq) {
  // About one 16-wave workgroup per CU (256 CUs) in all: a group's blocks are
  // cut into equal ranges, in whole 16-block tiles, at least one tile per
  // wave (256 blocks) and at most the LDS staging area.
  const int64_t groups = (int64_t)batch * kv_heads;
  const int64_t per_group = (256 + groups - 1) / groups;
  int64_t bpw = ((int64_t)max_blocks_seq + per_group - 1) / per_group;
  bpw = (bpw + 15) / 16 * 16;
  if (bpw < 256) bpw = 256;
  if (bpw > kMaxBlocksPerWg) bpw = kMaxBlocksPerWg;
  return (int32_t)bpw;
}

int32_t select_hist_words(int32_t batch, int32_t kv_heads, int32_t max_blocks_seq) {
  // A bound on the workgroups per group that never decreases as the length
  // grows (the count itself can, by a few, as the ranges are rounded to
  // tiles), so a workspace sized for a longer length fits every shorter one:
  // at most ceil(M / 256) ranges, and at most max(per_group, ceil(M / 8192)).
  const int64_t groups = (int64_t)batch * kv_heads;
  const int64_t per_group = (256 + groups - 1) / groups;
  const int64_t m = max_blocks_seq > 0 ? max_blocks_seq : 0;
  int64_t wgs = (m + kMaxBlocksPerWg - 1) / kMaxBlocksPerWg;
  if (wgs < per_group) wgs = per_group;
  const int64_t most = (m + 255) / 256;
  if (wgs > most) wgs = most;
  return (int32_t)(wgs * kSlotWords);
}

}  // namespace resa
