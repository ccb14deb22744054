// Block selection (Sec. 2.1) device code shared by the selection kernels and
// the fused decode step: average-pooled group query, Quest block score
// (Eq. 4) and the dynamic top-n (Eq. 5) with local forcing.
#pragma once

#include <type_traits>

#include "resa_device.h"
#include "resa_internal.h"

namespace resa {
namespace {

constexpr int kBins1 = 256;                       // first digit: key bits 31..24
constexpr int kSlotWords = 256;                   // per-workgroup slot: two 256-bin 16-bit histograms
constexpr int kBins2 = 4096;                      // next digits: bits 23..12, then 11..0
constexpr int kMaxSelectBlocks = 32768;          // fused top-n: M <= 32768 (keys in registers)
constexpr int kMaxBlocksPerWg = 8192;             // scores staged in LDS per workgroup (32 KiB)

// The top-n's in-window path (and the scoring's above-window bits and
// in-window lists it reads) is used when its workgroup holds at least 16384
// keys (NJ keys per thread, NT threads): below that, reading all keys costs
// less than the lists' extra round trip and their write-through stores.
// The lists are also limited to score ranges of at most kListRange blocks:
// a range's list stores grow with its length (one scattered write-through
// store per in-window key before its ticket) while the tail's saving does
// not (256K, batch 8: 4 ranges of 4128 blocks per group, selection 104 ->
// 108 us with them; batch 1: 31 ranges of 544 blocks, 27.4 -> 25.1 us).
__host__ __device__ constexpr bool window_lists(int nj, int nt) { return nj * nt >= 16384; }
constexpr int kListRange = 1024;

__device__ __forceinline__ uint32_t block_key(int m, int forced_from, float s) {
  return m >= forced_from ? 0xFFFFFFFFu : order_key(s);
}

// A buffer resource over a workgroup-uniform range (marked uniform for the
// compiler: in the persistent step kernel the group index comes from LDS,
// and a resource in vector registers would take a loop over the lanes).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(wave_uniform(p)), (short)0,
                                           (int)__builtin_amdgcn_readfirstlane(bytes), kBufWord3);
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

// Exclusive prefix sum over the NT threads of the workgroup; returns the
// thread's exclusive prefix and writes the total to *total. Waves scan with
// DPP, publish their totals, and every thread adds the totals of the waves
// before its own.
template <int NT>
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* lds16, uint32_t* total) {
  const int lane = thread_id() & 63, wave = thread_id() >> 6;
  const uint32_t x = wave_incl_scan(v);
  if (lane == 63) lds16[wave] = x;
  lds_sync();
  uint32_t off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    const uint32_t t = lds16[w];
    off += w < wave ? t : 0u;
    tot += t;
  }
  *total = tot;
  lds_sync();  // lds16 may be reused by the next scan
  return off + x - v;
}

// Among `nbins` counted digits (a larger digit is a larger key), finds the
// digit holding the k-th largest key, with the NT threads of the group:
// thread t owns `per` consecutive digits in descending order, waves scan
// their sums with lane shuffles, and every thread adds the totals of the
// waves before its own (two barriers). Leaves {digit, rank within the digit,
// count of the digit} in misc[0..2].
template <int NT>
__device__ void find_digit(const uint32_t* hist, int nbins, uint32_t k, uint32_t* lds32,
                           uint32_t* misc) {
  const int tid = thread_id(), lane = tid & 63, wave = tid >> 6;
  const int per = nbins >= NT ? nbins / NT : 1;
  const int owners = nbins / per;
  uint32_t cnt[kBins2 / NT];
  uint32_t sum = 0;
#pragma unroll
  for (int j = 0; j < kBins2 / NT; ++j) {
    cnt[j] = (tid < owners && j < per) ? hist[nbins - 1 - (tid * per + j)] : 0u;
    sum += cnt[j];
  }
  const uint32_t x = wave_incl_scan(sum);
  if (lane == 63) lds32[wave] = x;
  lds_sync();
  uint32_t cum = x - sum;
  for (int w = 0; w < wave; ++w) cum += lds32[w];
#pragma unroll
  for (int j = 0; j < kBins2 / NT; ++j) {
    if (tid < owners && j < per && cum < k && cum + cnt[j] >= k) {
      misc[0] = nbins - 1 - (tid * per + j);
      misc[1] = k - cum;
      misc[2] = cnt[j];
    }
    cum += cnt[j];
  }
  lds_sync();
}

// Sum over the 64 lanes of a wave (every lane active); wave-uniform.
__device__ __forceinline__ uint32_t wave_sum(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(x), 63);
}

// The digit of the k-th largest key (1 <= k <= total) among 256 counted
// digits, by one wave: lane i holds the counts of digits 4i .. 4i + 3 in
// c[0..3] (a larger digit is a larger key). Returns the digit, k's rank
// inside it and its count, all wave-uniform.
struct WaveDigit {
  uint32_t d = 0, k = 0, cnt = 0;
};
__device__ __forceinline__ WaveDigit wave_find_digit(const uint32_t (&c)[4], uint32_t k, int lane) {
  const uint32_t incl = wave_incl_scan(c[0] + c[1] + c[2] + c[3]);
  const uint32_t all = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
  uint32_t above = all - incl;  // keys in digits above this lane's
  uint32_t d = 0, r = 0, cn = 0;
  bool hit = false;
#pragma unroll
  for (int j = 3; j >= 0; --j) {
    if (!hit && above < k && above + c[j] >= k) {
      hit = true;
      d = 4 * lane + j;
      r = k - above;
      cn = c[j];
    }
    above += c[j];
  }
  const unsigned long long b = __ballot(hit);
  const int src = b != 0ull ? __builtin_ctzll(b) : 0;
  WaveDigit out;
  out.d = (uint32_t)__builtin_amdgcn_readlane((int)d, src);
  out.k = (uint32_t)__builtin_amdgcn_readlane((int)r, src);
  out.cnt = (uint32_t)__builtin_amdgcn_readlane((int)cn, src);
  return out;
}

// Keys [id0, id0 + NJ) of a group's key row (agent-scope loads; past the
// row they read 0).
template <int NJ>
__device__ __forceinline__ void load_keys(uint32_t (&key)[NJ], __amdgpu_buffer_rsrc_t rs, int id0) {
  if constexpr (NJ % 4 == 0) {
#pragma unroll
    for (int i = 0; i < NJ / 4; ++i) {
      const U4 v = __builtin_bit_cast(U4, __builtin_amdgcn_raw_buffer_load_b128(rs, (id0 + 4 * i) * 4, 0, kSc1));
      key[4 * i] = v.x;
      key[4 * i + 1] = v.y;
      key[4 * i + 2] = v.z;
      key[4 * i + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < NJ; ++i) key[i] = __builtin_amdgcn_raw_buffer_load_b32(rs, (id0 + i) * 4, 0, kSc1);
  }
}

constexpr uint32_t kMaxCand = 256;  // bucket size resolved by ranking (NT / 256 threads per candidate)

// Exact top-n of one group by its last workgroup (M <= NT * NJ). Thread t
// holds the keys of ids [t NJ, t NJ + NJ) in registers, so id order is
// thread order. The slot loads are issued first, then the key loads; while
// the keys are in flight the workgroup sums the group's slots into the counts
// of the keys' 8 high bits (or of 8 more bits inside the window hint), and one
// wave finds the threshold digit. When that digit lies in the window, the
// in-window path (see below) may finish from the scoring's above-window bits
// and in-window lists, and the key loads are then put off until it cannot.
// A bucket too large to rank is
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
//
// The ids and the count go out with agent-scope stores. With `ready` set
// (the fused decode step), the sequence length is left to the caller and,
// once every store of the workgroup is acknowledged, ready[grp] is set for
// the decode work of the group; otherwise the last group of a sequence
// stores its new length (fused append).
template <int NJ, int NT>
__device__ __forceinline__ void select_tail(const SelectArgs& a, size_t grp, int M, int forced_from, int W,
                                            uint32_t win, uint32_t* s_hist, uint32_t* lds32, uint32_t* misc,
                                            int32_t* s_out, int bb, int L, uint32_t* ready) {
  static_assert(NJ <= 64 && NT % 256 == 0, "tail shape");
  using Mask = std::conditional_t<(NJ > 32), unsigned long long, uint32_t>;
  constexpr int kMaskBits = 8 * sizeof(Mask);
  const int tid = thread_id();
  // Publishes the group's selection to the decode work of a fused step.
  auto publish = [&]() {
    if (ready == nullptr) return;
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) __hip_atomic_store(ready + grp, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };
  const int n = count_selected(M, a.keep_ppm, a.min_blocks, a.n_local);
  int32_t* out = a.block_idx + grp * a.n_cap;
  if (n == 0 || n >= M) {
    if (tid == 0) {
      __hip_atomic_store(a.num_sel + grp, n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.counters + grp, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (a.k_new != nullptr && ready == nullptr)
        finish_append(a, bb, L, __hip_atomic_fetch_add(a.seq_counters + bb, 1u, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT));
    }
    for (int i = tid; i < a.n_cap; i += NT)
      __hip_atomic_store(out + i, i < n ? i : -1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    publish();
    return;
  }
  const int id0 = tid * NJ;
  // The row is padded to a multiple of 4 keys, so each 16-byte load is
  // wholly inside the row or wholly past it (then it reads 0); ids past M
  // are never used.
  const __amdgpu_buffer_rsrc_t rs = buf_rsrc(a.keys + grp * a.score_stride, (uint32_t)((M + 3) & ~3) * 4);
  // The digit search needs only the group's W slots, summed as packed words:
  // word d holds the counts of bins 2d and 2d + 1 in its two halves, and a
  // bin's total over the group is at most M <= kMaxSelectBlocks < 2^16, so
  // adding whole words never carries from one half into the other. Wave v
  // sums slots v, v + NT / 64, ... with one 16-byte load per lane and slot
  // (slots past W read 0 through the buffer's range check, so the loads go
  // out back to back). They are issued before the key loads, so the sums can
  // be formed while the keys are still arriving.
  constexpr int kWaves = NT / 64;
  constexpr int kSlotRound = (32 + kWaves - 1) / kWaves;  // slots per wave in the first round (W <= 32)
  const __amdgpu_buffer_rsrc_t rh = buf_rsrc(a.hist + grp * W * kSlotWords, (uint32_t)W * kSlotWords * 4);
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6), lane4 = (tid & 63) * 4;
  auto slot_load = [&](int w) -> U4 {
    return __builtin_bit_cast(U4, __builtin_amdgcn_raw_buffer_load_b128(rh, (w * kSlotWords + lane4) * 4, 0, kSc1));
  };
  U4 sv[kSlotRound];
#pragma unroll
  for (int j = 0; j < kSlotRound; ++j) sv[j] = slot_load(wv + j * kWaves);
  // The keys as the scoring stored them (forced blocks hold the largest key).
  // With the window hint set and at most 32 ranges (their slots held in sv),
  // the in-window path below may finish without them: their loads are then
  // put off until it cannot. (Only where the scoring wrote the lists, and
  // not with more than 32 keys per thread, whose registers would not last
  // across that path.)
  const bool lazy = window_lists(NJ, NT) && NJ <= 32 && a.blocks_per_wg <= kListRange && (win >> 31) != 0 &&
                    W <= kSlotRound * kWaves;
  uint32_t key[NJ];
  if (!lazy) load_keys<NJ>(key, rs, id0);

  // Stores go out after the loads: a wave's memory counter drains in issue
  // order, so a store issued before a load would make the load's consumer
  // wait for the store's acknowledgement too. Every workgroup of the group
  // has taken its ticket, so the counter can be reset for the next call.
  // Every workgroup of the group has read the old length (all took their
  // tickets), so the sequence's counter is bumped now; its result is only
  // looked at after the selection, so the round trip overlaps the tail.
  uint32_t seq_ticket = 0;
  if (tid == 0) {
    if (a.k_new != nullptr && ready == nullptr)
      seq_ticket = __hip_atomic_fetch_add(a.seq_counters + bb, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(a.num_sel + grp, n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(a.counters + grp, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // The group's packed counts (words 512..767 of s_hist): word d holds the
  // counts of bins 2d and 2d + 1, bins 0..255 being the top byte and
  // 256..511 the window.
  uint32_t* packed = s_hist + 2 * kSlotWords;
  {
    if (tid < kSlotWords) packed[tid] = 0;
    if (tid == 0) misc[4] = 0;  // candidate counter of the ranking step (misc[3] holds the ticket)
    lds_sync();
    U4 acc = sv[0];
#pragma unroll
    for (int j = 1; j < kSlotRound; ++j) acc = U4{acc.x + sv[j].x, acc.y + sv[j].y, acc.z + sv[j].z, acc.w + sv[j].w};
    for (int w = wv + kSlotRound * kWaves; w < W; w += kWaves) {
      const U4 v = slot_load(w);
      acc = U4{acc.x + v.x, acc.y + v.y, acc.z + v.z, acc.w + v.w};
    }
    if (wv < W) {
      atomicAdd(&packed[lane4], acc.x);
      atomicAdd(&packed[lane4 + 1], acc.y);
      atomicAdd(&packed[lane4 + 2], acc.z);
      atomicAdd(&packed[lane4 + 3], acc.w);
    }
    lds_sync();
  }


  // Window hint: keys whose top 9 bits equal W9 were also counted by bits
  // 22..15. When the n-th largest key falls inside that window, those counts
  // pin 17 bits at once; otherwise the top-byte counts give 8. One wave reads
  // the packed counts (lane i: digits 4i .. 4i + 3 of both histograms) and
  // finds the digit; the workgroup waits for it at one barrier.
  if (wv == 0) {
    const int lane = tid;
    const uint32_t p0 = packed[2 * lane], p1 = packed[2 * lane + 1];
    const uint32_t q0 = packed[kSlotWords / 2 + 2 * lane], q1 = packed[kSlotWords / 2 + 2 * lane + 1];
    const uint32_t top[4] = {p0 & 0xFFFFu, p0 >> 16, p1 & 0xFFFFu, p1 >> 16};
    const uint32_t wnd[4] = {q0 & 0xFFFFu, q0 >> 16, q1 & 0xFFFFu, q1 >> 16};
    const uint32_t kk = (uint32_t)n;
    WaveDigit dg;
    uint32_t pre = 0, kn = 8;
    bool found = false;
    if (win >> 31) {
      const uint32_t w9 = win & 0x1FFu, w8 = w9 >> 1;
      // Keys in the window, and keys above it (the other half of the
      // window's top byte lies above it when W9 is even).
      uint32_t y = 0, t8 = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        y += (uint32_t)(4 * lane + j) > w8 ? top[j] : 0u;
        t8 = (uint32_t)j == (w8 & 3u) ? top[j] : t8;
      }
      const uint32_t inw = wave_sum(wnd[0] + wnd[1] + wnd[2] + wnd[3]);
      uint32_t above = wave_sum(y);
      if ((w9 & 1u) == 0) above += (uint32_t)__builtin_amdgcn_readlane((int)t8, (int)(w8 >> 2)) - inw;
      if (above < kk && kk <= above + inw) {
        dg = wave_find_digit(wnd, kk - above, lane);
        pre = (w9 << 23) | (dg.d << 15);
        kn = 17;
        found = true;
      }
    }
    if (!found) {
      dg = wave_find_digit(top, kk, lane);
      pre = dg.d << 24;
    }
    if (lane == 0) {
      misc[0] = pre;
      misc[1] = dg.k;
      misc[2] = dg.cnt;
      misc[5] = kn;
    }
  }
  lds_sync();
  uint32_t prefix = misc[0], k = misc[1], cnt = misc[2];
  int known = (int)misc[5];
  uint32_t pmask = known == 17 ? 0xFFFF8000u : 0xFF000000u;
  const int nv = min(max(M - id0, 0), NJ);  // this thread's valid keys: j < nv
  const Mask valid = nv >= kMaskBits ? ~Mask(0) : (Mask(1) << nv) - Mask(1);
  Mask take = 0, inb = 0;
  uint32_t thr = prefix;  // the threshold key (its known bits), for the next call's window
  // Bucket ranking: candidates are stored as (key << 32 | ~id), so (key
  // descending, id ascending) is plain 64-bit descending order; a candidate
  // is kept iff fewer than k candidates come before it, which keeps every key
  // above the threshold T and the lowest ids among the keys equal to T. The
  // kept ones set their id's bit in an LDS bitmap (ids < 32768: 1024 words);
  // T goes to misc[0]. TPC threads per candidate (adjacent lanes of one wave)
  // each count over a share of the bucket; the shares are added with DPP
  // quad swaps.
  constexpr int TPC = NT / (int)kMaxCand;  // threads per candidate: 4 or 2
  uint64_t* cv = reinterpret_cast<uint64_t*>(s_hist);  // words [0, 2 kMaxCand)
  uint32_t* bits = s_hist + 2048;                      // words [2048, 3072)
  auto rank_bucket = [&]() {
    const uint32_t cand = (uint32_t)tid / TPC, part = (uint32_t)tid % TPC;
    uint32_t before = 0;
    uint64_t vt = 0;
    if (cand < cnt) {
      vt = cv[cand];
      const uint32_t qlen = (cnt + TPC - 1) / TPC;
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
    if constexpr (TPC == 4)
      before += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)before, kDppXor2, 0xf, 0xf, true);
    if (cand < cnt && part == 0 && before < k) {
      const uint32_t id = ~(uint32_t)vt;
      atomicOr(&bits[id >> 5], 1u << (id & 31u));
      if (before == k - 1) misc[0] = (uint32_t)(vt >> 32);  // T
    }
  };
  // This thread's ids [id0, id0 + NJ) from the bitmap: they span at most two
  // words (for every instantiated NJ, (id0 mod 32) + NJ <= 64).
  auto bits_of_thread = [&]() -> Mask {
    const uint32_t w0 = (uint32_t)id0 >> 5, sh = (uint32_t)id0 & 31u;
    uint64_t pair = bits[w0];
    if (sh + NJ > 32) pair |= (uint64_t)bits[w0 + 1] << 32;
    return (Mask)(pair >> sh) & valid;
  };
  // 0: the whole bucket is kept; 1: its candidates were ranked; 2: every key
  // of the bucket equals the threshold and the k lowest ids are kept.
  int mode = 0;
  bool done = false;
  if (lazy && known == 17 && cnt <= kMaxCand) {
    // In-window path: the n-th largest key lies in the window, so every key
    // above the window is kept (the scoring's above-window bits), and of the
    // in-window keys (each range's list, digits descending) those with a digit
    // above d are kept and those with digit d form the bucket. Per range r:
    // A_r keys with a digit above d and B_r with digit d, from the window
    // counts of its slot (words 128..255, held by lanes 32..63 of the wave
    // that loaded it: word 4 l + q holds digits 8 (l - 32) + 2 q and + 1).
    const uint32_t d = (prefix >> 15) & 0xFFu;
    uint32_t* ab = s_hist + 3 * kSlotWords;  // words [768, 1024): A, B, prefixes, total
    const int ln = tid & 63;
#pragma unroll
    for (int j = 0; j < kSlotRound; ++j) {
      const uint32_t wd[4] = {sv[j].x, sv[j].y, sv[j].z, sv[j].w};
      uint32_t gt = 0, eq = 0;
      if (ln >= 32) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const uint32_t dg = 8u * (uint32_t)(ln - 32) + 2u * q + h, c = (wd[q] >> (16 * h)) & 0xFFFFu;
            gt += dg > d ? c : 0u;
            eq += dg == d ? c : 0u;
          }
      }
      const uint32_t A = wave_sum(gt), B = wave_sum(eq);
      const int w = wv + j * kWaves;
      if (ln == 0 && w < W) {
        ab[w] = A;
        ab[32 + w] = B;
      }
    }
    lds_sync();
    if (wv == 0) {
      const uint32_t A = ln < W ? ab[ln] : 0u, B = ln < W ? ab[32 + ln] : 0u, C = A + B;
      const uint32_t cpre = wave_incl_scan(C) - C, bpre = wave_incl_scan(B) - B, ctot = wave_sum(C);
      if (ln < W) {
        ab[64 + ln] = cpre;
        ab[96 + ln] = bpre;
      }
      if (ln == 0) ab[128] = ctot;
    }
    lds_sync();
    const uint32_t E = ab[128];  // list entries needed: at most one per thread
    if (E <= (uint32_t)NT) {
      done = true;
      // Diagnostic: calls of this group whose top-n finished on this path.
      if (tid == 0) __hip_atomic_fetch_add(a.stats + grp, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      // Requests: the group's above-window bits and this thread's entry
      // (entry e of range r, r the last range with prefix <= e).
      constexpr int kBitWords = 1024 / NT;
      const int words = (M + 31) / 32;
      const uint32_t* gb = a.above_bits + grp * a.bits_stride;
      uint32_t bw[kBitWords];
#pragma unroll
      for (int u = 0; u < kBitWords; ++u) {
        const int wi = tid + u * NT;
        bw[u] = wi < words ? __hip_atomic_load(gb + wi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
      }
      int er = -1;
      uint32_t ej = 0;
      uint64_t ent = 0;
      if ((uint32_t)tid < E) {
        int r = 0;
#pragma unroll
        for (int st = 16; st > 0; st >>= 1)
          if (r + st < W && ab[64 + r + st] <= (uint32_t)tid) r += st;
        er = r;
        ej = (uint32_t)tid - ab[64 + r];
        ent = __hip_atomic_load(a.win_keys + grp * a.score_stride + (size_t)r * a.blocks_per_wg + ej,
                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
#pragma unroll
      for (int u = 0; u < kBitWords; ++u) bits[tid + u * NT] = bw[u];
      lds_sync();
      if (er >= 0) {
        const uint32_t id = (uint32_t)ent;
        if (ej < ab[er] || cnt == k)  // above the bucket, or the whole bucket is kept
          atomicOr(&bits[id >> 5], 1u << (id & 31u));
        else
          cv[ab[96 + er] + (ej - ab[er])] = (ent & 0xFFFFFFFF00000000ull) | (uint32_t)~id;
      }
      lds_sync();
      if (cnt != k) {
        rank_bucket();
        lds_sync();
        thr = misc[0];
      }
      take = bits_of_thread();
    }
  }
  if (!done) {
    if (lazy) load_keys<NJ>(key, rs, id0);
    // A bucket too large to rank is narrowed by the next 12 bits (rare once
    // the window hint follows the threshold).
    while (known < 32 && cnt != k && cnt > kMaxCand) {
      const int width = min(12, 32 - known), shift = 32 - known - width;
      const uint32_t dmask = (1u << width) - 1u;
      for (int i = tid; i < (1 << width); i += NT) s_hist[i] = 0;
      lds_sync();
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        if (j < nv && (key[j] & pmask) == prefix) atomicAdd(&s_hist[(key[j] >> shift) & dmask], 1u);
      lds_sync();
      find_digit<NT>(s_hist, 1 << width, k, lds32, misc);
      prefix |= misc[0] << shift;
      pmask |= dmask << shift;
      known += width;
      k = misc[1];
      cnt = misc[2];
    }

    // One pass over the keys: bit j of `take` marks key j above the bucket of
    // the n-th largest key, bit j of `inb` key j inside it.
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const uint32_t km = key[j] & pmask;
      take |= km > prefix ? Mask(1) << j : Mask(0);
      inb |= km == prefix ? Mask(1) << j : Mask(0);
    }
    take &= valid;
    inb &= valid;
    thr = prefix;
    mode = cnt == k ? 0 : (cnt <= kMaxCand ? 1 : 2);
    if (mode == 0) {
      take |= inb;
    } else if (mode == 1) {
      for (int i = tid; i < 1024; i += NT) bits[i] = 0;
      const uint32_t mine = __builtin_popcountll(inb);
      const uint32_t incl = wave_incl_scan(mine);
      const uint32_t wave_tot = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
      uint32_t base = 0;
      if ((tid & 63) == 63 && wave_tot != 0) base = atomicAdd(&misc[4], wave_tot);
      uint32_t at = (uint32_t)__builtin_amdgcn_readlane((int)base, 63) + incl - mine;
      if constexpr (NJ <= 32) {
        // Only the key slots j that hold a bucket key in some lane of the
        // wave are visited (a wave-uniform loop, typically a few passes
        // instead of NJ; j indexes the key registers).
        for (Mask wm = (Mask)wave_or((uint32_t)inb); wm != 0; wm &= wm - Mask(1)) {
          const int j = __builtin_ctzll(wm);
          if ((inb >> j) & Mask(1)) {
            cv[at] = ((uint64_t)key[j] << 32) | (uint32_t)~(uint32_t)(id0 + j);
            ++at;
          }
        }
      } else {
        // 64 keys per thread: constant indices keep the keys in registers.
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          if ((inb >> j) & Mask(1)) {
            cv[at] = ((uint64_t)key[j] << 32) | (uint32_t)~(uint32_t)(id0 + j);
            ++at;
          }
        }
      }
      lds_sync();
      rank_bucket();
      lds_sync();
      thr = misc[0];
      take |= bits_of_thread();
    }
  }
  // The next call's window: the top 9 bits of this threshold. The stores
  // here go out before the compaction so their latency overlaps it.
  if (tid == 0) {
    if (a.k_new != nullptr && ready == nullptr) finish_append(a, bb, L, seq_ticket);
    a.window[grp] = 0x80000000u | (thr >> 23);
  }

  // Output positions: one scan of the packed per-thread counts (kept keys in
  // the high half; in mode 2 also the bucket keys, which are kept in id
  // order up to k, in the low half; totals <= M < 2^16).
  const uint32_t nb = mode == 2 ? (uint32_t)__builtin_popcountll(inb) : 0u;
  uint32_t tot;
  const uint32_t before = block_exclusive_scan<NT>(((uint32_t)__builtin_popcountll(take) << 16) | nb, lds32, &tot);
  uint32_t pos = before >> 16;
  if (mode == 2) {
    // Bucket keys kept by earlier threads, then by this one. Written so that
    // no subtraction can wrap: the form `k > e ? k - e : 0` was compiled into
    // an unguarded k - e.
    const uint32_t eb = min(before & 0xFFFFu, k);
    uint32_t keep = min(k - eb, nb);
    Mask m = inb;
    for (; keep > 0; --keep) {
      take |= m & (Mask(0) - m);  // lowest remaining bucket id
      m &= m - Mask(1);
    }
    pos += eb;
  }
  // Kept ids in ascending order. Rows shorter than the workgroup's score
  // staging area (free by now) are assembled there and written out coalesced.
  const bool staged = a.n_cap < kMaxBlocksPerWg;
  for (Mask m = take; m != 0; m &= m - Mask(1)) {
    const int32_t id = id0 + __builtin_ctzll(m);
    if (pos < (uint32_t)a.n_cap) {  // never past the row, whatever the scores
      if (staged) s_out[pos] = id;
      else __hip_atomic_store(out + pos, id, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    ++pos;
  }
  if (staged) {
    lds_sync();
    for (int i = tid; i < a.n_cap; i += NT)
      __hip_atomic_store(out + i, i < n ? s_out[i] : -1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  } else {
    for (int i = n + tid; i < a.n_cap; i += NT)
      __hip_atomic_store(out + i, -1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  publish();
}

// What the scoring workgroups of a group read of its sequence: the length
// (with the appended row), its blocks M, the first forced local block, and
// the window hint. The group's tail takes the same values.
// Blocks per scoring tile: two wave-wide loads of kmin and two of kmax (4 KB
// per tile and wave). With 16 waves per CU streaming at once, smaller tiles
// keep fewer bytes in flight, which the memory system serves faster:
// selection 29.7 -> 28.8 us at 64K and 24.2 -> 24.0 us at 256K against
// 16-block tiles, with one tile in flight beyond the one scored (4-block
// tiles and deeper prefetch measured slower).
constexpr int kTileRows = 8;
constexpr int kTileLoads = kTileRows / 4;

struct RangeInfo {
  SeqLen sl;
  int M, forced_from;
  uint32_t win;
};

// Pooled query (Fig. 3) and Quest scores (Eq. 4) of the blocks of range
// `range` of group (bb, hk), one of the group's `nranges`, by a workgroup of
// NW waves; returns what it read of the sequence. Lane (r, c) handles dims
// [8c, 8c + 8) of kTileRows-block tiles, so each wave-wide load is four whole
// 256-byte summary rows, and the next PF tiles' loads are in flight while one
// is scored. Per dimension the larger of q*kmax and q*kmin is the product
// with kmax when q >= 0 and with kmin otherwise (exactly, as fp32 rounding is
// monotone), so the summary row is selected before the multiply. Scores are
// staged in LDS (s_score) and written out coalesced as order-preserving keys
// with write-through stores; with `a.fused` the workgroup also counts its
// keys' 8 high bits (and 8 more inside the window hint) into its own
// histogram slot, and with kLists writes the in-window path's above-window
// bits and in-window list, all with agent-scope stores. Returns with those
// stores issued (the caller waits for them before its ticket).
template <int NW, int PF, bool kOpaque, bool kLists>
__device__ __forceinline__ RangeInfo score_range(const SelectArgs& a, int bb, int hk, int range, int nranges,
                                                 uint32_t* s_hist, float* s_score) {
  const int tid = tid_of<kOpaque>(), lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const size_t grp = (size_t)bb * a.c.kv_heads + hk;
  const int r = lane >> 4, c = lane & 15, col = c * 8;
  const int b0 = range * a.blocks_per_wg;

  // The first tiles are requested before the sequence length, the query and
  // the new key have arrived, bounded by the range's end at full length
  // (b1_cap, rows of the summary array in bounds); rows past the true end
  // are never scored. Rows past an end read the last row before it.
  const int b1_cap = min(b0 + a.blocks_per_wg, min(a.max_blocks_seq, a.c.max_blocks));
  const uint16_t* kmin = a.c.kmin + grp * a.c.max_blocks * kHeadDim + col;
  const uint16_t* kmax = a.c.kmax + grp * a.c.max_blocks * kHeadDim + col;
  auto load_tile = [&](int t, int end, U4 (&lo4)[kTileLoads], U4 (&hi4)[kTileLoads]) {
#pragma unroll
    for (int u = 0; u < kTileLoads; ++u) {
      const int m = min(b0 + kTileRows * t + 4 * u + r, end - 1);
      lo4[u] = ld16_stream(kmin + (size_t)m * kHeadDim);
      hi4[u] = ld16_stream(kmax + (size_t)m * kHeadDim);
    }
  };
  constexpr int P = PF + 1;
  U4 lo4[P][kTileLoads], hi4[P][kTileLoads];
#pragma unroll
  for (int k = 0; k < P; ++k)
    if (b0 + kTileRows * (wave + k * NW) < b1_cap) load_tile(wave + k * NW, b1_cap, lo4[k], hi4[k]);

  RangeInfo info;
  info.sl = seq_len_of(a, bb);
  const SeqLen sl = info.sl;
  // Lengths beyond max_seq_len are clamped so every access stays in bounds.
  const int M = max(0, min(min((sl.L + a.c.block_size - 1) / a.c.block_size, a.max_blocks_seq), a.c.max_blocks));
  const int forced_from = M - a.n_local;
  const int b1 = min(b0 + a.blocks_per_wg, M);
  // Window hint left by the previous call on this workspace (any value is
  // valid: it only chooses which key bits get a second histogram).
  const uint32_t win = a.fused ? a.window[grp] : 0u;
  info.M = M;
  info.forced_from = forced_from;
  info.win = win;
  const bool win_on = (win >> 31) != 0;
  const uint32_t w9 = win & 0x1FFu;

  // Fused append (Alg. 1): the first workgroup of the group writes the new
  // K and V rows; the workgroup owning block pos / b folds the new key into
  // that block's summary (or starts it) before scoring it, and stores it.
  const int m_new = sl.pos >= 0 ? sl.pos / a.c.block_size : -1;
  const bool opening = sl.pos >= 0 && sl.pos % a.c.block_size == 0;
  const bool row_writer = sl.pos >= 0 && range == 0 && tid < 32;
  const int64_t new_row = row_writer ? kv_row(a.c, bb, hk, sl.pos) : -1;
  U4 knew = U4{0, 0, 0, 0}, vnew = U4{0, 0, 0, 0};
  if (sl.pos >= 0) {
    knew = ld16(a.k_new + grp * kHeadDim + col);
    if (row_writer && tid >= 16) vnew = ld16(a.v_new + grp * kHeadDim + col);
  }
  // The appended block's updated summary row, held by the lanes that score
  // it and stored after the loop (a store inside it would hold up that
  // wave's next tile: the memory counter drains in issue order).
  U4 new_lo = U4{0, 0, 0, 0}, new_hi = U4{0, 0, 0, 0};
  bool owns_row = false;
  {
    U4 qv[kMaxGroup];
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h)
      qv[h] = h < a.group ? ld16(a.q + ((size_t)bb * a.q_heads + (size_t)hk * a.group + h) * kHeadDim + col)
                          : U4{0, 0, 0, 0};
    if (a.fused) {
      for (int i = tid; i < 2 * kSlotWords; i += NW * 64) s_hist[i] = 0;
      lds_sync();
    }
    const int ntiles = b1 > b0 ? (b1 - b0 + kTileRows - 1) / kTileRows : 0;
    int t = wave;
    float qb[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) qb[j] = 0.f;
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
      const uint32_t w[4] = {qv[h].x, qv[h].y, qv[h].z, qv[h].w};
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
    // Tile t of this wave's tiles t = wave, wave + NW, ...: scored from its
    // buffers; PF more tiles are in flight meanwhile (a ring of PF + 1).
    auto score_tile = [&](int t, U4 (&lo4)[kTileLoads], U4 (&hi4)[kTileLoads]) {
#pragma unroll
      for (int u = 0; u < kTileLoads; ++u) {
        const int m = b0 + kTileRows * t + 4 * u + r;
        if (m == m_new && m < b1) {
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
        if (c == 0 && m < b1) {
          s_score[m - b0] = s;
          if (a.fused) {
            const uint32_t key = block_key(m, forced_from, s);
            atomicAdd(&s_hist[key >> 24], 1u);
            if (win_on && (key >> 23) == w9) atomicAdd(&s_hist[256 + ((key >> 15) & 0xFFu)], 1u);
          }
        }
      }
    };
    while (t < ntiles) {
#pragma unroll
      for (int k = 0; k < P; ++k) {
        if (t < ntiles) {
          score_tile(t, lo4[k], hi4[k]);
          __builtin_amdgcn_sched_barrier(0);
          if (t + P * NW < ntiles) load_tile(t + P * NW, b1, lo4[k], hi4[k]);
          __builtin_amdgcn_sched_barrier(0);
          t += NW;
        }
      }
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
  // Coalesced write-out of this range: the blocks' order-preserving keys to
  // the workspace rows (16-byte aligned, write-through at agent scope), so
  // the top-n reads keys and converts nothing, and, if asked, the scores to
  // scores_out.
  const int nb = max(b1 - b0, 0);
  if (nb > 0) {
    const __amdgpu_buffer_rsrc_t rs = buf_rsrc(a.keys + grp * a.score_stride + b0, (uint32_t)nb * 4);
    for (int i = 4 * tid; i < nb; i += 4 * NW * 64) {
      const f4_t v = *reinterpret_cast<const f4_t*>(&s_score[i]);
      const int m = b0 + i;
      const U4 kv = U4{block_key(m, forced_from, v.x), block_key(m + 1, forced_from, v.y),
                       block_key(m + 2, forced_from, v.z), block_key(m + 3, forced_from, v.w)};
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(__attribute__((ext_vector_type(4))) unsigned, kv),
                                             rs, i * 4, 0, kSc1);
    }
    if (a.scores_out != nullptr) {
      float* so = a.scores_out + grp * a.max_blocks_seq + b0;
      for (int i = tid; i < nb; i += NW * 64) so[i] = s_score[i];
    }
  }
  if (!a.fused) return info;
  if (kLists && win_on && nb > 0 && a.blocks_per_wg <= kListRange) {
    // For the top-n's in-window path: a bit per block whose key lies above
    // the window (one ballot per 64 blocks; the range starts on a word), and
    // the range's in-window keys as (key, id) pairs grouped by digit (bits
    // 22..15), larger digits first, at the range's first block in the list
    // row. Wave 0 turns the window counts into each digit's first position.
    uint32_t* woff = s_hist + 2 * kSlotWords;
    if (wave == 0) {
      uint32_t cw[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) cw[j] = s_hist[kSlotWords + 255 - 4 * lane - j];
      const uint32_t tot = cw[0] + cw[1] + cw[2] + cw[3];
      uint32_t run = wave_incl_scan(tot) - tot;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        woff[255 - 4 * lane - j] = run;
        run += cw[j];
      }
    }
    lds_sync();
    uint64_t* lst = a.win_keys + grp * a.score_stride + b0;
    uint32_t* bits = a.above_bits + grp * a.bits_stride + b0 / 32;
    const int words = (nb + 31) / 32;
    for (int i0 = wave * 64; i0 < nb; i0 += NW * 64) {
      const int i = i0 + lane;
      bool above = false;
      if (i < nb) {
        const uint32_t key = block_key(b0 + i, forced_from, s_score[i]);
        above = (key >> 23) > w9;
        if ((key >> 23) == w9) {
          const uint32_t at = atomicAdd(&woff[(key >> 15) & 0xFFu], 1u);
          __hip_atomic_store(lst + at, ((uint64_t)key << 32) | (uint32_t)(b0 + i), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
        }
      }
      const unsigned long long bal = __ballot(above);
      if (lane == 0) {
        if (i0 / 32 < words)
          __hip_atomic_store(bits + i0 / 32, (uint32_t)bal, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (i0 / 32 + 1 < words)
          __hip_atomic_store(bits + i0 / 32 + 1, (uint32_t)(bal >> 32), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  // This workgroup's digit counts go to its own slot: no shared counters.
  // Counts fit in 16 bits (at most kMaxBlocksPerWg per workgroup): two per word.
  uint32_t* slot = a.hist + (grp * nranges + range) * kSlotWords;
  for (int i = tid; i < kSlotWords; i += NW * 64)
    __hip_atomic_store(slot + i, s_hist[2 * i] | (s_hist[2 * i + 1] << 16), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  return info;
}

}  // namespace
}  // namespace resa
