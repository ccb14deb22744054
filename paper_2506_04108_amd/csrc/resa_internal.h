// Internal interface between the C-ABI layer (api.cpp) and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "resa.h"

namespace resa {

// Eq. 5 (Sec. 2.1) in integer arithmetic; `keep_ppm` = round((1 - s) * 1e6).
// n = min(M, max(min_blocks, n_local, ceil(M * keep_ppm / 1e6))); 0 if M <= 0.
__host__ __device__ inline int32_t count_selected(int32_t M, int32_t keep_ppm,
                                                  int32_t min_blocks, int32_t n_local) {
  if (M <= 0) return 0;
  int64_t n = ((int64_t)M * keep_ppm + 999999) / 1000000;
  if (n < min_blocks) n = min_blocks;
  if (n < n_local) n = n_local;
  if (n > M) n = M;
  return (int32_t)n;
}

// Plain-value view of a resa_kv_cache_t for kernel arguments.
struct CacheArgs {
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* kmin;
  uint16_t* kmax;
  int32_t batch, kv_heads, capacity, block_size, max_blocks;  // max_blocks = capacity / b
  int32_t log2_block;        // log2(block_size)
  const int32_t* table;      // paged layout: block table [batch, max_blocks], else nullptr
  int32_t num_pages;
};

// Row (of head_dim elements) of k / v that holds token t of group (bb, hk),
// or -1 when the block table sends its block outside the page pool.
__device__ __forceinline__ int64_t kv_row(const CacheArgs& c, int bb, int hk, int t) {
  if (c.table == nullptr) return ((int64_t)bb * c.kv_heads + hk) * c.capacity + t;
  const int m = t >> c.log2_block;
  const int page = c.table[(size_t)bb * c.max_blocks + m];
  if ((unsigned)page >= (unsigned)c.num_pages) return -1;
  return ((int64_t)page * c.kv_heads + hk) * c.block_size + (t - (m << c.log2_block));
}

struct SelectArgs {
  CacheArgs c;
  const uint16_t* q;
  int32_t q_heads, group;      // group = q_heads / kv_heads
  const int32_t* seq_lens;
  int32_t max_blocks_seq;      // ceil(max_seq_len / b): row stride of the score array
  int32_t keep_ppm, min_blocks, n_local;
  uint32_t* keys;              // workspace [B, Hkv, score_stride]: order-preserving keys, 16-byte aligned rows
  int32_t score_stride;        // max_blocks_seq rounded up to a multiple of 4
  float* scores_out;           // optional [B, Hkv, max_blocks_seq]
  int32_t* block_idx;          // [B, Hkv, n_cap]
  int32_t* num_sel;            // [B, Hkv]
  int32_t n_cap;
  uint32_t* hist;              // [B, Hkv, workgroups, 256] per-workgroup key-digit counts
  uint32_t* counters;          // [B, Hkv], zero between calls
  int32_t blocks_per_wg;
  int32_t fused;               // top-n in the scoring kernel's last workgroup
  // Append fused in front of the selection (null k_new: plain selection).
  const uint16_t* k_new;       // [B, Hkv, D] key of the new token
  const uint16_t* v_new;       // [B, Hkv, D] value of the new token
  int32_t* lens_out;           // seq_lens, written once every group of the sequence is done
  uint32_t* seq_counters;      // [B], zero between calls
  uint32_t* window;            // [B, Hkv] digit-window hint kept across calls (any value is valid)
  uint32_t* stats;             // [B, Hkv] calls whose top-n finished on the in-window path (diagnostic)
  // Written by the scoring when the hint is set (fused top-n), for the
  // top-n's in-window path: per block, a bit for a key above the window,
  // and each range's in-window keys grouped by digit, descending.
  uint32_t* above_bits;        // [B, Hkv, bits_stride]
  int32_t bits_stride;         // words per group: ceil(max_blocks_seq / 32) rounded to 4
  uint64_t* win_keys;          // [B, Hkv, score_stride]: range r's list at its first block
};

struct DecodeArgs {
  CacheArgs c;
  const uint16_t* q;
  int32_t q_heads, group;
  const int32_t* seq_lens;
  const int32_t* block_idx;
  const int32_t* num_sel;
  int32_t n_cap, num_splits;
  float scale_log2;            // sm_scale * log2(e)
  float* out;                  // [B, Hq, D]
  float* lse;                  // [B, Hq] or null
  float* part_o;               // [B, Hkv, S, G, D]
  float* part_lse;             // [B, Hkv, S, G]
  uint32_t* counters;          // [B, Hkv] split tickets, zero between calls
  uint32_t* epochs;            // [B, Hkv] merged calls so far (kept from call to call)
  uint64_t* flags;             // [B, Hkv, S] split partial published: (epoch + 1) << 32 | S
  const uint16_t* k_new;       // fused step: [B, Hkv, D] token appended in the same launch
  const uint16_t* v_new;
};

// Fused decode step (append + selection + decode in one persistent launch).
struct StepArgs {
  SelectArgs s;
  DecodeArgs d;
  uint32_t* queue;             // [4]: score claims, decode claims, exits (zero between calls), error flag
  uint32_t* ready;             // [B, Hkv]: selection of the group published (zero between calls)
  int32_t nranges;             // score ranges per group (blocks_per_wg each)
  int32_t score_items, dec_items;
  uint32_t max_spins;          // bound of a decode split's wait for its group's selection
};

struct RectifyArgs {
  CacheArgs c;
  const uint16_t* q_f;         // [B, Hq, f, D]
  const uint16_t* k_f;         // [B, Hkv, f, D]
  const uint16_t* v_f;
  int32_t q_heads, group, f;
  const int32_t* seq_lens;
  int32_t max_seq_len;
  int32_t chunk;               // keys per split
  int32_t num_splits;          // ceil(max_seq_len / chunk)
  float scale_log2;
  float* out;                  // [B, Hq, f, D]
  float* lse;                  // [B, Hq, f] or null
  float* part_o;               // [B, Hkv, S, G*f, D]
  float* part_lse;             // [B, Hkv, S, G*f]
  int32_t refresh;
  const int32_t* seq_mask;     // [B]: sequences with 0 are left untouched (null: every sequence)
};

// Launchers: enqueue on `stream`; return the hipError_t of the launch.
hipError_t launch_summarize(const CacheArgs& c, const int32_t* seq_lens, int32_t blk_begin,
                            int32_t blk_end, hipStream_t stream);
hipError_t launch_summarize_tail(const CacheArgs& c, const int32_t* seq_lens, int32_t f,
                                 const int32_t* seq_mask, hipStream_t stream);
hipError_t launch_append(const CacheArgs& c, const uint16_t* k_new, const uint16_t* v_new,
                         int32_t* seq_lens, hipStream_t stream);
hipError_t launch_select(const SelectArgs& a, hipStream_t stream);
hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream);
hipError_t launch_step(const StepArgs& a, hipStream_t stream);
hipError_t launch_rectify(const RectifyArgs& a, hipStream_t stream);
hipError_t launch_clear(void* p, size_t bytes, hipStream_t stream);
hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, uint32_t match,
                              int32_t workgroups, hipStream_t stream);

// Split-count and chunk heuristics (host).
int32_t select_fused_max_blocks();
int32_t select_blocks_per_wg(int32_t batch, int32_t kv_heads, int32_t max_blocks_seq);
int32_t select_hist_words(int32_t batch, int32_t kv_heads, int32_t max_blocks_seq);
int32_t decode_auto_splits(int32_t batch, int32_t kv_heads, int32_t n_cap, int32_t block_size);
int32_t step_blocks_per_range(int32_t batch, int32_t kv_heads, int32_t max_blocks_seq);
int32_t step_hist_words(int32_t batch, int32_t kv_heads, int32_t max_blocks_seq);
int32_t step_max_blocks();
int32_t rectify_num_qblocks(int32_t group, int32_t f);
int32_t rectify_chunk(int32_t batch, int32_t kv_heads, int32_t nqblk, int32_t max_seq_len);
// An upper bound on the key splits of any call with lengths up to
// max_seq_len, non-decreasing in max_seq_len (workspace sizing).
int32_t rectify_max_splits(int32_t batch, int32_t kv_heads, int32_t nqblk, int32_t max_seq_len);

}  // namespace resa
