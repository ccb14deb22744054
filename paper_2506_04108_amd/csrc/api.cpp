// C ABI of the ReSA decode library: argument validation (before any HIP call),
// workspace layout, launch configuration and error reporting.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <mutex>
#include <string>

#include "resa_internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return RESA_OK;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

size_t round256(size_t x) { return (x + 255) & ~size_t(255); }

#define RESA_CHECK_PTR(p, align)                                                        \
  do {                                                                                  \
    if ((p) == nullptr) return fail(RESA_ERR_INVALID_ARG, "%s is NULL", #p);            \
    if (!aligned((p), (align)))                                                         \
      return fail(RESA_ERR_INVALID_ARG, "%s is not %d-byte aligned", #p, (int)(align)); \
  } while (0)

int check_cache(const resa_kv_cache_t* c) {
  if (c == nullptr) return fail(RESA_ERR_INVALID_ARG, "cache descriptor is NULL");
  RESA_CHECK_PTR(c->k, 16);
  RESA_CHECK_PTR(c->v, 16);
  RESA_CHECK_PTR(c->kmin, 16);
  RESA_CHECK_PTR(c->kmax, 16);
  if (c->head_dim != RESA_HEAD_DIM)
    return fail(RESA_ERR_UNSUPPORTED, "head_dim %d unsupported (only 128)", c->head_dim);
  if (c->block_size != 16 && c->block_size != 32 && c->block_size != 64)
    return fail(RESA_ERR_UNSUPPORTED, "block_size %d unsupported (16, 32 or 64)", c->block_size);
  if (c->batch < 1 || c->num_kv_heads < 1)
    return fail(RESA_ERR_INVALID_ARG, "batch (%d) and num_kv_heads (%d) must be >= 1", c->batch,
                c->num_kv_heads);
  if ((int64_t)c->batch * c->num_kv_heads > 65535)
    return fail(RESA_ERR_UNSUPPORTED, "batch * num_kv_heads = %lld exceeds 65535",
                (long long)c->batch * c->num_kv_heads);
  if (c->capacity < c->block_size || c->capacity % c->block_size != 0)
    return fail(RESA_ERR_INVALID_ARG, "capacity %d must be a positive multiple of block_size %d",
                c->capacity, c->block_size);
  if (c->block_table != nullptr) {
    if (!aligned(c->block_table, 4))
      return fail(RESA_ERR_INVALID_ARG, "block_table is not 4-byte aligned");
    if (c->num_pages < 1)
      return fail(RESA_ERR_INVALID_ARG, "num_pages %d must be >= 1 with a block table",
                  c->num_pages);
    if ((int64_t)c->num_pages * c->num_kv_heads * c->block_size >= ((int64_t)1 << 31))
      return fail(RESA_ERR_UNSUPPORTED, "page pool of %d pages x %d heads x %d rows exceeds 2^31 rows",
                  c->num_pages, c->num_kv_heads, c->block_size);
  }
  return RESA_OK;
}

resa::CacheArgs cache_args(const resa_kv_cache_t* c) {
  resa::CacheArgs a;
  a.k = static_cast<const uint16_t*>(c->k);
  a.v = static_cast<const uint16_t*>(c->v);
  a.kmin = static_cast<uint16_t*>(c->kmin);
  a.kmax = static_cast<uint16_t*>(c->kmax);
  a.batch = c->batch;
  a.kv_heads = c->num_kv_heads;
  a.capacity = c->capacity;
  a.block_size = c->block_size;
  a.max_blocks = c->capacity / c->block_size;
  a.log2_block = c->block_size == 16 ? 4 : c->block_size == 32 ? 5 : 6;
  a.table = c->block_table;
  a.num_pages = c->block_table != nullptr ? c->num_pages : 0;
  return a;
}

int check_heads(const resa_kv_cache_t* c, int32_t num_q_heads, int32_t* group) {
  if (num_q_heads < 1 || num_q_heads % c->num_kv_heads != 0)
    return fail(RESA_ERR_INVALID_ARG, "num_q_heads %d is not a positive multiple of num_kv_heads %d",
                num_q_heads, c->num_kv_heads);
  const int32_t g = num_q_heads / c->num_kv_heads;
  if (g > RESA_MAX_GROUP)
    return fail(RESA_ERR_UNSUPPORTED, "group size %d exceeds %d", g, RESA_MAX_GROUP);
  *group = g;
  return RESA_OK;
}

bool parse_sparsity(double s, int32_t* keep_ppm) {
  if (!(s >= 0.0 && s <= 1.0)) return false;
  const long long sp = llround(s * 1e6);
  *keep_ppm = (int32_t)(1000000 - sp);
  return true;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(RESA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

struct SelectLayout {
  size_t counters, seq_counters, window, stats, hist, keys, above_bits, win_keys, total;
};

size_t bits_stride(size_t mseq) { return ((mseq + 31) / 32 + 3) & ~size_t(3); }

// Workspace of resa_select_blocks / resa_append_select: one ticket per group
// and one per sequence (zero between calls), one digit-window hint per group
// (kept from call to call; any value is valid), one diagnostic counter per
// group (calls whose top-n finished on the in-window path), per-workgroup
// key-digit counts, the blocks' keys (rows padded to 4 words), and for the
// top-n's in-window path a bit per block and a (key, id) list per group.
SelectLayout select_layout_words(int32_t batch, int32_t kv_heads, size_t mseq, size_t hist_words) {
  SelectLayout l;
  const size_t groups = (size_t)batch * kv_heads;
  l.counters = 0;
  l.seq_counters = groups * 4;
  l.window = (groups + (size_t)batch) * 4;
  l.stats = (2 * groups + (size_t)batch) * 4;
  l.hist = round256((3 * groups + (size_t)batch) * 4);
  l.keys = l.hist + round256(groups * hist_words * 4);
  l.above_bits = l.keys + round256(groups * ((mseq + 3) & ~size_t(3)) * sizeof(uint32_t));
  l.win_keys = l.above_bits + round256(groups * bits_stride(mseq) * 4);
  l.total = l.win_keys + groups * ((mseq + 3) & ~size_t(3)) * sizeof(uint64_t);
  return l;
}

SelectLayout select_layout(int32_t batch, int32_t kv_heads, int32_t max_seq_len, int32_t block_size) {
  const size_t mseq = ((size_t)max_seq_len + block_size - 1) / block_size;
  return select_layout_words(batch, kv_heads, mseq,
                             (size_t)resa::select_hist_words(batch, kv_heads, (int32_t)mseq));
}

// Workspace of resa_sparse_decode: per group a ticket counter (zero between
// calls) and a count of the calls merged so far, one ready flag per split
// (tagged with that count and the split count, so flags of earlier calls
// never match and need no reset), then the split partials.
struct DecodeLayout {
  size_t counters, epochs, flags, lse, o, total;
};

DecodeLayout decode_layout(int32_t batch, int32_t kv_heads, int32_t group, int32_t splits) {
  DecodeLayout d;
  const size_t groups = (size_t)batch * kv_heads;
  d.counters = 0;
  d.epochs = groups * 4;
  d.flags = (groups * 8 + 7) & ~size_t(7);
  d.lse = round256(d.flags + groups * splits * 8);
  d.o = d.lse + round256(groups * splits * group * 4);
  d.total = d.o + groups * splits * group * RESA_HEAD_DIM * 4;
  return d;
}

// Workspace of resa_decode_step: claim counters and per-group ready flags,
// then a selection workspace (score ranges of the step) and a decode
// workspace.
struct StepLayout {
  size_t queue, ready, sel, dec, total;
  SelectLayout s;
  DecodeLayout d;
};

StepLayout step_layout(int32_t batch, int32_t kv_heads, int32_t group, int32_t sel_len,
                       int32_t block_size, int32_t splits) {
  StepLayout l;
  const size_t groups = (size_t)batch * kv_heads;
  const size_t mseq = ((size_t)sel_len + block_size - 1) / block_size;
  l.queue = 0;
  l.ready = 256;
  l.sel = l.ready + round256(groups * 4);
  l.s = select_layout_words(batch, kv_heads, mseq,
                            (size_t)resa::step_hist_words(batch, kv_heads, (int32_t)mseq));
  l.dec = l.sel + round256(l.s.total);
  l.d = decode_layout(batch, kv_heads, group, splits);
  l.total = l.dec + l.d.total;
  return l;
}

struct RectifyLayout {
  int32_t nq, chunk, splits;
  size_t lse, o, total;
};

RectifyLayout rectify_layout(int32_t batch, int32_t kv_heads, int32_t group, int32_t f,
                             int32_t max_seq_len) {
  RectifyLayout r;
  r.nq = resa::rectify_num_qblocks(group, f);
  r.chunk = resa::rectify_chunk(batch, kv_heads, r.nq, max_seq_len);
  r.splits = (max_seq_len + r.chunk - 1) / r.chunk;
  if (r.splits < 1) r.splits = 1;
  const size_t groups = (size_t)batch * kv_heads;
  const size_t rows = (size_t)group * f;
  r.lse = 0;
  r.o = round256(groups * r.splits * rows * 4);
  r.total = r.o + groups * r.splits * rows * RESA_HEAD_DIM * 4;
  if (r.splits == 1) r.total = 0;  // one split writes out / lse itself
  return r;
}

}  // namespace

extern "C" {

const char* resa_version(void) { return "0.1.0"; }

const char* resa_last_error(void) { return g_err.c_str(); }

int32_t resa_num_selected(int32_t num_blocks, double sparsity, int32_t min_blocks,
                          int32_t n_local) {
  int32_t keep = 0;
  if (num_blocks < 0 || min_blocks < 0 || n_local < 0 || !parse_sparsity(sparsity, &keep)) {
    fail(RESA_ERR_INVALID_ARG, "resa_num_selected: invalid argument");
    return -1;
  }
  return resa::count_selected(num_blocks, keep, min_blocks, n_local);
}

int resa_block_summarize(const resa_kv_cache_t* c, const int32_t* seq_lens, int32_t blk_begin,
                         int32_t blk_end, void* stream) {
  if (int e = check_cache(c)) return e;
  RESA_CHECK_PTR(seq_lens, 4);
  const int32_t mb = c->capacity / c->block_size;
  if (blk_begin < 0 || blk_begin > mb)
    return fail(RESA_ERR_INVALID_ARG, "blk_begin %d outside [0, %d]", blk_begin, mb);
  if (blk_end != -1 && (blk_end < blk_begin || blk_end > mb))
    return fail(RESA_ERR_INVALID_ARG, "blk_end %d outside [blk_begin, %d] (or -1)", blk_end, mb);
  hipError_t e = resa::launch_summarize(cache_args(c), seq_lens, blk_begin, blk_end,
                                        static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "resa_block_summarize launch");
  return ok();
}

int resa_append_kv(const resa_kv_cache_t* c, const void* k_new, const void* v_new,
                   int32_t* seq_lens, int32_t max_seq_len, void* stream) {
  if (int e = check_cache(c)) return e;
  RESA_CHECK_PTR(k_new, 16);
  RESA_CHECK_PTR(v_new, 16);
  RESA_CHECK_PTR(seq_lens, 4);
  if (max_seq_len < 0) return fail(RESA_ERR_INVALID_ARG, "max_seq_len %d < 0", max_seq_len);
  if (max_seq_len >= c->capacity)
    return fail(RESA_ERR_CAPACITY, "cache full: max_seq_len %d, capacity %d", max_seq_len,
                c->capacity);
  hipError_t e = resa::launch_append(cache_args(c), static_cast<const uint16_t*>(k_new),
                                     static_cast<const uint16_t*>(v_new), seq_lens,
                                     static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "resa_append_kv launch");
  return ok();
}

size_t resa_select_workspace_size(int32_t batch, int32_t num_kv_heads, int32_t max_seq_len,
                                  int32_t block_size) {
  if (batch < 1 || num_kv_heads < 1 || max_seq_len < 0 || block_size < 1) return 0;
  return select_layout(batch, num_kv_heads, max_seq_len, block_size).total;
}

namespace {

// Shared by resa_select_blocks and resa_append_select. `sel_len` is the host
// bound of the lengths the selection sees (one more than the stored bound
// when an append is fused in front).
int select_common(const resa_kv_cache_t* c, const void* q, int32_t num_q_heads,
                  const int32_t* seq_lens, int32_t sel_len, const resa_select_params_t* params,
                  int32_t* block_idx, int32_t* num_sel, int32_t n_cap, float* scores_out,
                  void* workspace, size_t workspace_bytes, const void* k_new, const void* v_new,
                  void* stream, const char* what) {
  int32_t group = 0;
  if (int e = check_heads(c, num_q_heads, &group)) return e;
  RESA_CHECK_PTR(q, 16);
  RESA_CHECK_PTR(seq_lens, 4);
  RESA_CHECK_PTR(block_idx, 4);
  RESA_CHECK_PTR(num_sel, 4);
  if (params == nullptr) return fail(RESA_ERR_INVALID_ARG, "params is NULL");
  int32_t keep = 0;
  if (!parse_sparsity(params->sparsity, &keep))
    return fail(RESA_ERR_INVALID_ARG, "sparsity %g outside [0, 1]", params->sparsity);
  if (params->min_blocks < 0 || params->n_local < 0)
    return fail(RESA_ERR_INVALID_ARG, "min_blocks (%d) and n_local (%d) must be >= 0",
                params->min_blocks, params->n_local);
  const int32_t mseq = (sel_len + c->block_size - 1) / c->block_size;
  const int32_t need = resa::count_selected(mseq, keep, params->min_blocks, params->n_local);
  if (n_cap < need)
    return fail(RESA_ERR_CAPACITY, "n_cap %d < %d blocks selectable at %d tokens", n_cap, need,
                sel_len);
  if (scores_out != nullptr) RESA_CHECK_PTR(scores_out, 4);
  const SelectLayout lay = select_layout(c->batch, c->num_kv_heads, sel_len, c->block_size);
  if (workspace == nullptr || workspace_bytes < lay.total)
    return fail(RESA_ERR_WORKSPACE, "select workspace needs %zu bytes, got %zu", lay.total,
                workspace == nullptr ? (size_t)0 : workspace_bytes);
  if (!aligned(workspace, 16)) return fail(RESA_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  char* ws = static_cast<char*>(workspace);
  resa::SelectArgs a;
  a.c = cache_args(c);
  a.q = static_cast<const uint16_t*>(q);
  a.q_heads = num_q_heads;
  a.group = group;
  a.seq_lens = seq_lens;
  a.max_blocks_seq = mseq;
  a.keep_ppm = keep;
  a.min_blocks = params->min_blocks;
  a.n_local = params->n_local;
  a.keys = reinterpret_cast<uint32_t*>(ws + lay.keys);
  a.score_stride = (mseq + 3) & ~3;
  a.scores_out = scores_out;
  a.block_idx = block_idx;
  a.num_sel = num_sel;
  a.n_cap = n_cap;
  a.counters = reinterpret_cast<uint32_t*>(ws + lay.counters);
  a.hist = reinterpret_cast<uint32_t*>(ws + lay.hist);
  a.blocks_per_wg = resa::select_blocks_per_wg(c->batch, c->num_kv_heads, mseq);
  a.fused = mseq <= resa::select_fused_max_blocks() ? 1 : 0;
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.lens_out = const_cast<int32_t*>(seq_lens);
  a.seq_counters = reinterpret_cast<uint32_t*>(ws + lay.seq_counters);
  a.window = reinterpret_cast<uint32_t*>(ws + lay.window);
  a.stats = reinterpret_cast<uint32_t*>(ws + lay.stats);
  a.above_bits = reinterpret_cast<uint32_t*>(ws + lay.above_bits);
  a.bits_stride = (int32_t)bits_stride(mseq);
  a.win_keys = reinterpret_cast<uint64_t*>(ws + lay.win_keys);
  hipError_t e = resa::launch_select(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, what);
  return ok();
}

}  // namespace

int resa_select_blocks(const resa_kv_cache_t* c, const void* q, int32_t num_q_heads,
                       const int32_t* seq_lens, int32_t max_seq_len,
                       const resa_select_params_t* params, int32_t* block_idx, int32_t* num_sel,
                       int32_t n_cap, float* scores_out, void* workspace, size_t workspace_bytes,
                       void* stream) {
  if (int e = check_cache(c)) return e;
  if (max_seq_len < 0 || max_seq_len > c->capacity)
    return fail(RESA_ERR_INVALID_ARG, "max_seq_len %d outside [0, capacity %d]", max_seq_len,
                c->capacity);
  return select_common(c, q, num_q_heads, seq_lens, max_seq_len, params, block_idx, num_sel, n_cap,
                       scores_out, workspace, workspace_bytes, nullptr, nullptr, stream,
                       "resa_select_blocks launch");
}

int resa_append_select(const resa_kv_cache_t* c, const void* k_new, const void* v_new,
                       const void* q, int32_t num_q_heads, int32_t* seq_lens, int32_t max_seq_len,
                       const resa_select_params_t* params, int32_t* block_idx, int32_t* num_sel,
                       int32_t n_cap, float* scores_out, void* workspace, size_t workspace_bytes,
                       void* stream) {
  if (int e = check_cache(c)) return e;
  RESA_CHECK_PTR(k_new, 16);
  RESA_CHECK_PTR(v_new, 16);
  if (max_seq_len < 0) return fail(RESA_ERR_INVALID_ARG, "max_seq_len %d < 0", max_seq_len);
  if (max_seq_len >= c->capacity)
    return fail(RESA_ERR_CAPACITY, "cache full: max_seq_len %d, capacity %d", max_seq_len,
                c->capacity);
  return select_common(c, q, num_q_heads, seq_lens, max_seq_len + 1, params, block_idx, num_sel,
                       n_cap, scores_out, workspace, workspace_bytes, k_new, v_new, stream,
                       "resa_append_select launch");
}

size_t resa_select_stats_offset(int32_t batch, int32_t num_kv_heads) {
  if (batch < 1 || num_kv_heads < 1) return 0;
  return select_layout_words(batch, num_kv_heads, 1, 1).stats;
}

size_t resa_step_stats_offset(int32_t batch, int32_t num_kv_heads) {
  if (batch < 1 || num_kv_heads < 1) return 0;
  return step_layout(batch, num_kv_heads, 1, 1, 16, 1).sel + select_layout_words(batch, num_kv_heads, 1, 1).stats;
}

int32_t resa_decode_num_splits(int32_t batch, int32_t num_kv_heads, int32_t n_cap,
                               int32_t block_size) {
  if (batch < 1 || num_kv_heads < 1 || n_cap < 0 || block_size < 16) return 1;
  return resa::decode_auto_splits(batch, num_kv_heads, n_cap, block_size);
}

size_t resa_decode_workspace_size(int32_t batch, int32_t num_kv_heads, int32_t num_q_heads,
                                  int32_t n_cap, int32_t block_size, int32_t num_splits) {
  if (batch < 1 || num_kv_heads < 1 || num_q_heads < num_kv_heads || num_splits < 0) return 0;
  const int32_t s = num_splits > 0 ? num_splits
                                   : resa_decode_num_splits(batch, num_kv_heads, n_cap, block_size);
  return decode_layout(batch, num_kv_heads, num_q_heads / num_kv_heads, s).total;
}

}  // extern "C"

namespace {

// Argument checks of resa_sparse_decode and resa_sparse_decode_noalloc
// (everything but the workspace); fills the split count and the workspace
// layout the call needs.
int decode_check(const resa_kv_cache_t* c, const void* q, int32_t num_q_heads,
                 const int32_t* seq_lens, const int32_t* block_idx, const int32_t* num_sel,
                 int32_t n_cap, int32_t num_splits, float sm_scale, const float* out,
                 const float* lse, int32_t* group, int32_t* splits, DecodeLayout* lay) {
  if (int e = check_cache(c)) return e;
  if (int e = check_heads(c, num_q_heads, group)) return e;
  RESA_CHECK_PTR(q, 16);
  RESA_CHECK_PTR(seq_lens, 4);
  RESA_CHECK_PTR(block_idx, 4);
  RESA_CHECK_PTR(num_sel, 4);
  RESA_CHECK_PTR(out, 4);
  if (lse != nullptr && !aligned(lse, 4)) return fail(RESA_ERR_INVALID_ARG, "lse is not 4-byte aligned");
  if (n_cap < 0) return fail(RESA_ERR_INVALID_ARG, "n_cap %d < 0", n_cap);
  if (num_splits < 0 || num_splits > 256)
    return fail(RESA_ERR_INVALID_ARG, "num_splits %d outside [0, 256]", num_splits);
  if (!std::isfinite(sm_scale)) return fail(RESA_ERR_INVALID_ARG, "sm_scale is not finite");
  *splits = num_splits > 0 ? num_splits
                           : resa::decode_auto_splits(c->batch, c->num_kv_heads, n_cap, c->block_size);
  *lay = decode_layout(c->batch, c->num_kv_heads, *group, *splits);
  return RESA_OK;
}

// Enqueues the decode on checked arguments with the workspace at `ws`.
// `clear_counters` first zero-fills the merge counters with a kernel (the
// allocation-free variant, whose scratch every call on the device shares).
int decode_launch(const resa_kv_cache_t* c, const void* q, int32_t num_q_heads,
                  const int32_t* seq_lens, const int32_t* block_idx, const int32_t* num_sel,
                  int32_t n_cap, int32_t group, int32_t splits, float sm_scale, float* out,
                  float* lse, char* ws, const DecodeLayout& lay, bool clear_counters, void* stream,
                  const char* what) {
  resa::DecodeArgs a;
  a.c = cache_args(c);
  a.q = static_cast<const uint16_t*>(q);
  a.q_heads = num_q_heads;
  a.group = group;
  a.seq_lens = seq_lens;
  a.block_idx = block_idx;
  a.num_sel = num_sel;
  a.n_cap = n_cap;
  a.num_splits = splits;
  a.scale_log2 = sm_scale * 1.4426950408889634f;
  a.out = out;
  a.lse = lse;
  a.counters = reinterpret_cast<uint32_t*>(ws + lay.counters);
  a.epochs = reinterpret_cast<uint32_t*>(ws + lay.epochs);
  a.flags = reinterpret_cast<uint64_t*>(ws + lay.flags);
  a.part_lse = reinterpret_cast<float*>(ws + lay.lse);
  a.part_o = reinterpret_cast<float*>(ws + lay.o);
  a.k_new = nullptr;
  a.v_new = nullptr;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (clear_counters) {
    hipError_t e = resa::launch_clear(ws + lay.counters, lay.lse - lay.counters, st);
    if (e != hipSuccess) return hip_fail(e, what);
  }
  hipError_t e = resa::launch_decode(a, st);
  if (e != hipSuccess) return hip_fail(e, what);
  return ok();
}

// Scratch of resa_sparse_decode_noalloc: one array per device, held for the
// life of the process. In host code `scratch` names a host-side stand-in,
// never the device memory: its device address comes from
// hipGetSymbolAddress, once per device, and only that address is passed on.
constexpr size_t kStaticScratchBytes = size_t(4) << 20;
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array (looked up on the
// first call on that device); nullptr with an error message on failure.
void* device_scratch(int* status) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    *status = hip_fail(e, "resa_sparse_decode_noalloc: hipGetDevice");
    return nullptr;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    *status = fail(RESA_ERR_UNSUPPORTED, "device %d beyond the %d the static scratch serves", dev,
                   kMaxDevices);
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || ptr == nullptr) {
      *status = hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol,
                         "resa_sparse_decode_noalloc: hipGetSymbolAddress(scratch)");
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

int resa_sparse_decode(const resa_kv_cache_t* c, const void* q, int32_t num_q_heads,
                       const int32_t* seq_lens, const int32_t* block_idx, const int32_t* num_sel,
                       int32_t n_cap, int32_t num_splits, float sm_scale, float* out, float* lse,
                       void* workspace, size_t workspace_bytes, void* stream) {
  int32_t group = 0, splits = 0;
  DecodeLayout lay;
  if (int e = decode_check(c, q, num_q_heads, seq_lens, block_idx, num_sel, n_cap, num_splits,
                           sm_scale, out, lse, &group, &splits, &lay))
    return e;
  if (workspace == nullptr || workspace_bytes < lay.total)
    return fail(RESA_ERR_WORKSPACE, "decode workspace needs %zu bytes, got %zu", lay.total,
                workspace == nullptr ? (size_t)0 : workspace_bytes);
  if (!aligned(workspace, 16)) return fail(RESA_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  return decode_launch(c, q, num_q_heads, seq_lens, block_idx, num_sel, n_cap, group, splits,
                       sm_scale, out, lse, static_cast<char*>(workspace), lay, false, stream,
                       "resa_sparse_decode launch");
}

size_t resa_sparse_decode_noalloc_max_bytes(void) { return kStaticScratchBytes; }

int resa_sparse_decode_noalloc(const resa_kv_cache_t* c, const void* q, int32_t num_q_heads,
                               const int32_t* seq_lens, const int32_t* block_idx,
                               const int32_t* num_sel, int32_t n_cap, int32_t num_splits,
                               float sm_scale, float* out, float* lse, void* stream) {
  int32_t group = 0, splits = 0;
  DecodeLayout lay;
  if (int e = decode_check(c, q, num_q_heads, seq_lens, block_idx, num_sel, n_cap, num_splits,
                           sm_scale, out, lse, &group, &splits, &lay))
    return e;
  if (lay.total > kStaticScratchBytes)
    return fail(RESA_ERR_WORKSPACE,
                "resa_sparse_decode_noalloc needs %zu bytes of scratch, above its static %zu "
                "(use resa_sparse_decode with a workspace, or fewer splits)",
                lay.total, kStaticScratchBytes);
  int status = RESA_OK;
  void* ptr = device_scratch(&status);
  if (ptr == nullptr) return status;
  return decode_launch(c, q, num_q_heads, seq_lens, block_idx, num_sel, n_cap, group, splits,
                       sm_scale, out, lse, static_cast<char*>(ptr), lay, true, stream,
                       "resa_sparse_decode_noalloc launch");
}

size_t resa_step_workspace_size(int32_t batch, int32_t num_kv_heads, int32_t num_q_heads,
                                int32_t max_seq_len, int32_t block_size, int32_t n_cap,
                                int32_t num_splits) {
  if (batch < 1 || num_kv_heads < 1 || num_q_heads < num_kv_heads || max_seq_len < 0 ||
      block_size < 16 || num_splits < 0)
    return 0;
  const int32_t s = num_splits > 0 ? num_splits
                                   : resa::decode_auto_splits(batch, num_kv_heads, n_cap, block_size);
  return step_layout(batch, num_kv_heads, num_q_heads / num_kv_heads, max_seq_len + 1, block_size, s)
      .total;
}

int resa_decode_step(const resa_kv_cache_t* c, const void* k_new, const void* v_new, const void* q,
                     int32_t num_q_heads, int32_t* seq_lens, int32_t max_seq_len,
                     const resa_select_params_t* params, int32_t* block_idx, int32_t* num_sel,
                     int32_t n_cap, int32_t num_splits, float sm_scale, float* out, float* lse,
                     void* workspace, size_t workspace_bytes, void* stream) {
  if (int e = check_cache(c)) return e;
  int32_t group = 0;
  if (int e = check_heads(c, num_q_heads, &group)) return e;
  RESA_CHECK_PTR(k_new, 16);
  RESA_CHECK_PTR(v_new, 16);
  RESA_CHECK_PTR(q, 16);
  RESA_CHECK_PTR(seq_lens, 4);
  RESA_CHECK_PTR(block_idx, 4);
  RESA_CHECK_PTR(num_sel, 4);
  RESA_CHECK_PTR(out, 4);
  if (lse != nullptr && !aligned(lse, 4)) return fail(RESA_ERR_INVALID_ARG, "lse is not 4-byte aligned");
  if (max_seq_len < 0) return fail(RESA_ERR_INVALID_ARG, "max_seq_len %d < 0", max_seq_len);
  if (max_seq_len >= c->capacity)
    return fail(RESA_ERR_CAPACITY, "cache full: max_seq_len %d, capacity %d", max_seq_len,
                c->capacity);
  if (params == nullptr) return fail(RESA_ERR_INVALID_ARG, "params is NULL");
  int32_t keep = 0;
  if (!parse_sparsity(params->sparsity, &keep))
    return fail(RESA_ERR_INVALID_ARG, "sparsity %g outside [0, 1]", params->sparsity);
  if (params->min_blocks < 0 || params->n_local < 0)
    return fail(RESA_ERR_INVALID_ARG, "min_blocks (%d) and n_local (%d) must be >= 0",
                params->min_blocks, params->n_local);
  if (num_splits < 0 || num_splits > 256)
    return fail(RESA_ERR_INVALID_ARG, "num_splits %d outside [0, 256]", num_splits);
  if (!std::isfinite(sm_scale)) return fail(RESA_ERR_INVALID_ARG, "sm_scale is not finite");
  const int32_t sel_len = max_seq_len + 1;
  const int32_t mseq = (sel_len + c->block_size - 1) / c->block_size;
  if (mseq > resa::step_max_blocks())
    return fail(RESA_ERR_UNSUPPORTED, "%d blocks per sequence exceed the fused step's %d", mseq,
                resa::step_max_blocks());
  const int32_t need = resa::count_selected(mseq, keep, params->min_blocks, params->n_local);
  if (n_cap < need)
    return fail(RESA_ERR_CAPACITY, "n_cap %d < %d blocks selectable at %d tokens", n_cap, need,
                sel_len);
  const int32_t splits = num_splits > 0 ? num_splits
                                        : resa::decode_auto_splits(c->batch, c->num_kv_heads, n_cap,
                                                                   c->block_size);
  const StepLayout lay = step_layout(c->batch, c->num_kv_heads, group, sel_len, c->block_size, splits);
  if (workspace == nullptr || workspace_bytes < lay.total)
    return fail(RESA_ERR_WORKSPACE, "step workspace needs %zu bytes, got %zu", lay.total,
                workspace == nullptr ? (size_t)0 : workspace_bytes);
  if (!aligned(workspace, 16)) return fail(RESA_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  char* ws = static_cast<char*>(workspace);
  char* wsel = ws + lay.sel;
  char* wdec = ws + lay.dec;
  const int64_t groups = (int64_t)c->batch * c->num_kv_heads;
  resa::StepArgs a;
  resa::SelectArgs& sa = a.s;
  sa.c = cache_args(c);
  sa.q = static_cast<const uint16_t*>(q);
  sa.q_heads = num_q_heads;
  sa.group = group;
  sa.seq_lens = seq_lens;
  sa.max_blocks_seq = mseq;
  sa.keep_ppm = keep;
  sa.min_blocks = params->min_blocks;
  sa.n_local = params->n_local;
  sa.keys = reinterpret_cast<uint32_t*>(wsel + lay.s.keys);
  sa.score_stride = (mseq + 3) & ~3;
  sa.scores_out = nullptr;
  sa.block_idx = block_idx;
  sa.num_sel = num_sel;
  sa.n_cap = n_cap;
  sa.counters = reinterpret_cast<uint32_t*>(wsel + lay.s.counters);
  sa.hist = reinterpret_cast<uint32_t*>(wsel + lay.s.hist);
  sa.blocks_per_wg = resa::step_blocks_per_range(c->batch, c->num_kv_heads, mseq);
  sa.fused = 1;
  sa.k_new = static_cast<const uint16_t*>(k_new);
  sa.v_new = static_cast<const uint16_t*>(v_new);
  sa.lens_out = seq_lens;
  sa.seq_counters = reinterpret_cast<uint32_t*>(wsel + lay.s.seq_counters);
  sa.window = reinterpret_cast<uint32_t*>(wsel + lay.s.window);
  sa.stats = reinterpret_cast<uint32_t*>(wsel + lay.s.stats);
  sa.above_bits = reinterpret_cast<uint32_t*>(wsel + lay.s.above_bits);
  sa.bits_stride = (int32_t)bits_stride(mseq);
  sa.win_keys = reinterpret_cast<uint64_t*>(wsel + lay.s.win_keys);
  resa::DecodeArgs& d = a.d;
  d.c = sa.c;
  d.q = sa.q;
  d.q_heads = num_q_heads;
  d.group = group;
  d.seq_lens = seq_lens;
  d.block_idx = block_idx;
  d.num_sel = num_sel;
  d.n_cap = n_cap;
  d.num_splits = splits;
  d.scale_log2 = sm_scale * 1.4426950408889634f;
  d.out = out;
  d.lse = lse;
  d.counters = reinterpret_cast<uint32_t*>(wdec + lay.d.counters);
  d.epochs = reinterpret_cast<uint32_t*>(wdec + lay.d.epochs);
  d.flags = reinterpret_cast<uint64_t*>(wdec + lay.d.flags);
  d.part_lse = reinterpret_cast<float*>(wdec + lay.d.lse);
  d.part_o = reinterpret_cast<float*>(wdec + lay.d.o);
  d.k_new = sa.k_new;
  d.v_new = sa.v_new;
  a.queue = reinterpret_cast<uint32_t*>(ws + lay.queue);
  a.ready = reinterpret_cast<uint32_t*>(ws + lay.ready);
  a.nranges = (mseq + sa.blocks_per_wg - 1) / sa.blocks_per_wg;
  if (a.nranges < 1) a.nranges = 1;
  a.score_items = (int32_t)(groups * a.nranges);
  a.dec_items = (int32_t)(groups * splits);
  // Bound of a decode split's wait for its group's selection (polls of about
  // 128 cycles each, ~1 s): a guard a correct launch never reaches. Tests of
  // the guard lower it through RESA_STEP_MAX_SPINS.
  a.max_spins = 1u << 20;
  if (const char* env = std::getenv("RESA_STEP_MAX_SPINS")) a.max_spins = (uint32_t)std::strtoul(env, nullptr, 10);
  hipError_t e = resa::launch_step(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "resa_decode_step launch");
  return ok();
}

size_t resa_rectify_workspace_size(int32_t batch, int32_t num_kv_heads, int32_t num_q_heads,
                                   int32_t f, int32_t max_seq_len) {
  if (batch < 1 || num_kv_heads < 1 || num_q_heads < num_kv_heads || f < 1 || max_seq_len < 1)
    return 0;
  // Sized for the largest split count of any length up to max_seq_len, so a
  // workspace sized once serves every shorter call (the layout of a call is
  // never larger: its offsets grow with its own split count).
  const int32_t group = num_q_heads / num_kv_heads;
  const int32_t nq = resa::rectify_num_qblocks(group, f);
  const int32_t most = resa::rectify_max_splits(batch, num_kv_heads, nq, max_seq_len);
  if (most == 1) return 0;  // every such call has one split, written to out / lse directly
  const size_t groups = (size_t)batch * num_kv_heads;
  const size_t rows = (size_t)group * f;
  return round256(groups * most * rows * 4) + groups * most * rows * RESA_HEAD_DIM * 4;
}

int resa_dense_rectify(const resa_kv_cache_t* c, const void* q_f, const void* k_f,
                       const void* v_f, int32_t num_q_heads, int32_t f, const int32_t* seq_lens,
                       const int32_t* seq_mask, int32_t max_seq_len, float sm_scale, float* out,
                       float* lse, int32_t refresh_summaries, void* workspace,
                       size_t workspace_bytes, void* stream) {
  if (int e = check_cache(c)) return e;
  int32_t group = 0;
  if (int e = check_heads(c, num_q_heads, &group)) return e;
  RESA_CHECK_PTR(q_f, 16);
  RESA_CHECK_PTR(k_f, 16);
  RESA_CHECK_PTR(v_f, 16);
  RESA_CHECK_PTR(seq_lens, 4);
  if (seq_mask != nullptr && !aligned(seq_mask, 4))
    return fail(RESA_ERR_INVALID_ARG, "seq_mask is not 4-byte aligned");
  RESA_CHECK_PTR(out, 16);
  if (lse != nullptr && !aligned(lse, 4)) return fail(RESA_ERR_INVALID_ARG, "lse is not 4-byte aligned");
  if (f < 1 || f > RESA_MAX_RECTIFY_ROWS)
    return fail(RESA_ERR_INVALID_ARG, "f %d outside [1, %d]", f, RESA_MAX_RECTIFY_ROWS);
  if (max_seq_len < f || max_seq_len > c->capacity)
    return fail(RESA_ERR_INVALID_ARG, "max_seq_len %d outside [f = %d, capacity %d]", max_seq_len,
                f, c->capacity);
  if (!std::isfinite(sm_scale)) return fail(RESA_ERR_INVALID_ARG, "sm_scale is not finite");
  const RectifyLayout lay = rectify_layout(c->batch, c->num_kv_heads, group, f, max_seq_len);
  if (lay.total > 0 && (workspace == nullptr || workspace_bytes < lay.total))
    return fail(RESA_ERR_WORKSPACE, "rectify workspace needs %zu bytes, got %zu", lay.total,
                workspace == nullptr ? (size_t)0 : workspace_bytes);
  if (workspace != nullptr && !aligned(workspace, 16))
    return fail(RESA_ERR_INVALID_ARG, "workspace is not 16-byte aligned");
  char* ws = static_cast<char*>(workspace);
  resa::RectifyArgs a;
  a.c = cache_args(c);
  a.q_f = static_cast<const uint16_t*>(q_f);
  a.k_f = static_cast<const uint16_t*>(k_f);
  a.v_f = static_cast<const uint16_t*>(v_f);
  a.q_heads = num_q_heads;
  a.group = group;
  a.f = f;
  a.seq_lens = seq_lens;
  a.max_seq_len = max_seq_len;
  a.chunk = lay.chunk;
  a.num_splits = lay.splits;
  a.scale_log2 = sm_scale * 1.4426950408889634f;
  a.out = out;
  a.lse = lse;
  a.part_lse = reinterpret_cast<float*>(ws + lay.lse);
  a.part_o = reinterpret_cast<float*>(ws + lay.o);
  a.refresh = refresh_summaries ? 1 : 0;
  a.seq_mask = seq_mask;
  hipError_t e = resa::launch_rectify(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "resa_dense_rectify launch");
  return ok();
}

int resa_workspace_clear(void* workspace, size_t workspace_bytes, void* stream) {
  if (workspace_bytes == 0) return ok();
  RESA_CHECK_PTR(workspace, 16);
  hipError_t e = resa::launch_clear(workspace, workspace_bytes, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "resa_workspace_clear launch");
  return ok();
}

int resa_stream_read(const void* buffer, size_t bytes, uint32_t* sink, uint32_t match,
                     int32_t workgroups, void* stream) {
  RESA_CHECK_PTR(buffer, 16);
  RESA_CHECK_PTR(sink, 4);
  if (bytes % 16 != 0) return fail(RESA_ERR_INVALID_ARG, "bytes %zu is not a multiple of 16", bytes);
  if (workgroups < 1 || workgroups > 65536)
    return fail(RESA_ERR_INVALID_ARG, "workgroups %d outside [1, 65536]", workgroups);
  if (bytes == 0) return ok();
  hipError_t e = resa::launch_stream_read(buffer, bytes, sink, match, workgroups,
                                          static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "resa_stream_read launch");
  return ok();
}

}  // extern "C"
