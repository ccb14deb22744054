/*
 * resa.h - C ABI of the ReSA decode library for AMD Instinct MI355X (gfx950).
 *
 * Rectified Sparse Attention ("ReSA", arXiv 2506.04108) decodes with
 * group block-sparse attention (Sec. 2.1) and periodically re-encodes the
 * most recent f tokens densely (Sec. 2.2, Alg. 1). This library implements
 * one attention layer's share of that loop on one GPU:
 *
 *   resa_block_summarize  Eq. 3   block key summaries (element-wise min/max)
 *   resa_append_kv        Alg. 1  append one token, update its block summary
 *   resa_select_blocks    Eq. 4-5 pooled-query Quest score + dynamic top-n
 *   resa_append_select    Alg. 1 + Eq. 4-5  append fused with the selection
 *   resa_sparse_decode    Eq. 2, Alg. 2  split flash-decoding over the
 *                                 selected blocks with log-sum-exp combine
 *   resa_decode_step      Alg. 1 one decode token: append + select +
 *                                 sparse decode in one persistent launch
 *   resa_dense_rectify    Sec. 2.2  rewrite the last f cache rows, dense
 *                                 causal attention of their queries over the
 *                                 whole cache, refresh the touched summaries
 *
 * Conventions shared by every call
 * --------------------------------
 * - Every tensor argument is a DEVICE pointer to caller-owned memory
 *   (usually allocated by PyTorch). The library never allocates, frees or
 *   synchronises; scratch comes from a caller workspace sized by the matching
 *   resa_*_workspace_size() call.
 * - Calls are asynchronous on the HIP stream passed as `stream` (a
 *   hipStream_t; NULL is the default stream). A call returns once its kernels
 *   are enqueued.
 * - Return value: RESA_OK, or an error code; resa_last_error() then gives a
 *   message (per host thread). Argument checks run before any HIP call, so a
 *   rejected call touches neither the device nor the stream.
 * - Data types: bf16 caches and queries (uint16 bit patterns), fp32 outputs,
 *   int32 lengths and indices. bf16 tensors, workspaces and the rectify
 *   output must be 16-byte aligned; other int32/fp32 arrays 4-byte aligned.
 * - Supported shapes: head_dim 128; block_size 16, 32 or 64; capacity a
 *   multiple of block_size; 1 <= num_q_heads / num_kv_heads <= 8.
 * - Layouts (row-major, last index fastest):
 *     k, v        [batch, num_kv_heads, capacity, head_dim]
 *     kmin, kmax  [batch, num_kv_heads, capacity / block_size, head_dim]
 *     q           [batch, num_q_heads, head_dim]; query head h belongs to
 *                 kv head h / g, g = num_q_heads / num_kv_heads (GQA, Eq. 1)
 *     seq_lens    [batch] int32, current length L_b of each sequence
 * - A block m of sequence b covers tokens [m*block_size, (m+1)*block_size)
 *   cut at L_b; M_b = ceil(L_b / block_size) blocks exist.
 */
#ifndef RESA_H_
#define RESA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RESA_HEAD_DIM 128
#define RESA_MAX_GROUP 8
#define RESA_MAX_RECTIFY_ROWS 65536 /* largest f of resa_dense_rectify */

typedef enum resa_status {
  RESA_OK = 0,
  RESA_ERR_INVALID_ARG = 1,  /* null/misaligned pointer, bad size or range */
  RESA_ERR_UNSUPPORTED = 2,  /* valid in principle, not built (e.g. head_dim) */
  RESA_ERR_WORKSPACE = 3,    /* workspace missing or too small */
  RESA_ERR_CAPACITY = 4,     /* n_cap or cache capacity too small */
  RESA_ERR_HIP = 5           /* a HIP runtime call or launch failed */
} resa_status_t;

/* The KV cache of one attention layer and its block-key cache. */
typedef struct resa_kv_cache {
  void* k;              /* bf16 [batch, num_kv_heads, capacity, head_dim], or a page
                           pool (see block_table) */
  void* v;              /* bf16, same layout as k */
  void* kmin;           /* bf16 [batch, num_kv_heads, capacity / block_size, head_dim] */
  void* kmax;           /* bf16, same layout as kmin */
  int32_t batch;
  int32_t num_kv_heads;
  int32_t head_dim;     /* 128 */
  int32_t capacity;     /* tokens per sequence; multiple of block_size */
  int32_t block_size;   /* b: 16, 32 or 64 */
  /* Paged layout (serving; optional). NULL: k and v are contiguous per
   * sequence as above. Otherwise k and v are page pools, bf16
   * [num_pages, num_kv_heads, block_size, head_dim]: one page holds one
   * selection block (b tokens) of every kv head, and block_table (device
   * int32 [batch, capacity / block_size]) names the page of logical block m
   * of sequence s at block_table[s * (capacity / block_size) + m]. Block ids
   * (selection output, Eq. 5) stay logical; the kernels translate them.
   * Summaries stay per sequence (kmin / kmax layout above). Entries of the
   * blocks a call touches must lie in [0, num_pages); an entry outside it is
   * never dereferenced (its rows read as absent or zero and writes to them
   * are dropped), and that sequence's results are then unspecified.
   * num_pages * num_kv_heads * block_size must stay below 2^31. */
  const int32_t* block_table;
  int32_t num_pages;    /* pages in each pool (ignored when block_table is NULL) */
} resa_kv_cache_t;

/* Block-selection parameters (Sec. 2.1, Eq. 5). */
typedef struct resa_select_params {
  double sparsity;      /* s in [0, 1]: share of blocks skipped; keep = 1 - s.
                           Rounded to the nearest multiple of 1e-6. */
  int32_t min_blocks;   /* n_min >= 0: minimum number of selected blocks */
  int32_t n_local;      /* >= 0: most recent blocks always selected */
} resa_select_params_t;

/* Library version string ("major.minor.patch"). */
const char* resa_version(void);

/* Message of the last failed call on this host thread ("" if none). */
const char* resa_last_error(void);

/*
 * Eq. 5 (Sec. 2.1), reading p as the kept fraction:
 *   n = min(M, max(min_blocks, n_local, ceil(M * (1 - sparsity))))
 * in exact integer arithmetic on sparsity rounded to 1e-6; 0 when M == 0.
 * The device-side selection uses the same arithmetic. Host only, no device
 * access. Returns -1 for invalid arguments (M < 0, sparsity outside [0, 1],
 * negative min_blocks or n_local).
 */
int32_t resa_num_selected(int32_t num_blocks, double sparsity, int32_t min_blocks,
                          int32_t n_local);

/*
 * Eq. 3 (Sec. 2.1, "Block Representation"): for every sequence b and kv head,
 * kmin/kmax of blocks [blk_begin, blk_end) become the element-wise min/max
 * of the block's valid keys (tokens < L_b). blk_end = -1 means "through the
 * last block of each sequence"; blocks at or past M_b are left untouched.
 * Exact: the min/max of bf16 values is a bf16 value. Reads c->k, writes
 * c->kmin and c->kmax. Used after prefill and by resa_dense_rectify.
 */
int resa_block_summarize(const resa_kv_cache_t* c, const int32_t* seq_lens,
                         int32_t blk_begin, int32_t blk_end, void* stream);

/*
 * Alg. 1, "Update KV cache / block key cache with t": for every sequence b,
 * writes k_new[b], v_new[b] ([batch, num_kv_heads, head_dim] bf16) at row
 * p = seq_lens[b] and folds the key into block p / block_size's summary
 * (initialising it when p opens the block), then sets seq_lens[b] = p + 1
 * in place. max_seq_len is a host-side upper bound of seq_lens before the
 * call; it must be < capacity (RESA_ERR_CAPACITY otherwise). A sequence whose
 * device length has reached capacity is left unchanged.
 */
int resa_append_kv(const resa_kv_cache_t* c, const void* k_new, const void* v_new,
                   int32_t* seq_lens, int32_t max_seq_len, void* stream);

/* Workspace bytes resa_select_blocks needs. */
size_t resa_select_workspace_size(int32_t batch, int32_t num_kv_heads,
                                  int32_t max_seq_len, int32_t block_size);

/*
 * Fig. 3 + Eq. 4 + Eq. 5 (Sec. 2.1, "Block Selection"), per (sequence b,
 * kv head i):
 *   qbar     = mean of the g query heads of group i             (fp32)
 *   score_m  = sum_j max(qbar_j * kmax_mj, qbar_j * kmin_mj)     (fp32)
 *   the last n_local blocks count as +inf; n = resa_num_selected(M_b, ...)
 *   block_idx[b, i, :n] = the n best blocks by (score desc, id asc),
 *                         written in ascending id order; the rest of the
 *                         row up to n_cap is set to -1
 *   num_sel[b, i] = n
 * q: bf16 [batch, num_q_heads, head_dim]. block_idx: int32 [batch,
 * num_kv_heads, n_cap]; num_sel: int32 [batch, num_kv_heads]. n_cap must be
 * >= resa_num_selected(ceil(max_seq_len / block_size), ...) (else
 * RESA_ERR_CAPACITY). scores_out (optional, may be NULL): fp32 [batch,
 * num_kv_heads, ceil(max_seq_len / block_size)], receives the Eq. 4 scores
 * before local forcing (entries past M_b are not written); the workspace
 * keeps the blocks' order-preserving keys either way.
 * One kernel scores the blocks and, in the last workgroup of each group to
 * finish, selects them (groups of more than 32768 blocks use a second
 * kernel). The workspace starts with one ticket per group: zero-fill it
 * before its first use (resa_workspace_clear); every call leaves the tickets
 * at zero again. It also keeps, per group, a hint from the previous call
 * (which bits of the scores to count twice); the hint never changes the
 * result, only how fast the threshold is found, so reusing one workspace per
 * attention layer keeps it matched to that layer's scores. Calls sharing a
 * workspace must be ordered on one stream.
 */
int resa_select_blocks(const resa_kv_cache_t* c, const void* q, int32_t num_q_heads,
                       const int32_t* seq_lens, int32_t max_seq_len,
                       const resa_select_params_t* params, int32_t* block_idx,
                       int32_t* num_sel, int32_t n_cap, float* scores_out,
                       void* workspace, size_t workspace_bytes, void* stream);

/*
 * Alg. 1 "update KV cache / block key cache with t", then Fig. 3 + Eq. 4 +
 * Eq. 5, in one launch: the same results as resa_append_kv followed by
 * resa_select_blocks with max_seq_len + 1. For every sequence b with
 * p = seq_lens[b] < capacity: k_new[b], v_new[b] (bf16 [batch,
 * num_kv_heads, head_dim]) are written at row p, the key is folded into
 * block p / block_size's summary (it starts the summary when p opens the
 * block), the blocks are scored and selected over p + 1 tokens, and
 * seq_lens[b] becomes p + 1 once every kv head of b is done. A sequence
 * already at capacity is left unchanged and selected over its stored length.
 * max_seq_len is a host-side upper bound of seq_lens before the call and must
 * be < capacity (RESA_ERR_CAPACITY otherwise). n_cap, scores_out and the
 * workspace are sized for max_seq_len + 1 tokens
 * (resa_select_workspace_size(batch, num_kv_heads, max_seq_len + 1,
 * block_size)); besides the per-group tickets the workspace holds one
 * counter per sequence, likewise zero-filled before first use and left at
 * zero by every call.
 */
int resa_append_select(const resa_kv_cache_t* c, const void* k_new, const void* v_new,
                       const void* q, int32_t num_q_heads, int32_t* seq_lens,
                       int32_t max_seq_len, const resa_select_params_t* params,
                       int32_t* block_idx, int32_t* num_sel, int32_t n_cap,
                       float* scores_out, void* workspace, size_t workspace_bytes,
                       void* stream);

/*
 * Diagnostics: byte offset, in a resa_select_blocks / resa_append_select
 * workspace (resa_select_stats_offset) or a resa_decode_step workspace
 * (resa_step_stats_offset), of uint32 [batch, num_kv_heads] counters of the
 * calls whose exact top-n finished on its in-window path (from the window
 * hint's bits and lists, without reading every key). They only grow (from the
 * zero-filled workspace) and never change a result.
 */
size_t resa_select_stats_offset(int32_t batch, int32_t num_kv_heads);
size_t resa_step_stats_offset(int32_t batch, int32_t num_kv_heads);

/* Split count resa_sparse_decode uses when num_splits = 0. */
int32_t resa_decode_num_splits(int32_t batch, int32_t num_kv_heads, int32_t n_cap,
                               int32_t block_size);

/* Workspace bytes resa_sparse_decode needs for the given split count
 * (0 = the automatic count). */
size_t resa_decode_workspace_size(int32_t batch, int32_t num_kv_heads,
                                  int32_t num_q_heads, int32_t n_cap,
                                  int32_t block_size, int32_t num_splits);

/*
 * Eq. 2 with Alg. 2 (App. A): block-sparse flash-decoding. For every
 * (sequence b, kv head i) the selected blocks block_idx[b, i, :num_sel[b, i]]
 * (ids in [0, M_b); any order; as written by resa_select_blocks) are cut
 * into 16-token chunks, dealt to num_splits parts one by one (part s takes
 * chunks s, s + num_splits, ...); each part runs an online softmax of the g
 * query heads over its chunks' valid tokens (t < L_b; others are excluded)
 * and the parts are merged by log-sum-exp. For query head h:
 *   out[b, h, :] = sum_t softmax_t(q_h . K_t * sm_scale) V_t     (fp32)
 *   lse[b, h]    = log sum_t exp(q_h . K_t * sm_scale)           (optional)
 * With no token selected, out is 0 and lse is -inf. Passing every block id
 * gives dense decoding. Value range: the fp32 accumulation keeps softmax
 * weights up to 2^8 over up to 2^20 tokens per split, so results are finite
 * for |v| <= 2^100. num_splits = 0 picks resa_decode_num_splits();
 * explicit counts must lie in [1, 256].
 * One kernel: each split writes a partial into the workspace and the last
 * split of a group to finish merges them (with 16 or more splits, the last g
 * splits to finish merge one query head each). The workspace starts with one
 * merge counter and one count of merged calls per group, which tags the
 * splits' ready flags of each call: zero-fill it before its first use
 * (resa_workspace_clear or any zeroing allocator); every call leaves the
 * counters at zero again and advances the counts.
 * Calls sharing a workspace must be ordered on one stream.
 */
int resa_sparse_decode(const resa_kv_cache_t* c, const void* q, int32_t num_q_heads,
                       const int32_t* seq_lens, const int32_t* block_idx,
                       const int32_t* num_sel, int32_t n_cap, int32_t num_splits,
                       float sm_scale, float* out, float* lse, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * resa_sparse_decode without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same arguments, kernels and results as
 * resa_sparse_decode (bit-identical for the same split count), minus the
 * workspace: the split partials and merge counters live in a static device
 * array of resa_sparse_decode_noalloc_max_bytes() bytes (4 MiB) that each GPU
 * the library runs on holds until the process ends. The call allocates and
 * frees nothing; it zero-fills the merge counters, call counts and ready
 * flags with a kernel before the decode. The first call on a device looks up that device's array address
 * (hipGetSymbolAddress). Every call on one GPU shares that GPU's array and
 * the array keeps the last call's contents, so calls that may overlap on one
 * GPU (different streams without ordering, concurrent host threads) race:
 * order them on one stream. Errors: as resa_sparse_decode; RESA_ERR_WORKSPACE
 * when the call's partials (resa_decode_workspace_size for the same shape and
 * split count) exceed the static array, RESA_ERR_HIP when the array's address
 * cannot be obtained.
 */
int resa_sparse_decode_noalloc(const resa_kv_cache_t* c, const void* q, int32_t num_q_heads,
                               const int32_t* seq_lens, const int32_t* block_idx,
                               const int32_t* num_sel, int32_t n_cap, int32_t num_splits,
                               float sm_scale, float* out, float* lse, void* stream);

/* Bytes of the static scratch resa_sparse_decode_noalloc works in. */
size_t resa_sparse_decode_noalloc_max_bytes(void);

/* Workspace bytes resa_decode_step needs; max_seq_len and num_splits as
 * passed to it (num_splits 0 = the automatic count). */
size_t resa_step_workspace_size(int32_t batch, int32_t num_kv_heads, int32_t num_q_heads,
                                int32_t max_seq_len, int32_t block_size, int32_t n_cap,
                                int32_t num_splits);

/*
 * One decode token of one attention layer (Alg. 1, decoding loop, without
 * the periodic rectification): resa_append_select followed by
 * resa_sparse_decode, in one launch. For every sequence b with
 * p = seq_lens[b] < capacity the token k_new[b], v_new[b] is appended (row p,
 * block summary updated), the blocks of the p + 1 tokens are scored and
 * selected (Eq. 4-5; block_idx / num_sel as resa_select_blocks), the g query
 * heads attend to the selected blocks (Eq. 2, Alg. 2; out / lse as
 * resa_sparse_decode) and seq_lens[b] becomes p + 1. A sequence already at
 * capacity is left unchanged and decoded over its stored length.
 * Arguments as for resa_append_select and resa_sparse_decode: max_seq_len is
 * a host bound of seq_lens before the call and must be < capacity
 * (RESA_ERR_CAPACITY otherwise), n_cap >= the Eq. 5 count at max_seq_len + 1
 * tokens, num_splits 0 (automatic) or in [1, 256]. Groups of more than 32768
 * blocks are RESA_ERR_UNSUPPORTED.
 * The selection and the decode are the same computations as the two calls
 * (selected ids identical, outputs equal up to fp32 summation order: the
 * split parts are cut the same way but summed by 8 waves instead of 4).
 * One workgroup per compute unit claims the work: score ranges first, then
 * decode splits, each waiting for its group's selection (so a group's decode
 * overlaps the selection of later groups). The workspace
 * (resa_step_workspace_size) holds claim counters, per-group flags and
 * tickets and the selection hint: zero-fill it before its first use
 * (resa_workspace_clear); every call leaves the counters and the ready flags
 * at zero (the decode's split flags carry a per-call tag instead).
 * Calls sharing a workspace must be ordered on one stream.
 * Status: the uint32 at byte offset 12 of the workspace becomes 1 if a decode
 * split gave up waiting for its group's selection (a bounded wait, a guard
 * that a correct launch never trips); that split then decodes nothing and the
 * outputs of that call are unspecified. The word is sticky: zero-fill the
 * workspace to clear it.
 */
int resa_decode_step(const resa_kv_cache_t* c, const void* k_new, const void* v_new,
                     const void* q, int32_t num_q_heads, int32_t* seq_lens, int32_t max_seq_len,
                     const resa_select_params_t* params, int32_t* block_idx, int32_t* num_sel,
                     int32_t n_cap, int32_t num_splits, float sm_scale, float* out, float* lse,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes resa_dense_rectify needs for any call whose max_seq_len
 * is at most the one given (the size never decreases as max_seq_len grows,
 * so a workspace sized once for the longest context serves every call): 0
 * when one key split covers every such window (long windows such as
 * prefill), and then workspace may be NULL. */
size_t resa_rectify_workspace_size(int32_t batch, int32_t num_kv_heads,
                                   int32_t num_q_heads, int32_t f, int32_t max_seq_len);

/*
 * Dense rectification (Sec. 2.2; Alg. 1, "DenseForward" every f steps) of
 * one layer. For every sequence b with length L = seq_lens[b] >= f that the
 * call covers (seq_mask == NULL: every sequence; else those with
 * seq_mask[b] != 0):
 *   1. rows [L - f, L) of k and v become k_f[b], v_f[b]
 *      (bf16 [batch, num_kv_heads, f, head_dim]);
 *   2. query row r of q_f[b, h] (bf16 [batch, num_q_heads, f, head_dim]) sits
 *      at position L - f + r and attends causally to tokens t <= L - f + r:
 *        out[b, h, r, :] = sum_t softmax_t(q . K_t * sm_scale) V_t   (fp32)
 *        lse[b, h, r]    = log sum_t exp(...)            (optional, may be NULL)
 *   3. if refresh_summaries, blocks floor((L - f) / b) .. M_b - 1 are
 *      re-summarised (Eq. 3).
 * 1 <= f <= RESA_MAX_RECTIFY_ROWS and f <= max_seq_len <= capacity.
 * max_seq_len bounds every seq_lens[b] (host side, for launch sizing). A
 * sequence with seq_lens[b] < f is left untouched and its out rows are 0 (lse
 * -inf). The workspace holds split partials and needs no initialisation.
 * Per-request phases (Sec. 2.2, compatibility with serving systems: each
 * request is rectified every f of its own steps, so in a continuous batch
 * requests reach their rectification at different steps): seq_mask (device
 * int32 [batch], or NULL) selects the sequences this call rectifies. A
 * sequence with seq_mask[b] == 0 is not touched at all: its cache rows,
 * summaries, out and lse rows keep their contents, and its q_f / k_f / v_f
 * rows are not read.
 * Value range: any finite bf16 V gives a finite out. P . V runs on fp16
 * matrix cores with P in [0, 2^8]; V enters at its own scale (exact for
 * |v| in 2^-14 .. 65280, fp16 subnormal spacing 2^-24 below), and a head
 * dimension holding larger values is scaled by a power of two for the
 * whole call from the first tile that needs it (its smaller values then lose
 * the bits below 2^-24 of the scale, far below 2e-3 of the dimension's
 * largest magnitude).
 * Errors: RESA_ERR_INVALID_ARG for the ranges above or misaligned pointers,
 * RESA_ERR_WORKSPACE when a needed workspace is missing or too small.
 * The same call serves (chunked) prefill (Alg. 1, prefill step): with
 * seq_lens[b] already counting a prompt chunk of f tokens, the chunk's keys
 * and values are written, its queries attend causally to the cache before
 * it and to themselves, and its blocks are summarised; with f = L the whole
 * prompt is prefilled and every block summary built.
 */
int resa_dense_rectify(const resa_kv_cache_t* c, const void* q_f, const void* k_f,
                       const void* v_f, int32_t num_q_heads, int32_t f,
                       const int32_t* seq_lens, const int32_t* seq_mask, int32_t max_seq_len,
                       float sm_scale, float* out, float* lse, int32_t refresh_summaries,
                       void* workspace, size_t workspace_bytes, void* stream);

/* Zero-fills a workspace with a kernel (safe under stream capture). */
int resa_workspace_clear(void* workspace, size_t workspace_bytes, void* stream);

/*
 * Measurement helper, not part of the attention method: reads every byte of
 * `buffer` (device, 16-byte aligned, `bytes` a multiple of 16) once with the
 * 16-byte non-temporal loads the decode kernel uses for K and V, spread over
 * `workgroups` workgroups of 256 threads (1 .. 65536). The XOR of all words
 * read is stored to sink[0] (device uint32) only if it equals `match`, so the
 * loads cannot be elided and the sink is normally untouched. Timing it gives
 * the HBM read ceiling the decode bandwidth is compared with.
 * Errors: RESA_ERR_INVALID_ARG for a null or misaligned pointer, a size that
 * is not a multiple of 16 or a workgroup count out of range.
 */
int resa_stream_read(const void* buffer, size_t bytes, uint32_t* sink, uint32_t match,
                     int32_t workgroups, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RESA_H_ */
