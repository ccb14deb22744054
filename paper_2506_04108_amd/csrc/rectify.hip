// Dense rectification (Sec. 2.2; Alg. 1 "DenseForward" every f steps) on
// gfx950 matrix cores.
//
// The f re-encoded query rows of a (sequence, kv head) group, times its g
// heads, are R = g * f rows (row rho = r * g + h sits at position L - f + r).
// Against the whole cache they form a dense contraction, so this is the one
// place the library uses MFMA (v_mfma_f32_16x16x32_bf16).
//
// Grid (num_splits, ceil(R / rows), batch * kv_heads) with 4 waves (rows =
// 128, windows of up to 128 rows) or 8 waves (rows = 256, longer windows
// such as prefill) per workgroup, each wave owning 32 query rows (two
// 16-row tiles). A workgroup walks its key range in tiles of 32 keys (4
// waves) or 64 keys (8 waves) through four LDS stages: K and V rows go from HBM straight into LDS
// (buffer loads with the LDS destination, no registers), three tiles ahead
// of the one being computed, and one barrier per tile publishes a tile and
// frees the stage read before it. Per tile and wave:
//   S^T = K . Q^T        (keys x queries; lane l holds query l % 16 and keys
//                          16 kt + 4 (l / 16) + i)
//   online softmax per query row in the log2 domain against a reference
//   that moves only in steps of more than 2^8, so P lies in [0, 2^8]; P is
//   rounded to fp16 (11 significant bits)
//   O^T += V^T . P^T     (dims x queries, fp16 MFMA; the contraction index is
//                          ordered so that P^T is already in the B-operand
//                          layout, and V^T comes from the row-major V tile
//                          through the LDS transpose read)
// V tiles are converted from bf16 to fp16 in LDS, before the barrier, by
// the threads that loaded them, each head dimension d multiplied by a power
// of two 2^-E_d first (E_d = 0 until a value needs it). Every bf16 value of
// magnitude 2^-14 .. 65280 is an fp16 value (8 significant bits fit in 11),
// so in that range the conversion is exact; smaller values keep fp16's
// subnormal spacing of 2^-24 (an error of at most 2^-24 * P per key). A
// thread that finds a scaled value above 65504 flags the tile; on a flagged
// tile every thread reloads its V pieces from HBM, E_d rises for the
// dimensions that need it (so that max |v| 2^-E_d < 2^16), those
// accumulator rows are multiplied by the change, and the tile is converted
// again. Rows are multiplied back by 2^E_d after the normalisation by the
// softmax sum, so every finite bf16 V gives a finite result (products
// P V 2^-E_d stay below 2^24 and their sums far below the fp32 range).
// Masking (causal cut, end of the split) is only evaluated on the tiles that
// reach it. A second kernel merges the splits by log-sum-exp (Alg. 2,
// "Combine"), spread over many workgroups.
#include <type_traits>

#include "resa_device.h"
#include "resa_internal.h"

namespace resa {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4_t __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kRowsPerWave = 32;
// Workgroups of 4 waves (128 rows) for short windows; long windows (prefill)
// use 8 waves (256 rows), so each K / V tile brought into LDS serves twice
// the rows.
template <int kWaves>
constexpr int rows_per_wg() { return kWaves * kRowsPerWave; }
__host__ __device__ constexpr int waves_for_rows(int rows) { return rows > 128 ? 8 : 4; }
// Keys per tile: 32 for 4-wave workgroups (two per CU share the LDS), 64 for
// 8-wave ones (one per CU: fewer barriers, load issues and softmax
// bookkeeping per key where the matrix work dominates).
template <int kWaves>
constexpr int key_tile() { return kWaves == 8 ? 64 : 32; }
constexpr int kMaxKeyTile = 64;
constexpr int kStages = 4;                        // LDS stages: the tile computed, three in flight
constexpr int kRowBytes = kHeadDim * 2;           // one K or V row (16-bit values)
constexpr int kPageRing = 8;                      // page ids per wave held in LDS
typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));

// Tile rows are stored unpadded (256 B); 16-byte piece p of row r sits in
// slot p ^ swz(r). swz is a bijection on r % 16, so the K operand reads (16
// rows, one piece) hit 16 distinct slots; its bits 1..3 follow r % 8 and
// its low bit r / 8, so the V transpose reads (4 aligned rows, two
// neighbouring pieces) hit 8 distinct slots: no LDS bank conflicts.
__host__ __device__ constexpr int swz(int r) { return ((r & 7) << 1) | ((r >> 3) & 1); }

// s_waitcnt immediates (vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
constexpr int wait_vm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0F70; }
constexpr int kWaitLgkm0 = 0xC07F;
// Buffer resource over `bytes` bytes at p (stride 0, 32-bit format), for
// values the caller knows are uniform across the wave: read from the first
// lane, so the resource sits in scalar registers. Offsets at or past
// `bytes` read as zero.
__device__ __forceinline__ i32x4_t rsrc_words(const void* p, int bytes) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  return i32x4_t{(int32_t)__builtin_amdgcn_readfirstlane((uint32_t)u),
                 (int32_t)(__builtin_amdgcn_readfirstlane((uint32_t)(u >> 32)) & 0xffffu),
                 __builtin_amdgcn_readfirstlane(bytes), kBufWord3};
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t uniform_rsrc(const void* p, int bytes) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  void* q = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(q, (short)0, __builtin_amdgcn_readfirstlane(bytes), kBufWord3);
}
// LDS byte address of an LDS object.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
// Buffer loads straight into LDS (no registers): lane i's 16 (4) bytes at
// offset voff land at LDS byte address lds + 16 i (lds + 4 i); M0 carries
// the LDS address. Written as assembly so that the compiler does not track
// them: it would otherwise make every V transpose read wait for all of them.
// Their completion is ordered by hand (vmcnt waits, then a barrier). M0 is
// saved and restored around each group of loads, so whatever the compiler
// keeps in it survives; one wait state follows each write of M0 that a load
// reads.
//
// A wave's rows of one tile: two 1 KB loads of K (rows +0 and +4 of its
// LDS rows, global offsets voff0 / voff1 in rk) and the same two of V (LDS
// address + kTile, rv).
template <int kTile>
__device__ __forceinline__ void lds_load_rows8(uint32_t lds, uint32_t voff0, uint32_t voff1, i32x4_t rk,
                                               i32x4_t rv) {
  uint32_t saved;
  __asm__ volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\ts_nop 0\n\tbuffer_load_dwordx4 %2, %4, 0 offen nt lds\n\t"
      "s_add_i32 m0, %1, %6\n\ts_nop 0\n\tbuffer_load_dwordx4 %2, %5, 0 offen nt lds\n\t"
      "s_add_i32 m0, %1, 1024\n\ts_nop 0\n\tbuffer_load_dwordx4 %3, %4, 0 offen nt lds\n\t"
      "s_add_i32 m0, %1, %7\n\ts_nop 0\n\tbuffer_load_dwordx4 %3, %5, 0 offen nt lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds), "v"(voff0), "v"(voff1), "s"(rk), "s"(rv), "n"(kTile), "n"(kTile + 1024)
      : "memory", "scc");
}
__device__ __forceinline__ void lds_load4(uint32_t lds, uint32_t voff, i32x4_t rs) {
  uint32_t saved;
  __asm__ volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
      "buffer_load_dword %2, %3, 0 offen lds\n\ts_mov_b32 m0, %0"
      : "=&s"(saved) : "s"(lds), "v"(voff), "s"(rs) : "memory");
}
// Keeps the compiler from moving memory accesses across this point; the
// hardware ordering comes from the explicit waits and barriers around it.
__device__ __forceinline__ void compiler_fence() { __asm__ volatile("" ::: "memory"); }
constexpr int kMaxRectSplits = 1024;     // splits per group (bounded by the host)
constexpr float kRefSlack = 8.f;         // log2-domain headroom of the softmax reference

__device__ __forceinline__ f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma16(f16x8_t a, f16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// LDS transpose read of a 4-key x 16-dim block of 16-bit values by each
// 16-lane group: lane c of the group passes the address of key
// kbase + c / 4, dims dbase + 4 (c % 4) .. + 4; lane i of the group receives
// dim dbase + i of keys kbase .. kbase + 3.
__device__ __forceinline__ f16x4_t lds_read_tr(const uint8_t* p) {
  typedef __attribute__((address_space(3))) i16x4_t lds_i16x4;
  const i16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_i16x4*)(const_cast<uint8_t*>(p)));
  return __builtin_bit_cast(f16x4_t, v);
}

// Writes the re-encoded rows k_f, v_f over cache rows [L - f, L).
// Grid (ceil(f / 16), batch * kv_heads): each workgroup copies 16 rows.
__global__ __launch_bounds__(256) void k_rectify_rows(RectifyArgs a) {
  const int grp = blockIdx.y;
  const int bb = grp / a.c.kv_heads;
  if (a.seq_mask != nullptr && a.seq_mask[bb] == 0) return;
  const int L = a.seq_lens[bb];
  if (L < a.f || L > a.c.capacity) return;
  uint16_t* k = const_cast<uint16_t*>(a.c.k);
  uint16_t* v = const_cast<uint16_t*>(a.c.v);
  const int s = blockIdx.x * 256 + threadIdx.x;
  if (s < a.f * 16) {
    const int row = s >> 4, part = s & 15;
    const size_t src = ((size_t)grp * a.f + row) * kHeadDim + part * 8;
    const int64_t kr = kv_row(a.c, bb, grp % a.c.kv_heads, L - a.f + row);
    if (kr >= 0) {
      const size_t dst = (size_t)kr * kHeadDim + part * 8;
      st16(k + dst, ld16(a.k_f + src));
      st16(v + dst, ld16(a.v_f + src));
    }
  }
}

template <int kWaves, bool kPaged>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_rectify_attn(RectifyArgs a) {
  constexpr int kRowsPerWg = rows_per_wg<kWaves>();
  constexpr int kKT = key_tile<kWaves>();
  constexpr int kTileBytes = kKT * kRowBytes;    // K (and V) bytes of a tile
  constexpr int kLoadRows = kKT / kWaves;        // tile rows whose K and V each wave loads
  constexpr int kLoads = kLoadRows / 4;          // 1 KB load instructions per wave, tensor and tile
  // Loads a wave issues per tile (K, V and, paged, one page id). When tile t
  // is waited for, those of tiles t + 1 and t + 2 may still be in flight
  // (page ids run three tiles ahead of the data they locate).
  constexpr int kOpsPerTile = 2 * kLoads + (kPaged ? 1 : 0);
  constexpr int kWaitTile = wait_vm(2 * kOpsPerTile);
  // All of the workgroup's LDS is one object. With several, the compiler
  // tags each access with the object it touches and then makes every LDS
  // read of the tile buffers wait for all loads into them (the newest
  // included), which would drain the pipeline; here the explicit waits and
  // barriers below order the loads into LDS against the reads.
  struct Lds {
    uint8_t kv[kStages][2][kTileBytes];  // [stage][K, V] tile rows
    int page[kWaves][kPageRing];         // page ids of each wave's rows
    // V range handling: flag[st] = first key of the tile in stage st when
    // one of its scaled values is above the fp16 range (else an older
    // tile's key, or -1); vscale[cur][d] = 2^-E_d; vmax[d] = max |v| of
    // dimension d over a flagged tile (fp32 bits: non-negative values order
    // as integers).
    int flag[kStages];
    float vscale[2][kHeadDim];
    uint32_t vmax[kHeadDim];
  };
  __shared__ __attribute__((aligned(1024))) Lds lds;
  auto& s_kv = lds.kv;
  auto& s_page = lds.page;
  auto& s_flag = lds.flag;
  auto& s_vscale = lds.vscale;
  auto& s_vmax = lds.vmax;
  // The wave index is uniform per wave (readfirstlane tells the compiler), so
  // the load addressing below stays in scalar registers.
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int split = blockIdx.x, qblk = blockIdx.y, grp = blockIdx.z;
  const int bb = grp / a.c.kv_heads, hk = grp % a.c.kv_heads;
  // A sequence left out of this call: nothing is read or written (uniform
  // across the workgroup, before any barrier).
  if (a.seq_mask != nullptr && a.seq_mask[bb] == 0) return;
  const int G = a.group, f = a.f, R = G * f;
  const int S = a.num_splits;
  const int L = a.seq_lens[bb];
  const bool seq_ok = L >= f && L <= a.c.capacity;
  const int k0 = split * a.chunk;
  // Keys past the last causal limit of this workgroup's rows are never
  // needed (row rho sits at L - f + rho / G): long windows (chunked prefill)
  // skip them instead of masking them.
  const int last_row = min(R - 1, (qblk + 1) * kRowsPerWg - 1);
  const int k1 = seq_ok ? min(min(k0 + a.chunk, L), L - f + last_row / G + 1) : k0;
  const int ntiles = k1 > k0 ? (k1 - k0 + kKT - 1) / kKT : 0;
  const int j = lane >> 4, lq = lane & 15;
  const int row_base = qblk * kRowsPerWg + wave * kRowsPerWave;
  const float ninf = -__builtin_inff();
  const float c = a.scale_log2;

  // Q^T operand (B of the S^T product): lane holds query row lq of each tile,
  // dims 32 s + 8 j .. + 8 for k-step s.
  bf16x8_t qb[2][4];
  int lim[2];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int rho = row_base + 16 * qt + lq;
    if (rho < R && seq_ok) {
      const int h = rho % G, r = rho / G;
      lim[qt] = L - f + r;
      const uint16_t* qp = a.q_f + (((size_t)bb * a.q_heads + (size_t)hk * G + h) * f + r) * kHeadDim;
#pragma unroll
      for (int s = 0; s < 4; ++s) qb[qt][s] = __builtin_bit_cast(bf16x8_t, ld16(qp + 32 * s + 8 * j));
    } else {
      lim[qt] = -1;
#pragma unroll
      for (int s = 0; s < 4; ++s) qb[qt][s] = __builtin_bit_cast(bf16x8_t, U4{0, 0, 0, 0});
    }
  }
  // Keys at or past `cut` need the mask: the causal cut of the first row of
  // this wave (the smallest limit) or the end of the split.
  const int cut = min(k1, L - f + row_base / G);

  f32x4_t o[8][2];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) o[dt][qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m[2] = {ninf, ninf}, l[2] = {0.f, 0.f};

  // Wave w loads tile rows kLoadRows w .. + kLoadRows; load instruction e
  // covers four of them: lane i fills LDS slot i % 16 of row
  // kLoadRows w + 4 e + i / 16, fetching the row's piece (i % 16) ^ swz(row).
  const int wrow = kLoadRows * wave;
  const int lrow = lane >> 4, lslot = lane & 15;
  // Buffer resources over this wave's rows of tile ti: rows at or past k1
  // and rows of a page outside the pool fall outside them and read as zero.
  auto tile_src = [&](int ti, const uint16_t*& pk, const uint16_t*& pv, int& nrec) __attribute__((always_inline)) {
    const int key = k0 + ti * kKT + wrow;
    nrec = min(max(k1 - key, 0), kLoadRows) * kRowBytes;
    size_t row;
    if constexpr (kPaged) {
      const int page = __builtin_amdgcn_readfirstlane(s_page[wave][ti & (kPageRing - 1)]);
      if ((unsigned)page >= (unsigned)a.c.num_pages) nrec = 0;
      row = ((size_t)page * a.c.kv_heads + hk) * a.c.block_size + (key & (a.c.block_size - 1));
    } else {
      row = ((size_t)bb * a.c.kv_heads + hk) * a.c.capacity + key;
    }
    pk = a.c.k + row * kHeadDim;
    pv = a.c.v + row * kHeadDim;
  };
  auto src_off = [&](int e) __attribute__((always_inline)) {
    return (uint32_t)((4 * e + lrow) * kRowBytes + 16 * (lslot ^ swz(wrow + 4 * e + lrow)));
  };
  const uint32_t lds_kv = __builtin_amdgcn_readfirstlane(lds_addr(&s_kv[0][0][0]));
  // Tile ti's K and V rows of this wave, straight into stage ti % kStages.
  auto issue = [&](int ti) __attribute__((always_inline)) {
    const uint16_t *pk, *pv;
    int nrec;
    tile_src(ti, pk, pv, nrec);
    const i32x4_t rk = rsrc_words(pk, nrec), rv = rsrc_words(pv, nrec);
    const uint32_t dk = lds_kv + (uint32_t)((ti & (kStages - 1)) * 2 * kTileBytes + wrow * kRowBytes);
    static_assert(kLoads == 2, "eight rows per wave and tile");
    lds_load_rows8<kTileBytes>(dk, src_off(0), src_off(1), rk, rv);
  };
  // Page id of this wave's rows of tile ti (its rows lie in one block), into
  // the ring; blocks past the table read as page 0 (only tiles past k1 ask).
  auto issue_page = [&](int ti) __attribute__((always_inline)) {
    if constexpr (kPaged) {
      const int mb = (k0 + ti * kKT + wrow) >> a.c.log2_block;
      const i32x4_t rt = rsrc_words(a.c.table + (size_t)bb * a.c.max_blocks, a.c.max_blocks * 4);
      const uint32_t dst = __builtin_amdgcn_readfirstlane(lds_addr(&s_page[wave][ti & (kPageRing - 1)]));
      if (lane == 0) lds_load4(dst, (uint32_t)mb * 4, rt);
    }
  };

  // V scale state, uniform across the workgroup: `scaled` once any E_d > 0,
  // `cur` the current half of s_vscale.
  bool scaled = false;
  int cur = 0;
  // Converts a 16-byte piece of V (8 bf16 values) to fp16, times the
  // per-dimension factors when `use_sc`; vmax collects the largest scaled
  // magnitude.
  auto to_h8 = [&](const U4& w, const float (&sc)[8], bool use_sc, float& vmax) __attribute__((always_inline)) {
    float x[8] = {bf_lo(w.x), bf_hi(w.x), bf_lo(w.y), bf_hi(w.y),
                  bf_lo(w.z), bf_hi(w.z), bf_lo(w.w), bf_hi(w.w)};
    uint32_t h[4];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (use_sc) x[i] *= sc[i];
      vmax = fmaxf(vmax, fabsf(x[i]));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f16x2_t p = {(_Float16)x[2 * i], (_Float16)x[2 * i + 1]};
      h[i] = __builtin_bit_cast(uint32_t, p);
    }
    return U4{h[0], h[1], h[2], h[3]};
  };
  // Converts the V pieces this thread loaded for the tile in stage st
  // (first key t0) in place; a thread with a scaled value outside the fp16
  // range flags the tile.
  auto convert = [&](int st, int t0) __attribute__((always_inline)) {
    float vmax = 0.f;
#pragma unroll
    for (int e = 0; e < kLoads; ++e) {
      uint8_t* p = s_kv[st][1] + (wrow + 4 * e) * kRowBytes + 16 * lane;
      const U4 w = ld16(p);
      float sc[8];
      if (scaled) {
        const int piece = lslot ^ swz(wrow + 4 * e + lrow);
#pragma unroll
        for (int i = 0; i < 8; ++i) sc[i] = s_vscale[cur][8 * piece + i];
        st16(p, to_h8(w, sc, true, vmax));
      } else {
        st16(p, to_h8(w, sc, false, vmax));
      }
    }
    if (!(vmax <= 65504.f)) s_flag[st] = t0;
  };
  // A flagged tile (uniform: every wave reads the same flag). This thread's
  // raw V pieces are reloaded, the per-dimension maxima are gathered, E_d
  // rises where max |v| 2^-E_d would reach 2^16, the accumulator rows of
  // those dimensions follow, and the pieces are converted again in place.
  auto fix_tile = [&](int ti, int st) __attribute__((always_inline)) {
    const uint16_t *pk, *pv;
    int nrec;
    tile_src(ti, pk, pv, nrec);
    const __amdgpu_buffer_rsrc_t rv = uniform_rsrc(pv, nrec);
    U4 vv[kLoads];
#pragma unroll
    for (int e = 0; e < kLoads; ++e)
      vv[e] = __builtin_bit_cast(U4, __builtin_amdgcn_raw_buffer_load_b128(rv, src_off(e), 0, 0));
#pragma unroll
    for (int e = 0; e < kLoads; ++e) {
      const int piece = lslot ^ swz(wrow + 4 * e + lrow);
      const float x[8] = {bf_lo(vv[e].x), bf_hi(vv[e].x), bf_lo(vv[e].y), bf_hi(vv[e].y),
                          bf_lo(vv[e].z), bf_hi(vv[e].z), bf_lo(vv[e].w), bf_hi(vv[e].w)};
#pragma unroll
      for (int i = 0; i < 8; ++i) atomicMax(&s_vmax[8 * piece + i], __float_as_uint(fabsf(x[i])));
    }
    lds_sync();
    if (tid < kHeadDim) {
      const uint32_t mb = s_vmax[tid];
      // max |v| < 2^(ex + 1); E = ex - 15 keeps the scaled maximum below 2^16.
      const int ex = (int)((mb >> 23) & 0xff) - 127;
      const int E = ex > 15 ? ex - 15 : 0;
      s_vscale[cur ^ 1][tid] = fminf(s_vscale[cur][tid], __uint_as_float((uint32_t)(127 - E) << 23));
    }
    lds_sync();
    float unused = 0.f;
#pragma unroll
    for (int e = 0; e < kLoads; ++e) {
      const int piece = lslot ^ swz(wrow + 4 * e + lrow);
      float ns[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) ns[i] = s_vscale[cur ^ 1][8 * piece + i];
      st16(s_kv[st][1] + (wrow + 4 * e) * kRowBytes + 16 * lane, to_h8(vv[e], ns, true, unused));
    }
    lds_sync();
    if (tid < kHeadDim) s_vmax[tid] = 0u;
    // Accumulator row d (lane dims 16 dt + 4 j + i) times 2^(E_old - E_new).
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = 16 * dt + 4 * j + i;
        const float r = s_vscale[cur ^ 1][d] / s_vscale[cur][d];
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) o[dt][qt][i] *= r;
      }
    }
    cur ^= 1;
    scaled = true;
  };

  // LDS byte offsets of this lane's operand reads within a stage. K (A of
  // S^T): row 16 kt + lq, piece 4 s + j. V^T (A of O^T, transpose read):
  // rows 4 j + lq / 4 and 16 + 4 j + lq / 4 (the same swizzle), dims
  // 16 dt + 4 (lq % 4) .. + 4, i.e. piece 2 dt + (lq % 4) / 2, byte
  // 8 (lq % 2) within it.
  const int swq = swz(lq);
  const int vrow = 4 * j + (lq >> 2), swv = swz(vrow);
  // One tile: scores, softmax update, P.V. kMasked evaluates the causal cut
  // and the split end per key.
  auto tile = [&](int ti, int st, auto masked) __attribute__((always_inline)) {
    constexpr bool kMasked = decltype(masked)::value;
    constexpr int KT16 = kKT / 16, KT32 = kKT / 32;
    const int t0 = k0 + ti * kKT;
    const uint8_t* tk = s_kv[st][0];
    const uint8_t* tv = s_kv[st][1];
    const int flag = s_flag[st];  // read now, used after the scores
    f32x4_t sacc[KT16][2];
#pragma unroll
    for (int kt = 0; kt < KT16; ++kt)
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) sacc[kt][qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // The matrix-core sections run at wave priority 1 (the softmax and the
    // conversion at 0): a SIMD's other wave, at another point of its tile,
    // then fills the gaps with vector work instead of delaying the MFMAs.
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
      for (int kt = 0; kt < KT16; ++kt) {
        const bf16x8_t ka = *reinterpret_cast<const bf16x8_t*>(
            tk + (16 * kt + lq) * kRowBytes + 16 * ((4 * s + j) ^ swq));
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) sacc[kt][qt] = mfma16(ka, qb[qt][s], sacc[kt][qt]);
      }
    }

    __builtin_amdgcn_s_setprio(0);
    f16x8_t ph[2][KT32];  // [qt][32-key step ks]: keys 32 ks + 4 j + (0..3), then + 16
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      float x[4 * KT16];
      float tmax = ninf;
#pragma unroll
      for (int kt = 0; kt < KT16; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float y = sacc[kt][qt][i];
          if constexpr (kMasked) {
            const int key = t0 + 16 * kt + 4 * j + i;
            y = (key > lim[qt] || key >= k1) ? ninf : y;
          }
          x[4 * kt + i] = y;
          tmax = fmaxf(tmax, y);
        }
      // Raw scores times c are log2-domain logits (c > 0 keeps the maximum).
      // The reference m moves only when the tile's maximum exceeds it by
      // more than kRefSlack, so the accumulator rescale is rare; every
      // weight stays <= 2^kRefSlack, well inside fp16 and fp32 range, and
      // the normalisation by l uses the same reference. A query's keys of
      // the tile sit in four lanes (lq + 16 j): the row maximum across them is only
      // needed when one of them exceeds the reference, so the cross-lane
      // reduction runs on those (rare) tiles only.
      float alpha = 1.f;
      if (__any(tmax * c > m[qt] + kRefSlack)) {
        tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
        const float tm = tmax * c;
        if (tm > m[qt] + kRefSlack) {
          alpha = fast_exp2(m[qt] - tm);  // 0 when m was -inf
          m[qt] = tm;
        }
      }
      const float mref = m[qt] == ninf ? 0.f : m[qt];
      float ps = 0.f;
#pragma unroll
      for (int e = 0; e < 4 * KT16; ++e) {
        const float pe = fast_exp2(fmaf(x[e], c, -mref));
        ps += pe;
        ph[qt][e >> 3][e & 7] = (_Float16)pe;
      }
      l[qt] = fmaf(l[qt], alpha, ps);
      if (__any(alpha != 1.f)) {
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) o[dt][qt] *= alpha;
      }
    }

    if (__builtin_amdgcn_readfirstlane(flag) == t0) fix_tile(ti, st);
    __builtin_amdgcn_s_setprio(1);

    // P^T for 32-key step ks: lane keys 32 ks + 4 j + (0..3) then
    // 32 ks + 16 + 4 j + (0..3) (S^T tiles kt = 2 ks, 2 ks + 1); V^T rows of
    // the same keys come from two transpose reads (rows 32 ks + r keep the
    // swizzle of row r).
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const int off = 16 * ((2 * dt + ((lq & 3) >> 1)) ^ swv) + 8 * (lq & 1);
#pragma unroll
      for (int ks = 0; ks < KT32; ++ks) {
        const f16x4_t v0 = lds_read_tr(tv + (32 * ks + vrow) * kRowBytes + off);
        const f16x4_t v1 = lds_read_tr(tv + (32 * ks + vrow + 16) * kRowBytes + off);
        const f16x8_t va = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) o[dt][qt] = mfma16(va, ph[qt][ks], o[dt][qt]);
      }
    }
    __builtin_amdgcn_s_setprio(0);
  };

  if (tid < kHeadDim) {
    s_vscale[0][tid] = 1.f;
    s_vmax[tid] = 0u;
  }
  if (tid < kStages) s_flag[tid] = -1;
  lds_sync();
  // The Q operand has landed before the pipeline starts: no load that
  // writes registers is pending inside the loop, whose waits then only
  // follow the tile loads.
  __builtin_amdgcn_s_waitcnt(wait_vm(0));
  if (ntiles > 0) {
    // Pipeline start: page ids of tiles 0 .. 2 (waited for), then for tiles
    // i = 0 .. kStages - 2 the page id of tile i + 3 and the rows of tile i.
    if constexpr (kPaged) {
      issue_page(0);
      issue_page(1);
      issue_page(2);
      __builtin_amdgcn_s_waitcnt(wait_vm(0));
      compiler_fence();
    }
#pragma unroll
    for (int i = 0; i < kStages - 1; ++i) {
      issue_page(i + 3);
      issue(i);
    }
  }
  for (int ti = 0; ti < ntiles; ++ti) {
    const int st = ti & (kStages - 1);
    // This wave's rows of tile ti (and the page id of tile ti + 3) have
    // landed: convert its V pieces, then one barrier publishes the whole
    // tile. Every wave finished reading stage (ti - 1) % kStages before it,
    // so that stage takes tile ti + kStages - 1; phantom tiles past the end
    // read nothing (empty resources) and keep the load count per tile fixed.
    __builtin_amdgcn_s_waitcnt(kWaitTile);
    compiler_fence();
    convert(st, k0 + ti * kKT);
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    compiler_fence();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    issue_page(ti + kStages + 2);
    issue(ti + kStages - 1);
    if (k0 + ti * kKT + kKT > cut)
      tile(ti, st, std::true_type{});
    else
      tile(ti, st, std::false_type{});
  }
  // No load may still be writing LDS when the workgroup ends.
  __builtin_amdgcn_s_waitcnt(wait_vm(0));
  compiler_fence();

  // This split's normalised partial rows and their lse (log2 domain).
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    float lt = l[qt];
    lt += __shfl_xor(lt, 16);
    lt += __shfl_xor(lt, 32);
    const int rho = row_base + 16 * qt + lq;
    if (rho < R) {
      const float inv = lt > 0.f ? 1.f / lt : 0.f;
      const float l2 = lt > 0.f ? m[qt] + fast_log2(lt) : ninf;
      // With a single split (long windows, e.g. prefill) this is the final
      // row: it goes straight to out / lse and the combine is skipped.
      const size_t oi = ((size_t)bb * a.q_heads + (size_t)hk * G + rho % G) * f + rho / G;
      float* po = S == 1 ? a.out + oi * kHeadDim
                         : a.part_o + (((size_t)grp * S + split) * R + rho) * kHeadDim;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        f32x4_t y = o[dt][qt] * inv;
        if (scaled) {  // back to the values' own scale: times 2^E_d
#pragma unroll
          for (int i = 0; i < 4; ++i) y[i] *= 1.f / s_vscale[cur][16 * dt + 4 * j + i];
        }
        *reinterpret_cast<f32x4_t*>(po + 16 * dt + 4 * j) = y;
      }
      if (j == 0) {
        if (S > 1)
          a.part_lse[((size_t)grp * S + split) * R + rho] = l2;
        else if (a.lse)
          a.lse[oi] = lt > 0.f ? l2 * kLn2 : ninf;
      }
    }
  }

}

// Log-sum-exp merge of the splits (Alg. 2, "Combine") spread over many
// workgroups: each takes kCombineRows query rows of one group.
constexpr int kCombineRows = 8;

__global__ __launch_bounds__(256) void k_rectify_combine(RectifyArgs a) {
  __shared__ float s_w[kMaxRectSplits * kCombineRows];
  __shared__ f4_t s_red[256];
  const int grp = blockIdx.y;
  const int bb = grp / a.c.kv_heads, hk = grp % a.c.kv_heads;
  if (a.seq_mask != nullptr && a.seq_mask[bb] == 0) return;
  const int G = a.group, f = a.f, R = G * f, S = a.num_splits;
  const int rho0 = blockIdx.x * kCombineRows;
  const int rows = min(kCombineRows, R - rho0);
  if (rows <= 0) return;
  auto out_index = [&](int r) {
    const int rho = rho0 + r;
    return ((size_t)bb * a.q_heads + (size_t)hk * G + rho % G) * f + rho / G;
  };
  merge_splits<false>(a.part_o + ((size_t)grp * S * R + rho0) * kHeadDim, (size_t)R * kHeadDim,
               a.part_lse + (size_t)grp * S * R + rho0, (size_t)R, S, rows, s_w, s_red,
               [&](int r) { return a.out + out_index(r) * kHeadDim; },
               [&](int r, float v) { if (a.lse) a.lse[out_index(r)] = v; });
}

}  // namespace

int32_t rectify_num_qblocks(int32_t group, int32_t f) {
  const int rows = group * f;
  const int per = waves_for_rows(rows) * kRowsPerWave;
  return (rows + per - 1) / per;
}

// Key splits per group the attention aims for: about 512 workgroups in all.
static int64_t rectify_target_splits(int32_t batch, int32_t kv_heads, int32_t nqblk) {
  const int64_t wgs = (int64_t)batch * kv_heads * nqblk;
  const int64_t target = (512 + wgs - 1) / wgs;
  return target < 1 ? 1 : target;
}
// Short caches still fill the chip (4K, batch 1: 32 splits of 128 keys,
// 30.4 against 34.0 us per call with a 512-key minimum).
constexpr int kMinRectChunk = 128;

int32_t rectify_chunk(int32_t batch, int32_t kv_heads, int32_t nqblk, int32_t max_seq_len) {
  const int64_t target = rectify_target_splits(batch, kv_heads, nqblk);
  int64_t chunk = (max_seq_len + target - 1) / target;
  chunk = (chunk + kMaxKeyTile - 1) / kMaxKeyTile * kMaxKeyTile;
  if (chunk < kMinRectChunk) chunk = kMinRectChunk;
  // At most kMaxRectSplits splits, so the combine's weights fit in LDS.
  const int64_t least = ((int64_t)max_seq_len + kMaxRectSplits - 1) / kMaxRectSplits;
  if (chunk < least) chunk = (least + kMaxKeyTile - 1) / kMaxKeyTile * kMaxKeyTile;
  return (int32_t)chunk;
}

int32_t rectify_max_splits(int32_t batch, int32_t kv_heads, int32_t nqblk, int32_t max_seq_len) {
  // ceil(L / chunk) with chunk >= 128 and chunk >= ceil(L / target) (target
  // <= 512 < kMaxRectSplits): at most min(ceil(L / 128), target), a bound
  // that never decreases as L grows, while the split count itself can (the
  // chunk is rounded up to whole 64-key tiles: 512 splits at L = 65536, 342
  // at 65537 for one group and one query block).
  const int64_t by_len = ((int64_t)max_seq_len + kMinRectChunk - 1) / kMinRectChunk;
  const int64_t target = rectify_target_splits(batch, kv_heads, nqblk);
  const int64_t s = by_len < target ? by_len : target;
  return (int32_t)(s < 1 ? 1 : s);
}

hipError_t launch_rectify(const RectifyArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(k_rectify_rows, dim3((a.f + 15) / 16, a.c.batch * a.c.kv_heads), dim3(256), 0,
                     stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.refresh) {
    e = launch_summarize_tail(a.c, a.seq_lens, a.f, a.seq_mask, stream);
    if (e != hipSuccess) return e;
  }
  const int32_t nq = rectify_num_qblocks(a.group, a.f);
  const dim3 grid(a.num_splits, nq, a.c.batch * a.c.kv_heads);
  const bool paged = a.c.table != nullptr;
  if (waves_for_rows(a.group * a.f) == 8) {
    if (paged)
      hipLaunchKernelGGL((k_rectify_attn<8, true>), grid, dim3(512), 0, stream, a);
    else
      hipLaunchKernelGGL((k_rectify_attn<8, false>), grid, dim3(512), 0, stream, a);
  } else {
    if (paged)
      hipLaunchKernelGGL((k_rectify_attn<4, true>), grid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL((k_rectify_attn<4, false>), grid, dim3(256), 0, stream, a);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.num_splits == 1) return hipSuccess;  // the attention kernel wrote out / lse
  const int32_t rows = a.group * a.f;
  hipLaunchKernelGGL(k_rectify_combine, dim3((rows + kCombineRows - 1) / kCombineRows,
                     a.c.batch * a.c.kv_heads), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace resa
