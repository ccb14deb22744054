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
// 16-row tiles). A workgroup walks its key
// range in tiles of 64 keys: K and V rows go from registers (loaded one tile
// ahead) into one of two LDS buffers, row-major, so one barrier per tile
// separates filling a buffer from reading it. Per tile and wave:
//   S^T = K . Q^T        (keys x queries; lane l holds query l % 16 and keys
//                          16 kt + 4 (l / 16) + i)
//   online softmax per query row in the log2 domain against a reference
//   that moves only in steps of more than 2^8, so P lies in [0, 2^8]; P is
//   rounded to fp16 (11 significant bits)
//   O^T += V^T . P^T     (dims x queries, fp16 MFMA; the contraction index is
//                          ordered so that P^T is already in the B-operand
//                          layout, and V^T comes from the row-major V tile
//                          through the LDS transpose read)
// V tiles are converted from bf16 to fp16 on their way into LDS, each head
// dimension d multiplied by a power of two 2^-E_d first (E_d = 0 until a
// value needs it). Every bf16 value of magnitude 2^-14 .. 65280 is an fp16
// value (8 significant bits fit in 11), so in that range the conversion is
// exact; smaller values keep fp16's subnormal spacing of 2^-24 (an error of at
// most 2^-24 * P per key). A thread that finds a scaled value above 65504
// flags the tile; on a flagged tile every wave reloads the tile's V, raises
// E_d of the dimensions that need it (so that max |v| 2^-E_d < 2^16),
// multiplies those accumulator rows by the change, and converts the tile
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
constexpr int kKeyTile = 64;
constexpr int kStride = kHeadDim + 8;    // bf16 per K or V row in LDS (272 B, 16-B aligned)
constexpr int kTileElems = kKeyTile * kStride;
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
__device__ __forceinline__ f16x4_t lds_read_tr(const uint16_t* p) {
  typedef __attribute__((address_space(3))) i16x4_t lds_i16x4;
  const i16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_i16x4*)(const_cast<uint16_t*>(p)));
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

template <int kWaves>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_rectify_attn(RectifyArgs a) {
  constexpr int kRowsPerWg = rows_per_wg<kWaves>();
  constexpr int kThreads = 64 * kWaves;
  constexpr int kPieces = kKeyTile * 16 / kThreads;  // 16-byte pieces of K (and of V) per thread per tile
  constexpr int kRowStep = kThreads / 16;           // tile rows covered by one pass of the threads
  __shared__ __attribute__((aligned(16))) uint16_t sK[2][kTileElems];
  __shared__ __attribute__((aligned(16))) uint16_t sV[2][kTileElems];
  // V range handling: s_flag[buf] = first key of the tile in buffer buf when
  // one of its scaled values is above the fp16 range (else an older tile's
  // key, or -1); s_vscale[cur][d] = 2^-E_d; s_vmax[d] = max |v| of dimension
  // d over a flagged tile (fp32 bits: non-negative values order as integers).
  __shared__ int s_flag[2];
  __shared__ __attribute__((aligned(16))) float s_vscale[2][kHeadDim];
  __shared__ uint32_t s_vmax[kHeadDim];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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

  // Thread tid moves 16-byte pieces tid + kThreads e (e < kPieces) of a
  // tile's K and V: key (tid + kThreads e) / 16, dims 8 (tid % 16) .. + 8.
  const int part = tid & 15;
  U4 rk[kPieces], rv[kPieces];
  // Cache rows of the next tile to load. With a block table they are looked
  // up one load ahead (gload(t0) loads tile t0 and looks up tile t0 + 64, the
  // next one loaded), so the table read is not on the path of the data loads.
  int64_t nrow[kPieces];
  auto lookup = [&](int t0) {
#pragma unroll
    for (int e = 0; e < kPieces; ++e) {
      const int kk = t0 + (tid >> 4) + kRowStep * e;
      nrow[e] = kk < k1 ? kv_row(a.c, bb, hk, kk) : -1;
    }
  };
  auto gload = [&](int t0) {
#pragma unroll
    for (int e = 0; e < kPieces; ++e) {
      if (nrow[e] >= 0) {
        rk[e] = ld16_stream(a.c.k + (size_t)nrow[e] * kHeadDim + part * 8);
        rv[e] = ld16_stream(a.c.v + (size_t)nrow[e] * kHeadDim + part * 8);
      } else {
        rk[e] = U4{0, 0, 0, 0};
        rv[e] = U4{0, 0, 0, 0};
      }
    }
    lookup(t0 + kKeyTile);
  };
  // V scale state, uniform across the workgroup: `scaled` once any E_d > 0,
  // `cur` the current half of s_vscale.
  bool scaled = false;
  int cur = 0;
  // Converts a 16-byte piece of V (8 bf16 values of dims part*8 ..) to fp16,
  // times the per-dimension factors when `scaled`; vmax collects the largest
  // scaled magnitude.
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
  // Stores the loaded tile (first key `tag`) into buffer buf; a thread with a
  // scaled V value outside the fp16 range flags the tile.
  auto lstore = [&](int buf, int tag) __attribute__((always_inline)) {
    float sc[8];
    if (scaled) {
#pragma unroll
      for (int i = 0; i < 8; ++i) sc[i] = s_vscale[cur][part * 8 + i];
    }
    float vmax = 0.f;
#pragma unroll
    for (int e = 0; e < kPieces; ++e) {
      const int off = ((tid >> 4) + kRowStep * e) * kStride + part * 8;
      st16(&sK[buf][off], rk[e]);
      st16(&sV[buf][off], scaled ? to_h8(rv[e], sc, true, vmax) : to_h8(rv[e], sc, false, vmax));
    }
    if (!(vmax <= 65504.f)) s_flag[buf] = tag;
  };
  // A flagged tile (uniform: every wave reads the same flag). The tile's V is
  // reloaded, the per-dimension maxima are gathered, E_d rises where
  // max |v| 2^-E_d would reach 2^16, the accumulator rows of those dimensions
  // follow, and the tile is converted again into its buffer.
  auto fix_tile = [&](int t0, int buf) __attribute__((always_inline)) {
    U4 vv[kPieces];
#pragma unroll
    for (int e = 0; e < kPieces; ++e) {
      const int kk = t0 + (tid >> 4) + kRowStep * e;
      const int64_t row = kk < k1 ? kv_row(a.c, bb, hk, kk) : -1;
      vv[e] = row >= 0 ? ld16(a.c.v + (size_t)row * kHeadDim + part * 8) : U4{0, 0, 0, 0};
    }
    float dm[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int e = 0; e < kPieces; ++e) {
      const float x[8] = {bf_lo(vv[e].x), bf_hi(vv[e].x), bf_lo(vv[e].y), bf_hi(vv[e].y),
                          bf_lo(vv[e].z), bf_hi(vv[e].z), bf_lo(vv[e].w), bf_hi(vv[e].w)};
#pragma unroll
      for (int i = 0; i < 8; ++i) dm[i] = fmaxf(dm[i], fabsf(x[i]));
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) atomicMax(&s_vmax[part * 8 + i], __float_as_uint(dm[i]));
    lds_sync();
    float ns[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t mb = s_vmax[part * 8 + i];
      // max |v| < 2^(ex + 1); E = ex - 15 keeps the scaled maximum below 2^16.
      const int ex = (int)((mb >> 23) & 0xff) - 127;
      const int E = ex > 15 ? ex - 15 : 0;
      ns[i] = fminf(s_vscale[cur][part * 8 + i], __uint_as_float((uint32_t)(127 - E) << 23));
    }
    if (tid < 16) {  // part == tid: one thread per 8 dimensions publishes them
#pragma unroll
      for (int i = 0; i < 8; ++i) s_vscale[cur ^ 1][part * 8 + i] = ns[i];
    }
    float unused = 0.f;
#pragma unroll
    for (int e = 0; e < kPieces; ++e) {
      const int off = ((tid >> 4) + kRowStep * e) * kStride + part * 8;
      st16(&sV[buf][off], to_h8(vv[e], ns, true, unused));
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

  // One tile: scores, softmax update, P.V. kMasked evaluates the causal cut
  // and the split end per key.
  auto tile = [&](int t0, int buf, auto masked) {
    constexpr bool kMasked = decltype(masked)::value;
    const uint16_t* tk = sK[buf];
    const uint16_t* tv = sV[buf];
    const int flag = s_flag[buf];  // read now, used after the scores
    f32x4_t sacc[4][2];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) sacc[kt][qt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const bf16x8_t ka = *reinterpret_cast<const bf16x8_t*>(&tk[(16 * kt + lq) * kStride + 32 * s + 8 * j]);
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) sacc[kt][qt] = mfma16(ka, qb[qt][s], sacc[kt][qt]);
      }
    }

    f16x8_t ph[2][2];  // [qt][32-key step]
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      float x[16];
      float tmax = ninf;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
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
      // the normalisation by l uses the same reference. A query's 64 keys
      // sit in four lanes (lq + 16 j): the row maximum across them is only
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
      for (int e = 0; e < 16; ++e) {
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

    if (__builtin_amdgcn_readfirstlane(flag) == t0) fix_tile(t0, buf);

    // P^T for 32-key step ks: lane keys 32 ks + 4 j + (0..3) then
    // 32 ks + 16 + 4 j + (0..3) (S^T tiles kt = 2 ks, 2 ks + 1); V^T rows of
    // the same keys come from two transpose reads.
    const int tr_key = 4 * j + (lq >> 2), tr_dim = 4 * (lq & 3);
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const f16x4_t v0 = lds_read_tr(&tv[(32 * ks + tr_key) * kStride + 16 * dt + tr_dim]);
        const f16x4_t v1 = lds_read_tr(&tv[(32 * ks + 16 + tr_key) * kStride + 16 * dt + tr_dim]);
        const f16x8_t va = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) o[dt][qt] = mfma16(va, ph[qt][ks], o[dt][qt]);
      }
    }
  };

  if (k0 < k1) {
    lookup(k0);
    gload(k0);
  }
  if (tid < kHeadDim) {
    s_vscale[0][tid] = 1.f;
    s_vmax[tid] = 0u;
  }
  if (tid < 2) s_flag[tid] = -1;
  lds_sync();
  if (k0 < k1) {
    lstore(0, k0);
    if (k0 + kKeyTile < k1) gload(k0 + kKeyTile);
    lds_sync();
  }
  int buf = 0;
  for (int t0 = k0; t0 < k1; t0 += kKeyTile) {
    if (t0 + kKeyTile > cut)
      tile(t0, buf, std::true_type{});
    else
      tile(t0, buf, std::false_type{});
    // The other buffer was last read in the previous tile, before the
    // barrier that ended it: fill it with the next tile, start the loads of
    // the one after, and publish.
    if (t0 + kKeyTile < k1) lstore(buf ^ 1, t0 + kKeyTile);
    if (t0 + 2 * kKeyTile < k1) gload(t0 + 2 * kKeyTile);
    lds_sync();
    buf ^= 1;
  }

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
constexpr int kCombineRows = 2;

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

int32_t rectify_chunk(int32_t batch, int32_t kv_heads, int32_t nqblk, int32_t max_seq_len) {
  const int64_t wgs = (int64_t)batch * kv_heads * nqblk;
  int64_t target = (512 + wgs - 1) / wgs;
  if (target < 1) target = 1;
  int64_t chunk = (max_seq_len + target - 1) / target;
  chunk = (chunk + kKeyTile - 1) / kKeyTile * kKeyTile;
  if (chunk < 512) chunk = 512;
  // At most kMaxRectSplits splits, so the combine's weights fit in LDS.
  const int64_t least = ((int64_t)max_seq_len + kMaxRectSplits - 1) / kMaxRectSplits;
  if (chunk < least) chunk = (least + kKeyTile - 1) / kKeyTile * kKeyTile;
  return (int32_t)chunk;
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
  if (waves_for_rows(a.group * a.f) == 8)
    hipLaunchKernelGGL(k_rectify_attn<8>, grid, dim3(512), 0, stream, a);
  else
    hipLaunchKernelGGL(k_rectify_attn<4>, grid, dim3(256), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.num_splits == 1) return hipSuccess;  // the attention kernel wrote out / lse
  const int32_t rows = a.group * a.f;
  hipLaunchKernelGGL(k_rectify_combine, dim3((rows + kCombineRows - 1) / kCombineRows,
                     a.c.batch * a.c.kv_heads), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace resa
