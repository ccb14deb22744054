// Group block-sparse flash-decoding (Eq. 2; App. A, Alg. 2) for gfx950.
//
// Device code shared by the decode kernel and the fused decode step. The
// selected blocks of a (sequence, kv head) group are cut into 16-token chunks
// and the chunks are dealt to num_splits splits one by one (split s takes
// chunk slots s, s + S, ...); wave w of a split's workgroup of NW waves takes
// the split's slots w, w + NW, ..., with kDepth chunks' loads in flight per
// wave while one is consumed.
//
// Lane layout inside a wave: lane = 16 * r + c. Lane (r, c) owns dims
// [8c, 8c + 8) of the chunk's rows r, r + 4, r + 8, r + 12, for K and for V,
// so every wave-wide 16-byte load covers four consecutive 256-byte rows
// (1 KiB contiguous) and one chunk is 4 K loads + 4 V loads per lane.
// q.k partial sums use v_dot2 on bf16 pairs, then a 16-lane DPP reduction.
// Each row group r keeps its own online-softmax state (running max m, sum l,
// accumulator over its 8 dims) for the g query heads of the group, in the
// log2 domain; the row groups and waves of a workgroup are merged by
// log-sum-exp through LDS, and the split holding the last ticket of its group
// merges the others' published partials with its own (a single split writes
// the output directly).
#pragma once

#include <utility>

#include "resa_device.h"
#include "resa_internal.h"

namespace resa {
namespace {


constexpr int kIdxBatch = 1024;  // chunk start tokens staged in LDS per pass
constexpr int kMaxSplits = 256;  // splits per group (bounded by the host)

// One 16-token chunk of K and V for this lane: four K rows (in the lane's
// permuted order) and V rows r, r+4, r+8, r+12.
struct Chunk {
  U4 k[4], v[4];
};

// The chunk's rows from row row0 on (wave-uniform) of the K and V arrays at
// kp / vp (wave-uniform): non-temporal buffer loads over the chunk's 4 KB of
// each, at the lane's offset loff (elements) into a row. The resource base
// is a scalar sum and the offsets 32-bit (measured 0.3 – 0.7 us per launch
// faster than 64-bit global addressing at 64K and 256K, and 1 – 2 us faster
// in the persistent step kernel).
__device__ __forceinline__ void load_chunk(Chunk& ch, const uint16_t* kp, const uint16_t* vp,
                                           const int (&krow)[4], int row0, int loff) {
  constexpr int kBytes = kChunk * kHeadDim * 2;
  const size_t base = (size_t)row0 * kHeadDim;
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(kp + base), (short)0, kBytes, kBufWord3);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(vp + base), (short)0, kBytes, kBufWord3);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ch.k[i] = __builtin_bit_cast(U4, __builtin_amdgcn_raw_buffer_load_b128(
                                         rk, (uint32_t)((krow[i] * kHeadDim + loff) * 2), 0, kPolicyNt));
    ch.v[i] = __builtin_bit_cast(U4, __builtin_amdgcn_raw_buffer_load_b128(
                                         rv, (uint32_t)((4 * i * kHeadDim + loff) * 2), 0, kPolicyNt));
  }
}

// Heads padded to GP (4 or 8), so a row group's 4 rows x GP heads are 16 or
// 32 values: one or two per lane after the transpose-reduce.
template <int G>
struct Pad {
  static constexpr int GP = G <= 4 ? 4 : 8;
};

// Per-lane online-softmax state: after the transpose-reduce lane c of a row
// group owns head c % GP, so m and l are one value per lane.
struct Soft {
  float m, l;
};

// The softmax reference m of a head moves only when a chunk's maximum cm
// exceeds it by more than kRefSlack (log2 domain): weights stay <= 2^kRefSlack
// and the accumulator rescale (returned factor != 1) is rare. The output is
// normalised by l under the same reference, so the result does not depend on
// where m sits.
constexpr float kRefSlack = 8.f;

__device__ __forceinline__ float move_ref(float& m, float cm) {
  if (cm > m + kRefSlack) {
    const float alpha = fast_exp2(m - cm);  // 0 when m was -inf
    m = cm;
    return alpha;
  }
  return 1.f;
}

// One chunk for this lane's row group (rows r + 4i of the chunk).
//   logits: v_dot2 over the lane's 8 dims for 4 rows x GP heads, laid out so
//           that slot s holds value n = s ^ c (n = row * GP + head), then one
//           transpose-reduce leaves lane c with the logit of value n = c
//           (and n = c + 16 when GP = 8);
//   softmax: max and sum over the 4 rows of a head by row rotations, one
//           exp per value instead of one per value and lane;
//   P.V: p and the rescale factor are broadcast from the owning lanes, and
//        every lane updates its 8 dims of the g heads.
// Rows with token >= L, every row of an invalid chunk (t0 < 0) and padded
// heads are excluded.
template <int G>
__device__ __forceinline__ void consume_chunk(const Chunk& ch, int t0, int r, int c, int L,
                                              float scale, const uint32_t (&q)[Pad<G>::GP][4],
                                              Soft& st, float (&acc)[G][8]) {
  constexpr int GP = Pad<G>::GP;
  const float ninf = -__builtin_inff();
  float val[4 * GP];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int h = 0; h < GP; ++h) {
      float d = dot2_bf16(q[h][0], ch.k[i].x, 0.f);
      d = dot2_bf16(q[h][1], ch.k[i].y, d);
      d = dot2_bf16(q[h][2], ch.k[i].z, d);
      d = dot2_bf16(q[h][3], ch.k[i].w, d);
      val[i * GP + h] = d;
    }
  }
#pragma unroll
  for (int u = 0; u < GP / 4; ++u) transpose_reduce16(val + 16 * u);

  const int head = c & (GP - 1);
  float ab[G], pb[4][G], ab_own;
  if constexpr (GP == 4) {
    const int row = c >> 2;
    const bool ok = t0 >= 0 && t0 + r + 4 * row < L && head < G;
    const float x = ok ? val[0] * scale : ninf;
    float cm = fmaxf(x, dpp<kDppRor4>(x));
    cm = fmaxf(cm, dpp<kDppRor8>(cm));
    const float alpha = move_ref(st.m, cm);
    ab_own = alpha;
    const float mref = st.m == ninf ? 0.f : st.m;
    const float p = fast_exp2(x - mref);
    float ps = p + dpp<kDppRor4>(p);
    ps += dpp<kDppRor8>(ps);
    st.l = fmaf(st.l, alpha, ps);
    [&]<int... H>(std::integer_sequence<int, H...>) {
      ((ab[H] = dpp<kDppBcast0 + H>(alpha)), ...);
      ((pb[0][H] = dpp<kDppBcast0 + H>(p)), ...);
      ((pb[1][H] = dpp<kDppBcast0 + 4 + H>(p)), ...);
      ((pb[2][H] = dpp<kDppBcast0 + 8 + H>(p)), ...);
      ((pb[3][H] = dpp<kDppBcast0 + 12 + H>(p)), ...);
    }(std::make_integer_sequence<int, G>{});
  } else {
    const int row0 = c >> 3;  // rows row0 and row0 + 2
    const bool ok0 = t0 >= 0 && t0 + r + 4 * row0 < L && head < G;
    const bool ok1 = t0 >= 0 && t0 + r + 4 * (row0 + 2) < L && head < G;
    const float x0 = ok0 ? val[0] * scale : ninf;
    const float x1 = ok1 ? val[16] * scale : ninf;
    float cm = fmaxf(x0, x1);
    cm = fmaxf(cm, dpp<kDppRor8>(cm));
    const float alpha = move_ref(st.m, cm);
    ab_own = alpha;
    const float mref = st.m == ninf ? 0.f : st.m;
    const float p0 = fast_exp2(x0 - mref);
    const float p1 = fast_exp2(x1 - mref);
    float ps = p0 + p1;
    ps += dpp<kDppRor8>(ps);
    st.l = fmaf(st.l, alpha, ps);
    [&]<int... H>(std::integer_sequence<int, H...>) {
      ((ab[H] = dpp<kDppBcast0 + H>(alpha)), ...);
      ((pb[0][H] = dpp<kDppBcast0 + H>(p0)), ...);
      ((pb[1][H] = dpp<kDppBcast0 + 8 + H>(p0)), ...);
      ((pb[2][H] = dpp<kDppBcast0 + H>(p1)), ...);
      ((pb[3][H] = dpp<kDppBcast0 + 8 + H>(p1)), ...);
    }(std::make_integer_sequence<int, G>{});
  }

  // Rescale only when some running max moved (alpha == 1 exactly otherwise);
  // after the first chunks of a split that is rare, and the test is uniform.
  if (__any(ab_own != 1.f)) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int d = 0; d < 8; ++d) acc[h][d] *= ab[h];
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float v[8];
    v[0] = bf_lo(ch.v[i].x); v[1] = bf_hi(ch.v[i].x);
    v[2] = bf_lo(ch.v[i].y); v[3] = bf_hi(ch.v[i].y);
    v[4] = bf_lo(ch.v[i].z); v[5] = bf_hi(ch.v[i].z);
    v[6] = bf_lo(ch.v[i].w); v[7] = bf_hi(ch.v[i].w);
#pragma unroll
    for (int h = 0; h < G; ++h) {
#pragma unroll
      for (int d = 0; d < 8; ++d) acc[h][d] = fmaf(pb[i][h], v[d], acc[h][d]);
    }
  }
}

// Merge of a group's S split partials by its last workgroup (Alg. 2,
// "Combine"), in one round of loads: every thread issues its lse loads (kept
// in LDS) and its 128-bit partial loads together, all with agent scope
// (buffer loads with the sc1 policy, bounds-checked by the buffer size). The
// merging workgroup's own split (`own`) never went to memory: its partial and
// lse are read from LDS. Float4 column u of head r = u / 32 gets
// T = NT / (32 G) threads, each summing splits ph, ph + T, ...; the T sums
// are added through LDS.
constexpr int kTailBatch = 16;    // partial loads per thread per round

template <int G, int NT, bool kOpaque>
__device__ void merge_tail(const DecodeArgs& a, size_t grp, int S, int own, size_t ob,
                           const float* own_o, const float* own_l, float* s_lse, f4_t* s_red) {
  constexpr int U = G * (kHeadDim / 4);
  constexpr int T = U >= NT ? 1 : NT / U;
  constexpr int kLse = (kMaxSplits * G + NT - 1) / NT;
  const int tid = tid_of<kOpaque>();
  const float ninf = -__builtin_inff();
  const float* pl = wave_uniform(a.part_lse + grp * S * (size_t)G);
  const float* po = wave_uniform(a.part_o + grp * S * (size_t)(G * kHeadDim));
  const __amdgpu_buffer_rsrc_t rl = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(pl), (short)0, S * G * 4, kBufWord3);
  const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(po), (short)0, S * G * kHeadDim * 4, kBufWord3);

  // Every load is unconditional, so no pending load shares a register with
  // an LDS read on another path (which would serialise the loads): offsets
  // past the buffer read 0 through its range check, and the own split's slot
  // (stale) is replaced by its LDS copy once the values are used.
  constexpr int kOut = 0x7fffffff;  // an offset past every buffer
  uint32_t lraw[kLse];
#pragma unroll
  for (int j = 0; j < kLse; ++j) {
    const int i = tid + NT * j;
    lraw[j] = __builtin_amdgcn_raw_buffer_load_b32(rl, i < S * G ? i * 4 : kOut, 0, kSc1);
  }
  const bool active = tid < U * T;
  const int u = tid % U, ph = tid / U, r = u / (kHeadDim / 4), c4 = u % (kHeadDim / 4);
  const int nb = (S + T * kTailBatch - 1) / (T * kTailBatch);
  const f4_t own_v = *reinterpret_cast<const f4_t*>(own_o + r * kHeadDim + 4 * c4);
  f4_t part[kTailBatch];
  auto issue = [&](int b) {
#pragma unroll
    for (int k = 0; k < kTailBatch; ++k) {
      const int sp = b * T * kTailBatch + k * T + ph;
      // The builtins return integer types: reinterpret the bits, never convert.
      part[k] = __builtin_bit_cast(f4_t, __builtin_amdgcn_raw_buffer_load_b128(
                    ro, active && sp < S ? ((sp * G + r) * kHeadDim + 4 * c4) * 4 : kOut, 0, kSc1));
    }
  };
  issue(0);
  float lreg[kLse];
#pragma unroll
  for (int j = 0; j < kLse; ++j) {
    const int i = tid + NT * j;
    lreg[j] = i >= S * G ? ninf : i / G == own ? own_l[i % G] : __builtin_bit_cast(float, lraw[j]);
  }
  // lse of split sp, head h at s_lse[h * SP + sp] (SP = S rounded up to 4,
  // padded with -inf), so each head's values are contiguous: after one
  // barrier every thread reads its head's S values (broadcast 16-byte reads)
  // and forms the weights itself, with no further barrier.
  const int SP = (S + 3) & ~3;
#pragma unroll
  for (int j = 0; j < kLse; ++j) {
    const int i = tid + NT * j;
    if (i < S * G) s_lse[(i % G) * SP + i / G] = lreg[j];
    else if (i < SP * G) s_lse[(i % G) * SP + i / G] = ninf;
  }
  lds_sync();
  const f4_t* lh = reinterpret_cast<const f4_t*>(s_lse + r * SP);
  float mx = ninf;
  for (int v = 0; v < SP / 4; ++v) {
    const f4_t x = lh[v];
    mx = fmaxf(fmaxf(mx, fmaxf(x.x, x.y)), fmaxf(x.z, x.w));
  }
  float wsum = 0.f;
  if (mx != ninf)
    for (int v = 0; v < SP / 4; ++v) {
      const f4_t x = lh[v];
      wsum += fast_exp2(x.x - mx) + fast_exp2(x.y - mx) + fast_exp2(x.z - mx) + fast_exp2(x.w - mx);
    }
  f4_t acc = {0.f, 0.f, 0.f, 0.f};
  for (int b = 0; b < nb; ++b) {
    if (b > 0) issue(b);
#pragma unroll
    for (int k = 0; k < kTailBatch; ++k) {
      const int sp = b * T * kTailBatch + k * T + ph;
      if (active && sp < S) {
        const float l = s_lse[r * SP + sp];
        acc += (l == ninf ? 0.f : fast_exp2(l - mx)) * (sp == own ? own_v : part[k]);
      }
    }
  }
  acc *= wsum > 0.f ? 1.f / wsum : 0.f;
  if constexpr (T > 1) {
    s_red[tid] = acc;
    lds_sync();
    if (active && ph == 0) {
#pragma unroll
      for (int k = 1; k < T; ++k) acc += s_red[tid + k * U];
    }
  }
  if (active && ph == 0) {
    *reinterpret_cast<f4_t*>(a.out + (ob + r) * kHeadDim + 4 * c4) = acc;
    if (c4 == 0 && a.lse) a.lse[ob + r] = wsum > 0.f ? (mx + fast_log2(wsum)) * kLn2 : ninf;
  }
}

// Wave-wide maximum and sum (every lane active; every lane gets the result):
// the 16 lanes of each row by DPP, then the rows by lane swaps.
__device__ __forceinline__ float wave_max_f(float x) {
  x = fmaxf(x, dpp<kDppXor1>(x));
  x = fmaxf(x, dpp<kDppXor2>(x));
  x = fmaxf(x, dpp<kDppHalfMirror>(x));
  x = fmaxf(x, dpp<kDppMirror>(x));
  return max_xor32(max_xor16(x));
}
__device__ __forceinline__ float wave_sum_f(float x) { return sum_xor32(sum_xor16(row16_sum(x))); }

// Alg. 2, "Combine", for one query head h of the group, by one of the G
// merging workgroups of a group with many splits (each takes one head, so
// each loads 1 / G of the partials). Thread i < S forms split i's weight
// 2^(lse_i - max) once (wave maxima and sums through LDS: two barriers);
// float4 column u of the head gets T = NT / 32 threads, each summing splits
// ph, ph + T, ...; the T sums are added through LDS. The merging split's
// own partial and lse are read from LDS. s_w holds kMaxSplits + 2 NT / 64
// floats.
template <int G, int NT>
__device__ void merge_head(const DecodeArgs& a, size_t grp, int S, int own, int h, size_t ob,
                           const float* own_o, const float* own_l, float* s_w, f4_t* s_red) {
  constexpr int U = kHeadDim / 4;
  constexpr int T = NT / U;
  constexpr int NWv = NT / 64;
  static_assert(NT % U == 0 && NT >= kMaxSplits, "merge_head shape");
  constexpr int kOut = 0x7fffffff;  // an offset past every buffer
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float ninf = -__builtin_inff();
  const float* pl = wave_uniform(a.part_lse + grp * S * (size_t)G);
  const float* po = wave_uniform(a.part_o + grp * S * (size_t)(G * kHeadDim));
  const __amdgpu_buffer_rsrc_t rl = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(pl), (short)0, S * G * 4, kBufWord3);
  const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(po), (short)0, S * G * kHeadDim * 4, kBufWord3);
  // Every load is unconditional (offsets past the buffer read 0), and the
  // own split's slot is replaced by its LDS copy when used.
  const uint32_t lraw = __builtin_amdgcn_raw_buffer_load_b32(rl, tid < S ? (tid * G + h) * 4 : kOut, 0, kSc1);
  const int u = tid % U, ph = tid / U;
  const int nb = (S + T * kTailBatch - 1) / (T * kTailBatch);
  const f4_t own_v = *reinterpret_cast<const f4_t*>(own_o + h * kHeadDim + 4 * u);
  f4_t part[kTailBatch];
  auto issue = [&](int b) {
#pragma unroll
    for (int k = 0; k < kTailBatch; ++k) {
      const int sp = b * T * kTailBatch + k * T + ph;
      part[k] = __builtin_bit_cast(f4_t, __builtin_amdgcn_raw_buffer_load_b128(
                    ro, sp < S ? ((sp * G + h) * kHeadDim + 4 * u) * 4 : kOut, 0, kSc1));
    }
  };
  issue(0);
  const float l = tid >= S ? ninf : tid == own ? own_l[h] : __builtin_bit_cast(float, lraw);
  float* s_max = s_w + kMaxSplits;
  float* s_sum = s_max + NWv;
  const float wm = wave_max_f(l);
  if (lane == 0) s_max[wave] = wm;
  lds_sync();
  float mx = s_max[0];
#pragma unroll
  for (int w = 1; w < NWv; ++w) mx = fmaxf(mx, s_max[w]);
  const float wt = l == ninf ? 0.f : fast_exp2(l - mx);
  if (tid < kMaxSplits) s_w[tid] = wt;
  const float ws = wave_sum_f(wt);
  if (lane == 0) s_sum[wave] = ws;
  lds_sync();
  float wsum = s_sum[0];
#pragma unroll
  for (int w = 1; w < NWv; ++w) wsum += s_sum[w];
  f4_t acc = {0.f, 0.f, 0.f, 0.f};
  for (int b = 0; b < nb; ++b) {
    if (b > 0) issue(b);
#pragma unroll
    for (int k = 0; k < kTailBatch; ++k) {
      const int sp = b * T * kTailBatch + k * T + ph;
      if (sp < S) acc += s_w[sp] * (sp == own ? own_v : part[k]);
    }
  }
  acc *= wsum > 0.f ? 1.f / wsum : 0.f;
  s_red[tid] = acc;
  lds_sync();
  if (ph == 0) {
#pragma unroll
    for (int k = 1; k < T; ++k) acc += s_red[tid + k * U];
    *reinterpret_cast<f4_t*>(a.out + (ob + h) * kHeadDim + 4 * u) = acc;
    if (u == 0 && a.lse) a.lse[ob + h] = wsum > 0.f ? (mx + fast_log2(wsum)) * kLn2 : ninf;
  }
}

// LDS of one split: per-wave softmax states for the wave merge, the staged
// chunk list, and the merge of the splits.
// Row-group states kept for the merge of the waves: all four row groups of
// each wave (RG = 4) or, for 8-wave workgroups, whose LDS is shared with the
// selection, the two pairs left by one lane swap (RG = 2).
template <int NW>
constexpr int kRowGroups = NW <= 4 ? 4 : 2;

// Entry e = w RG + r holds accumulator racc[w][r][h][:] and, per head h, its
// softmax reference rm[h][e] and sum rl[h][e] (contiguous per head).
template <int G, int NW>
struct DecodeLds {
  static constexpr int RG = kRowGroups<NW>;
  __attribute__((aligned(16))) float racc[NW][RG][G][kHeadDim];
  __attribute__((aligned(16))) float rm[G][NW * RG];
  __attribute__((aligned(16))) float rl[G][NW * RG];
  __attribute__((aligned(16))) float own_o[G * kHeadDim];   // the merging split's own partial
  float own_l[G];
  int tok[kIdxBatch];
  int row[kIdxBatch];
  __attribute__((aligned(16))) float w[kMaxSplits * G];
  f4_t red[64 * NW];
  uint32_t ticket;
};

// Bound of a merging split's wait for the other splits' flags (each poll
// sleeps about 64 cycles): the splits it waits for have taken their tickets
// and are finishing, so the bound is only a guard.
constexpr uint32_t kFlagSpins = 1u << 22;
// Splits from which the combine is spread over G merging workgroups, one
// query head each (merge_head), instead of done by the last one alone.
constexpr int kSpreadSplits = 16;

template <bool kCoherent>
__device__ __forceinline__ int ld_i32(const int32_t* p) {
  if constexpr (kCoherent) return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else return *p;
}


// Split `split` of group (bb, hk) by a workgroup of NW waves: wave w takes
// chunks c0 + w, c0 + w + NW, ... of the split's range. The group's length
// is lens[bb]; with `append` (the fused step) a sequence below capacity has
// one more token, appended in the same launch at row lens[bb], whose row is
// taken from a.k_new / a.v_new instead of the cache. kCoherent: the ids and
// the count were written by another workgroup of the same launch (agent-scope
// loads; also selects the opaque thread index of the persistent kernel).
// Every workgroup of the group writes its partial (several splits) and the
// last one to finish merges them; returns true in the workgroup that wrote
// the group's output. `empty`: the split decodes no chunk (it still takes
// part in the merge).
//
// Start-up: the count, the length, the query rows and the first pass's ids
// are all requested before anything waits for one of them (vector loads, so
// one wait covers them), which leaves one memory round trip between the
// kernel arguments and the first K / V loads.
template <int G, int BS, int NW, bool kCoherent, int kDepth>
__device__ __forceinline__ bool decode_split(const DecodeArgs& a, int bb, int hk, int split,
                                             const int32_t* lens, bool append, DecodeLds<G, NW>& lds,
                                             bool empty = false) {
  constexpr int GP = Pad<G>::GP;
  constexpr int CPB = BS / kChunk;  // chunks per block
  constexpr int NT = 64 * NW;
  constexpr int kPer = kIdxBatch / NT;  // ids per thread per pass
  const int tid = tid_of<kCoherent>();
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int S = a.num_splits;
  const size_t grp = (size_t)bb * a.c.kv_heads + hk;
  // The group's n_cap * CPB chunk slots are dealt to the splits one by one
  // (split s holds slots s, s + S, s + 2 S, ...), so the id loads do not wait
  // for the count n and any n leaves the splits balanced to one chunk (runs
  // of several slots per split left up to a run's difference, 14 % of a
  // split at 256K). Slots at or past n * CPB are skipped.
  auto slot_of = [&](int i) { return i * S + split; };
  auto count_below = [&](int T) {  // this split's slots below slot T
    return T > split ? (T - split + S - 1) / S : 0;
  };
  const int slots = count_below(a.n_cap * CPB);
  const int r = lane >> 4, c = lane & 15, col = c * 8;
  const int32_t* idx = a.block_idx + grp * a.n_cap;
  int blkv[kPer];
  auto load_ids = [&](int cb) {
    const int lim = min(slots, cb + kIdxBatch) - cb;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = tid + j * NT;
      blkv[j] = i < lim ? ld_i32<kCoherent>(idx + slot_of(cb + i) / CPB) : -1;
    }
  };
  load_ids(0);

  // Lane c's registers hold K row i ^ rperm and query head h ^ hperm, so
  // that logit slot s = i * GP + h is value n = s ^ c (see transpose_reduce16).
  const int hperm = c & (GP - 1);
  const int rperm = GP == 4 ? (c >> 2) & 3 : (c >> 3) & 1;
  int krow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) krow[i] = 4 * (i ^ rperm);
  uint32_t q[GP][4];
#pragma unroll
  for (int h = 0; h < GP; ++h) {
    const int head = h ^ hperm;
    U4 t = U4{0, 0, 0, 0};
    if (head < G) t = ld16(a.q + ((size_t)bb * a.q_heads + (size_t)hk * G + head) * kHeadDim + col);
    q[h][0] = t.x;
    q[h][1] = t.y;
    q[h][2] = t.z;
    q[h][3] = t.w;
  }
  // Contiguous layout: chunk rows are counted from the group's first row;
  // paged layout: from the start of the pool (the page's row is staged).
  const bool paged = a.c.table != nullptr;
  const size_t gbase = paged ? 0 : grp * (size_t)a.c.capacity * kHeadDim;
  const uint16_t* kp = wave_uniform(a.c.k + gbase);
  const uint16_t* vp = wave_uniform(a.c.v + gbase);
  const int loff = r * kHeadDim + col;  // this lane's element offset into a chunk row group
  const float scale = a.scale_log2;
  const float ninf = -__builtin_inff();
  // The count and the length are requested last: the first use of either
  // (a move into scalar registers) then waits for everything above at once.
  const int n_raw = ld_i32<true>(a.num_sel + grp);
  const int L0 = ld_i32<true>(lens + bb);
  // Calls of this group merged so far: tags this call's ready flags.
  // Requested with the count and the length (unconditionally: behind a
  // branch the compiler would move it into a scalar register, and so wait
  // for it, right there); nothing uses it before the tail.
  uint32_t epoch = __hip_atomic_load(a.epochs + grp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const bool app = append && L0 >= 0 && L0 < a.c.capacity;
  const int L = app ? L0 + 1 : L0;
  const int pos = app ? L0 : -1;
  const int M = min((L + BS - 1) / BS, a.c.max_blocks);
  const int n = empty ? 0 : max(0, min(n_raw, a.n_cap));
  const int C = n * CPB;
  const int valid = count_below(C);

  Soft st{ninf, 0.f};
  float acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int d = 0; d < 8; ++d) acc[h][d] = 0.f;

  // The first pass's ids were requested above; later passes (only while
  // slots with chunks remain) request theirs first thing.
  int cb = 0;
  do {
    if (cb > 0) load_ids(cb);
    const int ce = min(valid, cb + kIdxBatch);
    const int lim = min(slots, cb + kIdxBatch) - cb;
    // First token of each chunk of this pass (-1 for ids outside [0, M) and
    // for slots past the count) and the row holding it (0 for an invalid
    // chunk: in bounds, masked out). Paged: every table entry of the pass is
    // requested before any is used.
    int tk[kPer], rw[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = tid + j * NT;
      const int cc = slot_of(cb + i);
      const int blk = blkv[j];
      tk[j] = (i >= lim || cb + i >= valid || blk < 0 || blk >= M) ? -1 : blk * BS + (cc % CPB) * kChunk;
      rw[j] = tk[j];
    }
    if (paged) {
      int page[kPer];
#pragma unroll
      for (int j = 0; j < kPer; ++j)
        page[j] = tk[j] >= 0 ? a.c.table[(size_t)bb * a.c.max_blocks + blkv[j]] : -1;
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        const int cc = slot_of(cb + tid + j * NT);
        if (tk[j] >= 0) {
          if ((unsigned)page[j] < (unsigned)a.c.num_pages)
            rw[j] = (page[j] * a.c.kv_heads + hk) * BS + (cc % CPB) * kChunk;
          else
            tk[j] = -1;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = tid + j * NT;
      if (i < lim) {
        lds.tok[i] = tk[j];
        lds.row[i] = tk[j] < 0 ? 0 : rw[j];
      }
    }
    lds_sync();
    // Wave w takes slots cb + w, cb + w + W, ... (W waves). A ring of
    // kDepth + 1 chunk buffers keeps kDepth chunks' loads in flight while one
    // is consumed; an invalid chunk inside the pass reads row 0 (in bounds)
    // and is masked out entirely, and nothing is loaded past the pass. The
    // scheduling barriers keep the refills ahead of the compute.
    auto tok = [&](int cc) -> int { return cc < ce ? __builtin_amdgcn_readfirstlane(lds.tok[cc - cb]) : -1; };
    // The chunk holding token pos (appended in this launch) takes that row
    // from k_new / v_new: lane row r + 4 iv of the chunk is K slot iv ^ rperm
    // and V slot iv.
    auto patch = [&](Chunk& ch, int t0) {
      if (pos >= 0 && t0 >= 0 && pos >= t0 && pos < t0 + kChunk) {
        const int rr = pos - t0;
        if ((rr & 3) == r) {
          const U4 kn = ld16(a.k_new + grp * kHeadDim + col);
          const U4 vn = ld16(a.v_new + grp * kHeadDim + col);
          const int iv = rr >> 2;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (i == (iv ^ rperm)) ch.k[i] = kn;
            if (i == iv) ch.v[i] = vn;
          }
        }
      }
    };
    auto row_of = [&](int cc) -> int { return cc < ce ? __builtin_amdgcn_readfirstlane(lds.row[cc - cb]) : 0; };
    Chunk ring[kDepth + 1];
    int tring[kDepth + 1];
    int cc = cb + wave;
#pragma unroll
    for (int k = 0; k <= kDepth; ++k) {
      tring[k] = tok(cc + k * NW);
      if (cc + k * NW < ce) {  // no loads past the pass
        load_chunk(ring[k], kp, vp, krow, row_of(cc + k * NW), loff);
        patch(ring[k], tring[k]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    while (cc < ce) {
#pragma unroll
      for (int k = 0; k <= kDepth; ++k) {
        if (cc < ce) {
          consume_chunk<G>(ring[k], tring[k], r, c, L, scale, q, st, acc);
          __builtin_amdgcn_sched_barrier(0);
          tring[k] = tok(cc + (kDepth + 1) * NW);
          if (cc + (kDepth + 1) * NW < ce) {
            load_chunk(ring[k], kp, vp, krow, row_of(cc + (kDepth + 1) * NW), loff);
            patch(ring[k], tring[k]);
          }
          __builtin_amdgcn_sched_barrier(0);
          cc += NW;
        }
      }
    }
    lds_sync();
    cb += kIdxBatch;
  } while (cb < valid);

  // Tail. With several splits, one thread takes the split's ticket first:
  // its round trip overlaps the merge of the waves below. The ticket only
  // orders the splits' ends; the merging split(s) (below) wait for the
  // others' ready flags (their partials are in memory then) and merge.
  // Every K / V load of the loop has been consumed here; the compiler cannot
  // see that (refills are conditional), so without this explicit wait it
  // would place waits in the merge below that also cover the ticket.
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  const bool single = S == 1;
  uint32_t ticket = 0;
  if (!single && tid == 0)
    ticket = __hip_atomic_fetch_add(a.counters + grp, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  // Per-head state of this lane's row group: head h lives in lane 16 r + h
  // (a DPP row broadcast). With RG = 2, row groups r and r + 2 (lanes l and
  // l + 32) merge through one lane swap first. Every kept row-group state
  // goes to LDS.
  constexpr int RG = kRowGroups<NW>;
  constexpr int NE = NW * RG;
  float m_[G], l_[G];
  [&]<int... H>(std::integer_sequence<int, H...>) {
    ((m_[H] = dpp<kDppBcast0 + H>(st.m)), ...);
    ((l_[H] = dpp<kDppBcast0 + H>(st.l)), ...);
  }(std::make_integer_sequence<int, G>{});
  if constexpr (RG == 2) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mx = max_xor32(m_[h]);
      const float w = (m_[h] == ninf) ? 0.f : fast_exp2(m_[h] - mx);
      m_[h] = mx;
      l_[h] = sum_xor32(l_[h] * w);
#pragma unroll
      for (int d = 0; d < 8; ++d) acc[h][d] = sum_xor32(acc[h][d] * w);
    }
  }
  if (r < RG) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      f4_t* dst = reinterpret_cast<f4_t*>(&lds.racc[wave][r][h][col]);
      dst[0] = f4_t{acc[h][0], acc[h][1], acc[h][2], acc[h][3]};
      dst[1] = f4_t{acc[h][4], acc[h][5], acc[h][6], acc[h][7]};
    }
    if (c == 0) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        lds.rm[h][wave * RG + r] = m_[h];
        lds.rl[h][wave * RG + r] = l_[h];
      }
    }
  }
  lds_sync();

  // Merge the NE = 16 row-group states: this split's normalised partial and
  // its lse (log2 domain) for items it = tid + k NT of two dims each (head
  // it / 64, dims 2 (it % 64) ..). A wave's items share one head: each
  // 16-lane row holds the head's 16 states (lane e: state e), takes their
  // maximum and the weighted sum of l with DPP, and the 16 weights reach
  // every lane as wave-uniform values (one exp per lane, not 16).
  static_assert(NE == 16, "one row-group state per lane of a 16-lane row");
  constexpr int NT2 = 64 * NW;
  constexpr int kItems = (G * 64 + NT2 - 1) / NT2;
  f2_t val[kItems];
  float lg[kItems];
#pragma unroll
  for (int k = 0; k < kItems; ++k) {
    const int it = tid + k * NT2;
    val[k] = f2_t{0.f, 0.f};
    lg[k] = ninf;
    if (k * NT2 + wave * 64 < G * 64) {  // uniform across the wave
      const int h = it / 64, d = 2 * (it % 64), e0 = lane & 15;
      const float me = lds.rm[h][e0], le = lds.rl[h][e0];
      float mx = me;
      mx = fmaxf(mx, dpp<kDppXor1>(mx));
      mx = fmaxf(mx, dpp<kDppXor2>(mx));
      mx = fmaxf(mx, dpp<kDppHalfMirror>(mx));
      mx = fmaxf(mx, dpp<kDppMirror>(mx));
      const float fe = me == ninf ? 0.f : fast_exp2(me - mx);
      const float lsum = row16_sum(le * fe);
      f2_t x = {0.f, 0.f};
#pragma unroll
      for (int e = 0; e < NE; ++e) {
        const float f = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, fe), e));
        x += f * *reinterpret_cast<const f2_t*>(&lds.racc[e / RG][e % RG][h][d]);
      }
      if (lsum > 0.f) {
        val[k] = x * (1.f / lsum);
        lg[k] = mx + fast_log2(lsum);
      }
    }
  }
  const size_t ob = (size_t)bb * a.q_heads + (size_t)hk * G;
  if (single) {
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
      const int it = tid + k * NT2;
      if (it < G * 64) {
        *reinterpret_cast<f2_t*>(a.out + ob * kHeadDim + 2 * it) = val[k];
        if (it % 64 == 0 && a.lse) a.lse[ob + it / 64] = lg[k] == ninf ? ninf : lg[k] * kLn2;
      }
    }
    return true;
  }
  if (tid == 0) lds.ticket = ticket;
  lds_sync();
  // The call count read at the start is first used here: it stays in a
  // vector register until now, so no earlier instruction waits for it.
  __asm__ volatile("" : "+v"(epoch));
  // Merging splits: the one holding the last ticket, or with many splits
  // those holding the last G tickets, one query head each. A ready flag
  // carries this call's tag (the group's merged-call count + 1, and S), so
  // flags left by earlier calls never match and no flag is ever reset; the
  // split holding the last ticket returns the ticket counter to zero and
  // advances the count once every ticket is taken.
  const uint32_t tk = lds.ticket;
  const bool spread = !kCoherent && G >= 2 && S >= kSpreadSplits && S >= G;
  const uint32_t first = spread ? (uint32_t)(S - G) : (uint32_t)(S - 1);
  const uint64_t tag = ((uint64_t)(epoch + 1u) << 32) | (uint32_t)S;
  if (spread || tk < first) {
    // Publish: agent-scope stores write through to the level every L2 slice
    // reads (sc1), every thread waits for their acknowledgement, then one
    // thread raises the split's ready flag.
    float* po = a.part_o + (grp * S + split) * (size_t)(G * kHeadDim);
    float* pl = a.part_lse + (grp * S + split) * (size_t)G;
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
      const int it = tid + k * NT2;
      if (it < G * 64) {
        __hip_atomic_store(po + 2 * it, val[k].x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(po + 2 * it + 1, val[k].y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (it % 64 == 0) __hip_atomic_store(pl + it / 64, lg[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) __hip_atomic_store(a.flags + grp * S + split, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (tk < first) return false;
  }

  // Alg. 2, "Combine", in a merging split: its own partial stays in LDS;
  // every other split has taken its ticket and is publishing (or has), so
  // thread t < S waits for split t's flag (agent-scope loads), then the
  // partials are read with agent-scope loads and merged.
#pragma unroll
  for (int k = 0; k < kItems; ++k) {
    const int it = tid + k * NT2;
    if (it < G * 64) {
      *reinterpret_cast<f2_t*>(&lds.own_o[2 * it]) = val[k];
      if (it % 64 == 0) lds.own_l[it / 64] = lg[k];
    }
  }
  if (tid < S && tid != split) {
    const uint64_t* fl = a.flags + grp * S + tid;
    uint32_t spins = 0;
    while (__hip_atomic_load(fl, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != tag && ++spins < kFlagSpins)
      __builtin_amdgcn_s_sleep(1);
  }
  __syncthreads();
  if constexpr (!kCoherent && G >= 2) {
    if (spread)
      merge_head<G, 64 * NW>(a, grp, S, split, (int)(tk - first), ob, lds.own_o, lds.own_l, lds.w, lds.red);
    else
      merge_tail<G, 64 * NW, kCoherent>(a, grp, S, split, ob, lds.own_o, lds.own_l, lds.w, lds.red);
  } else {
    merge_tail<G, 64 * NW, kCoherent>(a, grp, S, split, ob, lds.own_o, lds.own_l, lds.w, lds.red);
  }
  const bool last = tk == (uint32_t)(S - 1);
  if (last && tid == 0) {
    __hip_atomic_store(a.counters + grp, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(a.epochs + grp, epoch + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  return last;
}

}  // namespace
}  // namespace resa
