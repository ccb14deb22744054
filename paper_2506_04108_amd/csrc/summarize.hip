// Block key summaries (Eq. 3), the per-token append with online summary
// update (Alg. 1), and the workspace clear kernel.
#include "resa_device.h"
#include "resa_internal.h"

namespace resa {
namespace {

// One wave summarises one block: lane (r, c) with r = lane / 16 and
// c = lane % 16 reads dims [8c, 8c + 8) of rows r, r + 4, ... of the block,
// so each wave-wide load covers four whole 256-byte rows (1 KiB contiguous).
//
// With rel_f > 0 the range is per sequence: blocks floor((L - rel_f) / b) ..
// M - 1, i.e. every block holding one of the last rel_f rows (rectify
// refresh); a sequence whose seq_mask entry is 0 is skipped (seq_mask may be
// null: every sequence).
template <int BS>
__global__ __launch_bounds__(256) void k_summarize(CacheArgs c, const int32_t* __restrict__ seq_lens,
                                                   int32_t blk_begin, int32_t blk_end, int32_t rel_f,
                                                   const int32_t* __restrict__ seq_mask) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int hk = blockIdx.y, bb = blockIdx.z;
  if (seq_mask != nullptr && seq_mask[bb] == 0) return;
  const int L = seq_lens[bb];
  if (rel_f > 0) {
    if (L < rel_f) return;
    blk_begin = (L - rel_f) / BS;
  }
  const int m = blk_begin + blockIdx.x * 4 + wave;
  const int M = (L + BS - 1) / BS;
  int end = blk_end < 0 ? M : min(blk_end, M);
  end = min(end, c.max_blocks);
  if (m >= end) return;

  const int r = lane >> 4, col = (lane & 15) * 8;
  const size_t grp = (size_t)bb * c.kv_heads + hk;
  const int64_t row0 = kv_row(c, bb, hk, m * BS);  // a block never straddles pages
  if (row0 < 0) return;
  const uint16_t* kb = c.k + (size_t)row0 * kHeadDim + col;
  float mn[8], mx[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    mn[j] = __builtin_inff();
    mx[j] = -__builtin_inff();
  }
  U4 rows[BS / 4];
#pragma unroll
  for (int i = 0; i < BS / 4; ++i) rows[i] = ld16(kb + (size_t)(r + 4 * i) * kHeadDim);
#pragma unroll
  for (int i = 0; i < BS / 4; ++i) {
    if (m * BS + r + 4 * i < L) {
      const uint32_t w[4] = {rows[i].x, rows[i].y, rows[i].z, rows[i].w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        mn[2 * j] = fminf(mn[2 * j], bf_lo(w[j]));
        mn[2 * j + 1] = fminf(mn[2 * j + 1], bf_hi(w[j]));
        mx[2 * j] = fmaxf(mx[2 * j], bf_lo(w[j]));
        mx[2 * j + 1] = fmaxf(mx[2 * j + 1], bf_hi(w[j]));
      }
    }
  }
  // Combine the four row groups (lanes c, c+16, c+32, c+48 hold the same dims).
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    mn[j] = fminf(mn[j], __shfl_xor(mn[j], 16));
    mx[j] = fmaxf(mx[j], __shfl_xor(mx[j], 16));
    mn[j] = fminf(mn[j], __shfl_xor(mn[j], 32));
    mx[j] = fmaxf(mx[j], __shfl_xor(mx[j], 32));
  }
  if (r == 0) {
    const size_t so = (grp * c.max_blocks + m) * kHeadDim + col;
    st16(c.kmin + so, U4{pack_exact(mn[0], mn[1]), pack_exact(mn[2], mn[3]),
                         pack_exact(mn[4], mn[5]), pack_exact(mn[6], mn[7])});
    st16(c.kmax + so, U4{pack_exact(mx[0], mx[1]), pack_exact(mx[2], mx[3]),
                         pack_exact(mx[4], mx[5]), pack_exact(mx[6], mx[7])});
  }
}

// One workgroup per sequence; wave w handles kv heads w, w + 4, ...
// Lanes 0-15 write the key row and update its block summary, lanes 16-31 the value row.
__global__ __launch_bounds__(256) void k_append(CacheArgs c, const uint16_t* __restrict__ k_new,
                                                const uint16_t* __restrict__ v_new,
                                                int32_t* __restrict__ seq_lens) {
  __shared__ int s_pos;
  const int bb = blockIdx.x;
  if (threadIdx.x == 0) s_pos = seq_lens[bb];
  __syncthreads();
  const int pos = s_pos;
  if (pos < 0 || pos >= c.capacity) return;  // uniform across the workgroup
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = (lane & 15) * 8;
  for (int hk = wave; hk < c.kv_heads; hk += 4) {
    const size_t grp = (size_t)bb * c.kv_heads + hk;
    const int64_t kr = kv_row(c, bb, hk, pos);
    if (kr < 0) continue;  // page outside the pool: nothing is written
    const size_t row = (size_t)kr * kHeadDim + col;
    const size_t src = grp * kHeadDim + col;
    if (lane < 16) {
      const U4 kv = ld16(k_new + src);
      st16(const_cast<uint16_t*>(c.k) + row, kv);
      const int m = pos / c.block_size;
      const size_t so = (grp * c.max_blocks + m) * kHeadDim + col;
      if (pos % c.block_size == 0) {
        st16(c.kmin + so, kv);
        st16(c.kmax + so, kv);
      } else {
        st16(c.kmin + so, u4_min(ld16(c.kmin + so), kv));
        st16(c.kmax + so, u4_max(ld16(c.kmax + so), kv));
      }
    } else if (lane < 32) {
      st16(const_cast<uint16_t*>(c.v) + row, ld16(v_new + src));
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) seq_lens[bb] = pos + 1;
}

__global__ void k_clear(uint8_t* p, size_t bytes) {
  const size_t n16 = bytes / 16;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    st16(p + 16 * i, U4{0, 0, 0, 0});
  const size_t tail = bytes - 16 * n16;
  if (blockIdx.x == 0 && threadIdx.x < tail) p[16 * n16 + threadIdx.x] = 0;
}

}  // namespace

static hipError_t summarize_grid(const CacheArgs& c, const int32_t* seq_lens, int32_t blk_begin,
                                 int32_t blk_end, int32_t rel_f, const int32_t* seq_mask, int32_t nblk,
                                 hipStream_t stream) {
  if (nblk <= 0) return hipSuccess;
  dim3 grid((nblk + 3) / 4, c.kv_heads, c.batch);
  switch (c.block_size) {
    case 16: hipLaunchKernelGGL(k_summarize<16>, grid, dim3(256), 0, stream, c, seq_lens, blk_begin, blk_end, rel_f, seq_mask); break;
    case 32: hipLaunchKernelGGL(k_summarize<32>, grid, dim3(256), 0, stream, c, seq_lens, blk_begin, blk_end, rel_f, seq_mask); break;
    case 64: hipLaunchKernelGGL(k_summarize<64>, grid, dim3(256), 0, stream, c, seq_lens, blk_begin, blk_end, rel_f, seq_mask); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_summarize(const CacheArgs& c, const int32_t* seq_lens, int32_t blk_begin,
                            int32_t blk_end, hipStream_t stream) {
  const int32_t last = blk_end < 0 ? c.max_blocks : blk_end;
  return summarize_grid(c, seq_lens, blk_begin, blk_end, 0, nullptr, last - blk_begin, stream);
}

hipError_t launch_summarize_tail(const CacheArgs& c, const int32_t* seq_lens, int32_t f,
                                 const int32_t* seq_mask, hipStream_t stream) {
  // Rows [L - f, L) touch at most ceil(f / b) + 1 blocks.
  const int32_t nblk = (f + c.block_size - 1) / c.block_size + 1;
  return summarize_grid(c, seq_lens, 0, -1, f, seq_mask, nblk, stream);
}

hipError_t launch_append(const CacheArgs& c, const uint16_t* k_new, const uint16_t* v_new,
                         int32_t* seq_lens, hipStream_t stream) {
  hipLaunchKernelGGL(k_append, dim3(c.batch), dim3(256), 0, stream, c, k_new, v_new, seq_lens);
  return hipGetLastError();
}

hipError_t launch_clear(void* p, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return hipSuccess;
  size_t n16 = bytes / 16 + 1;
  unsigned blocks = (unsigned)((n16 + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_clear, dim3(blocks), dim3(256), 0, stream, (uint8_t*)p, bytes);
  return hipGetLastError();
}

}  // namespace resa
