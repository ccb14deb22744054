// Group block-sparse flash-decoding (Eq. 2; App. A, Alg. 2) for gfx950:
// grid (num_splits, kv_heads, batch), one split per workgroup of 4 waves
// (decode_split).
#include "decode_impl.h"

namespace resa {
namespace {

constexpr int kDecodeWaves = 4;

// Chunks in flight per wave while one is consumed: one. Measured on MI355X
// with 256 workgroups streaming at once, fewer bytes in flight make the
// launch faster (depth 1 / 2 / 3 / 4: 41.1 / 41.7 / 42.4 / 43.0 us at 64K,
// 19.6 / 20.2 / 20.7 / 21.3 us at 256K; depth 0: 41.8 / 19.7 us): the memory
// system serves fewer, shorter queues better than it hides a longer wait.
constexpr int kDecodeDepth = 1;

template <int G, int BS>
__global__ __launch_bounds__(64 * kDecodeWaves) void k_decode(DecodeArgs a) {
  __shared__ DecodeLds<G, kDecodeWaves> lds;
  decode_split<G, BS, kDecodeWaves, false, kDecodeDepth>(a, blockIdx.z, blockIdx.y, blockIdx.x, a.seq_lens,
                                                         false, lds);
}

template <int G>
hipError_t launch_g(const DecodeArgs& a, hipStream_t stream) {
  dim3 grid(a.num_splits, a.c.kv_heads, a.c.batch);
  switch (a.c.block_size) {
    case 16: hipLaunchKernelGGL((k_decode<G, 16>), grid, dim3(64 * kDecodeWaves), 0, stream, a); break;
    case 32: hipLaunchKernelGGL((k_decode<G, 32>), grid, dim3(64 * kDecodeWaves), 0, stream, a); break;
    case 64: hipLaunchKernelGGL((k_decode<G, 64>), grid, dim3(64 * kDecodeWaves), 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int32_t decode_auto_splits(int32_t batch, int32_t kv_heads, int32_t n_cap, int32_t block_size) {
  const int64_t groups = (int64_t)batch * kv_heads;
  const int64_t chunks = (int64_t)n_cap * (block_size / kChunk);
  // About one workgroup per CU (256 CUs), with at least one chunk per wave.
  // Measured on MI355X: more splits than that lose to fewer, longer-running
  // workgroups at 64K and 256K (4 and 32 splits); small groups gain from the
  // full count (4K, batch 1: 16 splits 9.1 us against 11.5 us with 4, the
  // earlier cap of four chunks per wave).
  int64_t s = (256 + groups - 1) / groups;
  const int64_t most = chunks / kDecodeWaves;
  if (s > most) s = most;
  if (s > 256) s = 256;
  if (s < 1) s = 1;
  return (int32_t)s;
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  switch (a.group) {
    case 1: return launch_g<1>(a, stream);
    case 2: return launch_g<2>(a, stream);
    case 3: return launch_g<3>(a, stream);
    case 4: return launch_g<4>(a, stream);
    case 5: return launch_g<5>(a, stream);
    case 6: return launch_g<6>(a, stream);
    case 7: return launch_g<7>(a, stream);
    case 8: return launch_g<8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace resa
