// Layout of the split (many workgroups per sequence) summary path's
// workspace, shared by the Max-IDF (maxidf_split.hip) and scorer
// (scorers.hip) kernels.  Per sequence: N presence bitmaps of
// W = ceil(V / 32) words (padded to 32 bytes), then the df table of 32 W
// bytes (a byte per id, or the nibble df - 1 per id for N <= 16).
#pragma once

#include "summary.hpp"

constexpr int kSplitThreads = 1024;

__host__ __device__ inline int64_t split_words(int vocab) { return ((int64_t)vocab + 31) / 32; }
__host__ __device__ inline int64_t split_df_bytes(int vocab) { return split_words(vocab) * 32; }
// the bitmaps, padded to 32 bytes so that the df table (and the next
// sequence) stays 32-byte aligned
__host__ __device__ inline int64_t split_bits_bytes(int num_blocks, int vocab) {
  return ((int64_t)num_blocks * split_words(vocab) * 4 + 31) & ~int64_t(31);
}
__host__ __device__ inline int64_t split_seq_bytes(int num_blocks, int vocab) {
  return split_bits_bytes(num_blocks, vocab) + split_df_bytes(vocab);
}

// Copy of n 16-byte units (K rounds of kSplitThreads, n > (K - 1) *
// kSplitThreads) from global memory into LDS: all K loads are issued before
// the first store.  Lanes past the end copy the last unit onto itself, so no
// lane branches on its own load or store.
template <int K>
__device__ __forceinline__ void copy_rounds(const uint4* __restrict__ src, uint4* dst, int n,
                                            int tid) {
  uint4 r[K];
#pragma unroll
  for (int k = 0; k < K; ++k) r[k] = src[min(k * kSplitThreads + tid, n - 1)];
#pragma unroll
  for (int k = 0; k < K; ++k) dst[min(k * kSplitThreads + tid, n - 1)] = r[k];
}

// The same for any n up to PULSAR_LDS_BYTES / 16 units (10 rounds).
__device__ __forceinline__ void copy_to_lds(const uint4* __restrict__ src, uint4* dst, int n,
                                            int tid) {
  static_assert(PULSAR_LDS_BYTES / 16 / kSplitThreads == 10, "copy rounds below");
  switch ((n + kSplitThreads - 1) / kSplitThreads) {
    case 1: copy_rounds<1>(src, dst, n, tid); break;
    case 2: copy_rounds<2>(src, dst, n, tid); break;
    case 3: copy_rounds<3>(src, dst, n, tid); break;
    case 4: copy_rounds<4>(src, dst, n, tid); break;
    case 5: copy_rounds<5>(src, dst, n, tid); break;
    case 6: copy_rounds<6>(src, dst, n, tid); break;
    case 7: copy_rounds<7>(src, dst, n, tid); break;
    case 8: copy_rounds<8>(src, dst, n, tid); break;
    case 9: copy_rounds<9>(src, dst, n, tid); break;
    default: copy_rounds<10>(src, dst, n, tid); break;
  }
}

// The presence and df kernels of the split path for a batch that
// maxidf_split_workspace admits: the workspace's df table of every sequence
// (nibbles for N <= 16, else bytes), and the IDF table if idf is given.
int launch_split_df(const int32_t* ids, int batch, int64_t L, int num_blocks, int vocab,
                    float* idf, void* workspace, hipStream_t stream);
