// Max-IDF summaries of few sequences across many compute units (Section 3.1
// "Summary generation", Eq. 2; Appendix "Corpus-Level IDF Table" and
// "Max-IDF").
//
// The one-workgroup-per-sequence kernels (maxidf.hip) are bound by one
// compute unit's LDS instruction rate, so a batch of a few sequences leaves
// the chip idle.  This path splits each sequence over its blocks and its
// vocabulary, in three launches that communicate through a caller workspace:
//
//   presence  one workgroup per (sequence, block j): marks the block's ids in
//             an LDS bitmap (atomic OR) and copies it to the workspace as P_j
//             (bit t of word t / 32).  Every word of P_j is written, so
//             nothing needs clearing beforehand.
//   df        one thread per 32 ids: df(t) = sum_j P_j[t], counted with
//             bit-sliced adders over the N words (one counter bit per plane),
//             written as bytes to the workspace df table (and IDF = ln(N /
//             max(df, 1)) when asked).
//   select    one workgroup per (sequence, block): looks up the df of each id
//             of the block, takes each chunk's minimum (lane groups, then an
//             LDS minimum across wavefronts for chunks wider than 64 ids), and
//             one wavefront picks the top-k chunks (select_block).
//
// Workspace per sequence: N bitmaps of W = ceil(V / 32) words (padded to 32
// bytes), then the df table of 32 W bytes.
#include "summary.hpp"

namespace {

constexpr int kSplitThreads = 1024;
constexpr int kDfThreads = 256;
constexpr int kMaxidfSplitBatch = 16;  // beyond this, one workgroup per sequence is as fast
constexpr int kU = 8;                  // loads in flight per thread

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

// Block j of sequence b: its ids set bits of a zeroed LDS bitmap (atomic
// OR; bit t of word t / 32), which is then copied out as P_j.
__global__ __launch_bounds__(kSplitThreads) void split_presence_kernel(
    const int32_t* __restrict__ ids, int64_t L, int num_blocks, int Lb, int vocab,
    uint8_t* __restrict__ ws, int64_t seq_bytes) {
  extern __shared__ __attribute__((aligned(16))) uint32_t bm[];
  const int tid = threadIdx.x;
  const int64_t b = blockIdx.x / num_blocks;
  const int j = blockIdx.x - (int)(b * num_blocks);
  const int W = (int)split_words(vocab);
  const uint32_t vmax = (uint32_t)(vocab - 1);
  for (int w = tid; w < W; w += kSplitThreads) bm[w] = 0u;
  __syncthreads();
  const int32_t* seq = ids + b * L + (int64_t)j * Lb;
  // An id at or above vocab is the caller's error: clamped into the bitmap.
  // kU ids per thread are loaded together before their atomics.
  for (int x0 = 0; x0 < Lb; x0 += kU * kSplitThreads) {
    uint32_t t[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int x = x0 + u * kSplitThreads + tid;
      t[u] = x < Lb ? min((uint32_t)seq[x], vmax) : vmax + 1;
    }
#pragma unroll
    for (int u = 0; u < kU; ++u)
      if (t[u] <= vmax) atomicOr(&bm[t[u] >> 5], 1u << (t[u] & 31));
  }
  __syncthreads();
  uint32_t* bits = reinterpret_cast<uint32_t*>(ws + b * seq_bytes) + (int64_t)j * W;
  for (int w = tid; w < W; w += kSplitThreads) bits[w] = bm[w];
}

// df of ids 32g .. 32g+31 of sequence b from the N presence words: bit-sliced
// counters (plane p holds bit p of the 32 counts), then each count becomes a
// byte of the df table.
template <int P>
__global__ __launch_bounds__(kDfThreads) void split_df_kernel(int num_blocks, int vocab,
                                                              int slices, uint8_t* __restrict__ ws,
                                                              int64_t seq_bytes,
                                                              float* __restrict__ idf) {
  const int64_t b = blockIdx.x / slices;
  const int g = (blockIdx.x - (int)(b * slices)) * kDfThreads + threadIdx.x;
  const int W = (int)split_words(vocab);
  if (g >= W) return;
  uint8_t* seq_ws = ws + b * seq_bytes;
  const uint32_t* bits = reinterpret_cast<const uint32_t*>(seq_ws);
  uint32_t c[P];
#pragma unroll
  for (int p = 0; p < P; ++p) c[p] = 0u;
  // kU blocks' words are loaded together before they are added
  for (int j0 = 0; j0 < num_blocks; j0 += kU) {
    uint32_t w[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) w[u] = j0 + u < num_blocks ? bits[(int64_t)(j0 + u) * W + g] : 0u;
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      uint32_t carry = w[u];
#pragma unroll
      for (int p = 0; p < P; ++p) {
        const uint32_t t = c[p] & carry;
        c[p] ^= carry;
        carry = t;
      }
    }
  }
  // bytes 4r .. 4r+3 of the 32 counts: bit p of count 4r+q is bit 4r+q of
  // plane p; (nibble * 0x00204081) & 0x01010101 spreads a nibble's bits to
  // the low bits of four bytes
  u32x4 out[2];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    uint32_t v = 0;
#pragma unroll
    for (int p = 0; p < P; ++p) v |= (((c[p] >> (4 * r)) & 0xFu) * 0x00204081u & 0x01010101u) << p;
    out[r >> 2][r & 3] = v;
  }
  u32x4* df = reinterpret_cast<u32x4*>(seq_ws + split_bits_bytes(num_blocks, vocab)) + 2 * (int64_t)g;
  df[0] = out[0];
  df[1] = out[1];
  if (idf) {
    const float n = (float)num_blocks;
    float* dst = idf + b * vocab;
#pragma unroll
    for (int k = 0; k < 32; ++k) {
      const int t = 32 * g + k;
      const uint32_t d = (out[k >> 4][(k >> 2) & 3] >> (8 * (k & 3))) & 0xFFu;
      if (t < vocab) dst[t] = logf(n / (float)(d > 1u ? d : 1u));
    }
  }
}

// Block j of sequence b: the df of each id, each chunk's minimum, the top-k
// chunks.  Chunk c of the block is ids c*m .. c*m+m-1; lane groups of
// min(m, 64) lanes take their minimum, and chunks wider than a wavefront
// combine their groups with an LDS atomic minimum.
__global__ __launch_bounds__(kSplitThreads) void split_select_kernel(
    const int32_t* __restrict__ ids, int64_t L, int num_blocks, int Lb, int chunk_log2, int topk,
    int vocab, const uint8_t* __restrict__ ws, int64_t seq_bytes, int32_t* __restrict__ sel,
    int32_t* __restrict__ chunk_mindf) {
  extern __shared__ __attribute__((aligned(16))) uint32_t cmin[];  // [C]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int64_t b = blockIdx.x / num_blocks;
  const int j = blockIdx.x - (int)(b * num_blocks);
  const int C = Lb >> chunk_log2;
  const uint32_t vmax = (uint32_t)(vocab - 1);
  const uint8_t* df = ws + b * seq_bytes + split_bits_bytes(num_blocks, vocab);
  const int32_t* seq = ids + b * L + (int64_t)j * Lb;
  const int group = min(1 << chunk_log2, 64);
  const bool wide = chunk_log2 > 6;
  if (wide)
    for (int c = tid; c < C; c += kSplitThreads) cmin[c] = 0xFFFFFFFFu;
  __syncthreads();
  // kU ids per thread at a time: their loads, then their df lookups, are
  // issued together.  Every lane of a wavefront runs the same trip count, so
  // all join the cross-lane minimum; ids past the block read as df 255.
  for (int x0 = 0; x0 < Lb; x0 += kU * kSplitThreads) {
    uint32_t t[kU], d[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int x = x0 + u * kSplitThreads + tid;
      t[u] = x < Lb ? min((uint32_t)seq[x], vmax) : vmax + 1;
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) d[u] = t[u] <= vmax ? (uint32_t)df[t[u]] : 0xFFu;
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int x = x0 + u * kSplitThreads + tid;
      const uint32_t m = group_min(d[u], group);
      if (x < Lb && (x & (group - 1)) == 0) {
        const int c = x >> chunk_log2;
        if (wide) atomicMin(&cmin[c], m);
        else cmin[c] = m;
      }
    }
  }
  __syncthreads();
  if (chunk_mindf)
    for (int c = tid; c < C; c += kSplitThreads)
      chunk_mindf[(b * num_blocks + j) * C + c] = (int32_t)cmin[c];
  if (tid < 64 && topk > 0) {
    int32_t* dst = sel + (b * num_blocks + j) * topk;
    if (C <= 4 * 64)
      select_block<4>(cmin, C, (uint32_t)num_blocks, topk, dst, lane);
    else
      select_block<0>(cmin, C, (uint32_t)num_blocks, topk, dst, lane);
  }
}

}  // namespace

// Workspace of the split path, or 0 where the one-workgroup-per-sequence
// kernels serve (larger batches, shapes the split kernels do not take).
size_t maxidf_split_workspace(int batch, int64_t L, int num_blocks, int chunk, int vocab) {
  if (batch < 1 || batch > kMaxidfSplitBatch || L < 1 || num_blocks < 2 || num_blocks > 255 ||
      vocab < 1 || chunk < 4 || chunk > 256 || L % num_blocks != 0)
    return 0;
  const int64_t Lb = L / num_blocks;
  if (Lb % chunk != 0 || Lb / chunk > 16384 || L >= ((int64_t)1 << 31)) return 0;
  if (split_words(vocab) * 4 > PULSAR_LDS_BYTES) return 0;  // the presence bitmap
  return (size_t)(batch * split_seq_bytes(num_blocks, vocab));
}

int launch_maxidf_split(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk,
                        int topk, int vocab, int32_t* sel, int32_t* chunk_mindf, float* idf,
                        void* workspace, hipStream_t stream) {
  int chunk_log2 = 0;
  while ((1 << chunk_log2) < chunk) ++chunk_log2;
  const int Lb = (int)(L / num_blocks);
  const int64_t seq_bytes = split_seq_bytes(num_blocks, vocab);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  const int64_t grid = (int64_t)batch * num_blocks;
  const size_t tab = (size_t)split_words(vocab) * 4;
  if (hipFuncSetAttribute((const void*)split_presence_kernel,
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)tab) != hipSuccess)
    return PULSAR_EHIP;
  hipLaunchKernelGGL(split_presence_kernel, dim3((unsigned)grid), dim3(kSplitThreads), tab, stream,
                     ids, L, num_blocks, Lb, vocab, ws, seq_bytes);
  if (hipGetLastError() != hipSuccess) return PULSAR_EHIP;
  const int slices = (int)((split_words(vocab) + kDfThreads - 1) / kDfThreads);
  const dim3 dgrid((unsigned)(batch * slices));
  // counter planes: enough bits for num_blocks (<= 255)
  if (num_blocks < 16)
    hipLaunchKernelGGL(split_df_kernel<4>, dgrid, dim3(kDfThreads), 0, stream, num_blocks, vocab,
                       slices, ws, seq_bytes, idf);
  else if (num_blocks < 32)
    hipLaunchKernelGGL(split_df_kernel<5>, dgrid, dim3(kDfThreads), 0, stream, num_blocks, vocab,
                       slices, ws, seq_bytes, idf);
  else
    hipLaunchKernelGGL(split_df_kernel<8>, dgrid, dim3(kDfThreads), 0, stream, num_blocks, vocab,
                       slices, ws, seq_bytes, idf);
  if (hipGetLastError() != hipSuccess) return PULSAR_EHIP;
  const size_t cl = (size_t)(Lb >> chunk_log2) * 4;
  if (hipFuncSetAttribute((const void*)split_select_kernel,
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)cl) != hipSuccess)
    return PULSAR_EHIP;
  hipLaunchKernelGGL(split_select_kernel, dim3((unsigned)grid), dim3(kSplitThreads), cl, stream,
                     ids, L, num_blocks, Lb, chunk_log2, topk, vocab, ws, seq_bytes, sel,
                     chunk_mindf);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}
