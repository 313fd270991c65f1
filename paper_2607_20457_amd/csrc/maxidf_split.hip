// Max-IDF summaries of few sequences across many compute units (Section 3.1
// "Summary generation", Eq. 2; Appendix "Corpus-Level IDF Table" and
// "Max-IDF").
//
// The one-workgroup-per-sequence kernels (maxidf.hip) are bound by one
// compute unit's LDS instruction rate, so a batch of a few sequences leaves
// the chip idle.  This path splits each sequence over its blocks and its
// vocabulary, in three launches that communicate through a caller workspace:
//
//   presence  one workgroup per (sequence, block j, vocabulary slice): the
//             block's ids in the slice write a 1 into a zeroed LDS table of
//             one byte per id (repeated ids write the same value, so plain
//             byte stores suffice; LDS atomic OR serialises on them), which
//             is packed into the slice's words of P_j (bit t of word t / 32).
//             Small batches take more slices, so that clearing and packing
//             the tables is short; every slice reads the block's ids.  Every
//             word of P_j is written, so nothing needs clearing beforehand.
//   df        one thread per 32 ids: df(t) = sum_j P_j[t], counted with
//             bit-sliced adders over the N words (one counter bit per plane),
//             written to the workspace df table: nibbles df - 1 for N <= 16,
//             else bytes (and IDF = ln(N / max(df, 1)) when asked).
//   select    one workgroup per (sequence, block): copies the df table into
//             LDS when it fits there, looks up the df of each id of the
//             block, takes each chunk's minimum (over the lane's 8 ids, then
//             its lane group), and one wavefront picks the top-k chunks
//             (select_block).
//
// A thread's id loads carry no bounds branch (a lane past the block re-reads
// its last ids), so all of them are in flight at once: with a branch around
// each load the compiler waits for each in turn.
//
// Workspace per sequence: N bitmaps of W = ceil(V / 32) words (padded to 32
// bytes), then the df table of 32 W bytes (16 W of them used by nibbles).
#include <algorithm>

#include "split.hpp"

namespace {

constexpr int kDfThreads = 256;
constexpr int kMaxidfSplitBatch = 16;  // beyond this, one workgroup per sequence is as fast
constexpr int kU = 8;                  // loads in flight per thread

// Block j of sequence b (blockIdx.x = b N + j), vocabulary slice
// s = blockIdx.y (words [s Ws, (s + 1) Ws) of the bitmap), with a byte per
// id: the block's ids in the slice write 1 into a zeroed LDS byte table
// (repeated ids write the same value, so plain byte stores suffice), then
// each 32 bytes are packed into the word of P_j.  Slicing keeps the table
// small, so that clearing and packing it are short; every slice reads the
// block's ids.  Needs 32 Ws + 16 bytes of LDS: ids outside the slice write
// the pad byte after the table, so the stores need no branch.
__global__ __launch_bounds__(kSplitThreads) void split_presence_bytes_kernel(
    const int32_t* __restrict__ ids, int64_t L, int num_blocks, int Lb, int vocab, int Ws,
    uint8_t* __restrict__ ws, int64_t seq_bytes) {
  extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
  uint8_t* const pb = reinterpret_cast<uint8_t*>(lds);
  uint4* const p16 = reinterpret_cast<uint4*>(lds);
  const int tid = threadIdx.x;
  const int64_t b = blockIdx.x / num_blocks;
  const int j = blockIdx.x - (int)(b * num_blocks);
  const int W = (int)split_words(vocab);
  const int w0 = blockIdx.y * Ws;
  const int nw = max(0, min(W, w0 + Ws) - w0);  // words of this slice
  const uint32_t t0 = 32u * (uint32_t)w0;       // its first id
  const uint32_t span = 32u * (uint32_t)nw;
  const uint32_t vmax = (uint32_t)(vocab - 1);
  const int32_t* seq = ids + b * L + (int64_t)j * Lb;
  auto load = [&](int x0, uint32_t (&t)[kU]) {
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int x = x0 + u * kSplitThreads + tid;
      // a lane past the block re-reads the block's last id: marking it again
      // changes nothing, and such lanes form no chunk (Lb is a multiple of
      // the chunk); without a branch all kU loads are issued together
      t[u] = min((uint32_t)seq[min(x, Lb - 1)], vmax);
    }
  };
  // the first ids are in flight while the table is cleared
  uint32_t t[kU];
  load(0, t);
  for (int w = tid; w < 2 * nw; w += kSplitThreads) p16[w] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  for (int x0 = 0; x0 < Lb; x0 += kU * kSplitThreads) {
    if (x0 > 0) load(x0, t);
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const uint32_t r = t[u] - t0;  // wraps for ids below the slice
      pb[min(r, span)] = 1;
    }
  }
  __syncthreads();
  // byte k of a 4-byte group (0 or 1) lands on bit 24 + k of x * 0x01020408
  // (the other partial products fall on distinct bits below 24)
  uint32_t* bits = reinterpret_cast<uint32_t*>(ws + b * seq_bytes) + (int64_t)j * W + w0;
  for (int w = tid; w < nw; w += kSplitThreads) {
    const uint4 lo = p16[2 * w], hi = p16[2 * w + 1];
    const uint32_t g[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    uint32_t v = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) v |= ((g[i] * 0x01020408u) >> 24) << (4 * i);
    bits[w] = v;
  }
}

// df of ids 32g .. 32g+31 of sequence b from the N presence words: bit-sliced
// counters (plane p holds bit p of the 32 counts), then each count becomes an
// entry of the df table: a byte, or with NIB (N <= 16) the nibble df - 1.
// Every id that is looked up occurs in its own block, so its df is 1 .. N and
// df - 1 fits in 4 bits; the nibble of an absent id is never read.
template <int P, bool NIB>
__global__ __launch_bounds__(kDfThreads) void split_df_kernel(int num_blocks, int vocab,
                                                              int slices, uint8_t* __restrict__ ws,
                                                              int64_t seq_bytes,
                                                              float* __restrict__ idf) {
  constexpr int KD = P <= 5 ? 16 : kU;  // words loaded together
  const int64_t b = blockIdx.x / slices;
  const int g = (blockIdx.x - (int)(b * slices)) * kDfThreads + threadIdx.x;
  const int W = (int)split_words(vocab);
  if (g >= W) return;
  uint8_t* seq_ws = ws + b * seq_bytes;
  const uint32_t* bits = reinterpret_cast<const uint32_t*>(seq_ws);
  uint32_t c[P];
#pragma unroll
  for (int p = 0; p < P; ++p) c[p] = 0u;
  for (int j0 = 0; j0 < num_blocks; j0 += KD) {
    uint32_t w[KD];
#pragma unroll
    for (int u = 0; u < KD; ++u) w[u] = j0 + u < num_blocks ? bits[(int64_t)(j0 + u) * W + g] : 0u;
#pragma unroll
    for (int u = 0; u < KD; ++u) {
      uint32_t carry = w[u];
#pragma unroll
      for (int p = 0; p < P; ++p) {
        const uint32_t t = c[p] & carry;
        c[p] ^= carry;
        carry = t;
      }
    }
  }
  uint8_t* const table = seq_ws + split_bits_bytes(num_blocks, vocab);
  if constexpr (NIB) {
    // planes of count - 1 (a borrow chain), then nibble k of the 16 bytes =
    // bit k of the four planes; spread() moves bit i of a byte to bit 4 i
    uint32_t e[4];
    uint32_t borrow = 0xFFFFFFFFu;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      e[p] = c[p] ^ borrow;
      borrow &= ~c[p];
    }
    auto spread = [](uint32_t x) {
      x = (x | (x << 12)) & 0x000F000Fu;
      x = (x | (x << 6)) & 0x03030303u;
      return (x | (x << 3)) & 0x11111111u;
    };
    u32x4 out;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      uint32_t v = 0;
#pragma unroll
      for (int p = 0; p < 4; ++p) v |= spread((e[p] >> (8 * r)) & 0xFFu) << p;
      out[r] = v;
    }
    reinterpret_cast<u32x4*>(table)[g] = out;
  } else {
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
    u32x4* df = reinterpret_cast<u32x4*>(table) + 2 * (int64_t)g;
    df[0] = out[0];
    df[1] = out[1];
  }
  if (idf) {
    const float n = (float)num_blocks;
    float* dst = idf + b * vocab;
#pragma unroll
    for (int k = 0; k < 32; ++k) {
      const int t = 32 * g + k;
      uint32_t d = 0;
#pragma unroll
      for (int p = 0; p < P; ++p) d |= ((c[p] >> k) & 1u) << p;
      if (t < vocab) dst[t] = logf(n / (float)(d > 1u ? d : 1u));
    }
  }
}

// Block j of sequence b: the df of each id, each chunk's minimum, the top-k
// chunks.  In round r thread tid holds the 8 consecutive ids
// 8 (1024 r + tid) .. +7 of the block (two 16-byte groups), so a chunk of m
// ids is one group (m = 4) or m / 8 adjacent lanes: the lane takes the
// minimum of its ids, then its lane group (at most 32 lanes, within one
// wavefront).  With DF_LDS the df table (32 W bytes, or 16 W of nibbles) is
// first copied into LDS with 16-byte loads, issued together with the ids'
// loads, and the look-ups read LDS; otherwise they gather from the
// workspace.
template <bool DF_LDS, bool NIB>
__global__ __launch_bounds__(kSplitThreads) void split_select_kernel(
    const int32_t* __restrict__ ids, int64_t L, int num_blocks, int Lb, int chunk_log2, int topk,
    int vocab, const uint8_t* __restrict__ ws, int64_t seq_bytes, int32_t* __restrict__ sel,
    int32_t* __restrict__ chunk_mindf) {
  extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int64_t b = blockIdx.x / num_blocks;
  const int j = blockIdx.x - (int)(b * num_blocks);
  const int C = Lb >> chunk_log2;
  const int W = (int)split_words(vocab);
  const uint32_t vmax = (uint32_t)(vocab - 1);
  const uint8_t* df = ws + b * seq_bytes + split_bits_bytes(num_blocks, vocab);
  const uint8_t* const dfl = reinterpret_cast<const uint8_t*>(lds);
  const int tab16 = NIB ? W : 2 * W;  // 16-byte units of the df table
  uint32_t* const cmin = DF_LDS ? lds + 4 * tab16 : lds;  // [C]
  const int4* seq4 = reinterpret_cast<const int4*>(ids + b * L + (int64_t)j * Lb);
  const int ngroups = Lb >> 2;  // 16-byte groups of the block (Lb is a multiple of 4)
  // Groups past the block re-read its last group: their lanes record no chunk
  // (Lb is a multiple of the chunk, so no chunk or lane group straddles it),
  // and without a branch every load is issued at once.
  auto load = [&](int r, int4 (&q)[2]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) q[h] = seq4[min(2 * (r * kSplitThreads + tid) + h, ngroups - 1)];
  };
  int4 q[2];
  load(0, q);
  if constexpr (DF_LDS) {
    copy_to_lds(reinterpret_cast<const uint4*>(df), reinterpret_cast<uint4*>(lds), tab16, tid);
    // the first ids arrive before the barrier, not after it
    asm volatile("" : "+v"(q[0].x), "+v"(q[0].y), "+v"(q[0].z), "+v"(q[0].w), "+v"(q[1].x),
                 "+v"(q[1].y), "+v"(q[1].z), "+v"(q[1].w));
    __syncthreads();
  }
  const int nrounds = (ngroups + 2 * kSplitThreads - 1) / (2 * kSplitThreads);
  for (int rd = 0; rd < nrounds; ++rd) {
    if (rd > 0) load(rd, q);
    const uint32_t t[8] = {(uint32_t)q[0].x, (uint32_t)q[0].y, (uint32_t)q[0].z, (uint32_t)q[0].w,
                           (uint32_t)q[1].x, (uint32_t)q[1].y, (uint32_t)q[1].z, (uint32_t)q[1].w};
    uint32_t d[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t ti = min(t[i], vmax);
      if (NIB) {
        const uint32_t x = DF_LDS ? dfl[ti >> 1] : df[ti >> 1];
        d[i] = ((x >> ((ti & 1u) << 2)) & 0xFu) + 1u;
      } else {
        d[i] = DF_LDS ? dfl[ti] : df[ti];
      }
    }
    const int g0 = 2 * (rd * kSplitThreads + tid);  // the lane's first group
    if (chunk_log2 == 2) {
      // chunks of 4 ids: each group is a chunk of its own
#pragma unroll
      for (int h = 0; h < 2; ++h)
        if (g0 + h < ngroups)
          cmin[g0 + h] = min(min(d[4 * h], d[4 * h + 1]), min(d[4 * h + 2], d[4 * h + 3]));
    } else {
      uint32_t m = d[0];
#pragma unroll
      for (int i = 1; i < 8; ++i) m = min(m, d[i]);
      const int lg = chunk_log2 - 3;  // log2 of the lanes per chunk
      m = group_min(m, 1 << lg);
      if (g0 < ngroups && (tid & ((1 << lg) - 1)) == 0) cmin[g0 >> (lg + 1)] = m;
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
  // vocab up to 1310720 (40960 words): at most 9 presence slices per block
  if (split_words(vocab) * 4 > PULSAR_LDS_BYTES) return 0;
  return (size_t)(batch * split_seq_bytes(num_blocks, vocab));
}

int launch_split_df(const int32_t* ids, int batch, int64_t L, int num_blocks, int vocab,
                    float* idf, void* workspace, hipStream_t stream) {
  const int Lb = (int)(L / num_blocks);
  const int64_t seq_bytes = split_seq_bytes(num_blocks, vocab);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  const int64_t grid = (int64_t)batch * num_blocks;
  // Vocabulary slices: enough for the byte table to fit in LDS; for a grid
  // of at most 32 workgroups, more (down to 512-word slices) while it stays
  // within one workgroup per CU.  (Larger grids gain nothing from slicing
  // once their ids come from HBM: every slice reads the block's ids.)
  constexpr int kSliceWords = 512;
  const int64_t W = split_words(vocab);
  const int64_t max_ws = (PULSAR_LDS_BYTES - 16) / 32;  // words of the largest table
  const int64_t fit = (W + max_ws - 1) / max_ws;
  const int64_t small = (W + kSliceWords - 1) / kSliceWords;
  const int64_t room = grid <= 32 ? 256 / grid : 1;
  const int vslices = (int)std::max(fit, std::min(small, room));
  const int64_t Ws = (W + vslices - 1) / vslices;
  const size_t bytes_tab = (size_t)Ws * 32 + 16;  // at most the LDS, by the choice of `fit`
  if (bytes_tab > PULSAR_LDS_BYTES) return PULSAR_EUNSUPPORTED;
  if (hipFuncSetAttribute((const void*)split_presence_bytes_kernel,
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes_tab) != hipSuccess)
    return PULSAR_EHIP;
  hipLaunchKernelGGL(split_presence_bytes_kernel, dim3((unsigned)grid, (unsigned)vslices),
                     dim3(kSplitThreads), bytes_tab, stream, ids, L, num_blocks, Lb, vocab, (int)Ws,
                     ws, seq_bytes);
  if (hipGetLastError() != hipSuccess) return PULSAR_EHIP;
  const int slices = (int)((split_words(vocab) + kDfThreads - 1) / kDfThreads);
  const dim3 dgrid((unsigned)(batch * slices));
  // counter planes: enough bits for num_blocks (<= 255); a nibble table for
  // up to 16 blocks
  if (num_blocks < 16)
    hipLaunchKernelGGL((split_df_kernel<4, true>), dgrid, dim3(kDfThreads), 0, stream, num_blocks,
                       vocab, slices, ws, seq_bytes, idf);
  else if (num_blocks == 16)
    hipLaunchKernelGGL((split_df_kernel<5, true>), dgrid, dim3(kDfThreads), 0, stream, num_blocks,
                       vocab, slices, ws, seq_bytes, idf);
  else if (num_blocks < 32)
    hipLaunchKernelGGL((split_df_kernel<5, false>), dgrid, dim3(kDfThreads), 0, stream, num_blocks,
                       vocab, slices, ws, seq_bytes, idf);
  else
    hipLaunchKernelGGL((split_df_kernel<8, false>), dgrid, dim3(kDfThreads), 0, stream, num_blocks,
                       vocab, slices, ws, seq_bytes, idf);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}

int launch_maxidf_split(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk,
                        int topk, int vocab, int32_t* sel, int32_t* chunk_mindf, float* idf,
                        void* workspace, hipStream_t stream) {
  int chunk_log2 = 0;
  while ((1 << chunk_log2) < chunk) ++chunk_log2;
  const int Lb = (int)(L / num_blocks);
  const int64_t seq_bytes = split_seq_bytes(num_blocks, vocab);
  const int64_t grid = (int64_t)batch * num_blocks;
  int st = launch_split_df(ids, batch, L, num_blocks, vocab, idf, workspace, stream);
  if (st != PULSAR_OK) return st;
  const bool nib = num_blocks <= 16;
  const size_t cl = (size_t)(Lb >> chunk_log2) * 4;
  const size_t df_tab = (size_t)split_words(vocab) * (nib ? 16 : 32);
  const bool df_lds = df_tab + cl <= PULSAR_LDS_BYTES;
  auto sk = df_lds ? (nib ? split_select_kernel<true, true> : split_select_kernel<true, false>)
                   : (nib ? split_select_kernel<false, true> : split_select_kernel<false, false>);
  const size_t sl = df_lds ? df_tab + cl : cl;
  if (hipFuncSetAttribute((const void*)sk, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sl) !=
      hipSuccess)
    return PULSAR_EHIP;
  hipLaunchKernelGGL(sk, dim3((unsigned)grid), dim3(kSplitThreads), sl, stream, ids, L, num_blocks,
                     Lb, chunk_log2, topk, vocab, static_cast<const uint8_t*>(workspace), seq_bytes,
                     sel, chunk_mindf);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}
