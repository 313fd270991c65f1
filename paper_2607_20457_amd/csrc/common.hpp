// Shared device-side types and helpers for the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/pulsar.h"

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define PULSAR_WAVE 64
#define PULSAR_LDS_BYTES 163840  // 160 KB local data share per compute unit on gfx950

// Row -> global position map of an assembled Phase-1 input (Eq. 3, sparse
// position ids).  The summary region is a sequence of runs of m consecutive
// positions, one run per selected chunk; run q = j*k + c starts at
// j*Lb + sel[j][c]*m.  Kernels stage these run starts in LDS once
// (build_run_table) and then map a row with a few integer operations.
enum MapMode : int { MAP_IDENTITY = 0, MAP_SUMMARY = 1, MAP_ANCHOR = 2, MAP_EVEN = 3 };

struct RowMap {
  int mode;
  int block_idx;   // i
  int Lb;          // block length
  int sink;        // s_sink
  int chunk;       // m
  int topk;        // k
  int prefix;      // rows of the summary region, i * k * m (summary mode)
  int n_runs;      // summary runs, i * k
  int nchunk;      // chunks per block, Lb / m
  int m_log2;      // log2(m) when m is a power of two, else -1
  float inv_chunk; // 1 / m
  int64_t offset;  // identity mode: position of row 0
  int sigma;           // Even-Spaced: points per earlier block, k * m
  float inv_sigma;     // 1 / sigma
  double inv_sigma1;   // 1 / (sigma - 1), sigma > 1
};

// run_base[q] = j*Lb + sel[j][c]*m for run q = j*k + c; a selection outside
// [0, Lb/m) is a caller error and is clamped so that every access stays
// inside block j.
__device__ __forceinline__ void build_run_table(const RowMap& mp, const int32_t* __restrict__ sel,
                                                int* run_base, int tid, int nthreads) {
  for (int q = tid; q < mp.n_runs; q += nthreads) {
    const int j = q / mp.topk;
    const int c = min(max(sel[q], 0), mp.nchunk - 1);
    run_base[q] = j * mp.Lb + c * mp.chunk;
  }
}

// Global position of assembled row r, in two parts: the index of the LDS
// run-table entry the row reads (-1 for none) and what to add to that entry
// (or the position itself when there is no entry).  Rows are below 2^24
// (checked on the host), so float quotient estimates are within one of the
// true quotient.  MODE is the map mode, known at compile time.
template <int MODE>
__device__ __forceinline__ int2 row_position_split(const RowMap& mp, int r) {
  if constexpr (MODE == MAP_IDENTITY) return int2{-1, (int)(mp.offset + r)};
  if constexpr (MODE == MAP_ANCHOR)
    return int2{-1, r < mp.Lb ? r : mp.block_idx * mp.Lb + (r - mp.Lb)};
  if (r < mp.sink) return int2{-1, r};
  const int t = r - mp.sink;
  if (t >= mp.prefix) return int2{-1, mp.block_idx * mp.Lb + (t - mp.prefix)};
  if constexpr (MODE == MAP_EVEN) {
    // point p of block j: j*Lb + floor(p (Lb - 1) / (sigma - 1)); both
    // quotients are estimated in floating point and corrected exactly
    const int sig = mp.sigma;
    int j = (int)((float)t * mp.inv_sigma);
    int p = t - j * sig;
    if (p < 0) {
      --j;
      p += sig;
    } else if (p >= sig) {
      ++j;
      p -= sig;
    }
    if (sig == 1) return int2{-1, j * mp.Lb};
    const int64_t num = (int64_t)p * (mp.Lb - 1);  // < 2^48: exact as a double
    int64_t off = (int64_t)((double)num * mp.inv_sigma1);
    if (off * (sig - 1) > num) --off;
    else if ((off + 1) * (sig - 1) <= num) ++off;
    return int2{-1, j * mp.Lb + (int)off};
  }
  // summary runs: run q starts at run_base[q]
  int q, w;
  if (mp.m_log2 >= 0) {
    q = t >> mp.m_log2;
    w = t & (mp.chunk - 1);
  } else {
    q = (int)((float)t * mp.inv_chunk);
    w = t - q * mp.chunk;
    if (w < 0) {
      --q;
      w += mp.chunk;
    } else if (w >= mp.chunk) {
      ++q;
      w -= mp.chunk;
    }
  }
  return int2{q, w};
}

template <int MODE>
__device__ __forceinline__ int row_position_m(const RowMap& mp, const int* run_base, int r) {
  const int2 s = row_position_split<MODE>(mp, r);
  return s.x >= 0 ? run_base[s.x] + s.y : s.y;
}

// The same with the mode read at run time.
__device__ __forceinline__ int row_position(const RowMap& mp, const int* run_base, int r) {
  switch (mp.mode) {
    case MAP_IDENTITY: return row_position_m<MAP_IDENTITY>(mp, run_base, r);
    case MAP_ANCHOR: return row_position_m<MAP_ANCHOR>(mp, run_base, r);
    case MAP_EVEN: return row_position_m<MAP_EVEN>(mp, run_base, r);
    default: return row_position_m<MAP_SUMMARY>(mp, run_base, r);
  }
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
  return x;
}

__device__ __forceinline__ int wave_sum_int(int x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

// Exclusive prefix sum across the 64 lanes of a wavefront.
__device__ __forceinline__ int wave_excl_scan(int x) {
  const int lane = threadIdx.x & 63;
  int incl = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  return incl - x;
}

// Host-side launch helpers (implemented in the per-kernel sources).
int launch_maxidf(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk, int topk,
                  int vocab, int32_t* sel, int32_t* chunk_mindf, float* idf, size_t lds_bytes,
                  hipStream_t stream);
size_t maxidf_lds_bytes(int64_t L, int num_blocks, int chunk, int vocab);
// Max-IDF of few sequences split over blocks and vocabulary slices (three
// launches through a workspace); 0 bytes where that path is not taken.
size_t maxidf_split_workspace(int batch, int64_t L, int num_blocks, int chunk, int vocab);
int launch_maxidf_split(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk,
                        int topk, int vocab, int32_t* sel, int32_t* chunk_mindf, float* idf,
                        void* workspace, hipStream_t stream);
int decode_parts(int n_shards, int64_t S, int Hkv);
bool decode_applies(int Tq, int Hq, int Hkv, int d);
// The generation shard of a decode step, folded into the same launch: rows
// [0, G) are the tokens appended earlier, row G + t is new token t's own, and
// token t sees rows 0 .. G + t.
struct DecodeGen {
  const uint16_t* K;  // bf16 [G + Tq, Hkv, d]
  const uint16_t* V;
  int64_t G;
  int nparts;         // key ranges (one partial each), after the shards' parts
};
int launch_decode(const uint16_t* q, const uint16_t* K, const uint16_t* V, int n_shards, int Tq,
                  int64_t S, int Hq, int Hkv, int d, float scale, float* o, float* lse,
                  int nparts, hipStream_t stream, const DecodeGen* gen = nullptr);
int launch_scorer(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk, int topk,
                  int vocab, int scorer, int32_t* sel, float* scores, hipStream_t stream);
size_t scorer_lds_bytes(int64_t L, int num_blocks, int chunk, int vocab, int scorer);
// The scorers' split path for a small batch (the workspace of
// maxidf_split_workspace): LDS of its score kernel, and the launch.
size_t scorer_split_lds_bytes(int64_t L, int num_blocks, int chunk, int vocab, int scorer);
int launch_scorer_split(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk,
                        int topk, int vocab, int scorer, int32_t* sel, float* scores,
                        void* workspace, hipStream_t stream);

int launch_positions(const RowMap& mp, const int32_t* sel, int64_t sel_bstride, int batch,
                     int n_rows, int32_t* pos, hipStream_t stream);
#define PULSAR_MAX_ROWS (1 << 24)  // longest assembled input the row map supports

struct AttnLaunch {
  const uint16_t* Q;
  const uint16_t* K;
  const uint16_t* V;
  int64_t q_zstride;    // elements between consecutive z entries of Q
  int64_t kv_zstride;   // elements between consecutive kv "batches" (sequence or shard)
  int Hq, Hkv, d;
  int n_q;              // query rows per z
  int n_kv;             // key rows per kv batch (phase 2: shard length S)
  int causal;
  int nsplit;           // key splits per kv batch (phase 2)
  int split_len;        // keys per split
  int nz_kv;            // number of kv batches (sequences or shards)
  RowMap map;           // applies to both query and key rows (phase 1)
  const int32_t* sel;   // [batch, N, k] or NULL
  int64_t sel_bstride;
  float scale_log2;     // softmax_scale * log2(e)
  void* O;              // [z][n_q][Hq][d]
  int o_bf16;
  int64_t o_zstride;
  float* lse;           // [z][Hq][n_q]
  int64_t lse_zstride;
};
int launch_attention(const AttnLaunch& a, hipStream_t stream);
int attn_rows_per_wg(int group, bool causal);  // query rows of one attention workgroup

int launch_lse_merge(const float* o_parts, const float* lse_parts, int H, int nz, int Tq, int Hq,
                     int d, int64_t part_ostride, int64_t part_lstride, float* o, float* lse,
                     hipStream_t stream);

// Rows of an assembled Phase-1 input gathered from a per-position tensor and
// rotated per pos_mode (a pulsar_pos_mode).
int launch_gather_rope(const uint16_t* X, uint16_t* Y, int batch, int n, int64_t L, int H, int d,
                       const RowMap& mp, const int32_t* sel, int64_t sel_bstride, int pos_mode,
                       const float* inv_freq, double base, hipStream_t stream);

// IDF of a context with no tokens: every entry ln(num_blocks / 1).
int launch_idf_fill(float* idf, int64_t n, int num_blocks, hipStream_t stream);

int launch_copy_rows(const void* src, int64_t src_pitch, void* dst, int64_t dst_pitch,
                     int64_t bytes_per_row, int rows, hipStream_t stream);
