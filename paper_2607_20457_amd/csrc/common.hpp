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

// Row -> global position map of an attention launch.
enum MapMode : int { MAP_IDENTITY = 0, MAP_SUMMARY = 1, MAP_ANCHOR = 2 };

struct RowMap {
  int mode;
  int block_idx;   // i
  int Lb;          // block length
  int sink;        // s_sink
  int chunk;       // m
  int topk;        // k
  int sigma;       // k * m
  int prefix;      // summary rows = i * sigma (summary mode)
  int nchunk;      // chunks per block, Lb / m
  int64_t offset;  // identity mode: position of row 0
  float inv_sigma; // 1 / sigma, for the quotient estimate below
  float inv_chunk; // 1 / chunk
};

// Quotient of two non-negative ints through a float estimate and an exact
// correction step (the estimate is off by at most one below 2^24).
__device__ __forceinline__ int div_fix(int a, int b, float inv_b, int* rem) {
  int q = (int)((float)a * inv_b);
  int r = a - q * b;
  while (r < 0) { --q; r += b; }
  while (r >= b) { ++q; r -= b; }
  *rem = r;
  return q;
}

// Global position of assembled row r (Eq. 3, sparse position ids).
// sel points at this sequence's [num_blocks, topk] selection.
__device__ __forceinline__ int row_position(const RowMap& mp, const int32_t* __restrict__ sel,
                                            int r) {
  if (mp.mode == MAP_IDENTITY) return (int)(mp.offset + r);
  if (mp.mode == MAP_ANCHOR) return r < mp.Lb ? r : mp.block_idx * mp.Lb + (r - mp.Lb);
  if (r < mp.sink) return r;
  int t = r - mp.sink;
  if (t < mp.prefix) {
    int w;
    int j = div_fix(t, mp.sigma, mp.inv_sigma, &w);
    int rr;
    int c = div_fix(w, mp.chunk, mp.inv_chunk, &rr);
    // a selection outside [0, Lb/m) is a caller error; clamping keeps every
    // access inside block j
    const int cs = min(max(sel[j * mp.topk + c], 0), mp.nchunk - 1);
    return j * mp.Lb + cs * mp.chunk + rr;
  }
  return mp.block_idx * mp.Lb + (t - mp.prefix);
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
size_t maxidf_lds_bytes(int64_t L, int chunk, int vocab);

int launch_positions(const RowMap& mp, const int32_t* sel, int64_t sel_bstride, int batch,
                     int n_rows, int32_t* pos, hipStream_t stream);

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
int attn_rows_per_wg(int group);  // query rows covered by one attention workgroup

int launch_lse_merge(const float* o_parts, const float* lse_parts, int H, int nz, int Tq, int Hq,
                     int d, int64_t part_ostride, int64_t part_lstride, float* o, float* lse,
                     hipStream_t stream);

int launch_copy_rows(const void* src, int64_t src_pitch, void* dst, int64_t dst_pitch,
                     int64_t bytes_per_row, int rows, hipStream_t stream);
