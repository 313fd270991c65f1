// Bandwidth-bound helper kernels: the materialised Eq. 3 position map, the
// KV(B_i) retention copy, and the Phase-2 online-softmax merge.
#include "common.hpp"

// ---------------------------------------------------------------------------
// Row -> global position map (Eq. 3, sparse position ids), with the same
// device function the attention kernel uses for its fused gather.
__global__ __launch_bounds__(256) void positions_kernel(RowMap mp, const int32_t* __restrict__ sel,
                                                        int64_t sel_bstride, int n_rows,
                                                        int32_t* __restrict__ pos) {
  extern __shared__ int run_base[];
  const int b = blockIdx.y;
  build_run_table(mp, sel ? sel + b * sel_bstride : nullptr, run_base, threadIdx.x, 256);
  __syncthreads();
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r >= n_rows) return;
  pos[(int64_t)b * n_rows + r] = row_position(mp, run_base, r);
}

int launch_positions(const RowMap& mp, const int32_t* sel, int64_t sel_bstride, int batch,
                     int n_rows, int32_t* pos, hipStream_t stream) {
  if (batch == 0 || n_rows == 0) return PULSAR_OK;
  const size_t lds = (size_t)mp.n_runs * 4;
  if (lds > PULSAR_LDS_BYTES) return PULSAR_EUNSUPPORTED;
  if (hipFuncSetAttribute((const void*)positions_kernel,
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return PULSAR_EHIP;
  dim3 grid((n_rows + 255) / 256, batch);
  hipLaunchKernelGGL(positions_kernel, grid, dim3(256), lds, stream, mp, sel, sel_bstride, n_rows,
                     pos);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}

// ---------------------------------------------------------------------------
// Strided row copy (KV(B_i) retention, Appendix "KV Cache Discard").  Rows are
// multiples of 16 bytes and 16-byte aligned (checked by the caller).
__global__ __launch_bounds__(256) void copy_rows_kernel(const u32x4* __restrict__ src,
                                                        int64_t src_pitch16,
                                                        u32x4* __restrict__ dst,
                                                        int64_t dst_pitch16, int64_t row16) {
  const int64_t row = blockIdx.y;
  const u32x4* s = src + row * src_pitch16;
  u32x4* d = dst + row * dst_pitch16;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < row16;
       i += (int64_t)gridDim.x * 256)
    d[i] = s[i];
}

int launch_copy_rows(const void* src, int64_t src_pitch, void* dst, int64_t dst_pitch,
                     int64_t bytes_per_row, int rows, hipStream_t stream) {
  if (rows == 0 || bytes_per_row == 0) return PULSAR_OK;
  const int64_t row16 = bytes_per_row / 16;
  int64_t blocks = (row16 + 255) / 256;
  if (blocks > 2048) blocks = 2048;
  hipLaunchKernelGGL(copy_rows_kernel, dim3((unsigned)blocks, rows), dim3(256), 0, stream,
                     (const u32x4*)src, src_pitch / 16, (u32x4*)dst, dst_pitch / 16, row16);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}

// ---------------------------------------------------------------------------
// IDF table of a context without tokens (Eq. idf with df = 0 everywhere):
// the value the Max-IDF kernels write for an id that occurs in no block.
__global__ __launch_bounds__(256) void idf_fill_kernel(float* __restrict__ idf, int64_t n,
                                                       float num_blocks) {
  const float v = logf(num_blocks / 1.0f);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    idf[i] = v;
}

int launch_idf_fill(float* idf, int64_t n, int num_blocks, hipStream_t stream) {
  if (n == 0) return PULSAR_OK;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(idf_fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, idf, n,
                     (float)num_blocks);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}

// ---------------------------------------------------------------------------
// Online-softmax merge (Appendix "Phase 2 Distributed Softmax Merge").
// Thread = four consecutive head_dim entries of one (z, query, head).  One
// pass over the parts, CH at a time (2, 4 or 8: the fewest that cover H, up
// to 8) with all their loads issued together: the running maximum m,
// s = sum_h exp(l_h - m) and a = sum_h exp(l_h - m) o_h are rescaled when m
// rises; then l = m + ln s and o = a / s.  -inf partials weigh zero.
template <int CH>
__global__ __launch_bounds__(256) void lse_merge_kernel(
    const float* __restrict__ o_parts, const float* __restrict__ lse_parts, int H, int Tq, int Hq,
    int d4, int64_t part_ostride, int64_t part_lstride, float* __restrict__ o,
    float* __restrict__ lse, int64_t total) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int dv = (int)(i % d4);
  int64_t rest = i / d4;
  const int h = (int)(rest % Hq);
  rest /= Hq;
  const int q = (int)(rest % Tq);
  const int64_t z = rest / Tq;

  const float* lp = lse_parts + z * (int64_t)H * part_lstride + (int64_t)h * Tq + q;
  const int64_t orow = (((int64_t)q * Hq + h) * d4 + dv);
  const f32x4* op = reinterpret_cast<const f32x4*>(o_parts) + z * (int64_t)H * (part_ostride / 4);
  float m = -INFINITY, sum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int p0 = 0; p0 < H; p0 += CH) {
    float l[CH];
    f32x4 v[CH];
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const int p = min(p0 + u, H - 1);  // a part past the last re-reads it, weighing zero
      l[u] = lp[p * part_lstride];
      v[u] = op[p * (part_ostride / 4) + orow];
    }
    float cm = -INFINITY;
#pragma unroll
    for (int u = 0; u < CH; ++u)
      if (p0 + u < H) cm = fmaxf(cm, l[u]);
    // branch-free, so that all 2 CH loads are issued before the first
    // wait; with no finite partial yet the weights are taken against 0 and
    // come out 0
    const float nm = fmaxf(m, cm);
    const float nm_use = nm == -INFINITY ? 0.f : nm;
    const float alpha = __expf(m - nm_use);  // 0 while m is -inf
    sum *= alpha;
    acc *= alpha;
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const float w = p0 + u < H ? __expf(l[u] - nm_use) : 0.f;
      sum += w;
      acc += w * v[u];
    }
    m = nm;
  }
  float ell = -INFINITY;
  if (m != -INFINITY) {
    ell = m + __logf(sum);
    acc *= 1.f / sum;
  }
  reinterpret_cast<f32x4*>(o)[z * (int64_t)Tq * Hq * d4 + orow] = acc;
  if (lse && dv == 0) lse[z * (int64_t)Hq * Tq + (int64_t)h * Tq + q] = ell;
}

// The same merge with one wavefront per output group of four values: lane
// l folds parts l, l + 64, ..., and the wavefront combines the lanes.  For
// few outputs and many parts (a decode step: 1024 outputs, tens to hundreds
// of parts), where a thread per output leaves most of the chip idle and
// walks the parts one after another.
__global__ __launch_bounds__(256) void lse_merge_wide_kernel(
    const float* __restrict__ o_parts, const float* __restrict__ lse_parts, int H, int Tq, int Hq,
    int d4, int64_t part_ostride, int64_t part_lstride, float* __restrict__ o,
    float* __restrict__ lse, int64_t total) {
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= total) return;  // wave-uniform
  const int dv = (int)(i % d4);
  int64_t rest = i / d4;
  const int h = (int)(rest % Hq);
  rest /= Hq;
  const int q = (int)(rest % Tq);
  const int64_t z = rest / Tq;

  const float* lp = lse_parts + z * (int64_t)H * part_lstride + (int64_t)h * Tq + q;
  float mx = -INFINITY;
  for (int p = lane; p < H; p += 64) mx = fmaxf(mx, lp[p * part_lstride]);
  mx = wave_max(mx);
  const int64_t orow = (((int64_t)q * Hq + h) * d4 + dv);
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float ell = -INFINITY;
  if (mx != -INFINITY) {
    float sum = 0.f;
    for (int p = lane; p < H; p += 64) sum += __expf(lp[p * part_lstride] - mx);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, 64);
    ell = mx + __logf(sum);
    const f32x4* op = reinterpret_cast<const f32x4*>(o_parts) + z * (int64_t)H * (part_ostride / 4);
    for (int p = lane; p < H; p += 64) {
      const float w = __expf(lp[p * part_lstride] - ell);
      acc += w * op[p * (part_ostride / 4) + orow];
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      acc.x += __shfl_xor(acc.x, off, 64);
      acc.y += __shfl_xor(acc.y, off, 64);
      acc.z += __shfl_xor(acc.z, off, 64);
      acc.w += __shfl_xor(acc.w, off, 64);
    }
  }
  if (lane == 0) {
    reinterpret_cast<f32x4*>(o)[z * (int64_t)Tq * Hq * d4 + orow] = acc;
    if (lse && dv == 0) lse[z * (int64_t)Hq * Tq + (int64_t)h * Tq + q] = ell;
  }
}

int launch_lse_merge(const float* o_parts, const float* lse_parts, int H, int nz, int Tq, int Hq,
                     int d, int64_t part_ostride, int64_t part_lstride, float* o, float* lse,
                     hipStream_t stream) {
  const int64_t total = (int64_t)nz * Tq * Hq * (d / 4);
  if (total == 0) return PULSAR_OK;
  if (H >= 8 && total <= 8192) {  // at most 32 workgroups of the per-output form
    const int64_t blocks = (total + 3) / 4;
    hipLaunchKernelGGL(lse_merge_wide_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                       o_parts, lse_parts, H, Tq, Hq, d / 4, part_ostride, part_lstride, o, lse,
                       total);
    return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
  }
  const int64_t blocks = (total + 255) / 256;
  const auto kern = H <= 2 ? lse_merge_kernel<2> : H <= 4 ? lse_merge_kernel<4> : lse_merge_kernel<8>;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), 0, stream, o_parts, lse_parts, H,
                     Tq, Hq, d / 4, part_ostride, part_lstride, o, lse, total);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}
