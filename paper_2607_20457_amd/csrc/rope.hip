// Rotary position embedding of query/key rows at given positions (Appendix
// "RoPE Position ID Assignment").  In the paper's sparse mode every token
// keeps its global position id, so one pass over a layer's Q and K of the
// whole context gives every block's Phase-1 input its rotated rows: the
// rotation of a row depends on its position alone, not on the block whose
// input it appears in.
//
// Rotate-half form: pair i < d/2 of a head vector is (x_i, x_{i+d/2}) and is
// turned by the angle p * w_i.
//
// One wavefront per row.  Lane (h, j) owns pairs 8j .. 8j+7 of heads h,
// h + 64/(d/16), ...: 16-byte loads of x[8j .. 8j+7] and
// x[d/2+8j .. d/2+8j+7], so that each load instruction reads contiguous
// runs of the row.  Each of the row's angles is formed once, in fp64
// (p * w_i, then reduced to [-pi, pi] with a two-part 2*pi), its sine and
// cosine taken in fp32 on the reduced angle, and handed to the lanes that
// use it.  The rotation is evaluated in fp32 and rounded once to
// bf16.  Bound by HBM: 2 * n_rows * H * d * 2 bytes per call.
#include <cmath>

#include "common.hpp"

namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kRopeThreads = 256;
constexpr int kMaxHalf = 64;  // d <= 128

struct RopeFreqs {
  double w[kMaxHalf];  // w_i, i < d/2
};

// 2*pi split into a double and the double nearest its remainder.
constexpr double kTwoPiHi = 6.283185307179586;
constexpr double kTwoPiLo = 2.4492935982947064e-16;
constexpr double kInvTwoPi = 0.15915494309189535;

// One row of H heads: 16-byte loads of src (already offset by this lane's
// 8 pairs), rotation by the angles of position p + p_add (ROTATE) or a plain
// copy, 16-byte stores to dst.  `w_pair` and `p` may still be loading: the
// first data is requested before they are used.
template <int D, bool ROTATE>
__device__ __forceinline__ void rope_row(const uint16_t* src, uint16_t* dst, int H, int64_t p,
                                         int64_t p_add, double w_pair, int lane) {
  constexpr int G = D / 16;     // lanes per head: pairs 8j .. 8j+7 each
  constexpr int HPW = 64 / G;   // heads per wavefront step
  constexpr int U = 4;          // steps whose loads are in flight together
  const int j = lane % G, hl = lane / G;
  // Heads hl, hl + HPW, ...: one step covers HPW heads of the row, its low
  // and high halves as two runs of contiguous 16-byte chunks.  Loads are
  // branch-free (a head past the last re-reads the last; it is not stored).
  u32x4 lo[U], hi[U];
  auto load = [&](int h0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int hh = min(h0 + u * HPW + hl, H - 1);
      lo[u] = *reinterpret_cast<const u32x4*>(src + (int64_t)hh * D);
      hi[u] = *reinterpret_cast<const u32x4*>(src + (int64_t)hh * D + D / 2);
    }
  };
  // The row's angles: lane (hl, j) forms that of pair 8j + hl % 8, then
  // each lane gathers the eight of its own pairs 8j .. 8j+7 from lanes
  // v * G + j.
  load(0);
  float c[8], s[8];
  if constexpr (ROTATE) {
    asm volatile("" : "+v"(w_pair), "+v"(p));
    p += p_add;
    float s1, c1;
    {
      const double a = (double)p * w_pair;
      const double k = rint(a * kInvTwoPi);
      double r = fma(-k, kTwoPiHi, a);
      r = fma(-k, kTwoPiLo, r);
      sincosf((float)r, &s1, &c1);
    }
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      s[v] = __shfl(s1, v * G + j, 64);
      c[v] = __shfl(c1, v * G + j, 64);
    }
  }
  auto rotate = [&](const u32x4 lo, const u32x4 hi, u32x4& olo, u32x4& ohi) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      // words hold elements 2w (low half) and 2w+1 (high half)
      const float x0a = __builtin_bit_cast(float, lo[w] << 16);
      const float x0b = __builtin_bit_cast(float, lo[w] & 0xffff0000u);
      const float x1a = __builtin_bit_cast(float, hi[w] << 16);
      const float x1b = __builtin_bit_cast(float, hi[w] & 0xffff0000u);
      const int va = 2 * w, vb = 2 * w + 1;
      const f32x2 ylo = {fmaf(x0a, c[va], -x1a * s[va]), fmaf(x0b, c[vb], -x1b * s[vb])};
      const f32x2 yhi = {fmaf(x1a, c[va], x0a * s[va]), fmaf(x1b, c[vb], x0b * s[vb])};
      olo[w] = __builtin_bit_cast(uint32_t, __builtin_convertvector(ylo, bf16x2));
      ohi[w] = __builtin_bit_cast(uint32_t, __builtin_convertvector(yhi, bf16x2));
    }
  };
  for (int h0 = 0; h0 < H; h0 += U * HPW) {
    u32x4 clo[U], chi[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      clo[u] = lo[u];
      chi[u] = hi[u];
    }
    if (h0 + U * HPW < H) load(h0 + U * HPW);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int hh = h0 + u * HPW + hl;
      if (hh < H) {
        u32x4 olo = clo[u], ohi = chi[u];
        if constexpr (ROTATE) rotate(clo[u], chi[u], olo, ohi);
        *reinterpret_cast<u32x4*>(dst + (int64_t)hh * D) = olo;
        *reinterpret_cast<u32x4*>(dst + (int64_t)hh * D + D / 2) = ohi;
      }
    }
  }
}

template <int D, bool HAS_POS>
__global__ __launch_bounds__(kRopeThreads) void rope_kernel(uint16_t* __restrict__ X,
                                                            int64_t rows, int64_t n_rows, int H,
                                                            const int32_t* __restrict__ pos,
                                                            int64_t pos_offset, RopeFreqs f) {
  constexpr int G = D / 16;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (kRopeThreads / 64) + (threadIdx.x >> 6);
  if (row >= rows) return;  // wave-uniform
  const int j = lane % G, hl = lane / G;
  uint16_t* base = X + row * (int64_t)H * D + 8 * j;
  // The frequency and the position are requested before the first data.
  const double w = f.w[8 * j + (hl & 7)];
  const int64_t p = HAS_POS ? (int64_t)pos[row] : row % n_rows;
  rope_row<D, true>(base, base, H, p, pos_offset, w, lane);
}

// Rows of block i's assembled Phase-1 input (Eq. 3), gathered from the
// per-position tensor X through the row -> position map and rotated by
// their global position (ROT = 1, sparse), by their row index (ROT = 2,
// contiguous), or copied unrotated (ROT = 0, for V).  One wavefront per
// output row; its position is formed by the whole wave (the selection entry
// of a summary row is one read from sel, clamped into the block as the
// attention kernel's run table does).
template <int D, int ROT>
__global__ __launch_bounds__(kRopeThreads) void gather_rope_kernel(
    const uint16_t* __restrict__ X, uint16_t* __restrict__ Y, int64_t rows, int n,
    int64_t x_bstride, int H, RowMap mp, const int32_t* __restrict__ sel, int64_t sel_bstride,
    RopeFreqs f) {
  constexpr int G = D / 16;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (kRopeThreads / 64) + (threadIdx.x >> 6);
  if (row >= rows) return;  // wave-uniform
  const int64_t b = row / n;
  const int r = (int)(row - b * n);
  int2 ps;
  switch (mp.mode) {
    case MAP_IDENTITY: ps = row_position_split<MAP_IDENTITY>(mp, r); break;
    case MAP_ANCHOR: ps = row_position_split<MAP_ANCHOR>(mp, r); break;
    case MAP_EVEN: ps = row_position_split<MAP_EVEN>(mp, r); break;
    default: ps = row_position_split<MAP_SUMMARY>(mp, r); break;
  }
  int p = ps.y;
  if (ps.x >= 0) {  // summary run q = ps.x: block q / k, chunk sel[q]
    const int q = ps.x;
    const int c = min(max(sel[b * sel_bstride + q], 0), mp.nchunk - 1);
    p = (q / mp.topk) * mp.Lb + c * mp.chunk + ps.y;
  }
  const int j = lane % G, hl = lane / G;
  const uint16_t* src = X + b * x_bstride + (int64_t)p * H * D + 8 * j;
  uint16_t* dst = Y + row * (int64_t)H * D + 8 * j;
  const double w = f.w[8 * j + (hl & 7)];
  rope_row<D, ROT != 0>(src, dst, H, ROT == 2 ? (int64_t)r : (int64_t)p, 0, w, lane);
}

// The table w_i: the caller's (checked finite) or base^(-2i/d).
int make_freqs(const float* inv_freq, double base, int d, RopeFreqs* f) {
  if (inv_freq) {
    for (int i = 0; i < d / 2; ++i) {
      if (!std::isfinite(inv_freq[i])) return PULSAR_EINVAL;
      f->w[i] = (double)inv_freq[i];
    }
  } else {
    if (!(base > 0.0) || !std::isfinite(base)) return PULSAR_EINVAL;
    for (int i = 0; i < d / 2; ++i) f->w[i] = std::pow(base, -2.0 * i / d);
  }
  return PULSAR_OK;
}

}  // namespace

int launch_gather_rope(const uint16_t* X, uint16_t* Y, int batch, int n, int64_t L, int H, int d,
                       const RowMap& mp, const int32_t* sel, int64_t sel_bstride, int pos_mode,
                       const float* inv_freq, double base, hipStream_t stream) {
  RopeFreqs f{};
  if (pos_mode != PULSAR_POS_NONE) {
    const int st = make_freqs(inv_freq, base, d, &f);
    if (st != PULSAR_OK) return st;
  }
  const int64_t rows = (int64_t)batch * n;
  if (rows == 0 || H == 0) return PULSAR_OK;
  const int64_t blocks = (rows + kRopeThreads / 64 - 1) / (kRopeThreads / 64);  // a wave per row
  if (blocks > 0x7fffffff) return PULSAR_EUNSUPPORTED;
  decltype(&gather_rope_kernel<128, 0>) kern;
  if (d == 128)
    kern = pos_mode == PULSAR_POS_SPARSE       ? gather_rope_kernel<128, 1>
           : pos_mode == PULSAR_POS_CONTIGUOUS ? gather_rope_kernel<128, 2>
                                               : gather_rope_kernel<128, 0>;
  else
    kern = pos_mode == PULSAR_POS_SPARSE       ? gather_rope_kernel<64, 1>
           : pos_mode == PULSAR_POS_CONTIGUOUS ? gather_rope_kernel<64, 2>
                                               : gather_rope_kernel<64, 0>;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kRopeThreads), 0, stream, X, Y, rows, n,
                     L * H * d, H, mp, sel, sel_bstride, f);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}

extern "C" {

int pulsar_rope(void* X, int batch, int64_t n_rows, int H, int d, const int32_t* pos,
                int64_t pos_offset, const float* inv_freq, double base, void* stream) {
  if (batch < 0 || n_rows < 0 || H < 0) return PULSAR_EINVAL;
  if (d != 64 && d != 128) return d > 0 && d % 2 == 0 ? PULSAR_EUNSUPPORTED : PULSAR_EINVAL;
  const int64_t rows = (int64_t)batch * n_rows;
  if (rows == 0 || H == 0) return PULSAR_OK;
  if (X == nullptr || (reinterpret_cast<uintptr_t>(X) & 15u) != 0) return PULSAR_EINVAL;
  RopeFreqs f{};
  const int fst = make_freqs(inv_freq, base, d, &f);
  if (fst != PULSAR_OK) return fst;
  const int64_t blocks = (rows + kRopeThreads / 64 - 1) / (kRopeThreads / 64);  // a wave per row
  if (blocks > 0x7fffffff) return PULSAR_EUNSUPPORTED;
  auto s = (hipStream_t)stream;
  const auto kern = d == 128 ? (pos ? rope_kernel<128, true> : rope_kernel<128, false>)
                             : (pos ? rope_kernel<64, true> : rope_kernel<64, false>);
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kRopeThreads), 0, s, (uint16_t*)X, rows,
                     n_rows, H, pos, pos_offset, f);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}

}  // extern "C"
