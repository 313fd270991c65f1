// Flash-style attention on gfx950 bf16 matrix cores, shared by
//  * Phase 1: index-causal attention over block i's assembled input
//    [S_sink || Sigma_0..Sigma_{i-1} || B_i] (Eq. 3, Eq. 1), whose rows are
//    gathered from the global Q/K/V through the row -> position map, and
//  * Phase 2: unmasked attention of the query over each retained KV shard,
//    split along the keys, giving (o, lse) partials (Algorithm 1, Phase 2).
//
// Work decomposition
//   A workgroup is 8 wavefronts (2 per SIMD), all reading the same
//   KV head.  When the group size Hq/Hkv is a multiple of 4, four consecutive
//   waves are 4 query heads of that group over the same 32*QT rows
//   (grouped-query sharing: one K/V tile in LDS feeds four heads); further
//   waves, or smaller groups, split the rows.
//   Workgroup ids run heaviest causal row tile first, and the KV head is the
//   fastest-varying index, so with 8 KV heads each XCD's L2 serves one head.
//
// Per wavefront, per 64-key tile, in two 32-key halves (32x32x16 bf16 MFMA,
// fp32 accumulate)
//   S^T = K Q^T   A = K rows from LDS, B = Q fragments held in registers;
//                 the lane of query q holds 16 scores of q per half.
//   softmax       log2 domain.  Scores are taken relative to a fixed per-row
//                 reference (the row's maximum over the first 32 keys), so the
//                 O accumulator is only ever touched by the matrix cores; the
//                 final division by the weight sum makes the result exact.
//                 Should a weight exceed 2^64 (a later score far above the
//                 reference), the workgroup repeats the pass with the classic
//                 online softmax, which raises the running maximum and
//                 rescales O.  P enters the PV product rounded to bf16; O is
//                 divided by the sum of those rounded weights (an exact convex
//                 combination), while the LSE uses the fp32 sum.
//   O^T += V^T P^T  A = V^T from LDS (V is transposed on its way into LDS),
//                 B = P, which is already in the B-operand layout because K
//                 rows are stored in LDS with bits 2 and 3 of the key index
//                 swapped.
//   K/V tiles are double-buffered: the next tile's global loads are issued
//   before the current tile's math and written to LDS after it.
#include <type_traits>

#include "common.hpp"

namespace {

constexpr int BN = 64;          // keys per tile
constexpr float MAX_SLACK = 8.0f;  // exact pass: log2 slack before the running max is raised
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
constexpr int kBufferFlags = 0x00020000;  // raw 32-bit buffer access (word 3 of the resource)
__device__ constexpr bf16x2 kOnes2 = {(__bf16)1.0f, (__bf16)1.0f};

template <int D>
struct Tile {
  static constexpr int K_STRIDE = D * 2 + 16;   // bytes per K row in LDS (padded)
  static constexpr int V_STRIDE = BN * 2 + 16;  // bytes per V^T row (one head_dim entry)
  static constexpr int K_BYTES = BN * K_STRIDE;
  static constexpr int V_BYTES = D * V_STRIDE;
  static constexpr int STAGE = K_BYTES + V_BYTES;
  static constexpr int LDS = 2 * STAGE + 2 * BN * 4;  // two stages + two position rows
  static constexpr int CPR = D / 8;               // 16-byte chunks per row
  static constexpr int V_UNITS = (BN / 4) * CPR;  // 4 keys x 8 dims per unit (<= threads)
};

struct KernelArgs {
  AttnLaunch a;
  int group;          // Hq / Hkv
  int heads_per_wg;   // query heads per workgroup (1, 2 or 4)
  int hsub;           // workgroups per KV head along the head axis
  int rows_per_wg;    // query rows per workgroup
  int n_row_tiles;
  int nz;             // z extent (sequences, or shards x splits)
};

__device__ __forceinline__ int swap_bits23(int r) {
  return (r & ~12) | ((r >> 1) & 4) | ((r << 1) & 8);
}

__device__ __forceinline__ uint32_t pack_lo(uint32_t a, uint32_t b) {
  return (a & 0xFFFFu) | (b << 16);
}
__device__ __forceinline__ uint32_t pack_hi(uint32_t a, uint32_t b) {
  return (a >> 16) | (b & 0xFFFF0000u);
}

template <int D, int QT, int WAVES, bool CAUSAL, bool LSE>
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(3 - QT, 3 - QT)))
void attn_fwd_kernel(KernelArgs ka) {
  constexpr int THREADS = 64 * WAVES;
  using T = Tile<D>;
  constexpr int QR = 32 * QT;        // rows per wavefront
  constexpr int DS = D / 16;         // k-steps of the S product
  constexpr int DT = D / 32;         // 32-row tiles of O^T
  constexpr int KR = BN * T::CPR / THREADS;  // consecutive K rows loaded per thread
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const AttnLaunch& a = ka.a;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int g = lane >> 5;

  // ---- workgroup -> (kv head, head slice, z, row tile) ---------------------
  int bid = blockIdx.x;
  const int kvh = bid % a.Hkv;
  bid /= a.Hkv;
  const int hs = bid % ka.hsub;
  bid /= ka.hsub;
  const int z = bid % ka.nz;
  bid /= ka.nz;
  const int row_tile = ka.n_row_tiles - 1 - bid;

  const int head = kvh * ka.group + hs * ka.heads_per_wg + (wave % ka.heads_per_wg);
  const int wg_row0 = row_tile * ka.rows_per_wg;
  const int row0 = wg_row0 + (wave / ka.heads_per_wg) * QR;

  const int zkv = z / a.nsplit;
  const int split = z - zkv * a.nsplit;
  const int kv_begin = split * a.split_len;
  int kv_end = min(a.n_kv, kv_begin + a.split_len);
  if (CAUSAL) kv_end = min(kv_end, wg_row0 + ka.rows_per_wg);
  const int n_keys = max(0, kv_end - kv_begin);
  const int ntiles = (n_keys + BN - 1) / BN;

  const int32_t* sel = a.sel ? a.sel + zkv * a.sel_bstride : nullptr;
  const int64_t q_row = (int64_t)a.Hq * D;
  const int64_t kv_row = (int64_t)a.Hkv * D;
  const uint16_t* Qz = a.Q + zkv * a.q_zstride + (int64_t)head * D;
  const uint16_t* Kz = a.K + zkv * a.kv_zstride + (int64_t)kvh * D;
  const uint16_t* Vz = a.V + zkv * a.kv_zstride + (int64_t)kvh * D;
  const float c2 = a.scale_log2;

  uint8_t* stage0 = smem;
  int32_t* lpos = reinterpret_cast<int32_t*>(smem + 2 * T::STAGE);  // [2][BN]
  int* run_base = lpos + 2 * BN;                                      // [map.n_runs]
  build_run_table(a.map, sel, run_base, tid, THREADS);
  __syncthreads();

  // K/V rows are read through buffer resources covering this sequence (or
  // shard); a padded key has position -1, whose offset falls outside the
  // resource, so the hardware returns zeros for it.
  const uint32_t row_bytes = (uint32_t)(a.Hkv * D * 2);
  const __amdgpu_buffer_rsrc_t k_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.K + zkv * a.kv_zstride), (short)0, (int)(a.kv_zstride * 2),
      kBufferFlags);
  const __amdgpu_buffer_rsrc_t v_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.V + zkv * a.kv_zstride), (short)0, (int)(a.kv_zstride * 2),
      kBufferFlags);
  const uint32_t head_off = (uint32_t)(kvh * D * 2);

  // ---- Q fragments (B operand of S^T = K Q^T) --------------------------------
  bf16x8 qf[QT][DS];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int r = row0 + t * 32 + l32;
    const int p = r < a.n_q ? row_position(a.map, run_base, r) : 0;
    const bf16x8* src = reinterpret_cast<const bf16x8*>(Qz + (int64_t)p * q_row) + g;
#pragma unroll
    for (int s = 0; s < DS; ++s) qf[t][s] = r < a.n_q ? src[2 * s] : bf16x8{};
  }
  // Wait for the Q loads here: passing each fragment through an empty asm
  // statement makes the compiler wait for it before the loop and treat it as
  // defined afterwards, so no wait inside the key loop is tied to the Q loads
  // (which would also wait for the next tile's prefetch issued after them).
#pragma unroll
  for (int t = 0; t < QT; ++t)
#pragma unroll
    for (int s = 0; s < DS; ++s) asm volatile("" : "+v"(qf[t][s]));

  f32x16 acc[DT][QT];
  float m_ref[QT], l_run[QT], lr_run[QT];  // reference max, fp32 weight sum, bf16 weight sum

  // ---- cooperative tile loads -----------------------------------------------
  // K: thread t loads rows KR*(t/CPR) .. +KR-1 at 16-byte chunk t%CPR.
  // V: thread t (t < 16*CPR) loads rows 4*(t%16) .. +3 at chunk t/16 and
  //    writes them transposed (head_dim-major) into LDS.
  auto tile_positions = [&](int j, int32_t* dst) {
    if (tid < BN) {
      const int k = kv_begin + j * BN + tid;
      dst[tid] = k < kv_end ? row_position(a.map, run_base, k) : -1;
    }
  };
  u32x4 kreg[KR];
  u32x4 vreg[4];
  const bool v_thread = tid < T::V_UNITS;
  auto load_regs = [&](const int32_t* pos) {
    const int kr0 = KR * (tid / T::CPR);
    int kp[KR];
    if constexpr (KR == 4) {
      const int4 p4 = *reinterpret_cast<const int4*>(pos + kr0);
      kp[0] = p4.x; kp[1] = p4.y; kp[2] = p4.z; kp[3] = p4.w;
    } else {
#pragma unroll
      for (int i = 0; i < KR; ++i) kp[i] = pos[kr0 + i];
    }
    const uint32_t kcol = head_off + (uint32_t)(tid % T::CPR) * 16;
#pragma unroll
    for (int i = 0; i < KR; ++i)
      kreg[i] = __builtin_amdgcn_raw_buffer_load_b128(k_rsrc, (int)((uint32_t)kp[i] * row_bytes + kcol),
                                                      0, 0);
    if (v_thread) {
      const int4 p4 = *reinterpret_cast<const int4*>(pos + 4 * (tid & 15));
      const int vp[4] = {p4.x, p4.y, p4.z, p4.w};
      const uint32_t vcol = head_off + (uint32_t)(tid >> 4) * 16;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr)
        vreg[rr] = __builtin_amdgcn_raw_buffer_load_b128(
            v_rsrc, (int)((uint32_t)vp[rr] * row_bytes + vcol), 0, 0);
    }
  };
  auto store_lds = [&](uint8_t* st) {
    const int kr0 = KR * (tid / T::CPR);
#pragma unroll
    for (int i = 0; i < KR; ++i)
      *reinterpret_cast<u32x4*>(st + swap_bits23(kr0 + i) * T::K_STRIDE + (tid % T::CPR) * 16) =
          kreg[i];
    if (v_thread) {
      uint8_t* sv = st + T::K_BYTES;
      const int kq = tid & 15;
      const int dc = tid >> 4;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        // head_dim entries 8*dc + 2w (low halves) and 8*dc + 2w + 1 (high halves)
        const u32x2 lo = {__builtin_amdgcn_perm(vreg[1][w], vreg[0][w], 0x05040100u),
                          __builtin_amdgcn_perm(vreg[3][w], vreg[2][w], 0x05040100u)};
        const u32x2 hi = {__builtin_amdgcn_perm(vreg[1][w], vreg[0][w], 0x07060302u),
                          __builtin_amdgcn_perm(vreg[3][w], vreg[2][w], 0x07060302u)};
        *reinterpret_cast<u32x2*>(sv + (8 * dc + 2 * w) * T::V_STRIDE + 8 * kq) = lo;
        *reinterpret_cast<u32x2*>(sv + (8 * dc + 2 * w + 1) * T::V_STRIDE + 8 * kq) = hi;
      }
    }
  };

  // ---- building blocks of one 32-key half --------------------------------------
  // S^T of keys u*32..u*32+31 of the tile in LDS against this wave's queries.
  auto s_product = [&](const uint8_t* sK, int u, f32x16 (&S)[QT]) {
#pragma unroll
    for (int t = 0; t < QT; ++t) S[t] = f32x16{};
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const bf16x8 kf = *reinterpret_cast<const bf16x8*>(sK + (u * 32 + l32) * T::K_STRIDE +
                                                         (16 * s + 8 * g) * 2);
#pragma unroll
      for (int t = 0; t < QT; ++t)
        S[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[t][s], S[t], 0, 0, 0);
    }
  };
  // -inf for keys after the query row (causal) or past the last key.
  auto apply_mask = [&](int kh, f32x16 (&S)[QT]) {
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      const int qrow = row0 + t * 32 + l32;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = kh + 16 * (v >> 3) + 8 * g + (v & 7);
        const bool masked = CAUSAL ? (key > qrow || key >= kv_end) : (key >= kv_end);
        if (masked) S[t][v] = -INFINITY;
      }
    }
  };
  auto row_max = [&](const f32x16& S) {
    float mx = S[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) mx = fmaxf(mx, S[v]);
    return fmaxf(mx, __shfl_xor(mx, 32, 64)) * c2;  // both lanes of a query agree
  };
  // Weights relative to m_ref, their bf16-rounded sum (which normalises O),
  // the fp32 sum when the LSE is wanted, and P in the B-operand layout of the
  // PV product.
  auto weights = [&](const f32x16 (&S)[QT], bf16x8 (&pf)[2][QT]) {
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      float psum = 0.f;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        f32x8 p;
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          p[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(S[t][8 * c + v], c2, -m_ref[t]));
          if (LSE) psum += p[v];
        }
        pf[c][t] = __builtin_convertvector(p, bf16x8);
        const bf16x8 w = pf[c][t];
#pragma unroll
        for (int v = 0; v < 8; v += 2)
          lr_run[t] = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{w[v], w[v + 1]}, kOnes2, lr_run[t],
                                                      false);
      }
      if (LSE) l_run[t] += psum;
    }
  };
  auto pv_product = [&](const uint8_t* sV, int u, const bf16x8 (&pf)[2][QT]) {
#pragma unroll
    for (int e = 0; e < DT; ++e)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const bf16x8 vf = *reinterpret_cast<const bf16x8*>(
            sV + (e * 32 + l32) * T::V_STRIDE + (u * 32 + 16 * c + 8 * g) * 2);
#pragma unroll
        for (int t = 0; t < QT; ++t)
          acc[e][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[c][t], acc[e][t], 0, 0, 0);
      }
  };

  auto reset = [&]() {
#pragma unroll
    for (int e = 0; e < DT; ++e)
#pragma unroll
      for (int t = 0; t < QT; ++t) acc[e][t] = f32x16{};
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      m_ref[t] = -INFINITY;
      l_run[t] = 0.f;
      lr_run[t] = 0.f;
    }
  };
  // Tile 0 written to stage 0 and tile 1's positions staged.
  auto prologue = [&]() {
    tile_positions(0, lpos);
    __syncthreads();
    if (ntiles > 1) tile_positions(1, lpos + BN);
    load_regs(lpos);
    store_lds(stage0);
  };
  // Iteration j: wait for tile j in LDS, prefetch tile j+1 into registers, run
  // `body`, then store tile j+1 into the other buffer.
  auto tile_loop = [&](auto&& body) {
    for (int j = 0; j < ntiles; ++j) {
      __syncthreads();
      const int buf = j & 1;
      if (j + 1 < ntiles) load_regs(lpos + (buf ^ 1) * BN);
      if (j + 2 < ntiles) tile_positions(j + 2, lpos + buf * BN);
      const uint8_t* sK = stage0 + buf * T::STAGE;
      body(kv_begin + j * BN, sK, sK + T::K_BYTES);
      if (j + 1 < ntiles) store_lds(stage0 + (buf ^ 1) * T::STAGE);
    }
  };

  // ---- fast pass: fixed per-row reference, O touched only by MFMA -----------
  // The reference is the row's maximum over the first 32 keys; only halves
  // that reach past a query row (or past the last key) are masked.
  bool overflow = false;
  reset();
  if (ntiles > 0) {
    prologue();
    __syncthreads();
    f32x16 S[QT];
    s_product(stage0, 0, S);
    apply_mask(kv_begin, S);
#pragma unroll
    for (int t = 0; t < QT; ++t) m_ref[t] = row_max(S[t]);
  }
  tile_loop([&](int kbase, const uint8_t* sK, const uint8_t* sV) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int kh = kbase + 32 * u;
      if (CAUSAL && kh > row0 + QR - 1) continue;  // every key after every row
      f32x16 S[QT];
      bf16x8 pf[2][QT];
      s_product(sK, u, S);
      if (CAUSAL ? (kh + 31 > row0) : (kh + 32 > kv_end)) apply_mask(kh, S);
      weights(S, pf);
      pv_product(sV, u, pf);
    }
  });
  // Every weight is at most the final sum, so a finite sum below 2^88 bounds
  // them all; above that (or not finite) the exact pass takes over.
#pragma unroll
  for (int t = 0; t < QT; ++t) overflow |= !(lr_run[t] <= 0x1p88f);

  // ---- exact pass: classic online softmax, only after an overflow flag --------
  // The running maximum is raised when a half's maximum exceeds it by more
  // than 2^8, and O and the sums are rescaled.
  if (__syncthreads_or(overflow)) {
    __syncthreads();
    reset();
    if (ntiles > 0) prologue();
    tile_loop([&](int kbase, const uint8_t* sK, const uint8_t* sV) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int kh = kbase + 32 * u;
        if (CAUSAL && kh > row0 + QR - 1) continue;
        f32x16 S[QT];
        bf16x8 pf[2][QT];
        s_product(sK, u, S);
        apply_mask(kh, S);
#pragma unroll
        for (int t = 0; t < QT; ++t) {
          const float mx = row_max(S[t]);
          const bool raise = mx > m_ref[t] + MAX_SLACK;
          const float m_use = raise ? mx : m_ref[t];
          if (__any(raise)) {
            const float alpha = __builtin_amdgcn_exp2f(m_ref[t] - m_use);
#pragma unroll
            for (int e = 0; e < DT; ++e) acc[e][t] *= alpha;
            l_run[t] *= alpha;
            lr_run[t] *= alpha;
          }
          m_ref[t] = m_use;
        }
        weights(S, pf);
        pv_product(sV, u, pf);
      }
    });
  }

  // ---- epilogue: normalise, write O and LSE ---------------------------------
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const float l_tot = l_run[t] + __shfl_xor(l_run[t], 32, 64);
    const float lr_tot = lr_run[t] + __shfl_xor(lr_run[t], 32, 64);
    const float inv = lr_tot > 0.f ? 1.f / lr_tot : 0.f;
    const int qrow = row0 + t * 32 + l32;
    if (qrow < a.n_q) {
      const int64_t obase = ((int64_t)z * a.o_zstride) + ((int64_t)qrow * a.Hq + head) * D;
#pragma unroll
      for (int e = 0; e < DT; ++e)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int dd = e * 32 + 8 * q4 + 4 * g;
          f32x4 o4 = {acc[e][t][4 * q4] * inv, acc[e][t][4 * q4 + 1] * inv,
                      acc[e][t][4 * q4 + 2] * inv, acc[e][t][4 * q4 + 3] * inv};
          if (a.o_bf16) {
            *reinterpret_cast<bf16x4*>(reinterpret_cast<uint16_t*>(a.O) + obase + dd) =
                __builtin_convertvector(o4, bf16x4);
          } else {
            *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(a.O) + obase + dd) = o4;
          }
        }
      if (LSE && g == 0) {
        const float lse = l_tot > 0.f ? (m_ref[t] + __log2f(l_tot)) * 0.69314718055994531f
                                      : -INFINITY;
        a.lse[(int64_t)z * a.lse_zstride + (int64_t)head * a.n_q + qrow] = lse;
      }
    }
  }
}

template <int D, int QT, int WAVES, bool CAUSAL, bool LSE>
int launch_impl(const KernelArgs& ka, hipStream_t stream) {
  const int64_t nwg = (int64_t)ka.n_row_tiles * ka.hsub * ka.a.Hkv * ka.nz;
  if (nwg == 0) return PULSAR_OK;
  if (nwg > 0x7fffffff) return PULSAR_EUNSUPPORTED;
  const int64_t lds = Tile<D>::LDS + (int64_t)ka.a.map.n_runs * 4;
  if (lds > PULSAR_LDS_BYTES) return PULSAR_EUNSUPPORTED;
  auto kern = attn_fwd_kernel<D, QT, WAVES, CAUSAL, LSE>;
  if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lds) != hipSuccess)
    return PULSAR_EHIP;
  hipLaunchKernelGGL(kern, dim3((unsigned)nwg), dim3(64 * WAVES), (size_t)lds, stream, ka);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}

}  // namespace

// Queries per wavefront = 32 * QT.  QT = 2 halves the LDS traffic per matrix
// instruction (each K/V fragment read from LDS feeds two products) but needs
// the whole register file of a SIMD; QT = 1 runs two wavefronts per SIMD.
#ifndef PULSAR_ATTN_QT
#define PULSAR_ATTN_QT 1
#endif
constexpr int kQT = PULSAR_ATTN_QT;

// Wavefronts per workgroup: 8, i.e. two 32-row groups of four heads, so that
// one K/V tile in LDS serves 64 rows of four heads (for Phase 2: all 64
// queries); the two wavefronts that share a SIMD interleave their matrix and
// vector work.
#ifndef PULSAR_CAUSAL_WAVES
#define PULSAR_CAUSAL_WAVES 8
#endif
constexpr int kCausalWaves = PULSAR_CAUSAL_WAVES;
constexpr int kPartialWaves = 8;

int attn_rows_per_wg(int group, bool causal) {
  const int heads_per_wg = group >= 4 ? 4 : group;
  const int waves = causal ? kCausalWaves : kPartialWaves;
  return 32 * kQT * (waves / heads_per_wg);
}

int launch_attention(const AttnLaunch& a, hipStream_t stream) {
  KernelArgs ka;
  ka.a = a;
  ka.group = a.Hq / a.Hkv;
  ka.heads_per_wg = ka.group >= 4 ? 4 : ka.group;
  ka.hsub = ka.group / ka.heads_per_wg;
  ka.rows_per_wg = attn_rows_per_wg(ka.group, a.causal != 0);
  ka.n_row_tiles = (a.n_q + ka.rows_per_wg - 1) / ka.rows_per_wg;
  ka.nz = a.nz_kv * a.nsplit;
  const bool lse = a.lse != nullptr;
  constexpr int CW = kCausalWaves, PW = kPartialWaves;
  if (a.d == 128) {
    if (a.causal)
      return lse ? launch_impl<128, kQT, CW, true, true>(ka, stream)
                 : launch_impl<128, kQT, CW, true, false>(ka, stream);
    return lse ? launch_impl<128, kQT, PW, false, true>(ka, stream)
               : launch_impl<128, kQT, PW, false, false>(ka, stream);
  }
  if (a.causal)
    return lse ? launch_impl<64, kQT, CW, true, true>(ka, stream)
               : launch_impl<64, kQT, CW, true, false>(ka, stream);
  return lse ? launch_impl<64, kQT, PW, false, true>(ka, stream)
             : launch_impl<64, kQT, PW, false, false>(ka, stream);
}
