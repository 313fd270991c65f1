// Flash-style attention on gfx950 bf16 matrix cores, shared by
//  * Phase 1: index-causal attention over block i's assembled input
//    [S_sink || Sigma_0..Sigma_{i-1} || B_i] (Eq. 3, Eq. 1), whose rows are
//    gathered from the global Q/K/V through the row -> position map, and
//  * Phase 2: unmasked attention of the query over each retained KV shard,
//    split along the keys, giving (o, lse) partials (Algorithm 1, Phase 2).
//
// Work decomposition
//   A work item is one row tile of one KV head (and head slice, sequence or
//   split); a workgroup is 8 wavefronts (2 per SIMD), all reading the same
//   KV head.  When the group size Hq/Hkv is a multiple of 4, four consecutive
//   waves are 4 query heads of that group over the same 32*QT rows
//   (grouped-query sharing: one K/V tile in LDS feeds four heads); further
//   waves, or smaller groups, split the rows.
//   Items run heaviest causal row tile first.  Causal launches are
//   persistent: one workgroup per CU takes items from a queue per KV head,
//   its home queue (blockIdx mod Hkv; workgroups are placed on the XCDs
//   round-robin, so with 8 KV heads each XCD's L2 serves one head) and, once
//   that is empty, the others' -- the XCDs run at different clocks, and a
//   fixed share per XCD left the fast ones idle for the last few percent.
//   Otherwise (Phase 2, or no counter slot) each workgroup is one item,
//   with the KV head the fastest-varying index of its id.
//
// Per wavefront, per 64-key tile, in two 32-key halves (32x32x16 bf16 MFMA,
// fp32 accumulate)
//   S^T = K Q^T   A = K rows from LDS, B = Q fragments held in registers;
//                 the lane of query q holds 16 scores of q per half.
//   softmax       log2 domain.  Scores are taken relative to a fixed per-row
//                 reference (the row's maximum over the first 32 keys), so the
//                 O accumulator is only ever touched by the matrix cores; the
//                 final division by the weight sum makes the result exact.
//                 Should the weight sum exceed 2^88 (a later score far above
//                 the reference), the workgroup repeats the pass with the
//                 classic online softmax, which raises the running maximum
//                 and rescales O.  P enters the PV product rounded to bf16; O is
//                 divided by the sum of those rounded weights (an exact convex
//                 combination), while the LSE uses the fp32 sum.
//   O^T += V^T P^T  A = V^T, read from the V tile (keys as rows) in LDS with
//                 transposing reads; B = P, which is already in the
//                 B-operand layout because K rows are stored in LDS with bits
//                 2 and 3 of the key index swapped.
//   K and V tiles move from HBM to LDS by buffer loads that write LDS
//   directly.  Three LDS stages; the K row padding (2d+16 B) and a chunk
//   swizzle of the V rows keep the fragment reads free of bank conflicts.
//   The two wavefronts of a SIMD run ping-pong: one multiplies (PV of the
//   previous tile, S of the current one) while the other computes weights,
//   with a workgroup barrier between phases.
//
// This header holds the kernel template; attn.hip chooses the instantiation
// and attn_d64.hip / attn_d128.hip instantiate it per head dimension.
#pragma once
#include <type_traits>

#include "common.hpp"

namespace pulsar_attn {

struct KernelArgs {
  AttnLaunch a;
  int group;          // Hq / Hkv
  int heads_per_wg;   // query heads per workgroup (1, 2 or 4)
  int hsub;           // workgroups per KV head along the head axis
  int rows_per_wg;    // query rows per workgroup
  int n_row_tiles;
  int nz;             // z extent (sequences, or shards x splits)
  // Persistent causal launch: the work counters of this launch (one per KV
  // head, then the count of finished workgroups; all zero before the launch
  // and left zero by it), or null for one workgroup per item.
  unsigned* sched;
  int grid;           // workgroups of a persistent launch (one per CU)
};

// Launch of one instantiation for head dimension D (defined in the per-D
// sources).
int launch_d64(const KernelArgs& ka, bool causal, bool lse, int mode, hipStream_t stream);
int launch_d128(const KernelArgs& ka, bool causal, bool lse, int mode, hipStream_t stream);

}  // namespace pulsar_attn

namespace {
using pulsar_attn::KernelArgs;

constexpr int BN = 64;          // keys per tile
constexpr float MAX_SLACK = 8.0f;  // exact pass: log2 slack before the running max is raised
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
constexpr int kBufferFlags = 0x00020000;  // raw 32-bit buffer access (word 3 of the resource)
__device__ constexpr bf16x2 kOnes2 = {(__bf16)1.0f, (__bf16)1.0f};

typedef __attribute__((address_space(3))) uint8_t lds_u8;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

template <int D>
struct Tile {
  static constexpr int CPR = D / 8;               // 16-byte data chunks per row
  static constexpr int K_CH = CPR + 1;            // K row: data + one pad chunk
  static constexpr int K_STRIDE = 16 * K_CH;      // bytes per K row in LDS
  static constexpr int K_BYTES = BN * K_STRIDE;   // = K_CH KiB
  static constexpr int V_BYTES = BN * D * 2;      // raw V: rows = keys
  static constexpr int STAGE = K_BYTES + V_BYTES;
  static constexpr int V_SEGS = V_BYTES / 1024;   // 1 KiB load segments of a V tile
  static constexpr int LDS = 3 * STAGE + 3 * BN * 4;  // three stages + three position rows
};



// One 16-byte-per-lane buffer load that writes LDS directly: lane l's 16
// bytes land at LDS byte lds_base + 16*l.  Issued from asm so that the
// compiler does not order the key loop's LDS reads after it (it cannot tell
// that they read the other stage); the loop waits for it explicitly
// (vmcnt) before the barrier that publishes the stage.
__device__ __forceinline__ void lds_dma16(__amdgpu_buffer_rsrc_t rsrc, uint32_t voffset,
                                          uint32_t lds_base) {
  asm volatile("buffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(voffset), "s"(rsrc), "{m0}"(lds_base)
               : "memory");
}

__device__ __forceinline__ int swap_bits23(int r) {
  return (r & ~12) | ((r >> 1) & 4) | ((r << 1) & 8);
}

// Matrix-phase fragment reads run this many matrix steps ahead.
constexpr int MDEPTH = 4;

template <int D, int QT, int WAVES, bool CAUSAL, bool LSE, int MODE>
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(3 - QT, 3 - QT)))
void attn_fwd_kernel(KernelArgs ka) {
  constexpr int THREADS = 64 * WAVES;
  using T = Tile<D>;
  constexpr int QR = 32 * QT;        // rows per wavefront
  constexpr int DS = D / 16;         // k-steps of the S product
  constexpr int DT = D / 32;         // 32-row tiles of O^T
  constexpr int SEG_PER_WAVE = (T::K_CH + 3) / 4;  // K segments per group-1 wave
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const AttnLaunch& a = ka.a;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // ---- work items ------------------------------------------------------------
  // Item k of the queue of KV head h is (head slice, z, row tile) with the
  // heaviest row tile first; a persistent workgroup holds item h * qlen + k,
  // one of a plain launch is item k * Hkv + h (its blockIdx).
  unsigned* const sched = CAUSAL ? ka.sched : nullptr;
  const bool persistent = sched != nullptr;
  const int qlen = ka.hsub * ka.nz * ka.n_row_tiles;
  const int home = blockIdx.x % a.Hkv;
  __shared__ int s_item;
  // thread 0: the next item from the home queue, else from the others (a
  // queue read as exhausted is skipped without an increment); -1 when all
  // are empty.  Every queue hands out each of its qlen items exactly once.
  auto claim = [&]() -> int {
    for (int i = 0; i < a.Hkv; ++i) {
      const int h = home + i < a.Hkv ? home + i : home + i - a.Hkv;
      if (__hip_atomic_load(&sched[h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >=
          (unsigned)qlen)
        continue;
      const unsigned k = atomicAdd(&sched[h], 1u);
      if (k < (unsigned)qlen) return h * qlen + (int)k;
    }
    return -1;
  };
  int item = blockIdx.x;
  if (persistent) {
    if (tid == 0) s_item = claim();
    __syncthreads();
    item = s_item;
  }
  int last_z = -1;
  while (item >= 0) {
  int next_item = -1;
  {  // one item
  // lane-derived values are re-formed per item from an opaque copy of the
  // thread index, so that the compiler does not hold them in registers
  // across items
  int tid_i = threadIdx.x;
  asm volatile("" : "+v"(tid_i));
  const int tid = tid_i;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int g = lane >> 5;
  const int kvh = persistent ? item / qlen : item % a.Hkv;
  int kk = persistent ? item - kvh * qlen : item / a.Hkv;
  const int hs = kk % ka.hsub;
  kk /= ka.hsub;
  const int z = kk % ka.nz;
  kk /= ka.nz;
  const int row_tile = ka.n_row_tiles - 1 - kk;

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
  const uint16_t* Qz = a.Q + zkv * a.q_zstride + (int64_t)head * D;
  const float c2 = a.scale_log2;

  lds_u8* const stage0 = (lds_u8*)smem;  // LDS address space: reads take immediate offsets
  int32_t* lpos = reinterpret_cast<int32_t*>(smem + 3 * T::STAGE);  // [3][BN]
  auto pos_of = [&](int t) { return lpos + (t % 3) * BN; };
  int* run_base = lpos + 3 * BN;                                      // [map.n_runs]
  __syncthreads();  // the previous item's LDS reads are done
  if constexpr (MODE == MAP_SUMMARY)
    if (z != last_z) build_run_table(a.map, sel, run_base, tid, THREADS);
  last_z = z;
  __syncthreads();

  // K/V rows are read through buffer resources covering this sequence (or
  // shard), with 32-bit byte offsets.
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
    const int p = r < a.n_q ? row_position_m<MODE>(a.map, run_base, r) : 0;
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
  // reference max, fp32 weight sum, and the bf16 weight sum in NSUM
  // independent partial sums (so the dot2 accumulations are not one chain)
  constexpr int NSUM = 4;
  float m_ref[QT], l_run[QT], lr_run[QT][NSUM];

  // ---- tile loads --------------------------------------------------------------
  // Wave 0 writes the global positions of a tile's 64 keys to LDS (-1 past
  // the end), except with the identity map, whose positions are the key
  // indices themselves.
  // K: the four group-1 waves move the K tile straight into LDS, in K_CH
  //   segments of 1 KiB (pad chunks included); wave 4+w issues segments w,
  //   w+4, ...  Lane l of segment sg fills the 16 bytes at byte 16*l of it:
  //   slot 64*sg + l, i.e. row slot / K_CH, chunk slot % K_CH.  K row r holds
  //   key swap_bits23(r).  A pad chunk re-reads chunk 0 of its row, and a key
  //   past the end reads row 0 of the sequence: both finite, never weighted.
  // V: the four group-0 waves move the V tile straight into LDS as well,
  //   keys as rows (2D bytes each): wave w issues segments w, w+4, ...; lane
  //   l of segment sg fills chunk position (64 sg + l) % CPR of row
  //   (64 sg + l) / CPR, which holds 16-byte chunk position ^ vswz(row) of
  //   that key.  The PV product reads V^T fragments from it with transposing
  //   reads (v_frag); the chunk swizzle puts the four rows that one 16-lane
  //   group of such a read touches in disjoint banks.  A key past the end
  //   reads row 0 of the sequence: finite, and its weight is zero.
  auto tile_positions = [&](int j, int32_t* dst) {
    if (MODE != MAP_IDENTITY && tid < BN) {
      const int k = kv_begin + j * BN + tid;
      dst[tid] = k < kv_end ? row_position_m<MODE>(a.map, run_base, k) : -1;
    }
  };
  // The same in two steps for the loop, run by wave 0 inside its matrix
  // phase (where its vector unit is idle): pos_start reads the run-table
  // entry of its key, pos_finish adds the offset and writes the position.
  int2 pos_pending = int2{-1, -1};
  int pos_raw = 0;
  auto pos_start = [&](int j) {
    const int k = kv_begin + j * BN + lane;
    pos_pending = k < kv_end ? row_position_split<MODE>(a.map, k) : int2{-1, -1};
    pos_raw = pos_pending.x >= 0 ? run_base[pos_pending.x] : 0;
  };
  auto pos_finish = [&](int j) { pos_of(j)[lane] = pos_raw + pos_pending.y; };
  // Position of key row `row` of tile t for the loads: from the LDS row of
  // the tile, or (identity map) directly; a key past the end reads row 0.
  auto kpos = [&](int t, int row) -> uint32_t {
    if constexpr (MODE == MAP_IDENTITY) {
      const int k = kv_begin + t * BN + row;
      return k < kv_end ? (uint32_t)(a.map.offset + k) : 0u;
    } else {
      return (uint32_t)max(pos_of(t)[row], 0);
    }
  };
  int dma_row[SEG_PER_WAVE];
  uint32_t dma_col[SEG_PER_WAVE];
  const int wk = wave - 4;  // group-1 wave index
#pragma unroll
  for (int i = 0; i < SEG_PER_WAVE; ++i) {
    const int slot = (wk + 4 * i) * 64 + lane;
    const int r = slot / T::K_CH;
    const int col = slot - r * T::K_CH;
    dma_row[i] = swap_bits23(r & (BN - 1));
    dma_col[i] = head_off + (uint32_t)(col < T::CPR ? col : 0) * 16;
  }
  auto issue_k = [&](int tile, lds_u8* st) {
    const uint32_t st_lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)st);
    // all positions first, unconditionally (dma_row is a valid row for every
    // i), so that the reads are issued together: each asm load orders later
    // LDS reads; only the load itself depends on the (wave-uniform) segment
    uint32_t p[SEG_PER_WAVE];
#pragma unroll
    for (int i = 0; i < SEG_PER_WAVE; ++i) p[i] = kpos(tile, dma_row[i]);
#pragma unroll
    for (int i = 0; i < SEG_PER_WAVE; ++i) {
      const int sg = wk + 4 * i;
      if (sg < T::K_CH)
        lds_dma16(k_rsrc, __umul24(p[i], row_bytes) + dma_col[i], st_lds + sg * 1024);
    }
  };
  constexpr int NVSEG = T::V_SEGS / 4;  // V segments per group-0 wave
  auto vswz = [](int r) { return (4 * ((r * T::CPR) / 16)) % T::CPR; };
  int vdma_row[NVSEG];
  uint32_t vdma_col[NVSEG];
#pragma unroll
  for (int i = 0; i < NVSEG; ++i) {
    const int slot = (wave + 4 * i) * 64 + lane;  // meaningful for group 0
    const int r = (slot / T::CPR) & (BN - 1);
    vdma_row[i] = r;
    vdma_col[i] = head_off + (uint32_t)((slot % T::CPR) ^ vswz(r)) * 16;
  }
  auto issue_v = [&](int tile, lds_u8* st) {
    const uint32_t st_lds =
        __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(st + T::K_BYTES));
    uint32_t p[NVSEG];  // all positions first: each asm load orders later LDS reads
#pragma unroll
    for (int i = 0; i < NVSEG; ++i) p[i] = kpos(tile, vdma_row[i]);
#pragma unroll
    for (int i = 0; i < NVSEG; ++i)
      lds_dma16(v_rsrc, __umul24(p[i], row_bytes) + vdma_col[i], st_lds + (wave + 4 * i) * 1024);
  };

  // ---- building blocks of one 32-key half --------------------------------------
  // S^T of keys u*32..u*32+31 of the tile in LDS against this wave's queries.
  auto k_frag = [&](const lds_u8* sK, int u, int s) {
    return *reinterpret_cast<const lds_bf16x8*>(sK + (u * 32 + l32) * T::K_STRIDE +
                                                (16 * s + 8 * g) * 2);
  };
  // V^T rows e*32.., keys u*32+16c.. of the tile, as the A operand of PV,
  // from the raw V tile with two transposing reads.  Within each 16-lane
  // group such a read hands lane i, for slot j, element i%4 of the four that
  // lane 4j + i/4 addressed; so lane 16a + 4j + q addresses key row
  // 8(a/2) + j (+4 for the second read) at head_dim 16(a%2) + 4q, and lane
  // 16a + i receives head_dim 16(a%2) + i of keys 8(a/2) .. +7.
  uint32_t vtr_base[DT];
  {
    const int a16 = lane >> 4, j = (lane >> 2) & 3, q = lane & 3;
    const int trow = 8 * (a16 >> 1) + j;  // vswz of every row read equals vswz(trow)
    const int cb = 2 * (a16 & 1) + (q >> 1);
#pragma unroll
    for (int e = 0; e < DT; ++e)
      vtr_base[e] = trow * (2 * D) + 16 * ((4 * e + cb) ^ vswz(trow)) + 8 * (q & 1);
  }
  auto v_frag = [&](const lds_u8* sV, int u, int c, int e) -> bf16x8 {
    const lds_u8* b = sV + vtr_base[e] + (u * 32 + 16 * c) * (2 * D);
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)b);
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(b + 4 * (2 * D)));
    return __builtin_bit_cast(bf16x8,
                              (s16x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
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
          lr_run[t][v / 2] = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{w[v], w[v + 1]}, kOnes2,
                                                             lr_run[t][v / 2], false);
      }
      if (LSE) l_run[t] += psum;
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
#pragma unroll
      for (int j = 0; j < NSUM; ++j) lr_run[t][j] = 0.f;
    }
  };
  // ---- ping-pong schedule ------------------------------------------------
  // Waves 0-3 (group 0) and 4-7 (group 1) share the four SIMDs pairwise.
  // Every wave alternates a matrix phase M_m (PV of tile m-1, then S of
  // tile m) and a vector phase V_m (the weights of tile m), with a workgroup
  // barrier after each phase; group 1 runs one phase behind group 0, so on
  // every SIMD one wave's exponentials overlap the other wave's matrix
  // instructions.  Between barriers k-1 and k, group 0 runs its phase k and
  // group 1 its phase k-1 (phase 2m = M_m, 2m+1 = V_m).
  //
  // A half past every row of the wave (causal) or past the last key is
  // still multiplied; the mask gives it zero weight.
  //
  // Tiles rotate through three LDS stages (tile t in stage t % 3).  Tile t's
  // K is read in phases 2t and 2t+1 of the workgroup (S by group 0, then by
  // group 1) and its V in phases 2t+2 and 2t+3 (PV).  Group 1 moves K_t
  // into LDS during its V_{t-2} and waits for it at the end of its M_{t-1};
  // group 0 moves V_t into LDS during its V_{t-1} and waits for it at the end
  // of its V_t.  Stage t % 3 last held tile t-3, whose last reader ran before
  // either load was issued.  Wave 0 writes tile t's key positions during
  // V_{t-2}.
  static_assert(WAVES == 8, "the ping-pong schedule pairs waves w and w+4 on one SIMD");
  const int grp = wave >> 2;
  // The stage offset goes through readfirstlane so that loop strength
  // reduction keeps it one scalar (fragment reads then take immediate
  // offsets from one base) instead of one induction variable per read.
  auto stage_of = [&](int t) {
    return stage0 + __builtin_amdgcn_readfirstlane((t % 3) * T::STAGE);
  };
  auto key_of = [&](int t, int u) { return kv_begin + t * BN + 32 * u; };
  auto edge = [&](int t, int u) {
    const int kh = key_of(t, u);
    return CAUSAL ? (kh + 31 > row0) : (kh + 32 > kv_end);
  };
  f32x16 S[2][QT];
  bf16x8 P[2][2][QT];
  // Matrix phase with every half live, as one block: PV of the previous
  // tile (four independent accumulators), then S of this tile (two chains).
  // Fragment reads run MDEPTH matrix steps ahead through a register ring,
  // and a scheduling fence after each step keeps that order.
  auto m_phase_full = [&](const lds_u8* sV, const lds_u8* sK, int pos_tile) {
    constexpr int NPV = 4 * DT, N = NPV + 2 * DS;
    auto frag = [&](int i) -> bf16x8 {
      if (i < NPV) return v_frag(sV, i / (2 * DT), (i / DT) % 2, i % DT);
      return k_frag(sK, (i - NPV) % 2, (i - NPV) / 2);
    };
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int t = 0; t < QT; ++t) S[u][t] = f32x16{};
    bf16x8 ring[MDEPTH];
#pragma unroll
    for (int i = 0; i < MDEPTH; ++i) ring[i] = frag(i);
    // wave 0 forms the key positions of tile pos_tile (if any) here
    const bool do_pos = MODE != MAP_IDENTITY && wave == 0 && pos_tile >= 0;
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if (i == 2 && do_pos) pos_start(pos_tile);
      if (i == N - 8 && do_pos) pos_finish(pos_tile);
      const bf16x8 f = ring[i % MDEPTH];
      if (i + MDEPTH < N) ring[i % MDEPTH] = frag(i + MDEPTH);
      if (i < NPV) {
        const int u = i / (2 * DT), c = (i / DT) % 2, e = i % DT;
#pragma unroll
        for (int t = 0; t < QT; ++t)
          acc[e][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f, P[u][c][t], acc[e][t], 0, 0, 0);
      } else {
        const int u = (i - NPV) % 2, sk = (i - NPV) / 2;
#pragma unroll
        for (int t = 0; t < QT; ++t)
          S[u][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f, qf[t][sk], S[u][t], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // EXACT = false: fixed per-row reference (the row's maximum over the
  // first 32 keys), O touched only by MFMA.  EXACT = true: classic online
  // softmax; the running maximum is raised when a tile's maximum exceeds it
  // by more than 2^8, and O and the sums are rescaled.
  auto run_pass = [&](auto exact_tag) {
    constexpr bool EXACT = decltype(exact_tag)::value;
    reset();
    tile_positions(0, pos_of(0));
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int t = 0; t < QT; ++t) P[u][c][t] = bf16x8{};
    for (int i = tid; i < T::V_BYTES / 16; i += THREADS)
      reinterpret_cast<__attribute__((address_space(3))) u32x4*>(stage_of(2) + T::K_BYTES)[i] =
          u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
    if (ntiles > 0) {
      if (grp == 1) issue_k(0, stage_of(0));
      if (grp == 0) issue_v(0, stage_of(0));
    }
    if (ntiles > 1) tile_positions(1, pos_of(1));
    if (grp == 1) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (grp == 1) {  // K of tile 1, then group 1's lag barrier
      if (ntiles > 1) issue_k(1, stage_of(1));
      __syncthreads();
    }
    // The matrix phase runs at raised wave priority, so that the SIMD's
    // arbiter issues its matrix instructions ahead of the partner wave's
    // vector instructions whenever both are ready.
    // Each phase ends in phase_barrier(): the scheduling fences keep
    // arithmetic from moving across the workgroup barrier (it only orders
    // memory), so that no phase's work leaks into the next interval.
    auto phase_barrier = [&]() {
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      __builtin_amdgcn_sched_barrier(0);
    };
    auto m_phase_begin = [&]() {
      __builtin_amdgcn_s_setprio(1);
      __builtin_amdgcn_sched_barrier(0);
    };
    auto m_phase_end = [&]() {
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(0);
      if (grp == 1) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      phase_barrier();
    };
    // V_m: weights of tile m (both halves; a half with no visible key is
    // fully masked and weighs zero).
    auto v_phase = [&](int m) {
      if (grp == 1 && m + 2 < ntiles) issue_k(m + 2, stage_of(m + 2));
      if (grp == 0 && m + 1 < ntiles) issue_v(m + 1, stage_of(m + 1));
#pragma unroll
      for (int u = 0; u < 2; ++u)
        if (EXACT || edge(m, u)) apply_mask(key_of(m, u), S[u]);
      if (EXACT) {
        // One raise per tile: both halves' weights enter O only in M_{m+1},
        // so they must share the reference.
#pragma unroll
        for (int t = 0; t < QT; ++t) {
          const float mx = fmaxf(row_max(S[0][t]), row_max(S[1][t]));
          const bool raise = mx > m_ref[t] + MAX_SLACK;
          const float m_use = raise ? mx : m_ref[t];
          if (__any(raise)) {
            const float alpha = __builtin_amdgcn_exp2f(m_ref[t] - m_use);
#pragma unroll
            for (int e = 0; e < DT; ++e) acc[e][t] *= alpha;
            l_run[t] *= alpha;
#pragma unroll
            for (int j = 0; j < NSUM; ++j) lr_run[t][j] *= alpha;
          }
          m_ref[t] = m_use;
        }
      } else if (m == 0) {  // half 0 of tile 0 always has a visible key
#pragma unroll
        for (int t = 0; t < QT; ++t) m_ref[t] = row_max(S[0][t]);
      }
      weights(S[0], P[0]);
      weights(S[1], P[1]);
      // V of tile m must be in LDS for M_{m+1}; only V of tile m+1 may still
      // be in flight.
      if (grp == 0) {
        if (m + 1 < ntiles) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NVSEG) : "memory");
        else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      }
      phase_barrier();
    };
    // Every matrix phase is the full one: M_0 multiplies the zeroed V of
    // stage 2 by P = 0, and M_ntiles computes an S that is never used (from
    // finite LDS data).
    for (int m = 0; m <= ntiles; ++m) {
      m_phase_begin();
      // group 0's M_m forms the positions of tile m + 2 (read by group 1's
      // K issue in its V_m and group 0's V issue in V_{m+1}); the row it
      // overwrites last served tile m - 1, whose last reader ran two
      // intervals earlier
      m_phase_full(stage_of(m + 2) + T::K_BYTES, stage_of(m), m + 2 < ntiles ? m + 2 : -1);
      m_phase_end();
      if (m < ntiles) v_phase(m);
    }
    if (grp == 0) __syncthreads();  // matches group 1's lag barrier
  };

  // ---- fast pass, then the exact pass only after an overflow flag -----------
  run_pass(std::false_type{});
  // Every weight is at most the final sum, so a finite sum below 2^88 bounds
  // them all; above that (or not finite) the exact pass takes over.
  bool overflow = false;
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const float lr = (lr_run[t][0] + lr_run[t][1]) + (lr_run[t][2] + lr_run[t][3]);
    overflow |= !(lr <= 0x1p88f);
  }
  if (__syncthreads_or(overflow)) run_pass(std::true_type{});

  // The next item is claimed only now (its latency overlaps the stores
  // below): claiming it earlier commits a workgroup to it before it is known
  // which workgroup frees up first, which spreads the end of the launch.
  if (persistent && tid == 0) next_item = claim();

  // ---- epilogue: normalise, write O and LSE ---------------------------------
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const float l_tot = l_run[t] + __shfl_xor(l_run[t], 32, 64);
    const float lr = (lr_run[t][0] + lr_run[t][1]) + (lr_run[t][2] + lr_run[t][3]);
    const float lr_tot = lr + __shfl_xor(lr, 32, 64);
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
  }  // one item
  if (!persistent) break;
  __syncthreads();
  if (threadIdx.x == 0) s_item = next_item;
  __syncthreads();
  item = s_item;
  }  // items
  // The last workgroup to finish (every claim of every workgroup is done by
  // then) leaves the counters zero for the next launch on this slot.
  if (persistent && threadIdx.x == 0 && atomicAdd(&sched[a.Hkv], 1u) == gridDim.x - 1) {
    for (int h = 0; h <= a.Hkv; ++h) atomicExch(&sched[h], 0u);
  }
}

template <int D, int QT, int WAVES, bool CAUSAL, bool LSE, int MODE>
int launch_impl(const KernelArgs& ka, hipStream_t stream) {
  int64_t nwg = (int64_t)ka.n_row_tiles * ka.hsub * ka.a.Hkv * ka.nz;
  if (nwg == 0) return PULSAR_OK;
  if (CAUSAL && ka.sched != nullptr && nwg > ka.grid) nwg = ka.grid;
  if (nwg > 0x7fffffff) return PULSAR_EUNSUPPORTED;
  const int64_t lds = Tile<D>::LDS + (int64_t)ka.a.map.n_runs * 4;
  // the kernel's static LDS (the item broadcast) comes on top, aligned
  if (lds + 16 > PULSAR_LDS_BYTES) return PULSAR_EUNSUPPORTED;
  auto kern = attn_fwd_kernel<D, QT, WAVES, CAUSAL, LSE, MODE>;
  if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lds) != hipSuccess)
    return PULSAR_EHIP;
  hipLaunchKernelGGL(kern, dim3((unsigned)nwg), dim3(64 * WAVES), (size_t)lds, stream, ka);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}


// Every (causal, lse, map mode) instantiation for head dimension D: the
// unmasked (Phase 2) kernels only see the identity map.
template <int D, int QT, int WAVES_C, int WAVES_P>
int launch_for_d(const KernelArgs& ka, bool causal, bool lse, int mode, hipStream_t stream) {
  if (!causal) {
    if (mode != MAP_IDENTITY) return PULSAR_EUNSUPPORTED;
    return lse ? launch_impl<D, QT, WAVES_P, false, true, MAP_IDENTITY>(ka, stream)
               : launch_impl<D, QT, WAVES_P, false, false, MAP_IDENTITY>(ka, stream);
  }
  switch (mode) {
    case MAP_IDENTITY:
      return lse ? launch_impl<D, QT, WAVES_C, true, true, MAP_IDENTITY>(ka, stream)
                 : launch_impl<D, QT, WAVES_C, true, false, MAP_IDENTITY>(ka, stream);
    case MAP_SUMMARY:
      return lse ? launch_impl<D, QT, WAVES_C, true, true, MAP_SUMMARY>(ka, stream)
                 : launch_impl<D, QT, WAVES_C, true, false, MAP_SUMMARY>(ka, stream);
    case MAP_ANCHOR:
      return lse ? launch_impl<D, QT, WAVES_C, true, true, MAP_ANCHOR>(ka, stream)
                 : launch_impl<D, QT, WAVES_C, true, false, MAP_ANCHOR>(ka, stream);
    case MAP_EVEN:
      return lse ? launch_impl<D, QT, WAVES_C, true, true, MAP_EVEN>(ka, stream)
                 : launch_impl<D, QT, WAVES_C, true, false, MAP_EVEN>(ka, stream);
    default: return PULSAR_EINVAL;
  }
}

}  // namespace

// Queries per wavefront = 32 * QT with QT = 1, so that two wavefronts fit
// on a SIMD (QT = 2 would halve the LDS reads per matrix instruction but
// needs the whole register file of a SIMD, giving up the ping-pong pairing).
constexpr int kQT = 1;

// Wavefronts per workgroup: 8, i.e. two 32-row groups of four heads, so that
// one K/V tile in LDS serves 64 rows of four heads (for Phase 2: all 64
// queries); the two wavefronts that share a SIMD interleave their matrix and
// vector work.
constexpr int kCausalWaves = 8;
constexpr int kPartialWaves = 8;
