// Phase-2 partial attention for few query tokens (Algorithm 1, Phase 2:
// (o_h, l_h) of new tokens over a retained shard; Appendix "Phase 2
// Distributed Softmax Merge").  Built for the generation loop, where one new
// token (or a few) attends to every shard: the work is bound by streaming
// K/V from HBM, and the query rows are too few for the Phase-1 tiles.
//
// Rows.  The query rows that read one KV head (token t, head kvh*group + h
// -> row t*group + h) form 32-row tiles of 32 / group tokens each; a decode
// step has one tile.
//
// Work.  Each wave takes one key range `part` of one (shard, KV head) for
// one row tile.  Waves are numbered KV head fastest, so the four waves of a
// workgroup read the same keys of four KV heads: one compute unit streams
// runs of 4 * 256 contiguous bytes of every K/V row (measured 6% faster
// than four key ranges of one head).  The tiles of a range write disjoint
// rows of its (o, lse) partial, and the caller merges the partials with the
// log-sum-exp merge.  The generation shard of a query step (rows [0, G)
// appended earlier, then the new tokens' own rows) may ride in the same
// launch: waves past the shards' take its key ranges, token t sees rows up
// to its own (G + t), and a tile's range ends at its last token's row.  A
// wave streams its keys in 32-key steps, on its own (no workgroup barrier):
//   K  straight into registers as the A operand of S^T = K Q^T (lane l32
//      loads key swap_bits23(l32) of the step, so that P comes out in the B
//      layout of the PV product);
//   V  into the wave's LDS double buffer by loads that write LDS directly,
//      keys as rows with a chunk swizzle, then read transposed as the A
//      operand of O^T += V^T P^T;
//   softmax  online, log2 domain: the running maximum per row, O and the
//      sums rescaled when it rises; P enters PV rounded to bf16, O is
//      divided by the sum of those rounded weights, the LSE uses the fp32
//      sum (as in the Phase-1 kernel).
// The next step's K and V loads are in flight while a step is multiplied.
#include <type_traits>

#include "common.hpp"

namespace {

constexpr int DEC_WAVES = 4;
constexpr int DEC_KEYS = 32;  // keys per step
constexpr int kDecBufferFlags = 0x00020000;  // raw 32-bit buffer access (word 3 of the resource)

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) uint8_t lds_u8;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
__device__ constexpr bf16x2 kOnes2 = {(__bf16)1.0f, (__bf16)1.0f};

// 16 bytes per lane from global memory straight into LDS at lds_base + 16*l.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rsrc, uint32_t voffset,
                                      uint32_t lds_base) {
  asm volatile("buffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(voffset), "s"(rsrc), "{m0}"(lds_base)
               : "memory");
}

__device__ __forceinline__ int swap23(int r) {
  return (r & ~12) | ((r >> 1) & 4) | ((r << 1) & 8);
}

struct DecodeArgs {
  const uint16_t* Q;  // bf16 [Tq, Hq, D]
  const uint16_t* K;  // bf16 [n_shards, S, Hkv, D]
  const uint16_t* V;
  int Tq, Hq, Hkv, group;
  int n_shards;
  int64_t S;
  int nparts;         // key ranges per shard (one wave each)
  int part_len;       // keys per range
  const uint16_t* Kg; // generation shard, bf16 [G + Tq, Hkv, D] (gen_parts > 0)
  const uint16_t* Vg;
  int G;
  int gen_parts;      // its key ranges (0: no generation shard)
  int gen_part_len;
  int tile_tokens;    // tokens per 32-row tile, 32 / group
  int row_tiles;      // tiles over the Tq tokens
  float scale_log2;
  float* O;           // [n_shards * nparts + gen_parts, Tq, Hq, D]
  float* lse;         // [n_shards * nparts + gen_parts, Hq, Tq]
};

template <int D>
__global__ __launch_bounds__(64 * DEC_WAVES) __attribute__((amdgpu_waves_per_eu(2, 2)))
void decode_attn_kernel(DecodeArgs a) {
  constexpr int CPR = D / 8;       // 16-byte chunks per row
  constexpr int DS = D / 16;       // k-steps of S
  constexpr int DT = D / 32;       // 32-row tiles of O^T
  constexpr int V_BYTES = DEC_KEYS * D * 2;
  constexpr int V_SEGS = V_BYTES / 1024;  // 1 KiB segments: one 16-byte load per lane each
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31;
  const int g = lane >> 5;
  // wave -> (KV head, shard or generation shard, key range, row tile)
  const int64_t wl = (int64_t)blockIdx.x * DEC_WAVES + wave;
  const int kvh = (int)(wl % a.Hkv);
  const int64_t rest = wl / a.Hkv;
  const int64_t shard_waves = (int64_t)a.nparts * a.row_tiles;
  const bool gen = rest >= (int64_t)a.n_shards * shard_waves;
  int wi, nparts, part_len;
  int64_t S;
  const uint16_t *Kz, *Vz;
  int shard = 0;
  if (!gen) {
    shard = (int)(rest / shard_waves);
    wi = (int)(rest - shard * shard_waves);
    nparts = a.nparts;
    part_len = a.part_len;
    S = a.S;
    Kz = a.K + shard * a.S * a.Hkv * D;
    Vz = a.V + shard * a.S * a.Hkv * D;
  } else {
    wi = (int)(rest - (int64_t)a.n_shards * shard_waves);
    nparts = a.gen_parts;
    part_len = a.gen_part_len;
    S = (int64_t)a.G + a.Tq;
    Kz = a.Kg;
    Vz = a.Vg;
  }
  const int part = wi / a.row_tiles, tile = wi - part * a.row_tiles;
  if (part >= nparts) return;  // wave-uniform; no barrier follows
  // partial of this key range; each row tile writes its own tokens' rows of it
  const int64_t z = (gen ? (int64_t)a.n_shards * a.nparts : (int64_t)shard * a.nparts) + part;
  const int tok0 = tile * a.tile_tokens;
  const int R = min(a.tile_tokens, a.Tq - tok0) * a.group;  // live rows of the tile
  const int kv_begin = part * part_len;
  int kv_end = (int)min((int64_t)kv_begin + part_len, S);
  // in the generation shard no row of the tile sees past its last token's own
  if (gen) kv_end = min(kv_end, a.G + tok0 + R / a.group);
  const int nsteps = max(0, (kv_end - kv_begin + DEC_KEYS - 1) / DEC_KEYS);
  const float c2 = a.scale_log2;
  // Keys from vis_end on weigh zero for this lane's query row: the range's
  // end, and in the generation shard the rows after the token's own.
  int vis_end = kv_end;
  if (gen) vis_end = min(vis_end, a.G + tok0 + l32 / a.group + 1);
  // a step whose keys all lie below mask_from needs no mask in any lane
  const int mask_from = gen ? min(kv_end, a.G + tok0 + 1) : kv_end;

  // K/V of this shard through buffer resources, 32-bit byte offsets.
  const int64_t zstride = S * a.Hkv * D;
  const uint32_t row_bytes = (uint32_t)(a.Hkv * D * 2);
  const uint32_t head_off = (uint32_t)(kvh * D * 2);
  const __amdgpu_buffer_rsrc_t k_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(Kz), (short)0, (int)(zstride * 2), kDecBufferFlags);
  const __amdgpu_buffer_rsrc_t v_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(Vz), (short)0, (int)(zstride * 2), kDecBufferFlags);

  // ---- Q fragments (B operand): column l32 = packed row (token, head) ----
  bf16x8 qf[DS];
  {
    const int r = l32;
    const int tl = r / a.group;
    const int tok = tok0 + tl;
    const int head = kvh * a.group + (r - tl * a.group);
    const bf16x8* src =
        reinterpret_cast<const bf16x8*>(a.Q + ((int64_t)tok * a.Hq + head) * D) + g;
#pragma unroll
    for (int s = 0; s < DS; ++s) qf[s] = r < R ? src[2 * s] : bf16x8{};
#pragma unroll
    for (int s = 0; s < DS; ++s) asm volatile("" : "+v"(qf[s]));
  }

  // ---- loads of one step ----------------------------------------------------
  // K: lane (l32, g) loads key swap23(l32) of the step, 16-byte chunks
  // 2s + g.  A key past the end reads the range's first key (finite; masked).
  auto load_k = [&](int j, bf16x8 (&kf)[DS]) {
    int key = kv_begin + j * DEC_KEYS + swap23(l32);
    key = key < kv_end ? key : kv_begin;
    const uint32_t base = (uint32_t)key * row_bytes + head_off + 16u * g;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(k_rsrc, base + 32u * s, 0, 0);
      kf[s] = __builtin_bit_cast(bf16x8, v);
    }
  };
  // V: keys as rows of 2D bytes in the wave's LDS stage; lane l of segment
  // sg fills chunk position (64 sg + l) % CPR of row (64 sg + l) / CPR with
  // chunk position ^ vswz(row) of that key's row.
  auto vswz = [](int r) { return (4 * ((r * CPR) / 16)) % CPR; };
  lds_u8* const wave_lds = (lds_u8*)smem + wave * 2 * V_BYTES;
  auto issue_v = [&](int j, int stage) {
    const uint32_t st = __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(wave_lds + stage * V_BYTES));
#pragma unroll
    for (int sg = 0; sg < V_SEGS; ++sg) {
      const int slot = sg * 64 + lane;
      const int r = slot / CPR;
      int key = kv_begin + j * DEC_KEYS + r;
      key = key < kv_end ? key : kv_begin;
      dma16(v_rsrc, (uint32_t)key * row_bytes + head_off + (uint32_t)((slot % CPR) ^ vswz(r)) * 16u,
            st + sg * 1024);
    }
  };
  // V^T fragment (rows e*32.., keys 16c..16c+15) by two transposing reads:
  // lane 16a + 4j + q addresses key row 8(a/2) + j (+4) at head_dim
  // 16(a%2) + 4q; lane 16a + i receives head_dim 16(a%2) + i of keys
  // 8(a/2) .. +7, the k-slots that P's B layout puts in lane a's half.
  uint32_t vtr_base[DT];
  {
    const int a16 = lane >> 4, jj = (lane >> 2) & 3, q = lane & 3;
    const int trow = 8 * (a16 >> 1) + jj;
    const int cb = 2 * (a16 & 1) + (q >> 1);
#pragma unroll
    for (int e = 0; e < DT; ++e)
      vtr_base[e] = trow * (2 * D) + 16 * ((4 * e + cb) ^ vswz(trow)) + 8 * (q & 1);
  }
  auto v_frag = [&](const lds_u8* sV, int c, int e) -> bf16x8 {
    const lds_u8* b = sV + vtr_base[e] + (16 * c) * (2 * D);
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)b);
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(b + 4 * (2 * D)));
    return __builtin_bit_cast(bf16x8,
                              (s16x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
  };

  f32x16 acc[DT];
#pragma unroll
  for (int e = 0; e < DT; ++e) acc[e] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f, lr_run = 0.f;

  // Step j's K lives in kbuf[j % 2] and V(j) in LDS stage j % 2.  Step j
  // multiplies S(j), then issues K(j+1) and V(j+1), so that they travel
  // while the weights and the PV product of step j run.  The compiler's own
  // wait for K(j) also covers V(j), which was issued before it.
  bf16x8 kbuf[2][DS];
  if (nsteps > 0) {
    load_k(0, kbuf[0]);
    issue_v(0, 0);
  }
  // one step; KB = j % 2, a compile-time index into the register buffers
  auto step = [&](int j, auto kb_tag) {
    constexpr int KB = decltype(kb_tag)::value;
    const bool v1 = j + 1 < nsteps;
    // S^T of this step: row i = key swap23(i), column = packed query row
    f32x16 S = f32x16{};
#pragma unroll
    for (int s = 0; s < DS; ++s)
      S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kbuf[KB][s], qf[s], S, 0, 0, 0);
    if (v1) {
      load_k(j + 1, kbuf[KB ^ 1]);
      issue_v(j + 1, KB ^ 1);
    }
    // keys from vis_end on weigh zero; lane (l32, g) holds rows
    // 8(v/4) + 4g + v%4, i.e. keys swap23 of those
    const int k0 = kv_begin + j * DEC_KEYS;
    if (k0 + DEC_KEYS > mask_from) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = 8 * (v >> 2) + 4 * g + (v & 3);
        if (k0 + swap23(row) >= vis_end) S[v] = -INFINITY;
      }
    }
    float mx = S[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) mx = fmaxf(mx, S[v]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * c2;
    // A row may have seen no key yet (a generation-shard range that starts
    // after its token's own row): its maximum stays -inf, and the weights
    // are taken against 0 so that they come out 0 rather than NaN.
    const float m_new = fmaxf(m_run, mx);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
#pragma unroll
    for (int e = 0; e < DT; ++e) acc[e] *= alpha;
    l_run *= alpha;
    lr_run *= alpha;
    m_run = m_new;
    bf16x8 P[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      f32x8 p;
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        p[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(S[8 * c + v], c2, -m_use));
        l_run += p[v];
      }
      P[c] = __builtin_convertvector(p, bf16x8);
#pragma unroll
      for (int v = 0; v < 8; v += 2)
        lr_run = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{P[c][v], P[c][v + 1]}, kOnes2, lr_run,
                                                 false);
    }
    // V(j) is in LDS once only the loads issued after it are outstanding
    if (v1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(DS + V_SEGS) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    const lds_u8* sV = wave_lds + KB * V_BYTES;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int e = 0; e < DT; ++e)
        acc[e] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v_frag(sV, c, e), P[c], acc[e], 0, 0, 0);
  };
  for (int j = 0; j < nsteps; j += 2) {
    step(j, std::integral_constant<int, 0>{});
    if (j + 1 < nsteps) step(j + 1, std::integral_constant<int, 1>{});
  }

  // ---- this part's (o, lse) ---------------------------------------------------
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float lr_tot = lr_run + __shfl_xor(lr_run, 32, 64);
  const float inv = lr_tot > 0.f ? 1.f / lr_tot : 0.f;
  const int r = l32;
  if (r < R) {
    const int tl = r / a.group;
    const int tok = tok0 + tl;
    const int head = kvh * a.group + (r - tl * a.group);
    float* o = a.O + z * (int64_t)a.Tq * a.Hq * D + ((int64_t)tok * a.Hq + head) * D;
#pragma unroll
    for (int e = 0; e < DT; ++e)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int dd = e * 32 + 8 * q4 + 4 * g;
        *reinterpret_cast<f32x4*>(o + dd) =
            f32x4{acc[e][4 * q4] * inv, acc[e][4 * q4 + 1] * inv, acc[e][4 * q4 + 2] * inv,
                  acc[e][4 * q4 + 3] * inv};
      }
    if (g == 0)
      a.lse[z * (int64_t)a.Hq * a.Tq + (int64_t)head * a.Tq + tok] =
          l_tot > 0.f ? (m_run + __log2f(l_tot)) * 0.69314718055994531f : -INFINITY;
  }
}

}  // namespace

// Key ranges per shard for the decode kernel: enough waves for one
// four-wave workgroup per compute unit (as fast as two per compute unit,
// measured, with half the partials to merge), at least 256 keys per range.
int decode_parts(int n_shards, int64_t S, int Hkv) {
  if (S <= 0 || n_shards <= 0 || Hkv <= 0) return 1;
  const int64_t waves = (int64_t)n_shards * Hkv;
  int64_t np = (256 * 4 + waves - 1) / waves;
  const int64_t max_by_len = (S + 255) / 256;
  if (np > max_by_len) np = max_by_len;
  if (np < 1) np = 1;
  if (np > 256) np = 256;
  return (int)np;
}

bool decode_applies(int Tq, int Hq, int Hkv, int d) {
  return (d == 64 || d == 128) && Tq >= 1 && (int64_t)Tq * (Hq / Hkv) <= 32;
}

int launch_decode(const uint16_t* q, const uint16_t* K, const uint16_t* V, int n_shards, int Tq,
                  int64_t S, int Hq, int Hkv, int d, float scale, float* o, float* lse,
                  int nparts, hipStream_t stream, const DecodeGen* gen) {
  DecodeArgs a{};
  a.Q = q;
  a.K = K;
  a.V = V;
  a.Tq = Tq;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.group = Hq / Hkv;
  a.n_shards = n_shards;
  a.S = S;
  a.nparts = nparts;
  a.part_len = (int)((S + nparts - 1) / nparts);
  a.tile_tokens = 32 / a.group;
  if (a.tile_tokens < 1) return PULSAR_EUNSUPPORTED;
  a.row_tiles = (Tq + a.tile_tokens - 1) / a.tile_tokens;
  if (gen != nullptr && gen->nparts > 0) {
    const int64_t rows = gen->G + Tq;
    a.Kg = gen->K;
    a.Vg = gen->V;
    a.G = (int)gen->G;
    a.gen_parts = gen->nparts;
    a.gen_part_len = (int)((rows + gen->nparts - 1) / gen->nparts);
  }
  a.scale_log2 = scale * 1.4426950408889634f;
  a.O = o;
  a.lse = lse;
  const int64_t nwaves =
      (int64_t)Hkv * ((int64_t)n_shards * nparts + a.gen_parts) * a.row_tiles;
  const int64_t nwg = (nwaves + DEC_WAVES - 1) / DEC_WAVES;
  if (nwg == 0) return PULSAR_OK;
  if (nwg > 0x7fffffff) return PULSAR_EUNSUPPORTED;
  const size_t lds = (size_t)DEC_WAVES * 2 * DEC_KEYS * d * 2;  // two V stages per wave
  const auto kern = d == 128 ? decode_attn_kernel<128> : decode_attn_kernel<64>;
  if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lds) != hipSuccess)
    return PULSAR_EHIP;
  hipLaunchKernelGGL(kern, dim3((unsigned)nwg), dim3(64 * DEC_WAVES), lds, stream, a);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}
