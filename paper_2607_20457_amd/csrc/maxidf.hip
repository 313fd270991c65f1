// Max-IDF summary construction on gfx950 (Section 3.1 "Summary generation",
// Eq. 2; Appendix "Corpus-Level IDF Table" and "Max-IDF").
//
// One 1024-thread workgroup per sequence keeps the whole document-frequency
// table of that sequence in the compute unit's local data share (LDS), so the
// table never touches HBM:
//
//   pass 1  for every block j: clear a vocab-sized bitmap, stream the block's
//           ids with 16-byte loads, atomically set each id's bit; the thread
//           that sets a bit first adds one to that id's df byte (df <= 255).
//   pass 2  look up the df of every id; lanes of one chunk (chunk/4 lanes)
//           take the minimum with cross-lane operations.  The chunk minima go
//           to LDS (and optionally to HBM).
//   select  one wavefront per block picks the top-k chunks (select_topk).
//
// Three variants share these steps:
//   * general  (any vocab that fits): df bytes, then a scattered bitmap;
//     pass 2 streams the ids from HBM a second time;
//   * compact  (vocab <= 131072): a fixed 4096-word bitmap whose word is
//     t & 4095 (the most frequent, low ids spread over all banks) and the df
//     bytes behind it; pass 2 streams the ids again;
//   * resident (compact, L <= 131072, blocks of a multiple of 8192 ids): pass
//     1 keeps every thread's 128 ids in registers, packed, and pass 2 reads
//     them back from there, so the ids cross HBM once; two bitmaps alternate
//     between blocks, one barrier per block.
//
// A chunk's Max-IDF score ln(N / mindf) is strictly decreasing in mindf, so
// ranking by (mindf ascending, index ascending) is ranking by (score
// descending, index ascending).
#include "common.hpp"

#define MAXIDF_THREADS 1024
#define MAXIDF_WAVES (MAXIDF_THREADS / PULSAR_WAVE)

static inline int64_t round_up4(int64_t x) { return (x + 3) & ~int64_t(3); }

// Bitmap words of the general layout: a power of two at least vocab/32 when
// that still fits next to the df table, so that the bitmap can be scattered
// (see mark_tokens); otherwise exactly ceil(vocab/32), unscattered.
static int64_t bitmap_words(int vocab) {
  const int64_t need = ((int64_t)vocab + 31) / 32;
  int64_t w = 1;
  while (w < need) w <<= 1;
  return round_up4(vocab) + w * 4 <= PULSAR_LDS_BYTES ? w : need;
}

// Compact layout for vocab <= 131072: a fixed 4096-word bitmap at LDS byte
// 0, where token t owns bit t >> 12 of word t & 4095 (the most frequent, low
// ids fall in different words and banks), and the df bytes at byte 16384, an
// offset the LDS instructions carry as an immediate.  The chunk minima reuse
// the bitmap bytes when they fit there, else follow the df table.
constexpr int kFastWordsLog2 = 12;
constexpr int kFastWords = 1 << kFastWordsLog2;
constexpr int kFastBitmapBytes = kFastWords * 4;
constexpr int kFastVocab = kFastWords * 32;
// Register-resident variant (see maxidf_resident_kernel): rounds of 2 groups
// of 4 ids per thread, at most RES_ROUNDS of them per sequence.
constexpr int RES_ROUNDS = 16;
constexpr int RES_ROUND_TOKENS = MAXIDF_THREADS * 8;
// The resident variant alternates two compact bitmaps (block j marks bitmap
// j % 2 and clears the other), so its df bytes start at byte 32768.
constexpr int kResBitmapBytes = 2 * kFastBitmapBytes;

struct MaxidfPlan {
  bool fast;
  bool resident;     // compact layout with the ids held in registers
  int64_t lds_bytes;
  int64_t cmin_off;  // byte offset of the chunk minima
};

// General layout: df bytes [round_up4(vocab)], then a region reused as the
// per-block bitmap (pass 1) and the chunk minima (pass 2 / select).
static MaxidfPlan maxidf_plan(int64_t L, int num_blocks, int chunk, int vocab) {
  const int64_t df_bytes = round_up4(vocab);
  const int64_t chunk_bytes = round_up4(L / chunk);
  if (vocab <= kFastVocab) {
    if (L <= (int64_t)RES_ROUNDS * RES_ROUND_TOKENS && (L / num_blocks) % RES_ROUND_TOKENS == 0 &&
        chunk_bytes <= kResBitmapBytes)  // static LDS: bitmaps + the largest df table
      return {true, true, kResBitmapBytes + kFastVocab, 0};
    const bool in_bitmap = chunk_bytes <= kFastBitmapBytes;
    const int64_t lds = kFastBitmapBytes + df_bytes + (in_bitmap ? 0 : chunk_bytes);
    if (lds <= PULSAR_LDS_BYTES)
      return {true, false, lds, in_bitmap ? 0 : kFastBitmapBytes + df_bytes};
  }
  const int64_t bitmap_bytes = bitmap_words(vocab) * 4;
  return {false, false, df_bytes + (bitmap_bytes > chunk_bytes ? bitmap_bytes : chunk_bytes),
          df_bytes};
}

size_t maxidf_lds_bytes(int64_t L, int num_blocks, int chunk, int vocab) {
  return (size_t)maxidf_plan(L, num_blocks, chunk, vocab).lds_bytes;
}

// Token t owns bit t%32 of bitmap word (t/32) XOR ((t%32)*129 mod W): a
// bijection onto (word, bit) pairs that sends the 32 ids sharing a word --
// under a Zipf law the most frequent ids, half of all tokens -- to 32
// different words in 32 different banks, so their atomics do not serialise.
// The n ids of one thread are marked with all bitmap atomics issued before
// any result is used; the first setter of a bit adds one to the id's df
// byte.  A negative id marks nothing (the loader pads partial rounds with -1);
// an id at or above vocab is the caller's error, clamped into range so that
// no access leaves the table, with an unspecified result.
template <int n>
__device__ __forceinline__ void mark_tokens(const int (&t)[n], int vocab, int spread_mask,
                                            uint32_t* bits, uint32_t* dfw) {
  uint32_t bit[n], old[n];
  int word[n], ts[n];
#pragma unroll
  for (int i = 0; i < n; ++i) {
    ts[i] = (int)min((uint32_t)t[i], (uint32_t)(vocab - 1));
    const int b = ts[i] & 31;
    word[i] = (ts[i] >> 5) ^ (((b << 7) | b) & spread_mask);
    bit[i] = t[i] >= 0 ? 1u << b : 0u;  // -1 pads a partial round: marks nothing
  }
#pragma unroll
  for (int i = 0; i < n; ++i) old[i] = atomicOr(&bits[word[i]], bit[i]);
#pragma unroll
  for (int i = 0; i < n; ++i)
    if (bit[i] & ~old[i]) atomicAdd(&dfw[ts[i] >> 2], 1u << ((ts[i] << 3) & 31));
}

// Compact layout: the first setter of a token's bit in this block adds one
// to its df byte.  PAD: the round holds -1 padding, which marks nothing.  An
// id at or above vocab is clamped into the table (the caller's error;
// unspecified result, no access outside the table).
template <int n, bool PAD>
__device__ __forceinline__ void mark_tokens_compact(const int (&t)[n], uint32_t vmax,
                                                    uint32_t* bits, uint32_t* dfw) {
  uint32_t ts[n], bit[n], old[n];
#pragma unroll
  for (int i = 0; i < n; ++i) {
    ts[i] = min((uint32_t)t[i], vmax);
    bit[i] = 1u << (ts[i] >> kFastWordsLog2);
    if (PAD && t[i] < 0) bit[i] = 0u;
  }
#pragma unroll
  for (int i = 0; i < n; ++i) old[i] = atomicOr(&bits[ts[i] & (kFastWords - 1)], bit[i]);
#pragma unroll
  for (int i = 0; i < n; ++i)
    if (bit[i] & ~old[i]) atomicAdd(&dfw[ts[i] >> 2], 1u << ((ts[i] << 3) & 31));
}

__device__ __forceinline__ uint32_t df_of(int t, int vocab, const uint8_t* df8) {
  return df8[min((uint32_t)t, (uint32_t)(vocab - 1))];
}

// Minimum over aligned groups of `group` lanes (a power of two); DPP within
// rows of 16 lanes, cross-lane permutes beyond.
__device__ __forceinline__ uint32_t group_min(uint32_t x, int group) {
  if (group >= 2) x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0xB1, 0xF, 0xF, false));
  if (group >= 4) x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x4E, 0xF, 0xF, false));
  if (group >= 8) x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x141, 0xF, 0xF, false));
  if (group >= 16) x = min(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x140, 0xF, 0xF, false));
  if (group >= 32) x = min(x, (uint32_t)__shfl_xor((int)x, 16, 64));
  if (group >= 64) x = min(x, (uint32_t)__shfl_xor((int)x, 32, 64));
  return x;
}

// Optional IDF table (Eq. idf) of one sequence from its df bytes in LDS.
__device__ void write_idf(const uint8_t* df8, int vocab, int num_blocks, float* __restrict__ out,
                          int tid) {
  const float n = (float)num_blocks;
  for (int t = tid; t < vocab; t += MAXIDF_THREADS) {
    const uint32_t d = df8[t];
    out[t] = logf(n / (float)(d > 1u ? d : 1u));
  }
}

// Lanes below this one with their bit set in a wave mask.
__device__ __forceinline__ int count_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

// Top-k chunks of every block of sequence b from the chunk minima cmin
// ([num_blocks][C] bytes in LDS), written in ascending chunk order.  One
// wavefront per block; slot i of lane l is chunk 64*i + l, so chunk order is
// (slot, lane) order and every count is a ballot.  The threshold tau is the
// smallest df with at least k chunks at or below it (binary search over
// 1..N); every chunk below tau is kept, and the first k - #(< tau) chunks
// equal to tau in chunk order.
__device__ void select_topk(const uint8_t* cmin, int64_t b, int num_blocks, int C, int topk,
                            int32_t* __restrict__ sel, int wave, int lane) {
  if (topk == 0) return;
  const int slots = (C + 63) >> 6;
  for (int j = wave; j < num_blocks; j += MAXIDF_WAVES) {
    const uint8_t* cv = cmin + (int64_t)j * C;
    // a lane past the last chunk reads 256, above every df (<= 255)
    auto x_of = [&](int i) { return 64 * i + lane < C ? (int)cv[64 * i + lane] : 256; };
    int lo = 0, hi = num_blocks;  // #(mindf <= lo) < k <= #(mindf <= hi)
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      int cnt = 0;
      for (int i = 0; i < slots; ++i) cnt += __popcll(__ballot(x_of(i) <= mid));
      if (cnt >= topk) hi = mid; else lo = mid;
    }
    const int tau = hi;
    int n_lt = 0;
    for (int i = 0; i < slots; ++i) n_lt += __popcll(__ballot(x_of(i) < tau));
    const int need = topk - n_lt;  // chunks equal to tau that are kept
    int32_t* dst = sel + (b * num_blocks + j) * topk;
    int eq_before = 0, out_before = 0;
    for (int i = 0; i < slots; ++i) {
      const int x = x_of(i);
      const uint64_t m_eq = __ballot(x == tau);
      const bool keep = x < tau || (x == tau && eq_before + count_below(m_eq) < need);
      const uint64_t m_keep = __ballot(keep);
      if (keep) dst[out_before + count_below(m_keep)] = 64 * i + lane;
      eq_before += __popcll(m_eq);
      out_before += __popcll(m_keep);
    }
  }
}

template <bool COMPACT>
__global__ __launch_bounds__(MAXIDF_THREADS) void maxidf_kernel(
    const int32_t* __restrict__ ids, int64_t L, int num_blocks, int Lb, int chunk_log2,
    int topk, int vocab, int n_bitmap, int spread_mask, int cmin_off, int32_t* __restrict__ sel,
    int32_t* __restrict__ chunk_mindf, float* __restrict__ idf) {
  extern __shared__ uint32_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t b = blockIdx.x;
  const int chunk = 1 << chunk_log2;
  const int vocab_w4 = (vocab + 3) >> 2;
  uint8_t* const lds8 = reinterpret_cast<uint8_t*>(lds);
  uint8_t* df8 = lds8 + (COMPACT ? kFastBitmapBytes : 0);
  uint32_t* dfw = reinterpret_cast<uint32_t*>(df8);
  uint32_t* bits = COMPACT ? lds : lds + vocab_w4;
  uint8_t* cmin = lds8 + cmin_off;
  const uint32_t vmax = (uint32_t)(vocab - 1);

  const int32_t* seq = ids + b * L;

  for (int w = tid; w < vocab_w4; w += MAXIDF_THREADS) dfw[w] = 0u;
  // (the first round's barrier orders this against the atomics)

  // ---- pass 1: document frequency --------------------------------------
  // The blocks are streamed as rounds of MAXIDF_THREADS x ROUND int4 groups;
  // the loads of the next two rounds are in flight while a round's ids are
  // marked, so each thread overlaps its atomics with HBM latency.
  constexpr int ROUND = 2;
#ifndef MAXIDF_PREFETCH
#define MAXIDF_PREFETCH 2
#endif
  constexpr int PREFETCH = MAXIDF_PREFETCH;  // rounds of loads in flight
  const int nvec = Lb >> 2;  // int4 groups per block
  const int4* seq4 = reinterpret_cast<const int4*>(seq);
  const int rpb = (nvec + MAXIDF_THREADS * ROUND - 1) / (MAXIDF_THREADS * ROUND);
  const int rounds = num_blocks * rpb;
  auto load_round = [&](int rd, int4 (&t)[ROUND]) {
    const int j = rd / rpb;
    const int r = rd - j * rpb;
    const int4* blk = seq4 + (int64_t)j * nvec;
#pragma unroll
    for (int u = 0; u < ROUND; ++u) {
      const int v = (r * ROUND + u) * MAXIDF_THREADS + tid;
      const int4 x = blk[min(v, nvec - 1)];
      t[u] = v < nvec ? x : make_int4(-1, -1, -1, -1);
    }
  };
  // Loads run PREFETCH rounds ahead: cbuf[0] holds round rd, cbuf[i] round rd+i.
  int4 cbuf[PREFETCH + 1][ROUND];
#pragma unroll
  for (int i = 0; i < PREFETCH; ++i)
    if (i < rounds) load_round(i, cbuf[i]);
  for (int rd = 0; rd < rounds; ++rd) {
    if (rd % rpb == 0) {  // a new block: everyone is done with the previous bitmap
      __syncthreads();
      for (int w = tid; w < n_bitmap; w += MAXIDF_THREADS) bits[w] = 0u;
      __syncthreads();
    }
    if (rd + PREFETCH < rounds) load_round(rd + PREFETCH, cbuf[PREFETCH]);
    {
      int tk[4 * ROUND];
#pragma unroll
      for (int u = 0; u < ROUND; ++u) {
        tk[4 * u] = cbuf[0][u].x;
        tk[4 * u + 1] = cbuf[0][u].y;
        tk[4 * u + 2] = cbuf[0][u].z;
        tk[4 * u + 3] = cbuf[0][u].w;
      }
      if constexpr (COMPACT) {
        if ((rd - (rd / rpb) * rpb + 1) * ROUND * MAXIDF_THREADS <= nvec)
          mark_tokens_compact<4 * ROUND, false>(tk, vmax, bits, dfw);
        else
          mark_tokens_compact<4 * ROUND, true>(tk, vmax, bits, dfw);
      } else {
        mark_tokens(tk, vocab, spread_mask, bits, dfw);
      }
    }
#pragma unroll
    for (int u = 0; u < ROUND; ++u) {
#pragma unroll
      for (int i = 0; i < PREFETCH; ++i) cbuf[i][u] = cbuf[i + 1][u];
    }
  }
  __syncthreads();

  if (idf) write_idf(df8, vocab, num_blocks, idf + b * vocab, tid);

  // ---- pass 2: per-chunk minimum df -------------------------------------
  // Groups of PF int4 loads per thread, double-buffered: group g+1 is in
  // flight while group g is reduced.  Every lane runs the same trip count,
  // so all lanes join the cross-lane minimum.
#ifndef MAXIDF_PF2
#define MAXIDF_PF2 4
#endif
  constexpr int PF = MAXIDF_PF2;
  const int nvec_seq = (int)(L >> 2);  // L < 2^31 (checked by the caller)
  const int group = chunk >> 2;        // lanes per chunk (1..64)
  const int group_log2 = chunk_log2 - 2;
  const int nchunks_seq = (int)(L >> chunk_log2);
  const int n_iter = (nvec_seq + MAXIDF_THREADS - 1) / MAXIDF_THREADS;
  const int n_grp = (n_iter + PF - 1) / PF;
  auto load_group = [&](int gi, int4 (&t)[PF]) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int v = (gi * PF + p) * MAXIDF_THREADS + tid;
      t[p] = seq4[min(v, nvec_seq - 1)];
    }
  };
  auto reduce_group = [&](int gi, const int4 (&t)[PF]) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int it = gi * PF + p;
      if (it >= n_iter) break;  // uniform across the workgroup
      const int v = it * MAXIDF_THREADS + tid;
      uint32_t mn = min(min(df_of(t[p].x, vocab, df8), df_of(t[p].y, vocab, df8)),
                        min(df_of(t[p].z, vocab, df8), df_of(t[p].w, vocab, df8)));
      mn = group_min(mn, group);
      if ((lane & (group - 1)) == 0 && v < nvec_seq) {
        const int c = v >> group_log2;
        cmin[c] = (uint8_t)mn;
        if (chunk_mindf) chunk_mindf[b * nchunks_seq + c] = (int32_t)mn;
      }
    }
  };
  int4 ga[PF], gb[PF];
  if (n_grp > 0) load_group(0, ga);
  for (int gi = 0; gi < n_grp; gi += 2) {
    if (gi + 1 < n_grp) load_group(gi + 1, gb);
    reduce_group(gi, ga);
    if (gi + 2 < n_grp) load_group(gi + 2, ga);
    if (gi + 1 < n_grp) reduce_group(gi + 1, gb);
  }
  __syncthreads();

  // ---- select ------------------------------------------------------------
  select_topk(cmin, b, num_blocks, Lb >> chunk_log2, topk, sel, wave, lane);
}

// Register-resident variant for the compact layout when the sequence fits
// the register file: L <= 131072 and Lb a multiple of 8192, so that every
// thread owns exactly RES_ROUNDS x 2 16-byte groups of ids.  Pass 1 keeps
// each thread's ids in registers (the clamped id's low 16 bits packed two per
// register, bit 16 of all of them in four more registers), and pass 2 reads
// them back from there: the ids cross HBM once.  Thread tid's group u of
// round rd is the sequence's 16-byte group (2*rd + u)*1024 + tid, which is
// also the group pass 2 assigns to iteration 2*rd + u.
__global__ __launch_bounds__(MAXIDF_THREADS) void maxidf_resident_kernel(
    const int32_t* __restrict__ ids, int64_t L, int num_blocks, int Lb, int chunk_log2,
    int topk, int vocab, int32_t* __restrict__ sel, int32_t* __restrict__ chunk_mindf,
    float* __restrict__ idf) {
  // A fixed layout in static LDS, whose base the compiler knows, so every
  // table offset folds into the LDS instructions: two bitmaps, then the df
  // bytes (vocab <= 131072); the chunk minima (<= 32 KiB) reuse the bitmaps.
  __shared__ __attribute__((aligned(16))) uint32_t lds[(kResBitmapBytes + kFastVocab) / 4];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t b = blockIdx.x;
  uint8_t* const lds8 = reinterpret_cast<uint8_t*>(lds);
  uint8_t* df8 = lds8 + kResBitmapBytes;
  uint32_t* dfw = reinterpret_cast<uint32_t*>(df8);
  uint8_t* cmin = lds8;
  const uint32_t vmax = (uint32_t)(vocab - 1);
  const int vocab_w4 = (vocab + 3) >> 2;
  const int4* seq4 = reinterpret_cast<const int4*>(ids + b * L);
  const int rounds = (int)(L / RES_ROUND_TOKENS);  // <= RES_ROUNDS
  const int rpb = Lb / RES_ROUND_TOKENS;            // rounds per block

  for (int w = tid; w < vocab_w4; w += MAXIDF_THREADS) dfw[w] = 0u;
  for (int w = tid; w < 2 * kFastWords; w += MAXIDF_THREADS) lds[w] = 0u;
  __syncthreads();

  // ---- pass 1: document frequency, ids kept in registers ------------------
  constexpr int PREFETCH = 2;  // rounds of loads in flight
  int4 cbuf[PREFETCH + 1][2];
  uint32_t plo[RES_ROUNDS][2][2];         // low 16 bits, two ids per register
  uint32_t phi[RES_ROUNDS * 2 / 8] = {};  // bit 16 of every id, 32 per register
  auto load_round = [&](int rd, int4 (&t)[2]) {
#pragma unroll
    for (int u = 0; u < 2; ++u) t[u] = seq4[(2 * rd + u) * MAXIDF_THREADS + tid];
  };
#pragma unroll
  for (int i = 0; i < PREFETCH; ++i)
    if (i < rounds) load_round(i, cbuf[i]);
#pragma unroll
  for (int rd = 0; rd < RES_ROUNDS; ++rd) {
    if (rd < rounds) {
      // Block j marks bitmap j % 2.  At its start every wave is past block
      // j-1 (barrier), so the other bitmap is cleared for block j+1 while
      // this one is marked.
      const int j = rd / rpb;
      uint32_t* bits = lds + (j & 1) * kFastWords;
      if (rd % rpb == 0) {
        if (rd > 0) __syncthreads();
        uint32_t* other = lds + ((j + 1) & 1) * kFastWords;
        for (int w = tid; w < kFastWords; w += MAXIDF_THREADS) other[w] = 0u;
      }
      if (rd + PREFETCH < rounds)
        load_round(rd + PREFETCH, cbuf[(rd + PREFETCH) % (PREFETCH + 1)]);
      const int4 (&cur)[2] = cbuf[rd % (PREFETCH + 1)];
      int tk[8];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int4 x = cur[u];
        const uint32_t t0 = min((uint32_t)x.x, vmax), t1 = min((uint32_t)x.y, vmax);
        const uint32_t t2 = min((uint32_t)x.z, vmax), t3 = min((uint32_t)x.w, vmax);
        tk[4 * u] = (int)t0;
        tk[4 * u + 1] = (int)t1;
        tk[4 * u + 2] = (int)t2;
        tk[4 * u + 3] = (int)t3;
        plo[rd][u][0] = __builtin_amdgcn_perm(t1, t0, 0x05040100u);
        plo[rd][u][1] = __builtin_amdgcn_perm(t3, t2, 0x05040100u);
        const uint32_t h =
            ((t0 >> 16) & 1u) | ((t1 >> 15) & 2u) | ((t2 >> 14) & 4u) | ((t3 >> 13) & 8u);
        const int slot = 2 * rd + u;
        phi[slot >> 3] |= h << (4 * (slot & 7));
      }
      mark_tokens_compact<8, false>(tk, vmax, bits, dfw);
    }
  }
  __syncthreads();
  if (idf) write_idf(df8, vocab, num_blocks, idf + b * vocab, tid);

  // ---- pass 2: per-chunk minimum df from the registers --------------------
  const int group = 1 << (chunk_log2 - 2);  // lanes per chunk (1..64)
  const int group_log2 = chunk_log2 - 2;
  const int nchunks_seq = (int)(L >> chunk_log2);
#pragma unroll
  for (int slot = 0; slot < 2 * RES_ROUNDS; ++slot) {
    if (slot < 2 * rounds) {
      const uint32_t lo0 = plo[slot >> 1][slot & 1][0], lo1 = plo[slot >> 1][slot & 1][1];
      const uint32_t h = phi[slot >> 3] >> (4 * (slot & 7));
      const uint32_t t0 = (lo0 & 0xFFFFu) | ((h & 1u) << 16);
      const uint32_t t1 = (lo0 >> 16) | ((h & 2u) << 15);
      const uint32_t t2 = (lo1 & 0xFFFFu) | ((h & 4u) << 14);
      const uint32_t t3 = (lo1 >> 16) | ((h & 8u) << 13);
      uint32_t mn = min(min((uint32_t)df8[t0], (uint32_t)df8[t1]),
                        min((uint32_t)df8[t2], (uint32_t)df8[t3]));
      mn = group_min(mn, group);
      if ((lane & (group - 1)) == 0) {
        const int c = (slot * MAXIDF_THREADS + tid) >> group_log2;
        cmin[c] = (uint8_t)mn;
        if (chunk_mindf) chunk_mindf[b * nchunks_seq + c] = (int32_t)mn;
      }
    }
  }
  __syncthreads();
  select_topk(cmin, b, num_blocks, Lb >> chunk_log2, topk, sel, wave, lane);
}

int launch_maxidf(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk, int topk,
                  int vocab, int32_t* sel, int32_t* chunk_mindf, float* idf, size_t lds_bytes,
                  hipStream_t stream) {
  if (batch == 0) return PULSAR_OK;
  int chunk_log2 = 0;
  while ((1 << chunk_log2) < chunk) ++chunk_log2;
  const MaxidfPlan plan = maxidf_plan(L, num_blocks, chunk, vocab);
  if ((size_t)plan.lds_bytes != lds_bytes) return PULSAR_EINVAL;
  if (plan.resident) {  // static LDS only
    hipLaunchKernelGGL(maxidf_resident_kernel, dim3(batch), dim3(MAXIDF_THREADS), 0, stream, ids,
                       L, num_blocks, (int)(L / num_blocks), chunk_log2, topk, vocab, sel,
                       chunk_mindf, idf);
    return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
  }
  const auto kern = plan.fast ? maxidf_kernel<true> : maxidf_kernel<false>;
  if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lds_bytes) != hipSuccess)
    return PULSAR_EHIP;
  const int64_t nb = plan.fast ? kFastWords : bitmap_words(vocab);
  const bool pow2 = (nb & (nb - 1)) == 0;
  hipLaunchKernelGGL(kern, dim3(batch), dim3(MAXIDF_THREADS), lds_bytes, stream, ids, L,
                     num_blocks, (int)(L / num_blocks), chunk_log2, topk, vocab, (int)nb,
                     pow2 ? (int)(nb - 1) : 0, (int)plan.cmin_off, sel, chunk_mindf, idf);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}
