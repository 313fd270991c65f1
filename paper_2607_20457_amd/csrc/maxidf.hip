// Max-IDF summary construction on gfx950 (Section 3.1 "Summary generation",
// Eq. 2; Appendix "Corpus-Level IDF Table" and "Max-IDF").
//
// One 1024-thread workgroup per sequence keeps the whole document-frequency
// table of that sequence in the compute unit's local data share (LDS), so the
// table never touches HBM:
//
//   pass 1  the blocks in order, a workgroup barrier between two blocks:
//           stream the block's ids with 16-byte loads and count each id once
//           per block in its df entry.
//   pass 2  look up the df of every id; lanes of one chunk (chunk/4 lanes)
//           take the minimum with cross-lane operations.  The chunk minima go
//           to LDS (and optionally to HBM).
//   select  one wavefront per block picks the top-k chunks (select_topk).
//
// Pass 1 counts "once per block" in one of two ways:
//   * stamp code (N <= 16): one byte per id holds its df so far and the last
//     block it was seen in (see stamp_tokens).  A lane reads the byte and,
//     if the id is not yet stamped with the current block, writes the code of
//     (df + 1, this block).  Every lane that writes an id's byte during one
//     block writes the same value, so plain byte loads and stores suffice: no
//     atomics, and nothing to clear between blocks.
//   * bitmaps (any N <= 255): a per-block bitmap, set with atomic OR; the
//     lane that sets a bit first adds one to the id's df byte.
//
// Three kernels:
//   * resident (vocab <= 131072, L = 8192 times a power of two up to 16,
//     blocks of a multiple of 8192 ids, hence N <= 16): stamp code (with df
//     in the high nibble, see rstamp_tokens); pass 1 keeps every thread's
//     ids (up to 128) in registers, packed, and pass 2 reads them back from
//     there, so the ids cross HBM once; persistent over the batch, one
//     workgroup per compute unit;
//   * streaming, stamp code (N <= 16, table and chunk minima fit in LDS):
//     pass 2 streams the ids from HBM a second time;
//   * streaming, bitmaps: compact layout (vocab <= 131072: a fixed 4096-word
//     bitmap whose word is t & 4095) or general layout (scattered bitmap).
//
// A chunk's Max-IDF score ln(N / mindf) is strictly decreasing in mindf, so
// ranking by (mindf ascending, index ascending) is ranking by (score
// descending, index ascending).
#include "summary.hpp"


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
// of 4 ids per thread, a power of two up to RES_ROUNDS of them per sequence.
// Its static LDS holds the stamp-code table (vocab <= 131072 bytes) and,
// behind it, the chunk minima (at most kResChunkBytes).
constexpr int RES_ROUNDS = 16;
constexpr int RES_ROUND_TOKENS = MAXIDF_THREADS * 8;
constexpr int kResChunkBytes = PULSAR_LDS_BYTES - kFastVocab;

enum MaxidfMode { kGeneral = 0, kCompact = 1, kStamp = 2 };

struct MaxidfPlan {
  int mode;          // MaxidfMode of the streaming kernel
  bool resident;     // stamp code with the ids held in registers
  int64_t lds_bytes;
  int64_t cmin_off;  // byte offset of the chunk minima
};

// Streaming layouts: the df (or stamp-code) bytes [round_up4(vocab)] at LDS
// byte 0 (general, stamp) or 16384 (compact); the general layout reuses the
// region behind the table as the per-block bitmap (pass 1) and the chunk
// minima (pass 2 / select).
static MaxidfPlan maxidf_plan(int64_t L, int num_blocks, int chunk, int vocab) {
  const int64_t df_bytes = round_up4(vocab);
  const int64_t chunk_bytes = round_up4(L / chunk);
  // L = 8192 * (a power of two up to 16), blocks of a multiple of 8192 ids
  // (so N <= 16 and the rounds per block are a power of two)
  const int64_t res_rounds = L / RES_ROUND_TOKENS;
  if (vocab <= kFastVocab && L % RES_ROUND_TOKENS == 0 && res_rounds >= 1 &&
      res_rounds <= RES_ROUNDS &&
      (res_rounds & (res_rounds - 1)) == 0 && (L / num_blocks) % RES_ROUND_TOKENS == 0 &&
      chunk_bytes <= kResChunkBytes)
    return {kStamp, true, PULSAR_LDS_BYTES, kFastVocab};
  if (num_blocks <= kStampMaxBlocks && df_bytes + chunk_bytes <= PULSAR_LDS_BYTES)
    return {kStamp, false, df_bytes + chunk_bytes, df_bytes};
  if (vocab <= kFastVocab) {
    const bool in_bitmap = chunk_bytes <= kFastBitmapBytes;
    const int64_t lds = kFastBitmapBytes + df_bytes + (in_bitmap ? 0 : chunk_bytes);
    if (lds <= PULSAR_LDS_BYTES)
      return {kCompact, false, lds, in_bitmap ? 0 : kFastBitmapBytes + df_bytes};
  }
  const int64_t bitmap_bytes = bitmap_words(vocab) * 4;
  return {kGeneral, false, df_bytes + (bitmap_bytes > chunk_bytes ? bitmap_bytes : chunk_bytes),
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

// Optional IDF table (Eq. idf) of one sequence from its df bytes (STAMP:
// stamp codes) in LDS.
template <bool STAMP>
__device__ void write_idf(const uint8_t* df8, int vocab, int num_blocks, float* __restrict__ out,
                          int tid) {
  const float n = (float)num_blocks;
  for (int t = tid; t < vocab; t += MAXIDF_THREADS) {
    const uint32_t d = STAMP ? stamp_df(df8[t]) : df8[t];
    out[t] = logf(n / (float)(d > 1u ? d : 1u));
  }
}

template <int MODE>
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
  constexpr bool COMPACT = MODE == kCompact;
  constexpr bool STAMP = MODE == kStamp;
  uint8_t* df8 = lds8 + (COMPACT ? kFastBitmapBytes : 0);  // df bytes or stamp codes
  uint32_t* dfw = reinterpret_cast<uint32_t*>(df8);
  uint32_t* bits = COMPACT ? lds : lds + vocab_w4;
  uint8_t* cmin = lds8 + cmin_off;
  const uint32_t vmax = (uint32_t)(vocab - 1);

  const int32_t* seq = ids + b * L;

  const uint32_t init = STAMP ? kStampNever * 0x01010101u : 0u;
  for (int w = tid; w < vocab_w4; w += MAXIDF_THREADS) dfw[w] = init;
  // (the first round's barrier orders this against pass 1)

  // ---- pass 1: document frequency --------------------------------------
  // The blocks are streamed as rounds of MAXIDF_THREADS x ROUND int4 groups;
  // the loads of the next two rounds are in flight while a round's ids are
  // marked, so each thread overlaps its atomics with HBM latency.
  constexpr int ROUND = 2;
  constexpr int PREFETCH = 2;  // rounds of loads in flight
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
    if (rd % rpb == 0) {  // a new block: everyone is done with the previous one
      __syncthreads();
      if constexpr (!STAMP) {
        for (int w = tid; w < n_bitmap; w += MAXIDF_THREADS) bits[w] = 0u;
        __syncthreads();
      }
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
      const bool full = (rd - (rd / rpb) * rpb + 1) * ROUND * MAXIDF_THREADS <= nvec;
      if constexpr (STAMP) {
        if (full)
          stamp_tokens<4 * ROUND, false>(tk, rd / rpb, vmax, df8);
        else
          stamp_tokens<4 * ROUND, true>(tk, rd / rpb, vmax, df8);
      } else if constexpr (COMPACT) {
        if (full)
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

  if (idf) write_idf<STAMP>(df8, vocab, num_blocks, idf + b * vocab, tid);
  if constexpr (STAMP) {
    if (idf) __syncthreads();
    stamp_to_df(dfw, vocab_w4, tid);
    __syncthreads();
  }

  // ---- pass 2: per-chunk minimum df -------------------------------------
  // (STAMP: the table holds df - 1)
  // Groups of PF int4 loads per thread, double-buffered: group g+1 is in
  // flight while group g is reduced.  Every lane runs the same trip count,
  // so all lanes join the cross-lane minimum.
  constexpr int PF = 4;
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
      if (STAMP) mn += 1u;
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
  select_topk(cmin, b, num_blocks, Lb >> chunk_log2, (uint32_t)num_blocks, topk, sel, wave, lane);
}

// Stamp code of the resident kernel, block j: the high nibble of an id's byte
// holds df - 1 and the low nibble the stamp 15 - j of the last block j it was
// seen in; kStampNever (0xFF) before it is first seen.  The minimum of a
// chunk's codes then carries the chunk's minimum df - 1 in its high nibble,
// so pass 2 needs no conversion of the table.  A lane whose id is not yet
// stamped with j writes (df - 1 + 1, 15 - j); as with stamp_tokens, every
// writer of one byte during one block writes the same value.  CHECK_NEVER:
// kStampNever carries the stamp of block 0 in its low nibble, so a round that
// may belong to block 0 also tests for it.  nd: each id's df - 1 once this
// block is counted (final in the last block).
template <bool CHECK_NEVER>
__device__ __forceinline__ void rstamp_tokens(const int (&t)[4], int j, uint8_t* code,
                                              uint32_t (&nd)[4]) {
  uint32_t c[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) c[i] = code[t[i]];
  const uint32_t sj = 15u - (uint32_t)j;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bool stamped = (c[i] & 15u) == sj && (!CHECK_NEVER || c[i] != kStampNever);
    const uint32_t nc = ((c[i] + 16u) & 0xF0u) | sj;  // 0xFF + 16 wraps to df - 1 = 0
    nd[i] = (stamped ? c[i] : nc) >> 4;
    if (!stamped) code[t[i]] = (uint8_t)nc;
  }
}

// df of a resident stamp code (0 for an id never seen)
__device__ __forceinline__ uint32_t rstamp_df(uint32_t c) {
  return c == kStampNever ? 0u : (c >> 4) + 1u;
}

// Register-resident variant with the stamp code when the sequence fits the
// register file: L = ROUNDS * 8192 with ROUNDS a power of two up to 16, and
// Lb a multiple of 8192, so that every thread owns exactly ROUNDS x 2
// 16-byte groups of ids.  Pass 1 keeps each thread's ids in registers and
// pass 2 reads them back from there: the ids cross HBM once.  In round rd
// thread tid holds the 8 consecutive ids (rd*1024 + tid)*8 .. +7 (two
// adjacent 16-byte groups), so a chunk of m >= 8 ids spans m/8 lanes and
// pass 2 takes half of its minimum within the lane.
//
// Packing of the 4 clamped ids (< 2^17) of slot s: their low 16 bits two per
// register (plo), and their bit 16 in byte i of hb[s / 8] at bit s % 8 --
// each made and undone by byte permutes.
//
// Persistent: workgroup g takes sequences g, g + G, ... (G = gridDim.x, one
// workgroup per compute unit).  With CARRY_NEXT (more sequences than
// workgroups), pass 2 of one sequence frees the packed ids two rounds at a
// time and the first CARRY rounds of the next sequence are loaded into the
// freed registers, so HBM keeps streaming while the compute unit is busy
// with pass 2 and the top-k select.  Past the last sequence the next
// sequence's buffer resource covers no bytes, and those loads return zeros
// without touching memory.
//
// ROUNDS and the chunk's lane group (GL = log2(chunk / 4), or -1 for any)
// are template arguments, so that the loops are straight-line code: every
// load's wait is exact and the cross-lane minimum has no branches.  ONE: one
// round per block (Lb = 8192, N = ROUNDS), so the block of a round is known
// at compile time: block 0 writes its codes without reading them (every id
// is new), and the last block keeps each id's final df - 1 in the registers
// of its packed ids, so pass 2 looks up only the other blocks.
//
// The table of the next sequence is cleared while the select of the current
// one runs (the select reads only the chunk minima); the first sequence's,
// while its first ids are loading.
template <int ROUNDS, int GL, bool CARRY_NEXT, bool ONE>
__global__ __launch_bounds__(MAXIDF_THREADS) void maxidf_resident_kernel(
    const int32_t* __restrict__ ids, int batch, int num_blocks, int rpb_log2, int chunk_log2,
    int topk, int vocab, int32_t* __restrict__ sel, int32_t* __restrict__ chunk_mindf,
    float* __restrict__ idf) {
  // A fixed layout in static LDS, whose base the compiler knows, so every
  // table offset folds into the LDS instructions: the stamp codes (vocab <=
  // 131072 bytes), then the chunk minima (<= kResChunkBytes).
  __shared__ __attribute__((aligned(16))) uint32_t lds[PULSAR_LDS_BYTES / 4];
  constexpr int64_t L = (int64_t)ROUNDS * RES_ROUND_TOKENS;
  // rounds of the next sequence loaded during pass 2
  constexpr int CARRY = CARRY_NEXT ? ROUNDS / 2 : 0;
  constexpr int PREFETCH = 2;        // rounds of loads in flight during pass 1
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  uint8_t* const lds8 = reinterpret_cast<uint8_t*>(lds);
  uint8_t* code8 = lds8;
  uint8_t* cmin = lds8 + kFastVocab;
  const uint32_t vmax = (uint32_t)(vocab - 1);
  const int vocab_w4 = (vocab + 3) >> 2;
  const uint32_t lane_off = (uint32_t)tid * 32u;
  const int cl2 = GL >= 0 ? GL + 2 : chunk_log2;  // log2(chunk)
  const int nchunks_seq = (int)(L >> cl2);

  // a sequence's ids through a buffer resource (no bytes past the batch):
  // one lane offset, and each group's offset a scalar constant
  auto seq_rsrc = [&](int64_t b) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(ids + (b < batch ? b : 0) * L),
                                             (short)0, b < batch ? (int)(L * 4) : 0, kRawBuffer);
  };
  auto load_round = [&](__amdgpu_buffer_rsrc_t r, int rd, int4 (&t)[2]) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(
          r, lane_off, rd * MAXIDF_THREADS * 32 + u * 16, 0);
      t[u] = make_int4((int)v[0], (int)v[1], (int)v[2], (int)v[3]);
    }
  };

  auto clear_table = [&]() {
    const uint4 never = make_uint4(kStampNever * 0x01010101u, kStampNever * 0x01010101u,
                                   kStampNever * 0x01010101u, kStampNever * 0x01010101u);
    uint4* code16 = reinterpret_cast<uint4*>(lds);
    for (int w = tid; w < (vocab_w4 + 3) >> 2; w += MAXIDF_THREADS) code16[w] = never;
  };
  int4 nbuf[CARRY > 0 ? CARRY : 1][2];  // the next sequence's first CARRY rounds
  int4 cbuf[PREFETCH + 1][2];           // the rounds in flight during pass 1
  {
    // the first sequence's first rounds are in flight while its table is
    // cleared (without CARRY_NEXT a workgroup has one sequence, and its
    // first rounds are loaded here rather than in the loop)
    const __amdgpu_buffer_rsrc_t r0 = seq_rsrc(blockIdx.x);
#pragma unroll
    for (int rd = 0; rd < CARRY; ++rd) load_round(r0, rd, nbuf[rd]);
    if constexpr (!CARRY_NEXT) {
#pragma unroll
      for (int i = 0; i < PREFETCH && i < ROUNDS; ++i) load_round(r0, i, cbuf[i]);
    }
    clear_table();
  }
  for (int64_t b = blockIdx.x; b < batch; b += gridDim.x) {
    const __amdgpu_buffer_rsrc_t rsrc = seq_rsrc(b);
    const __amdgpu_buffer_rsrc_t rnext = seq_rsrc(b + gridDim.x);

    // ---- pass 1: document frequency, ids kept in registers ----------------
    uint32_t plo[ROUNDS][2][2];              // low 16 bits, two ids per register
    uint32_t hb[(ROUNDS * 2 + 7) / 8] = {};  // bit 16 of the ids of slot s: bit s % 8 of each byte
    if constexpr (CARRY_NEXT) {
#pragma unroll
      for (int i = CARRY; i < CARRY + PREFETCH && i < ROUNDS; ++i)
        load_round(rsrc, i, cbuf[i % (PREFETCH + 1)]);
    }
    __syncthreads();
#pragma unroll
    for (int rd = 0; rd < ROUNDS; ++rd) {
      // block j starts once every wave is past block j - 1
      const int j = rd >> rpb_log2;
      if (rd > 0 && (rd & ((1 << rpb_log2) - 1)) == 0) __syncthreads();
      if (rd >= CARRY && rd + PREFETCH < ROUNDS)
        load_round(rsrc, rd + PREFETCH, cbuf[(rd + PREFETCH) % (PREFETCH + 1)]);
      const int4 (&cur)[2] = rd < CARRY ? nbuf[rd < CARRY ? rd : 0] : cbuf[rd % (PREFETCH + 1)];
      // one 16-byte group at a time (measured faster than all 8 ids of the
      // round together)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int4 x = cur[u];
        const uint32_t t0 = min((uint32_t)x.x, vmax), t1 = min((uint32_t)x.y, vmax);
        const uint32_t t2 = min((uint32_t)x.z, vmax), t3 = min((uint32_t)x.w, vmax);
        const int tk[4] = {(int)t0, (int)t1, (int)t2, (int)t3};
        const int slot = 2 * rd + u;
        plo[rd][u][0] = __builtin_amdgcn_perm(t1, t0, 0x05040100u);
        plo[rd][u][1] = __builtin_amdgcn_perm(t3, t2, 0x05040100u);
        // byte i of h4 = bit 16 of id i
        const uint32_t h4 = __builtin_amdgcn_perm(t1, t0, 0x0C0C0602u) |
                            (__builtin_amdgcn_perm(t3, t2, 0x0C0C0602u) << 16);
        hb[slot >> 3] |= h4 << (slot & 7);
        // packed here, not next to pass 2: the compiler would otherwise keep
        // the unpacked ids alive
        asm volatile("" : "+v"(plo[rd][u][0]), "+v"(plo[rd][u][1]), "+v"(hb[slot >> 3]));
        if (ONE && rd == 0) {
          // block 0: every id is seen for the first time (df 1, stamp of
          // block 0), so its byte need not be read
#pragma unroll
          for (int i = 0; i < 4; ++i) code8[tk[i]] = (uint8_t)15u;
          if (ROUNDS == 1) plo[rd][u][0] = 0u;
        } else {
          uint32_t nd[4];
          if (ONE)
            rstamp_tokens<false>(tk, j, code8, nd);
          else
            rstamp_tokens<true>(tk, j, code8, nd);
          // the last block: the df - 1 read or written now is final, so
          // pass 2 takes it from here instead of the table
          if (ONE && rd == ROUNDS - 1)
            plo[rd][u][0] = nd[0] | (nd[1] << 8) | (nd[2] << 16) | (nd[3] << 24);
        }
      }
    }
    __syncthreads();
    if (idf) {
      const float nb = (float)num_blocks;
      float* out = idf + b * vocab;
      for (int t = tid; t < vocab; t += MAXIDF_THREADS) {
        const uint32_t d = rstamp_df(code8[t]);
        out[t] = logf(nb / (float)(d > 1u ? d : 1u));
      }
      __syncthreads();
    }

    // ---- pass 2: per-chunk minimum df from the registers ------------------
    // (the thread index is re-formed in every iteration: values derived from
    // it would otherwise be hoisted out of the sequence loop and held in
    // registers throughout)
    int tid_i = tid;
    asm volatile("" : "+v"(tid_i));
#pragma unroll
    for (int rd = 0; rd < ROUNDS; ++rd) {
      // the minimum df - 1 of each 16-byte half of the lane's 8 ids
      uint32_t mn[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int slot = 2 * rd + u;
        const uint32_t lo0 = plo[rd][u][0], lo1 = plo[rd][u][1];
        const uint32_t x = (hb[slot >> 3] >> (slot & 7)) & 0x01010101u;
        const uint32_t t0 = __builtin_amdgcn_perm(x, lo0, 0x0C040100u);
        const uint32_t t1 = __builtin_amdgcn_perm(x, lo0, 0x0C050302u);
        const uint32_t t2 = __builtin_amdgcn_perm(x, lo1, 0x0C060100u);
        const uint32_t t3 = __builtin_amdgcn_perm(x, lo1, 0x0C070302u);
        if (ONE && rd == ROUNDS - 1)
          mn[u] = min(min(lo0 & 0xFFu, (lo0 >> 8) & 0xFFu), min((lo0 >> 16) & 0xFFu, lo0 >> 24));
        else
          mn[u] = min(min((uint32_t)code8[t0], (uint32_t)code8[t1]),
                      min((uint32_t)code8[t2], (uint32_t)code8[t3])) >> 4;
      }
      const int g8 = rd * MAXIDF_THREADS + tid_i;  // the lane's 8-id group in the sequence
      if (cl2 == 2) {
        // chunks of 4 ids: each half is a chunk of its own
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          cmin[2 * g8 + u] = (uint8_t)(mn[u] + 1u);
          if (chunk_mindf) chunk_mindf[b * nchunks_seq + 2 * g8 + u] = (int32_t)(mn[u] + 1u);
        }
      } else {
        const int lg = cl2 - 3;  // log2 of the lanes per chunk, m / 8
        uint32_t m2 = min(mn[0], mn[1]);
        if constexpr (GL >= 1) m2 = group_min_c<GL - 1>(m2);
        else m2 = group_min(m2, 1 << lg);
        m2 += 1u;
        if ((tid_i & ((1 << lg) - 1)) == 0) {
          cmin[g8 >> lg] = (uint8_t)m2;
          if (chunk_mindf) chunk_mindf[b * nchunks_seq + (g8 >> lg)] = (int32_t)m2;
        }
      }
      // every second round frees two rounds of packed ids: load one round of
      // the next sequence in their place
      if ((rd & 1) == 1 && (rd >> 1) < CARRY) {
        __builtin_amdgcn_sched_barrier(0);
        load_round(rnext, rd >> 1, nbuf[(rd >> 1) < CARRY ? (rd >> 1) : 0]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __syncthreads();
    // the next sequence's table is cleared while the select runs (it reads
    // only the chunk minima)
    if (b + gridDim.x < batch) clear_table();
    select_topk(cmin, b, num_blocks, (int)(L / num_blocks) >> chunk_log2, (uint32_t)num_blocks, topk,
                sel, wave, lane);
  }
}

// Resident kernels by (rounds, chunk): the lane group is a template argument
// for chunks of 16 and 32 ids, the common sizes.
typedef void (*ResidentKernel)(const int32_t*, int, int, int, int, int, int, int32_t*, int32_t*,
                               float*);
template <int ROUNDS, bool CARRY_NEXT, bool ONE>
static ResidentKernel resident_for_chunk(int chunk_log2) {
  if (chunk_log2 == 5) return maxidf_resident_kernel<ROUNDS, 3, CARRY_NEXT, ONE>;
  if (chunk_log2 == 4) return maxidf_resident_kernel<ROUNDS, 2, CARRY_NEXT, ONE>;
  return maxidf_resident_kernel<ROUNDS, -1, CARRY_NEXT, ONE>;
}
template <int ROUNDS, bool CARRY_NEXT>
static ResidentKernel resident_for_chunk(int chunk_log2, int rpb_log2) {
  return rpb_log2 == 0 ? resident_for_chunk<ROUNDS, CARRY_NEXT, true>(chunk_log2)
                       : resident_for_chunk<ROUNDS, CARRY_NEXT, false>(chunk_log2);
}
template <bool CARRY_NEXT>
static ResidentKernel resident_kernel(int rounds, int chunk_log2, int rpb_log2) {
  switch (rounds) {
    case 16: return resident_for_chunk<16, CARRY_NEXT>(chunk_log2, rpb_log2);
    case 8: return resident_for_chunk<8, CARRY_NEXT>(chunk_log2, rpb_log2);
    case 4: return resident_for_chunk<4, CARRY_NEXT>(chunk_log2, rpb_log2);
    case 2: return resident_for_chunk<2, CARRY_NEXT>(chunk_log2, rpb_log2);
    case 1: return resident_for_chunk<1, CARRY_NEXT>(chunk_log2, rpb_log2);
    default: return nullptr;  // maxidf_plan admits only the round counts above
  }
}

int launch_maxidf(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk, int topk,
                  int vocab, int32_t* sel, int32_t* chunk_mindf, float* idf, size_t lds_bytes,
                  hipStream_t stream) {
  if (batch == 0 || L == 0) return PULSAR_OK;
  int chunk_log2 = 0;
  while ((1 << chunk_log2) < chunk) ++chunk_log2;
  const MaxidfPlan plan = maxidf_plan(L, num_blocks, chunk, vocab);
  if ((size_t)plan.lds_bytes != lds_bytes) return PULSAR_EINVAL;
  if (plan.resident) {  // static LDS only
    const int rounds = (int)(L / RES_ROUND_TOKENS);
    int rpb_log2 = 0;
    while ((RES_ROUND_TOKENS << rpb_log2) < L / num_blocks) ++rpb_log2;
    // one workgroup per compute unit (160 KB of LDS each), persistent over
    // the batch; the next sequence's ids are carried only when a workgroup
    // has more than one sequence
    int dev = 0, n_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n_cu < 1)
      return PULSAR_EHIP;
    const int grid = batch < n_cu ? batch : n_cu;
    const ResidentKernel kern = batch > grid ? resident_kernel<true>(rounds, chunk_log2, rpb_log2)
                                             : resident_kernel<false>(rounds, chunk_log2, rpb_log2);
    if (kern == nullptr) return PULSAR_EINVAL;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(MAXIDF_THREADS), 0, stream, ids, batch, num_blocks,
                       rpb_log2, chunk_log2, topk, vocab, sel, chunk_mindf, idf);
    return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
  }
  const auto kern = plan.mode == kStamp     ? maxidf_kernel<kStamp>
                    : plan.mode == kCompact ? maxidf_kernel<kCompact>
                                            : maxidf_kernel<kGeneral>;
  if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lds_bytes) != hipSuccess)
    return PULSAR_EHIP;
  const int64_t nb = plan.mode == kCompact ? kFastWords : bitmap_words(vocab);
  const bool pow2 = (nb & (nb - 1)) == 0;
  hipLaunchKernelGGL(kern, dim3(batch), dim3(MAXIDF_THREADS), lds_bytes, stream, ids, L,
                     num_blocks, (int)(L / num_blocks), chunk_log2, topk, vocab, (int)nb,
                     pow2 ? (int)(nb - 1) : 0, (int)plan.cmin_off, sel, chunk_mindf, idf);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}
