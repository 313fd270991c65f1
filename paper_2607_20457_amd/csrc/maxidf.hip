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
//   pass 2  stream the ids again; each lane looks up the df of its four ids,
//           and lanes of one chunk (chunk/4 lanes) take the minimum with
//           cross-lane shuffles.  The chunk minima go to LDS (and optionally
//           to HBM).
//   select  one wavefront per block finds the threshold tau, the smallest df
//           with at least k chunks at or below it (binary search over
//           1..N with wave-wide counts), keeps every chunk below tau and the
//           first k - #(< tau) chunks equal to tau in index order, and writes
//           the kept indices in ascending order with a wave prefix sum.
//
// A chunk's Max-IDF score ln(N / mindf) is strictly decreasing in mindf, so
// ranking by (mindf ascending, index ascending) is ranking by (score
// descending, index ascending).
#include "common.hpp"

#define MAXIDF_THREADS 1024
#define MAXIDF_WAVES (MAXIDF_THREADS / PULSAR_WAVE)

static inline int64_t round_up4(int64_t x) { return (x + 3) & ~int64_t(3); }

// Bitmap words: a power of two at least vocab/32 when that still fits next
// to the df table (vocab up to 131072 here), so that the bitmap can be
// scattered (see mark_token); otherwise exactly ceil(vocab/32), unscattered.
static int64_t bitmap_words(int vocab) {
  const int64_t need = ((int64_t)vocab + 31) / 32;
  int64_t w = 1;
  while (w < need) w <<= 1;
  return round_up4(vocab) + w * 4 <= PULSAR_LDS_BYTES ? w : need;
}

// LDS layout: df bytes [round_up4(vocab)], then a region reused as the
// per-block bitmap (pass 1) and the chunk minima (pass 2 / select).
size_t maxidf_lds_bytes(int64_t L, int chunk, int vocab) {
  int64_t df_bytes = round_up4(vocab);
  int64_t bitmap_bytes = bitmap_words(vocab) * 4;
  int64_t chunk_bytes = round_up4(L / chunk);
  return (size_t)(df_bytes + (bitmap_bytes > chunk_bytes ? bitmap_bytes : chunk_bytes));
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
    if (bit[i] & ~old[i]) atomicAdd(&dfw[ts[i] >> 2], 1u << ((ts[i] & 3) * 8));
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

__global__ __launch_bounds__(MAXIDF_THREADS) void maxidf_kernel(
    const int32_t* __restrict__ ids, int64_t L, int num_blocks, int Lb, int chunk_log2,
    int topk, int vocab, int n_bitmap, int spread_mask, int32_t* __restrict__ sel,
    int32_t* __restrict__ chunk_mindf, float* __restrict__ idf) {
  extern __shared__ uint32_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t b = blockIdx.x;
  const int chunk = 1 << chunk_log2;
  const int vocab_w4 = (vocab + 3) >> 2;
  uint32_t* dfw = lds;
  uint8_t* df8 = reinterpret_cast<uint8_t*>(lds);
  uint32_t* bits = lds + vocab_w4;
  uint8_t* cmin = reinterpret_cast<uint8_t*>(bits);

  const int32_t* seq = ids + b * L;

  for (int w = tid; w < vocab_w4; w += MAXIDF_THREADS) dfw[w] = 0u;
  // (the first round's barrier orders this against the atomics)

  // ---- pass 1: document frequency --------------------------------------
  // The blocks are streamed as rounds of MAXIDF_THREADS x ROUND int4 groups;
  // the loads of the next two rounds are in flight while a round's ids are
  // marked, so each thread overlaps its atomics with HBM latency.
  constexpr int ROUND = 2;
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
  int4 c0[ROUND], c1[ROUND], c2[ROUND];
  if (rounds > 0) load_round(0, c0);
  if (rounds > 1) load_round(1, c1);
  for (int rd = 0; rd < rounds; ++rd) {
    if (rd % rpb == 0) {  // a new block: everyone is done with the previous bitmap
      __syncthreads();
      for (int w = tid; w < n_bitmap; w += MAXIDF_THREADS) bits[w] = 0u;
      __syncthreads();
    }
    if (rd + 2 < rounds) load_round(rd + 2, c2);
    {
      int tk[4 * ROUND];
#pragma unroll
      for (int u = 0; u < ROUND; ++u) {
        tk[4 * u] = c0[u].x;
        tk[4 * u + 1] = c0[u].y;
        tk[4 * u + 2] = c0[u].z;
        tk[4 * u + 3] = c0[u].w;
      }
      mark_tokens(tk, vocab, spread_mask, bits, dfw);
    }
#pragma unroll
    for (int u = 0; u < ROUND; ++u) {
      c0[u] = c1[u];
      c1[u] = c2[u];
    }
  }
  __syncthreads();

  // ---- optional IDF table (Eq. idf) -------------------------------------
  if (idf) {
    const float n = (float)num_blocks;
    float* out = idf + b * vocab;
    for (int t = tid; t < vocab; t += MAXIDF_THREADS) {
      const uint32_t d = df8[t];
      out[t] = logf(n / (float)(d > 1u ? d : 1u));
    }
  }

  // ---- pass 2: per-chunk minimum df -------------------------------------
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

  // ---- select: top-k chunks per block, ascending order ------------------
  if (topk == 0) return;
  const int C = Lb >> chunk_log2;          // chunks per block
  const int per_lane = (C + 63) >> 6;      // contiguous chunks owned by a lane
  for (int j = wave; j < num_blocks; j += MAXIDF_WAVES) {
    const uint8_t* cv = cmin + (int64_t)j * C;
    const int c0 = lane * per_lane;
    const int c1 = min(C, c0 + per_lane);
    // smallest tau with #(mindf <= tau) >= topk; mindf lies in [1, num_blocks]
    int lo = 0, hi = num_blocks;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      int cnt = 0;
      for (int c = c0; c < c1; ++c) cnt += cv[c] <= mid;
      cnt = wave_sum_int(cnt);
      if (cnt >= topk) hi = mid; else lo = mid;
    }
    const int tau = hi;
    int n_lt = 0, n_eq = 0;
    for (int c = c0; c < c1; ++c) {
      n_lt += cv[c] < tau;
      n_eq += cv[c] == tau;
    }
    const int need = topk - wave_sum_int(n_lt);  // chunks equal to tau that are kept
    const int eq_base = wave_excl_scan(n_eq);     // equal-to-tau chunks in lower lanes
    int n_sel = 0;
    int r = eq_base;
    for (int c = c0; c < c1; ++c) {
      const int x = cv[c];
      if (x < tau) {
        ++n_sel;
      } else if (x == tau) {
        n_sel += r < need;
        ++r;
      }
    }
    int out = wave_excl_scan(n_sel);
    int32_t* dst = sel + (b * num_blocks + j) * topk;
    r = eq_base;
    for (int c = c0; c < c1; ++c) {
      const int x = cv[c];
      bool keep = x < tau;
      if (x == tau) {
        keep = r < need;
        ++r;
      }
      if (keep) dst[out++] = c;
    }
  }
}

int launch_maxidf(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk, int topk,
                  int vocab, int32_t* sel, int32_t* chunk_mindf, float* idf, size_t lds_bytes,
                  hipStream_t stream) {
  if (batch == 0) return PULSAR_OK;
  int chunk_log2 = 0;
  while ((1 << chunk_log2) < chunk) ++chunk_log2;
  if (hipFuncSetAttribute((const void*)maxidf_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lds_bytes) != hipSuccess)
    return PULSAR_EHIP;
  const int64_t nb = bitmap_words(vocab);
  const bool pow2 = (nb & (nb - 1)) == 0;
  hipLaunchKernelGGL(maxidf_kernel, dim3(batch), dim3(MAXIDF_THREADS), lds_bytes, stream, ids, L,
                     num_blocks, (int)(L / num_blocks), chunk_log2, topk, vocab, (int)nb,
                     pow2 ? (int)(nb - 1) : 0, sel, chunk_mindf, idf);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}
