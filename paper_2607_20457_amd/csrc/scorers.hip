// Chunk summaries under the other scorers of the paper (Appendix "Scoring
// Heuristic Details"): TF-IDF (Eq. tfidf), BM25 (Eq. bm25), Entropy
// (Eq. entropy), and Max-IDF again (Eq. maxidf) so that every scorer has the
// same interface.  They share the document-frequency pass with Max-IDF.
//
// One 1024-thread workgroup per sequence, N <= 16 blocks:
//   pass 1  the stamp-code df table in LDS (summary.hpp), then df - 1 per id;
//   pass 2  the ids streamed again, 4 per lane; the lanes of a chunk (chunk/4
//           of them) each add up their 4 positions and combine with
//           cross-lane operations;
//   select  the k best chunks of each block in positional order.
//
// Per position p of a chunk C with token t (df = df(t), tf = occurrences of
// t in C, m = |C|):
//   TF-IDF   ln(N / df) / m
//   BM25     IDF_BM25(df) (k1 + 1) / (tf + k1 D), IDF_BM25(df) = ln((N - df +
//            0.5) / (df + 0.5) + 1), k1 = 1.2, b = 0.75, D = 1 - b + b m /
//            l_bar = 1 (every chunk has the mean length); summed over the
//            positions of a token this is the paper's per-token term
//   Entropy  1 / tf, whose sum over C is the number of distinct tokens
//   Max-IDF  the chunk's minimum df (its score is ln(N / mindf))
// The sums are taken in fp64 and the score rounded once to fp32 (the paper
// scores from an fp32 IDF table); Entropy's sum is rounded to the integer it
// equals.  tf comes from comparing every position with the m tokens of its
// chunk, which each wave stages in LDS.
//
// Ranking keys (smaller is better; ties go to the lower chunk index): the
// minimum df for Max-IDF, m - distinct for Entropy, and the complemented bit
// pattern of the non-negative fp32 score for TF-IDF and BM25.
#include <cmath>

#include "split.hpp"

namespace {

constexpr double kK1 = 1.2;
constexpr double kB = 0.75;
constexpr int kStageBytes = MAXIDF_WAVES * 256 * 4;  // one 256-id slot per wave

struct ScorerLayout {
  int64_t key_off;    // uint32 chunk keys [L / m]
  int64_t tab_off;    // fp64 tables: per df value [N + 1], per tf value [m + 1]
  int64_t stage_off;  // tf staging, kStageBytes (BM25, Entropy)
  int64_t bytes;
};

bool needs_tf(int scorer) { return scorer == PULSAR_SCORE_BM25 || scorer == PULSAR_SCORE_ENTROPY; }

int64_t round_up16(int64_t x) { return (x + 15) & ~int64_t(15); }

ScorerLayout scorer_layout(int64_t L, int num_blocks, int chunk, int vocab, int scorer) {
  ScorerLayout s{};
  s.key_off = round_up16(vocab);
  s.tab_off = s.key_off + round_up16(L / chunk * 4);
  s.stage_off = s.tab_off + round_up16((int64_t)(num_blocks + 1 + chunk + 1) * 8);
  s.bytes = s.stage_off + (needs_tf(scorer) ? kStageBytes : 0);
  return s;
}

// Sum over aligned groups of 2^GL lanes (GL < 0: `group` lanes); every lane
// of a group ends with the same sum.
template <int GL, typename T>
__device__ __forceinline__ T group_sum(T x, int group) {
  auto mov = [](T v, auto ctrl) {
    if constexpr (sizeof(T) == 8) {
      const uint64_t u = __builtin_bit_cast(uint64_t, v);
      const uint64_t r = (uint64_t)dpp_mov<decltype(ctrl)::value>((uint32_t)u) |
                         ((uint64_t)dpp_mov<decltype(ctrl)::value>((uint32_t)(u >> 32)) << 32);
      return __builtin_bit_cast(T, r);
    } else {
      return __builtin_bit_cast(T, dpp_mov<decltype(ctrl)::value>(__builtin_bit_cast(uint32_t, v)));
    }
  };
  auto xor_shfl = [](T v, int mask) {
    if constexpr (sizeof(T) == 8) {
      const uint64_t u = __builtin_bit_cast(uint64_t, v);
      const uint64_t r = (uint64_t)(uint32_t)__shfl_xor((int)(uint32_t)u, mask, 64) |
                         ((uint64_t)(uint32_t)__shfl_xor((int)(uint32_t)(u >> 32), mask, 64) << 32);
      return __builtin_bit_cast(T, r);
    } else {
      return __builtin_bit_cast(T, __shfl_xor(__builtin_bit_cast(int, v), mask, 64));
    }
  };
  const int gl = GL >= 0 ? GL : __builtin_ctz((unsigned)group);
  if (gl >= 1) x = x + mov(x, std::integral_constant<int, 0xB1>{});   // lane ^ 1
  if (gl >= 2) x = x + mov(x, std::integral_constant<int, 0x4E>{});   // lane ^ 2
  if (gl >= 3) x = x + mov(x, std::integral_constant<int, 0x141>{});  // mirror within 8
  if (gl >= 4) x = x + mov(x, std::integral_constant<int, 0x140>{});  // mirror within 16
  if (gl >= 5) x = x + xor_shfl(x, 16);
  if (gl >= 6) x = x + xor_shfl(x, 32);
  return x;
}

template <int SCORER, int GL>
__global__ __launch_bounds__(MAXIDF_THREADS) void scorer_kernel(
    const int32_t* __restrict__ ids, int64_t L, int num_blocks, int Lb, int chunk_log2, int topk,
    int vocab, int key_off, int tab_off, int stage_off, int32_t* __restrict__ sel,
    float* __restrict__ scores) {
  extern __shared__ uint32_t lds[];
  uint8_t* const lds8 = reinterpret_cast<uint8_t*>(lds);
  uint8_t* code8 = lds8;
  uint32_t* keys = reinterpret_cast<uint32_t*>(lds8 + key_off);
  double* tab_df = reinterpret_cast<double*>(lds8 + tab_off);  // [N + 1] by df
  double* tab_tf = tab_df + num_blocks + 1;                     // [m + 1] by tf
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t b = blockIdx.x;
  const int m = 1 << chunk_log2;
  const int group_log2 = GL >= 0 ? GL : chunk_log2 - 2;  // lanes per chunk: 1..64
  const int group = 1 << group_log2;
  const uint32_t vmax = (uint32_t)(vocab - 1);
  const int vocab_w4 = (vocab + 3) >> 2;
  const int4* seq4 = reinterpret_cast<const int4*>(ids + b * L);
  const double N = (double)num_blocks;

  for (int w = tid; w < vocab_w4; w += MAXIDF_THREADS) lds[w] = kStampNever * 0x01010101u;
  // per-value tables (the first barrier of pass 1 orders them)
  if (tid <= num_blocks) {
    const double d = (double)tid;
    if (SCORER == PULSAR_SCORE_TFIDF) tab_df[tid] = log(N / fmax(d, 1.0));
    if (SCORER == PULSAR_SCORE_BM25) tab_df[tid] = log((N - d + 0.5) / (d + 0.5) + 1.0);
  }
  if (tid <= m && tid >= 1) {
    const double tf = (double)tid;
    const double D = 1.0 - kB + kB * (double)m / (double)m;  // every chunk has the mean length
    if (SCORER == PULSAR_SCORE_BM25) tab_tf[tid] = (kK1 + 1.0) / (tf + kK1 * D);
    if (SCORER == PULSAR_SCORE_ENTROPY) tab_tf[tid] = 1.0 / tf;
  }

  // ---- pass 1: document frequency ----------------------------------------
  stamp_pass_streaming(seq4, num_blocks, Lb, vmax, code8, tid);
  stamp_to_df(lds, vocab_w4, tid);
  __syncthreads();

  // ---- pass 2: per-chunk score and key --------------------------------------
  const int nvec_seq = (int)(L >> 2);
  const int n_iter = (nvec_seq + MAXIDF_THREADS - 1) / MAXIDF_THREADS;
  const int nchunks_seq = (int)(L >> chunk_log2);
  int4* stage = reinterpret_cast<int4*>(lds8 + stage_off) + wave * 64;
  const int gbase = lane & ~(group - 1);  // first lane of this lane's chunk
  // the next iteration's ids load while this one is scored; past the end a
  // lane re-reads the last group (without a branch), which it does not use
  auto load_it = [&](int it) { return seq4[min(it * MAXIDF_THREADS + tid, nvec_seq - 1)]; };
  auto body = [&](int it, const int4 x4) {
    const int v = it * MAXIDF_THREADS + tid;
    auto clamp = [&](int x) { return (uint32_t)x < vmax ? (uint32_t)x : vmax; };
    const uint32_t t[4] = {clamp(x4.x), clamp(x4.y), clamp(x4.z), clamp(x4.w)};
    uint32_t dfm1[4];  // df - 1
#pragma unroll
    for (int i = 0; i < 4; ++i) dfm1[i] = code8[t[i]];
    uint32_t key = 0;
    float score = 0.f;
    if constexpr (SCORER == PULSAR_SCORE_MAXIDF) {
      uint32_t mn = min(min(dfm1[0], dfm1[1]), min(dfm1[2], dfm1[3]));
      mn = (GL >= 0 ? group_min_c<GL >= 0 ? GL : 0>(mn) : group_min(mn, group)) + 1u;
      key = mn;
      score = (float)log(N / (double)mn);
    } else if constexpr (SCORER == PULSAR_SCORE_TFIDF) {
      double s = 0.0;
#pragma unroll
      for (int i = 0; i < 4; ++i) s += tab_df[dfm1[i] + 1];
      s = group_sum<GL>(s, group);
      score = (float)(s / (double)m);  // m a power of two: the division is exact
      key = ~__builtin_bit_cast(uint32_t, score);
    } else {
      // tf of each of the 4 positions within the chunk, from the chunk's m
      // tokens staged by the wave
      stage[lane] = make_int4((int)t[0], (int)t[1], (int)t[2], (int)t[3]);
      uint32_t tf[4] = {0u, 0u, 0u, 0u};
      const int4* cs = stage + gbase;
      for (int q = 0; q < group; ++q) {
        const int4 y = cs[q];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          tf[i] += (uint32_t)((uint32_t)y.x == t[i]);
          tf[i] += (uint32_t)((uint32_t)y.y == t[i]);
          tf[i] += (uint32_t)((uint32_t)y.z == t[i]);
          tf[i] += (uint32_t)((uint32_t)y.w == t[i]);
        }
      }
      // The counts stay opaque until here, so that the table index's scaling
      // is not distributed over the terms: each comparison is then one
      // compare and one add-with-carry.
#pragma unroll
      for (int i = 0; i < 4; ++i) asm volatile("" : "+v"(tf[i]));
      double s = 0.0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const double w = tab_tf[tf[i]];
        s += SCORER == PULSAR_SCORE_BM25 ? tab_df[dfm1[i] + 1] * w : w;
      }
      s = group_sum<GL>(s, group);
      if constexpr (SCORER == PULSAR_SCORE_BM25) {
        score = (float)s;
        key = ~__builtin_bit_cast(uint32_t, score);
      } else {
        const int distinct = (int)rint(s);  // a sum of 1/tf over the chunk
        score = (float)distinct / (float)m;  // m a power of two: exact
        key = (uint32_t)(m - distinct);
      }
    }
    if ((lane & (group - 1)) == 0 && v < nvec_seq) {
      const int c = v >> group_log2;
      keys[c] = key;
      if (scores) scores[b * nchunks_seq + c] = score;
    }
  };
  // unrolled by two, so that each buffer keeps its register while its load
  // is in flight (the same trip count in every lane)
  int4 xa = load_it(0), xb = load_it(1);
  for (int it = 0; it < n_iter; it += 2) {
    body(it, xa);
    xa = load_it(it + 2);
    if (it + 1 < n_iter) body(it + 1, xb);
    xb = load_it(it + 3);
  }
  __syncthreads();

  // ---- select ------------------------------------------------------------
  const uint32_t key_hi = SCORER == PULSAR_SCORE_MAXIDF   ? (uint32_t)num_blocks
                          : SCORER == PULSAR_SCORE_ENTROPY ? (uint32_t)m
                                                           : 0xFFFFFFFFu;
  select_topk(keys, b, num_blocks, Lb >> chunk_log2, key_hi, topk, sel, wave, lane);
}

// ---- split path: a small batch over many compute units ----------------------
// The presence and df kernels of the Max-IDF split path (split.hpp) leave the
// df table of each sequence in the workspace (a nibble df - 1 per id: the
// scorers take N <= 16); then one workgroup per (sequence, block) copies the
// table into LDS and scores the block's chunks.  In round r thread tid holds
// the 8 consecutive ids 8 (1024 r + tid) .. +7 of the block, so a chunk of m
// ids is one 16-byte group (m = 4) or m / 8 adjacent lanes: a lane adds up
// its 8 positions (each group of 4 for m = 4), then its lane group.  tf comes
// from comparing each position with the m tokens of its chunk, which each
// wave stages in LDS (for m = 4, the lane's own group).  The per-value tables
// and the rounding are those of scorer_kernel.
struct SplitScoreLayout {
  int64_t key_off;    // uint32 chunk keys [Lb / m]
  int64_t tab_off;    // fp64 tables: per df value [N + 1], per tf value [m + 1]
  int64_t stage_off;  // tf staging, 16 waves x 512 ids (BM25, Entropy)
  int64_t bytes;
};
constexpr int kSplitStageBytes = (kSplitThreads / 64) * 512 * 4;

SplitScoreLayout split_score_layout(int64_t L, int num_blocks, int chunk, int vocab, int scorer) {
  SplitScoreLayout s{};
  s.key_off = split_words(vocab) * 16;  // the nibble df table
  s.tab_off = s.key_off + round_up16(L / num_blocks / chunk * 4);
  s.stage_off = s.tab_off + round_up16((int64_t)(num_blocks + 1 + chunk + 1) * 8);
  s.bytes = s.stage_off + (needs_tf(scorer) ? kSplitStageBytes : 0);
  return s;
}

template <int SCORER>
__global__ __launch_bounds__(kSplitThreads) void split_score_kernel(
    const int32_t* __restrict__ ids, int64_t L, int num_blocks, int Lb, int chunk_log2, int topk,
    int vocab, const uint8_t* __restrict__ ws, int64_t seq_bytes, int key_off, int tab_off,
    int stage_off, int32_t* __restrict__ sel, float* __restrict__ scores) {
  extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
  uint8_t* const lds8 = reinterpret_cast<uint8_t*>(lds);
  uint32_t* const keys = reinterpret_cast<uint32_t*>(lds8 + key_off);
  double* const tab_df = reinterpret_cast<double*>(lds8 + tab_off);  // [N + 1] by df
  double* const tab_tf = tab_df + num_blocks + 1;                     // [m + 1] by tf
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t b = blockIdx.x / num_blocks;
  const int j = blockIdx.x - (int)(b * num_blocks);
  const int m = 1 << chunk_log2;
  const int C = Lb >> chunk_log2;
  const int W = (int)split_words(vocab);
  const uint32_t vmax = (uint32_t)(vocab - 1);
  const double N = (double)num_blocks;
  const uint8_t* df = ws + b * seq_bytes + split_bits_bytes(num_blocks, vocab);
  const int4* seq4 = reinterpret_cast<const int4*>(ids + b * L + (int64_t)j * Lb);
  const int ngroups = Lb >> 2;  // 16-byte groups of the block (Lb is a multiple of 4)
  // Groups past the block re-read its last group: their lanes record no
  // chunk (Lb is a multiple of the chunk), and no load needs a branch.
  auto load = [&](int r, int4 (&q)[2]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) q[h] = seq4[min(2 * (r * kSplitThreads + tid) + h, ngroups - 1)];
  };
  int4 q[2];
  load(0, q);
  copy_to_lds(reinterpret_cast<const uint4*>(df), reinterpret_cast<uint4*>(lds), W, tid);
  if (tid <= num_blocks) {
    const double d = (double)tid;
    if (SCORER == PULSAR_SCORE_TFIDF) tab_df[tid] = log(N / fmax(d, 1.0));
    if (SCORER == PULSAR_SCORE_BM25) tab_df[tid] = log((N - d + 0.5) / (d + 0.5) + 1.0);
  }
  if (tid <= m && tid >= 1) {
    const double tf = (double)tid;
    const double D = 1.0 - kB + kB * (double)m / (double)m;  // every chunk has the mean length
    if (SCORER == PULSAR_SCORE_BM25) tab_tf[tid] = (kK1 + 1.0) / (tf + kK1 * D);
    if (SCORER == PULSAR_SCORE_ENTROPY) tab_tf[tid] = 1.0 / tf;
  }
  // the first ids arrive before the barrier, not after it
  asm volatile("" : "+v"(q[0].x), "+v"(q[0].y), "+v"(q[0].z), "+v"(q[0].w), "+v"(q[1].x),
               "+v"(q[1].y), "+v"(q[1].z), "+v"(q[1].w));
  __syncthreads();

  const int64_t nchunks_seq = L >> chunk_log2;
  int4* const stage = reinterpret_cast<int4*>(lds8 + stage_off) + wave * 128;  // 64 lanes x 2
  const int nrounds = (ngroups + 2 * kSplitThreads - 1) / (2 * kSplitThreads);
  for (int rd = 0; rd < nrounds; ++rd) {
    if (rd > 0) load(rd, q);
    const uint32_t t[8] = {min((uint32_t)q[0].x, vmax), min((uint32_t)q[0].y, vmax),
                           min((uint32_t)q[0].z, vmax), min((uint32_t)q[0].w, vmax),
                           min((uint32_t)q[1].x, vmax), min((uint32_t)q[1].y, vmax),
                           min((uint32_t)q[1].z, vmax), min((uint32_t)q[1].w, vmax)};
    uint32_t dfm1[8];  // df - 1
#pragma unroll
    for (int i = 0; i < 8; ++i) dfm1[i] = (lds8[t[i] >> 1] >> ((t[i] & 1u) << 2)) & 0xFu;
    uint32_t tf[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    const int g0 = 2 * (rd * kSplitThreads + tid);  // the lane's first group
    const int lg = chunk_log2 - 3;                 // log2 of the lanes per chunk (m >= 8)
    if constexpr (SCORER == PULSAR_SCORE_BM25 || SCORER == PULSAR_SCORE_ENTROPY) {
      if (chunk_log2 == 2) {
        // chunks of 4: each group against itself
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int k = 0; k < 4; ++k) tf[4 * h + i] += (uint32_t)(t[4 * h + k] == t[4 * h + i]);
      } else {
        stage[2 * lane] = make_int4((int)t[0], (int)t[1], (int)t[2], (int)t[3]);
        stage[2 * lane + 1] = make_int4((int)t[4], (int)t[5], (int)t[6], (int)t[7]);
        const int4* cs = stage + 2 * (lane & ~((1 << lg) - 1));  // the chunk's first lane
        for (int y = 0; y < (m >> 2); ++y) {
          const int4 z = cs[y];
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            tf[i] += (uint32_t)((uint32_t)z.x == t[i]);
            tf[i] += (uint32_t)((uint32_t)z.y == t[i]);
            tf[i] += (uint32_t)((uint32_t)z.z == t[i]);
            tf[i] += (uint32_t)((uint32_t)z.w == t[i]);
          }
        }
      }
      // the counts stay opaque until here, so that each comparison is one
      // compare and one add-with-carry
#pragma unroll
      for (int i = 0; i < 8; ++i) asm volatile("" : "+v"(tf[i]));
    }
    // the score and ranking key of the positions 4 h0 .. 4 h1 - 1 of the lane
    auto score_of = [&](int h0, int h1, double& s, uint32_t& mn) {
      s = 0.0;
      mn = 0xFFFFFFFFu;
#pragma unroll
      for (int i = 4 * h0; i < 4 * h1; ++i) {
        if (SCORER == PULSAR_SCORE_MAXIDF) mn = min(mn, dfm1[i]);
        if (SCORER == PULSAR_SCORE_TFIDF) s += tab_df[dfm1[i] + 1];
        if (SCORER == PULSAR_SCORE_BM25) s += tab_df[dfm1[i] + 1] * tab_tf[tf[i]];
        if (SCORER == PULSAR_SCORE_ENTROPY) s += tab_tf[tf[i]];
      }
    };
    auto finish = [&](double s, uint32_t mn, float& score, uint32_t& key) {
      if constexpr (SCORER == PULSAR_SCORE_MAXIDF) {
        key = mn + 1u;
        score = (float)log(N / (double)key);
      } else if constexpr (SCORER == PULSAR_SCORE_TFIDF) {
        score = (float)(s / (double)m);  // m a power of two: the division is exact
        key = ~__builtin_bit_cast(uint32_t, score);
      } else if constexpr (SCORER == PULSAR_SCORE_BM25) {
        score = (float)s;
        key = ~__builtin_bit_cast(uint32_t, score);
      } else {
        const int distinct = (int)rint(s);  // a sum of 1/tf over the chunk
        score = (float)distinct / (float)m;  // m a power of two: exact
        key = (uint32_t)(m - distinct);
      }
    };
    if (chunk_log2 == 2) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        double s;
        uint32_t mn, key;
        float score;
        score_of(h, h + 1, s, mn);
        finish(s, mn, score, key);
        if (g0 + h < ngroups) {
          keys[g0 + h] = key;
          if (scores) scores[b * nchunks_seq + (int64_t)j * C + g0 + h] = score;
        }
      }
    } else {
      double s;
      uint32_t mn, key;
      float score;
      score_of(0, 2, s, mn);
      if (SCORER == PULSAR_SCORE_MAXIDF) mn = group_min(mn, 1 << lg);
      else s = group_sum<-1>(s, 1 << lg);
      finish(s, mn, score, key);
      if (g0 < ngroups && (tid & ((1 << lg) - 1)) == 0) {
        const int c = g0 >> (lg + 1);
        keys[c] = key;
        if (scores) scores[b * nchunks_seq + (int64_t)j * C + c] = score;
      }
    }
  }
  __syncthreads();
  if (tid < 64 && topk > 0) {
    const uint32_t key_hi = SCORER == PULSAR_SCORE_MAXIDF   ? (uint32_t)num_blocks
                            : SCORER == PULSAR_SCORE_ENTROPY ? (uint32_t)m
                                                             : 0xFFFFFFFFu;
    int32_t* dst = sel + (b * num_blocks + j) * topk;
    if (C <= 4 * 64)
      select_block<4>(keys, C, key_hi, topk, dst, lane);
    else
      select_block<0>(keys, C, key_hi, topk, dst, lane);
  }
}

typedef void (*ScorerKernel)(const int32_t*, int64_t, int, int, int, int, int, int, int, int,
                             int32_t*, float*);

template <int SCORER>
ScorerKernel scorer_for_chunk(int chunk_log2) {
  if (chunk_log2 == 5) return scorer_kernel<SCORER, 3>;
  if (chunk_log2 == 4) return scorer_kernel<SCORER, 2>;
  return scorer_kernel<SCORER, -1>;
}

}  // namespace

size_t scorer_lds_bytes(int64_t L, int num_blocks, int chunk, int vocab, int scorer) {
  return (size_t)scorer_layout(L, num_blocks, chunk, vocab, scorer).bytes;
}

int launch_scorer(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk, int topk,
                  int vocab, int scorer, int32_t* sel, float* scores, hipStream_t stream) {
  if (batch == 0) return PULSAR_OK;
  int chunk_log2 = 0;
  while ((1 << chunk_log2) < chunk) ++chunk_log2;
  const ScorerLayout lay = scorer_layout(L, num_blocks, chunk, vocab, scorer);
  ScorerKernel kern = nullptr;
  switch (scorer) {
    case PULSAR_SCORE_MAXIDF: kern = scorer_for_chunk<PULSAR_SCORE_MAXIDF>(chunk_log2); break;
    case PULSAR_SCORE_TFIDF: kern = scorer_for_chunk<PULSAR_SCORE_TFIDF>(chunk_log2); break;
    case PULSAR_SCORE_BM25: kern = scorer_for_chunk<PULSAR_SCORE_BM25>(chunk_log2); break;
    case PULSAR_SCORE_ENTROPY: kern = scorer_for_chunk<PULSAR_SCORE_ENTROPY>(chunk_log2); break;
    default: return PULSAR_EINVAL;
  }
  if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lay.bytes) != hipSuccess)
    return PULSAR_EHIP;
  hipLaunchKernelGGL(kern, dim3(batch), dim3(MAXIDF_THREADS), (size_t)lay.bytes, stream, ids, L,
                     num_blocks, (int)(L / num_blocks), chunk_log2, topk, vocab,
                     (int)lay.key_off, (int)lay.tab_off, (int)lay.stage_off, sel, scores);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}

size_t scorer_split_lds_bytes(int64_t L, int num_blocks, int chunk, int vocab, int scorer) {
  return (size_t)split_score_layout(L, num_blocks, chunk, vocab, scorer).bytes;
}

int launch_scorer_split(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk,
                        int topk, int vocab, int scorer, int32_t* sel, float* scores,
                        void* workspace, hipStream_t stream) {
  if (batch == 0) return PULSAR_OK;
  int chunk_log2 = 0;
  while ((1 << chunk_log2) < chunk) ++chunk_log2;
  const SplitScoreLayout lay = split_score_layout(L, num_blocks, chunk, vocab, scorer);
  typedef void (*K)(const int32_t*, int64_t, int, int, int, int, int, const uint8_t*, int64_t, int,
                    int, int, int32_t*, float*);
  K kern = nullptr;
  switch (scorer) {
    case PULSAR_SCORE_MAXIDF: kern = split_score_kernel<PULSAR_SCORE_MAXIDF>; break;
    case PULSAR_SCORE_TFIDF: kern = split_score_kernel<PULSAR_SCORE_TFIDF>; break;
    case PULSAR_SCORE_BM25: kern = split_score_kernel<PULSAR_SCORE_BM25>; break;
    case PULSAR_SCORE_ENTROPY: kern = split_score_kernel<PULSAR_SCORE_ENTROPY>; break;
    default: return PULSAR_EINVAL;
  }
  int st = launch_split_df(ids, batch, L, num_blocks, vocab, nullptr, workspace, stream);
  if (st != PULSAR_OK) return st;
  if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lay.bytes) != hipSuccess)
    return PULSAR_EHIP;
  hipLaunchKernelGGL(kern, dim3((unsigned)((int64_t)batch * num_blocks)), dim3(kSplitThreads),
                     (size_t)lay.bytes, stream, ids, L, num_blocks, (int)(L / num_blocks),
                     chunk_log2, topk, vocab, static_cast<const uint8_t*>(workspace),
                     split_seq_bytes(num_blocks, vocab), (int)lay.key_off, (int)lay.tab_off,
                     (int)lay.stage_off, sel, scores);
  return hipGetLastError() == hipSuccess ? PULSAR_OK : PULSAR_EHIP;
}
