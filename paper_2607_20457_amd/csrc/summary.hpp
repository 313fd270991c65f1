// Device pieces shared by the chunk-summary kernels (Max-IDF and the other
// scorers): the stamp-code document frequency, lane-group reductions, and the
// top-k select in positional order (Algorithm 1, summary step; Appendix
// "Scoring Heuristic Details").
#pragma once

#include "common.hpp"

#define MAXIDF_THREADS 1024
#define MAXIDF_WAVES (MAXIDF_THREADS / PULSAR_WAVE)

// Stamp code: one byte per id, 16 * (15 - j) + (df - 1) after the id was
// last seen in block j with df blocks so far (1 <= df <= j + 1 <= 16), or
// kStampNever before it is first seen.  Once pass 1 is over the low nibble of
// every seen id is df - 1 (stamp_to_df).
constexpr int kStampMaxBlocks = 16;
// word 3 of a buffer resource for raw 32-bit-offset access
constexpr int kRawBuffer = 0x00020000;
constexpr uint32_t kStampNever = 0xFFu;

// Stamp code, block j: an id whose byte is not yet stamped with j gets the
// code of (df + 1, j).  With base = 16 * (15 - j), the codes stamped with j
// are base .. base + j (df - 1 <= j); the code of an id last seen in an
// earlier block, and kStampNever, lie above that range, and their low nibble
// plus one (mod 16) is the new df - 1.  All lanes that write one byte during
// block j write the same value, whatever order their loads and stores take,
// so the count is exact without atomics as long as no two blocks run at once
// (the caller puts a workgroup barrier between blocks).  PAD: the round holds
// -1 padding, which stamps nothing.  An id at or above vocab is clamped into
// the table (the caller's error).
template <int n, bool PAD>
__device__ __forceinline__ void stamp_tokens(const int (&t)[n], int j, uint32_t vmax,
                                             uint8_t* code) {
  uint32_t ts[n], c[n];
#pragma unroll
  for (int i = 0; i < n; ++i) ts[i] = min((uint32_t)t[i], vmax);
#pragma unroll
  for (int i = 0; i < n; ++i) c[i] = code[ts[i]];
  const uint32_t base = 16u * (15u - (uint32_t)j);
#pragma unroll
  for (int i = 0; i < n; ++i) {
    const bool stamped = c[i] - base <= (uint32_t)j;
    if (!stamped && (!PAD || t[i] >= 0)) code[ts[i]] = (uint8_t)(base | ((c[i] + 1u) & 15u));
  }
}

// After pass 1: every stamp code becomes df - 1 (its low nibble), four ids
// per word.  Only ids never seen (kStampNever) read as df 16; no id of the
// sequence is one of them.
// The table starts 16-byte aligned; 16 bytes per access, then the words past
// the last full 16 bytes.
__device__ __forceinline__ void stamp_to_df(uint32_t* codew, int vocab_w4, int tid) {
  uint4* c16 = reinterpret_cast<uint4*>(codew);
  const int n16 = vocab_w4 >> 2;
  for (int w = tid; w < n16; w += MAXIDF_THREADS) {
    uint4 x = c16[w];
    x.x &= 0x0F0F0F0Fu;
    x.y &= 0x0F0F0F0Fu;
    x.z &= 0x0F0F0F0Fu;
    x.w &= 0x0F0F0F0Fu;
    c16[w] = x;
  }
  for (int w = 4 * n16 + tid; w < vocab_w4; w += MAXIDF_THREADS) codew[w] &= 0x0F0F0F0Fu;
}

// df of a stamp code after pass 1 (0 for an id never seen)
__device__ __forceinline__ uint32_t stamp_df(uint32_t c) {
  return c == kStampNever ? 0u : (c & 15u) + 1u;
}

// Pass 1 of a streaming kernel with the stamp code: the blocks of one
// sequence (seq4: its ids as 16-byte groups) in order, a workgroup barrier
// before each block, two rounds of loads in flight.  The table (code, vocab
// bytes) must hold kStampNever for every id on entry; on return every thread
// has passed a final barrier and the table holds the final stamp codes
// (stamp_to_df turns them into df - 1).
__device__ __forceinline__ void stamp_pass_streaming(const int4* __restrict__ seq4,
                                                     int num_blocks, int Lb, uint32_t vmax,
                                                     uint8_t* code, int tid) {
  constexpr int ROUND = 2;
  constexpr int PREFETCH = 2;
  const int nvec = Lb >> 2;  // int4 groups per block
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
  int4 cbuf[PREFETCH + 1][ROUND];
#pragma unroll
  for (int i = 0; i < PREFETCH; ++i)
    if (i < rounds) load_round(i, cbuf[i]);
  for (int rd = 0; rd < rounds; ++rd) {
    if (rd % rpb == 0) __syncthreads();  // a new block: everyone is done with the previous one
    if (rd + PREFETCH < rounds) load_round(rd + PREFETCH, cbuf[PREFETCH]);
    int tk[4 * ROUND];
#pragma unroll
    for (int u = 0; u < ROUND; ++u) {
      tk[4 * u] = cbuf[0][u].x;
      tk[4 * u + 1] = cbuf[0][u].y;
      tk[4 * u + 2] = cbuf[0][u].z;
      tk[4 * u + 3] = cbuf[0][u].w;
    }
    if ((rd - (rd / rpb) * rpb + 1) * ROUND * MAXIDF_THREADS <= nvec)
      stamp_tokens<4 * ROUND, false>(tk, rd / rpb, vmax, code);
    else
      stamp_tokens<4 * ROUND, true>(tk, rd / rpb, vmax, code);
#pragma unroll
    for (int u = 0; u < ROUND; ++u) {
#pragma unroll
      for (int i = 0; i < PREFETCH; ++i) cbuf[i][u] = cbuf[i + 1][u];
    }
  }
  __syncthreads();
}

// x moved across lanes by a DPP control (quad permutes, row mirrors)
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}

// Minimum over aligned groups of 2^GL lanes, the group size a compile-time
// constant; every lane of a group ends with the group's minimum.
template <int GL>
__device__ __forceinline__ uint32_t group_min_c(uint32_t x) {
  if (GL >= 1) x = min(x, dpp_mov<0xB1>(x));   // lane ^ 1
  if (GL >= 2) x = min(x, dpp_mov<0x4E>(x));   // lane ^ 2
  if (GL >= 3) x = min(x, dpp_mov<0x141>(x));  // mirror within 8
  if (GL >= 4) x = min(x, dpp_mov<0x140>(x));  // mirror within 16
  if (GL >= 5) x = min(x, (uint32_t)__shfl_xor((int)x, 16, 64));
  if (GL >= 6) x = min(x, (uint32_t)__shfl_xor((int)x, 32, 64));
  return x;
}

// Minimum over aligned groups of `group` lanes (a power of two); DPP within
// rows of 16 lanes, cross-lane permutes beyond.
__device__ __forceinline__ uint32_t group_min(uint32_t x, int group) {
  if (group >= 2) x = min(x, dpp_mov<0xB1>(x));
  if (group >= 4) x = min(x, dpp_mov<0x4E>(x));
  if (group >= 8) x = min(x, dpp_mov<0x141>(x));
  if (group >= 16) x = min(x, dpp_mov<0x140>(x));
  if (group >= 32) x = min(x, (uint32_t)__shfl_xor((int)x, 16, 64));
  if (group >= 64) x = min(x, (uint32_t)__shfl_xor((int)x, 32, 64));
  return x;
}

// Lanes below this one with their bit set in a wave mask.
__device__ __forceinline__ int count_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

// Top-k chunks of one block from their keys cv[C] in LDS (smaller key =
// better chunk; every key <= key_hi), written in ascending chunk order to
// dst.  Slot i of lane l is chunk 64*i + l, so chunk order is (slot, lane)
// order and every count is a ballot.  The threshold tau is the smallest key
// with at least k chunks at or below it (binary search over 0..key_hi);
// every chunk below tau is kept, and the first k - #(< tau) chunks equal to
// tau in chunk order, which is the lowest-index tie-break.  S > 0: the block
// has at most S slots and their keys are held in registers; S == 0: any
// number of slots, read from LDS each time.
template <int S, typename KeyT>
__device__ __forceinline__ void select_block(const KeyT* cv, int C, uint32_t key_hi, int topk,
                                             int32_t* __restrict__ dst, int lane) {
  const int slots = (C + 63) >> 6;
  const int n_slots = S > 0 ? S : slots;
  constexpr int R = S > 0 ? S : 1;
  // With S > 0 a slot past the block's chunks holds the key 0xFFFFFFFF, so
  // the tests need no validity term.  A bisection midpoint is always below
  // key_hi, so such a slot never counts as at or below it, nor below tau.
  // Should tau itself be 0xFFFFFFFF, these slots are the highest chunk
  // indices: they rank after every real chunk equal to tau, of which there
  // are at least k - #(< tau), so none of them is kept.
  uint32_t xr[R];
#pragma unroll
  for (int i = 0; i < R; ++i)
    xr[i] = (S > 0 && i < slots && 64 * i + lane < C) ? (uint32_t)cv[64 * i + lane] : 0xFFFFFFFFu;
  // valid: the slot holds a chunk of the block; key: its key
#define SEL_VALID(i) (S > 0 || 64 * (i) + lane < C)
#define SEL_KEY(i) (S > 0 ? xr[S > 0 ? (i) : 0] : (uint32_t)cv[64 * (i) + lane])
  // each slot loop is straight-line code with S slots in registers, a plain
  // loop over the LDS keys otherwise
  auto for_slots = [&](auto&& f) {
    if constexpr (S > 0) {
#pragma unroll
      for (int i = 0; i < S; ++i) f(i);
    } else {
      for (int i = 0; i < n_slots; ++i) f(i);
    }
  };
  uint32_t lo = 0, hi = key_hi;  // #(key <= hi) >= k; tau in [lo, hi]
  while (lo < hi) {
    const uint32_t mid = lo + ((hi - lo) >> 1);
    int cnt = 0;
    for_slots([&](int i) { cnt += __popcll(__ballot(SEL_VALID(i) && SEL_KEY(i) <= mid)); });
    if (cnt >= topk) hi = mid; else lo = mid + 1;
  }
  const uint32_t tau = lo;
  int n_lt = 0;
  for_slots([&](int i) { n_lt += __popcll(__ballot(SEL_VALID(i) && SEL_KEY(i) < tau)); });
  const int need = topk - n_lt;  // kept chunks equal to tau
  int eq_before = 0, out_before = 0;
  for_slots([&](int i) {
    const bool valid = SEL_VALID(i);
    const uint32_t x = valid ? SEL_KEY(i) : 0u;
    const uint64_t m_eq = __ballot(valid && x == tau);
    const bool keep = valid && (x < tau || (x == tau && eq_before + count_below(m_eq) < need));
    const uint64_t m_keep = __ballot(keep);
    if (keep) dst[out_before + count_below(m_keep)] = 64 * i + lane;
    eq_before += __popcll(m_eq);
    out_before += __popcll(m_keep);
  });
#undef SEL_VALID
#undef SEL_KEY
}

// Top-k chunks of every block of sequence b from the chunk keys ([num_blocks]
// [C] in LDS, every key <= key_hi); one wavefront per block.
template <typename KeyT>
__device__ __forceinline__ void select_topk(const KeyT* keys, int64_t b, int num_blocks, int C,
                                            uint32_t key_hi, int topk,
                                            int32_t* __restrict__ sel, int wave, int lane) {
  if (topk == 0) return;
  // the block loop is uniform across the wavefront: keep it scalar
  for (int j = __builtin_amdgcn_readfirstlane(wave); j < num_blocks; j += MAXIDF_WAVES) {
    const KeyT* cv = keys + (int64_t)j * C;
    int32_t* dst = sel + (b * num_blocks + j) * topk;
    if (C <= 4 * 64)
      select_block<4>(cv, C, key_hi, topk, dst, lane);
    else
      select_block<0>(cv, C, key_hi, topk, dst, lane);
  }
}
