// C ABI entry points: host-side validation, then kernel launches.
#include <math.h>

#include <algorithm>
#include <mutex>

#include "common.hpp"

namespace {

constexpr int kVersion = 5;

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

// Shape checks shared by the Phase-1 calls (Eq. 3 row counts).
int64_t phase1_len_checked(int64_t L, int num_blocks, int block_idx, int sink, int chunk, int topk,
                           int prefix_mode) {
  if (L < 0 || num_blocks < 1 || L % num_blocks != 0) return PULSAR_EINVAL;
  if (block_idx < 0 || block_idx >= num_blocks) return PULSAR_EINVAL;
  if (prefix_mode != PULSAR_PREFIX_SUMMARY && prefix_mode != PULSAR_PREFIX_ANCHOR &&
      prefix_mode != PULSAR_PREFIX_EVEN)
    return PULSAR_EINVAL;
  const int64_t Lb = L / num_blocks;
  if (sink < 0 || sink > Lb) return PULSAR_EINVAL;
  if (chunk < 1 || topk < 0 || (int64_t)topk * chunk > Lb) return PULSAR_EINVAL;
  if (block_idx == 0) return Lb;
  if (prefix_mode == PULSAR_PREFIX_ANCHOR) return 2 * Lb;
  return Lb + sink + (int64_t)block_idx * topk * chunk;
}

RowMap make_map(int64_t L, int num_blocks, int block_idx, int sink, int chunk, int topk,
                int prefix_mode) {
  RowMap mp{};
  const int Lb = (int)(L / num_blocks);
  mp.block_idx = block_idx;
  mp.Lb = Lb;
  mp.sink = sink;
  mp.chunk = chunk;
  mp.topk = topk;
  mp.nchunk = Lb / chunk;
  mp.m_log2 = is_pow2(chunk) ? __builtin_ctz(chunk) : -1;
  mp.inv_chunk = 1.0f / (float)chunk;
  if (block_idx == 0) {
    mp.mode = MAP_IDENTITY;
    mp.offset = 0;
  } else if (prefix_mode == PULSAR_PREFIX_ANCHOR) {
    mp.mode = MAP_ANCHOR;
  } else if (prefix_mode == PULSAR_PREFIX_EVEN) {
    mp.mode = MAP_EVEN;
    mp.sigma = topk * chunk;
    mp.prefix = block_idx * mp.sigma;
    mp.inv_sigma = mp.sigma > 0 ? 1.0f / (float)mp.sigma : 0.f;
    mp.inv_sigma1 = mp.sigma > 1 ? 1.0 / (double)(mp.sigma - 1) : 0.0;
  } else {
    mp.mode = MAP_SUMMARY;
    mp.n_runs = block_idx * topk;
    mp.prefix = mp.n_runs * chunk;
  }
  return mp;
}

bool needs_sel(int block_idx, int topk, int prefix_mode) {
  return block_idx > 0 && topk > 0 && prefix_mode == PULSAR_PREFIX_SUMMARY;
}

bool heads_supported(int Hq, int Hkv) {
  const int group = Hq / Hkv;
  return group == 1 || group == 2 || group % 4 == 0;
}

}  // namespace

extern "C" {

const char* pulsar_status_string(int status) {
  switch (status) {
    case PULSAR_OK: return "ok";
    case PULSAR_EINVAL: return "invalid argument";
    case PULSAR_EUNSUPPORTED: return "unsupported configuration";
    case PULSAR_EHIP: return "HIP runtime error";
    case PULSAR_EWORKSPACE: return "workspace missing or too small";
    case PULSAR_ETOOLARGE: return "partials exceed the static scratch of the no-allocation call";
    default: return "unknown status";
  }
}

int pulsar_version(void) { return kVersion; }

size_t pulsar_maxidf_workspace_bytes(int batch, int64_t L, int num_blocks, int chunk, int vocab) {
  return maxidf_split_workspace(batch, L, num_blocks, chunk, vocab);
}

int pulsar_maxidf_summaries(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk,
                            int topk, int vocab, int32_t* sel_chunks, int32_t* chunk_mindf,
                            float* idf, void* workspace, size_t workspace_bytes, void* stream) {
  if (batch < 0 || L < 0 || num_blocks < 1 || vocab < 1 || chunk < 1 || topk < 0)
    return PULSAR_EINVAL;
  if (L % num_blocks != 0) return PULSAR_EINVAL;
  const int64_t Lb = L / num_blocks;
  if (Lb % chunk != 0 || topk > Lb / chunk) return PULSAR_EINVAL;
  if ((int64_t)batch * L > 0 && (ids == nullptr || !aligned16(ids))) return PULSAR_EINVAL;
  if ((int64_t)batch * num_blocks * topk > 0 && sel_chunks == nullptr) return PULSAR_EINVAL;
  if (num_blocks > 255 || !is_pow2(chunk) || chunk < 4 || chunk > 256) return PULSAR_EUNSUPPORTED;
  if (L >= ((int64_t)1 << 31)) return PULSAR_EUNSUPPORTED;
  if ((int64_t)batch * L == 0) {
    // no tokens: every df is 0, so IDF(t) = ln(N / 1) and there are no chunks
    if (batch == 0 || idf == nullptr) return PULSAR_OK;
    return launch_idf_fill(idf, (int64_t)batch * vocab, num_blocks, (hipStream_t)stream);
  }
  const size_t need = maxidf_split_workspace(batch, L, num_blocks, chunk, vocab);
  if (need > 0 && workspace != nullptr) {
    if (workspace_bytes < need || !aligned16(workspace)) return PULSAR_EWORKSPACE;
    return launch_maxidf_split(ids, batch, L, num_blocks, chunk, topk, vocab, sel_chunks,
                               chunk_mindf, idf, workspace, (hipStream_t)stream);
  }
  const size_t lds = maxidf_lds_bytes(L, num_blocks, chunk, vocab);
  if (lds > PULSAR_LDS_BYTES) return PULSAR_EUNSUPPORTED;
  return launch_maxidf(ids, batch, L, num_blocks, chunk, topk, vocab, sel_chunks, chunk_mindf, idf,
                       lds, (hipStream_t)stream);
}

size_t pulsar_chunk_workspace_bytes(int batch, int64_t L, int num_blocks, int chunk, int vocab,
                                    int scorer) {
  // 0 wherever pulsar_chunk_summaries would refuse the shapes
  if (scorer < PULSAR_SCORE_MAXIDF || scorer > PULSAR_SCORE_ENTROPY || num_blocks > 16 ||
      num_blocks < 1 || chunk < 4 || !is_pow2(chunk) || vocab < 1 || L < 1 ||
      scorer_lds_bytes(L, num_blocks, chunk, vocab, scorer) > PULSAR_LDS_BYTES)
    return 0;
  const size_t need = maxidf_split_workspace(batch, L, num_blocks, chunk, vocab);
  if (need == 0 || scorer_split_lds_bytes(L, num_blocks, chunk, vocab, scorer) > PULSAR_LDS_BYTES)
    return 0;
  return need;
}

int pulsar_chunk_summaries(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk,
                           int topk, int vocab, int scorer, int32_t* sel_chunks,
                           float* chunk_scores, void* workspace, size_t workspace_bytes,
                           void* stream) {
  if (batch < 0 || L < 0 || num_blocks < 1 || vocab < 1 || chunk < 1 || topk < 0)
    return PULSAR_EINVAL;
  if (scorer < PULSAR_SCORE_MAXIDF || scorer > PULSAR_SCORE_ENTROPY) return PULSAR_EINVAL;
  if (L % num_blocks != 0) return PULSAR_EINVAL;
  const int64_t Lb = L / num_blocks;
  if (Lb % chunk != 0 || topk > Lb / chunk) return PULSAR_EINVAL;
  if ((int64_t)batch * L > 0 && (ids == nullptr || !aligned16(ids))) return PULSAR_EINVAL;
  if ((int64_t)batch * num_blocks * topk > 0 && sel_chunks == nullptr) return PULSAR_EINVAL;
  if (num_blocks > 16 || !is_pow2(chunk) || chunk < 4 || chunk > 256) return PULSAR_EUNSUPPORTED;
  if (L >= ((int64_t)1 << 31)) return PULSAR_EUNSUPPORTED;
  if (scorer_lds_bytes(L, num_blocks, chunk, vocab, scorer) > PULSAR_LDS_BYTES)
    return PULSAR_EUNSUPPORTED;
  if ((int64_t)batch * L == 0) return PULSAR_OK;
  const size_t need = pulsar_chunk_workspace_bytes(batch, L, num_blocks, chunk, vocab, scorer);
  if (need > 0 && workspace != nullptr) {
    if (workspace_bytes < need || !aligned16(workspace)) return PULSAR_EWORKSPACE;
    return launch_scorer_split(ids, batch, L, num_blocks, chunk, topk, vocab, scorer, sel_chunks,
                               chunk_scores, workspace, (hipStream_t)stream);
  }
  return launch_scorer(ids, batch, L, num_blocks, chunk, topk, vocab, scorer, sel_chunks,
                       chunk_scores, (hipStream_t)stream);
}

int64_t pulsar_phase1_len(int64_t L, int num_blocks, int block_idx, int sink, int chunk, int topk,
                          int prefix_mode) {
  return phase1_len_checked(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode);
}

int pulsar_phase1_positions(const int32_t* sel_chunks, int batch, int64_t L, int num_blocks,
                            int block_idx, int sink, int chunk, int topk, int prefix_mode,
                            int32_t* pos, void* stream) {
  const int64_t n = phase1_len_checked(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode);
  if (n < 0) return (int)n;
  if (batch < 0 || L >= ((int64_t)1 << 31)) return PULSAR_EINVAL;
  if (n >= PULSAR_MAX_ROWS) return PULSAR_EUNSUPPORTED;
  if (batch == 0 || n == 0) return PULSAR_OK;
  if (pos == nullptr) return PULSAR_EINVAL;
  if (needs_sel(block_idx, topk, prefix_mode) && sel_chunks == nullptr) return PULSAR_EINVAL;
  const RowMap mp = make_map(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode);
  const int32_t* sel = needs_sel(block_idx, topk, prefix_mode) ? sel_chunks : nullptr;
  return launch_positions(mp, sel, (int64_t)num_blocks * topk, batch, (int)n, pos,
                          (hipStream_t)stream);
}

int pulsar_phase1_gather(const void* X, int batch, int64_t L, int H, int d, int num_blocks,
                         int block_idx, int sink, int chunk, int topk, const int32_t* sel_chunks,
                         int prefix_mode, int pos_mode, const float* inv_freq, double base,
                         void* X_out, void* stream) {
  const int64_t n = phase1_len_checked(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode);
  if (n < 0) return (int)n;
  if (batch < 0 || H < 1 || d < 1 || L >= ((int64_t)1 << 31)) return PULSAR_EINVAL;
  if (pos_mode != PULSAR_POS_SPARSE && pos_mode != PULSAR_POS_CONTIGUOUS &&
      pos_mode != PULSAR_POS_NONE)
    return PULSAR_EINVAL;
  if (d != 64 && d != 128) return d % 2 == 0 ? PULSAR_EUNSUPPORTED : PULSAR_EINVAL;
  if (n >= PULSAR_MAX_ROWS) return PULSAR_EUNSUPPORTED;
  if (batch == 0 || n == 0) return PULSAR_OK;
  if (X == nullptr || X_out == nullptr || !aligned16(X) || !aligned16(X_out)) return PULSAR_EINVAL;
  if (needs_sel(block_idx, topk, prefix_mode) && sel_chunks == nullptr) return PULSAR_EINVAL;
  const RowMap mp = make_map(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode);
  const int32_t* sel = needs_sel(block_idx, topk, prefix_mode) ? sel_chunks : nullptr;
  return launch_gather_rope(static_cast<const uint16_t*>(X), static_cast<uint16_t*>(X_out), batch,
                            (int)n, L, H, d, mp, sel, (int64_t)num_blocks * topk, pos_mode,
                            inv_freq, base, (hipStream_t)stream);
}

int pulsar_phase1_attn(const void* Q, const void* K, const void* V, int batch, int64_t L, int Hq,
                       int Hkv, int d, int num_blocks, int block_idx, int sink, int chunk,
                       int topk, const int32_t* sel_chunks, int prefix_mode, float softmax_scale,
                       void* O, int o_dtype, float* lse, void* K_keep, void* V_keep,
                       void* stream) {
  const int64_t n = phase1_len_checked(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode);
  if (n < 0) return (int)n;
  if (batch < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || d < 1) return PULSAR_EINVAL;
  if (L >= ((int64_t)1 << 31)) return PULSAR_EINVAL;
  if (!(softmax_scale > 0.f) || !isfinite(softmax_scale)) return PULSAR_EINVAL;
  if (o_dtype != PULSAR_OUT_F32 && o_dtype != PULSAR_OUT_BF16) return PULSAR_EINVAL;
  if ((K_keep == nullptr) != (V_keep == nullptr)) return PULSAR_EINVAL;
  if (d != 64 && d != 128) return PULSAR_EUNSUPPORTED;
  if (!heads_supported(Hq, Hkv)) return PULSAR_EUNSUPPORTED;
  if (n >= PULSAR_MAX_ROWS || L * Hkv * d * 2 >= ((int64_t)1 << 31)) return PULSAR_EUNSUPPORTED;
  if (batch == 0 || n == 0) return PULSAR_OK;
  if (Q == nullptr || K == nullptr || V == nullptr || O == nullptr) return PULSAR_EINVAL;
  if (needs_sel(block_idx, topk, prefix_mode) && sel_chunks == nullptr) return PULSAR_EINVAL;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O)) return PULSAR_EINVAL;
  if (K_keep != nullptr && (!aligned16(K_keep) || !aligned16(V_keep))) return PULSAR_EINVAL;

  AttnLaunch a{};
  a.Q = static_cast<const uint16_t*>(Q);
  a.K = static_cast<const uint16_t*>(K);
  a.V = static_cast<const uint16_t*>(V);
  a.q_zstride = L * Hq * d;
  a.kv_zstride = L * Hkv * d;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.d = d;
  a.n_q = (int)n;
  a.n_kv = (int)n;
  a.causal = 1;
  a.nsplit = 1;
  a.split_len = (int)n;
  a.nz_kv = batch;
  a.map = make_map(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode);
  a.sel = needs_sel(block_idx, topk, prefix_mode) ? sel_chunks : nullptr;
  a.sel_bstride = (int64_t)num_blocks * topk;
  a.scale_log2 = softmax_scale * 1.4426950408889634f;
  a.O = O;
  a.o_bf16 = o_dtype == PULSAR_OUT_BF16;
  a.o_zstride = n * Hq * d;
  a.lse = lse;
  a.lse_zstride = (int64_t)Hq * n;
  int st = launch_attention(a, (hipStream_t)stream);
  if (st != PULSAR_OK || K_keep == nullptr) return st;

  // KV(B_i): the last Lb rows of Input_i are block i's own tokens.
  const int64_t Lb = L / num_blocks;
  const int64_t row_bytes = Lb * Hkv * d * 2;
  const int64_t src_off = (int64_t)block_idx * Lb * Hkv * d;
  const int64_t pitch = L * Hkv * d * 2;
  st = launch_copy_rows(static_cast<const uint16_t*>(K) + src_off, pitch, K_keep, row_bytes,
                        row_bytes, batch, (hipStream_t)stream);
  if (st != PULSAR_OK) return st;
  return launch_copy_rows(static_cast<const uint16_t*>(V) + src_off, pitch, V_keep, row_bytes,
                          row_bytes, batch, (hipStream_t)stream);
}

}  // extern "C"

// Phase-2 key splitting: each shard is cut into nsplit ranges so that the
// launch has enough workgroups to cover the chip; the partials of a shard are
// then merged with the same online-softmax merge as the shards themselves.
static int phase2_splits(int n_shards, int Tq, int64_t S, int Hq, int Hkv, int d) {
  if (S <= 0) return 1;
  if (decode_applies(Tq, Hq, Hkv, d)) return decode_parts(n_shards, S, Hkv);
  const int group = Hq / Hkv;
  const int heads_per_wg = group >= 4 ? 4 : group;
  const int rows_per_wg = attn_rows_per_wg(group, false);
  const int64_t row_tiles = (Tq + rows_per_wg - 1) / rows_per_wg;
  const int64_t base = row_tiles * (group / heads_per_wg) * Hkv * n_shards;
  const int64_t target = 256;  // one round of 8-wavefront workgroups over 256 CUs
  int64_t ns = (target + base - 1) / base;
  const int64_t max_by_len = (S + 511) / 512;  // keep at least 512 keys per split
  if (ns > max_by_len) ns = max_by_len;
  if (ns < 1) ns = 1;
  if (ns > 64) ns = 64;
  return (int)ns;
}

extern "C" {

size_t pulsar_phase2_workspace_bytes(int n_shards, int Tq, int64_t S, int Hq, int Hkv, int d) {
  if (n_shards < 0 || Tq < 0 || S < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || d < 1) return 0;
  const int ns = phase2_splits(n_shards, Tq, S, Hq, Hkv, d);
  if (ns <= 1) return 0;
  const int64_t per = (int64_t)n_shards * ns;
  return (size_t)(per * Tq * Hq * d * 4 + per * Hq * Tq * 4);
}

int pulsar_phase2_partial(const void* q, const void* K, const void* V, int n_shards, int Tq,
                          int64_t S, int Hq, int Hkv, int d, float softmax_scale, float* o_parts,
                          float* lse_parts, void* workspace, size_t workspace_bytes,
                          void* stream) {
  if (n_shards < 0 || Tq < 0 || S < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || d < 1)
    return PULSAR_EINVAL;
  if (!(softmax_scale > 0.f) || !isfinite(softmax_scale)) return PULSAR_EINVAL;
  if (d != 64 && d != 128) return PULSAR_EUNSUPPORTED;
  if (!heads_supported(Hq, Hkv)) return PULSAR_EUNSUPPORTED;
  if (S >= ((int64_t)1 << 31) || S * Hkv * d * 2 >= ((int64_t)1 << 31) ||
      Tq >= PULSAR_MAX_ROWS)
    return PULSAR_EUNSUPPORTED;
  if (n_shards == 0 || Tq == 0) return PULSAR_OK;
  if (q == nullptr || o_parts == nullptr || lse_parts == nullptr) return PULSAR_EINVAL;
  if (S > 0 && (K == nullptr || V == nullptr)) return PULSAR_EINVAL;
  if (!aligned16(q) || (S > 0 && (!aligned16(K) || !aligned16(V))) || !aligned16(o_parts))
    return PULSAR_EINVAL;
  const int ns = phase2_splits(n_shards, Tq, S, Hq, Hkv, d);
  const size_t need = pulsar_phase2_workspace_bytes(n_shards, Tq, S, Hq, Hkv, d);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need || !aligned16(workspace)))
    return PULSAR_EWORKSPACE;

  float* ws_o = static_cast<float*>(workspace);
  float* ws_l = ws_o + (int64_t)n_shards * ns * Tq * Hq * d;
  if (decode_applies(Tq, Hq, Hkv, d)) {
    // few query rows: the decode kernel, one key range per wave
    int st = launch_decode(static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(K),
                           static_cast<const uint16_t*>(V), n_shards, Tq, S, Hq, Hkv, d,
                           softmax_scale, ns > 1 ? ws_o : o_parts, ns > 1 ? ws_l : lse_parts, ns,
                           (hipStream_t)stream);
    if (st != PULSAR_OK || ns == 1) return st;
    return launch_lse_merge(ws_o, ws_l, ns, n_shards, Tq, Hq, d, (int64_t)Tq * Hq * d,
                            (int64_t)Hq * Tq, o_parts, lse_parts, (hipStream_t)stream);
  }

  AttnLaunch a{};
  a.Q = static_cast<const uint16_t*>(q);
  a.K = static_cast<const uint16_t*>(K);
  a.V = static_cast<const uint16_t*>(V);
  a.q_zstride = 0;
  a.kv_zstride = S * Hkv * d;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.d = d;
  a.n_q = Tq;
  a.n_kv = (int)S;
  a.causal = 0;
  a.nsplit = ns;
  a.split_len = (int)((S + ns - 1) / ns);
  a.nz_kv = n_shards;
  a.map = RowMap{};
  a.map.mode = MAP_IDENTITY;
  a.sel = nullptr;
  a.scale_log2 = softmax_scale * 1.4426950408889634f;
  a.o_bf16 = 0;
  a.o_zstride = (int64_t)Tq * Hq * d;
  a.lse_zstride = (int64_t)Hq * Tq;
  a.O = ns > 1 ? ws_o : o_parts;
  a.lse = ns > 1 ? ws_l : lse_parts;
  int st = launch_attention(a, (hipStream_t)stream);
  if (st != PULSAR_OK || ns == 1) return st;
  return launch_lse_merge(ws_o, ws_l, ns, n_shards, Tq, Hq, d, (int64_t)Tq * Hq * d,
                          (int64_t)Hq * Tq, o_parts, lse_parts, (hipStream_t)stream);
}

int pulsar_lse_merge(const float* o_parts, const float* lse_parts, int H, int Tq, int Hq, int d,
                     float* o, float* lse, void* stream) {
  if (H < 1 || Tq < 0 || Hq < 0 || d < 1 || d % 4 != 0) return PULSAR_EINVAL;
  if ((int64_t)Tq * Hq == 0) return PULSAR_OK;
  if (o_parts == nullptr || lse_parts == nullptr || o == nullptr) return PULSAR_EINVAL;
  if (!aligned16(o_parts) || !aligned16(o)) return PULSAR_EINVAL;
  return launch_lse_merge(o_parts, lse_parts, H, 1, Tq, Hq, d, (int64_t)Tq * Hq * d,
                          (int64_t)Hq * Tq, o, lse, (hipStream_t)stream);
}

// Phase-2 attention of new tokens: partials of the shards, of the G earlier
// appended rows and of the new tokens' own rows (causal), then one merge.
// Workspace: the partials, o then lse, each 16-byte aligned.
namespace {
inline size_t align16(size_t x) { return (x + 15) & ~(size_t)15; }
// Partials of a Phase-2 query step; every key range is its own partial and
// one merge folds them all.  With the decode kernel (few query rows) one
// launch covers the ranges of every shard and of the generation shard (the
// G appended rows and the new tokens' own).  Otherwise the attention kernel
// gives the key splits of the shards.  A generation shard of at most
// kGenDecodeRows rows, for at most kGenDecodeQueryRows (token, head) rows
// per KV head, then goes to the decode kernel in 32-row tiles (each token
// limited to the rows up to its own; every tile reads the shard's K/V once,
// so this is kept to 16 tiles).  Otherwise the attention kernel takes it:
// key splits of the G appended rows, and one index-causal partial over the
// new tokens' own rows.
constexpr int64_t kGenDecodeRows = 4096;
constexpr int64_t kGenDecodeQueryRows = 512;
struct QueryPlan {
  bool decode;      // everything in one decode launch
  bool gen_decode;  // the generation shard in a decode launch
  int np_shard, np_gen;  // key ranges per shard / of the generation shard's rows
  int parts;
};
QueryPlan query_plan(int n_shards, int Tq, int64_t S, int64_t G, int Hq, int Hkv, int d) {
  QueryPlan p{};
  p.decode = decode_applies(Tq, Hq, Hkv, d);
  p.gen_decode = p.decode || ((d == 64 || d == 128) && Hq / Hkv <= 32 && G + Tq <= kGenDecodeRows &&
                               (int64_t)Tq * (Hq / Hkv) <= kGenDecodeQueryRows);
  if (p.decode) {
    p.np_shard = decode_parts(n_shards, S, Hkv);
  } else {
    p.np_shard = n_shards > 0 ? phase2_splits(n_shards, Tq, S, Hq, Hkv, d) : 0;
  }
  if (p.gen_decode) {
    p.np_gen = decode_parts(1, G + Tq, Hkv);
    p.parts = n_shards * p.np_shard + p.np_gen;
  } else {
    p.np_gen = G > 0 ? phase2_splits(1, Tq, G, Hq, Hkv, d) : 0;
    p.parts = n_shards * p.np_shard + p.np_gen + 1;
  }
  return p;
}

// Unmasked attention of the Tq queries over nz key sets of S rows each, every
// one cut into ns key splits; split s of set z writes partial z * ns + s.
int launch_split_parts(const void* q, const void* K, const void* V, int nz, int Tq, int64_t S,
                       int Hq, int Hkv, int d, float scale, int ns, float* po, float* pl,
                       hipStream_t stream) {
  AttnLaunch a{};
  a.Q = static_cast<const uint16_t*>(q);
  a.K = static_cast<const uint16_t*>(K);
  a.V = static_cast<const uint16_t*>(V);
  a.q_zstride = 0;
  a.kv_zstride = S * Hkv * d;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.d = d;
  a.n_q = Tq;
  a.n_kv = (int)S;
  a.causal = 0;
  a.nsplit = ns;
  a.split_len = (int)((S + ns - 1) / ns);
  a.nz_kv = nz;
  a.map = RowMap{};
  a.map.mode = MAP_IDENTITY;
  a.sel = nullptr;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.o_bf16 = 0;
  a.o_zstride = (int64_t)Tq * Hq * d;
  a.lse_zstride = (int64_t)Hq * Tq;
  a.O = po;
  a.lse = pl;
  return launch_attention(a, stream);
}
}  // namespace

size_t pulsar_phase2_query_workspace_bytes(int n_shards, int Tq, int64_t S, int64_t G, int Hq,
                                           int Hkv, int d) {
  if (n_shards < 0 || Tq < 0 || S < 0 || G < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || d < 1)
    return 0;
  const QueryPlan plan = query_plan(n_shards, Tq, S, G, Hq, Hkv, d);
  const size_t parts = (size_t)plan.parts;
  return align16(parts * Tq * Hq * d * 4) + align16(parts * Hq * Tq * 4);
}

}  // extern "C"

namespace {
// Host-side checks of a Phase-2 query step, everything but the workspace.
int phase2_query_check(const void* q, const void* Kg, const void* Vg, int64_t G, const void* K,
                       const void* V, int n_shards, int Tq, int64_t S, int Hq, int Hkv, int d,
                       float softmax_scale, const float* o) {
  if (n_shards < 0 || Tq < 0 || S < 0 || G < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || d < 1)
    return PULSAR_EINVAL;
  if (!(softmax_scale > 0.f) || !isfinite(softmax_scale)) return PULSAR_EINVAL;
  if (d != 64 && d != 128) return PULSAR_EUNSUPPORTED;
  if (!heads_supported(Hq, Hkv)) return PULSAR_EUNSUPPORTED;
  if (G + Tq >= PULSAR_MAX_ROWS || (G + Tq) * Hkv * d * 2 >= ((int64_t)1 << 31))
    return PULSAR_EUNSUPPORTED;
  if (S * Hkv * d * 2 >= ((int64_t)1 << 31) || Tq >= PULSAR_MAX_ROWS)
    return PULSAR_EUNSUPPORTED;  // byte offsets within a shard must fit 32 bits
  if (Tq == 0) return PULSAR_OK;
  if (q == nullptr || Kg == nullptr || Vg == nullptr || o == nullptr) return PULSAR_EINVAL;
  if (n_shards > 0 && S > 0 && (K == nullptr || V == nullptr)) return PULSAR_EINVAL;
  if (!aligned16(q) || !aligned16(Kg) || !aligned16(Vg) || !aligned16(o)) return PULSAR_EINVAL;
  return PULSAR_OK;
}

// The no-allocation variant's partials: one array per device, for the life
// of the process.  In host code `scratch` names a host-side stand-in; the
// device address comes from hipGetSymbolAddress, once per device, and only
// that address is ever handed to a kernel.
__device__ __align__(256) uint8_t scratch[PULSAR_STATIC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices];  // device address of `scratch`, per device

int scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return PULSAR_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return PULSAR_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return PULSAR_EHIP;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return PULSAR_OK;
}
}  // namespace

extern "C" {

int pulsar_phase2_query(const void* q, const void* Kg, const void* Vg, int64_t G, const void* K,
                        const void* V, int n_shards, int Tq, int64_t S, int Hq, int Hkv, int d,
                        float softmax_scale, float* o, float* lse, void* workspace,
                        size_t workspace_bytes, void* stream) {
  const int chk = phase2_query_check(q, Kg, Vg, G, K, V, n_shards, Tq, S, Hq, Hkv, d,
                                     softmax_scale, o);
  if (chk != PULSAR_OK || Tq == 0) return chk;
  const size_t need = pulsar_phase2_query_workspace_bytes(n_shards, Tq, S, G, Hq, Hkv, d);
  if (workspace == nullptr || workspace_bytes < need || !aligned16(workspace))
    return PULSAR_EWORKSPACE;

  const QueryPlan plan = query_plan(n_shards, Tq, S, G, Hq, Hkv, d);
  const int parts = plan.parts;
  const int64_t ostride = (int64_t)Tq * Hq * d, lstride = (int64_t)Hq * Tq;
  float* po = static_cast<float*>(workspace);
  float* pl = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                       align16((size_t)parts * ostride * 4));
  int part = 0, st = PULSAR_OK;
  if (plan.decode) {
    // every key range its own partial, the shards' and then the generation
    // shard's, in one launch; then one merge
    const DecodeGen gen{static_cast<const uint16_t*>(Kg), static_cast<const uint16_t*>(Vg), G,
                        plan.np_gen};
    st = launch_decode(static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(K),
                       static_cast<const uint16_t*>(V), n_shards, Tq, S, Hq, Hkv, d,
                       softmax_scale, po, pl, plan.np_shard, (hipStream_t)stream, &gen);
    if (st != PULSAR_OK) return st;
    return launch_lse_merge(po, pl, parts, 1, Tq, Hq, d, ostride, lstride, o, lse,
                            (hipStream_t)stream);
  }
  if (n_shards > 0) {  // the shards' key splits
    st = launch_split_parts(q, K, V, n_shards, Tq, S, Hq, Hkv, d, softmax_scale, plan.np_shard,
                            po, pl, (hipStream_t)stream);
    if (st != PULSAR_OK) return st;
    part = n_shards * plan.np_shard;
  }
  if (plan.gen_decode) {  // the generation shard's rows, each token up to its own
    const DecodeGen gen{static_cast<const uint16_t*>(Kg), static_cast<const uint16_t*>(Vg), G,
                        plan.np_gen};
    st = launch_decode(static_cast<const uint16_t*>(q), nullptr, nullptr, 0, Tq, 0, Hq, Hkv, d,
                       softmax_scale, po + part * ostride, pl + part * lstride, 1,
                       (hipStream_t)stream, &gen);
    if (st != PULSAR_OK) return st;
    return launch_lse_merge(po, pl, parts, 1, Tq, Hq, d, ostride, lstride, o, lse,
                            (hipStream_t)stream);
  }
  if (G > 0) {  // the earlier appended rows, all visible, in key splits
    st = launch_split_parts(q, Kg, Vg, 1, Tq, G, Hq, Hkv, d, softmax_scale, plan.np_gen,
                            po + part * ostride, pl + part * lstride, (hipStream_t)stream);
    if (st != PULSAR_OK) return st;
    part += plan.np_gen;
  }
  // the new tokens' own rows: index-causal, square
  const int64_t row = (int64_t)Hkv * d;
  AttnLaunch a{};
  a.Q = static_cast<const uint16_t*>(q);
  a.K = static_cast<const uint16_t*>(Kg) + G * row;
  a.V = static_cast<const uint16_t*>(Vg) + G * row;
  a.q_zstride = 0;
  a.kv_zstride = Tq * row;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.d = d;
  a.n_q = Tq;
  a.n_kv = Tq;
  a.causal = 1;
  a.nsplit = 1;
  a.split_len = Tq;
  a.nz_kv = 1;
  a.map = RowMap{};
  a.map.mode = MAP_IDENTITY;
  a.sel = nullptr;
  a.scale_log2 = softmax_scale * 1.4426950408889634f;
  a.O = po + part * ostride;
  a.o_bf16 = 0;
  a.o_zstride = ostride;
  a.lse = pl + part * lstride;
  a.lse_zstride = lstride;
  st = launch_attention(a, (hipStream_t)stream);
  if (st != PULSAR_OK) return st;
  return launch_lse_merge(po, pl, parts, 1, Tq, Hq, d, ostride, lstride, o, lse,
                          (hipStream_t)stream);
}

int pulsar_phase2_query_noalloc(const void* q, const void* Kg, const void* Vg, int64_t G,
                                const void* K, const void* V, int n_shards, int Tq, int64_t S,
                                int Hq, int Hkv, int d, float softmax_scale, float* o, float* lse,
                                void* stream) {
  const int chk = phase2_query_check(q, Kg, Vg, G, K, V, n_shards, Tq, S, Hq, Hkv, d,
                                     softmax_scale, o);
  if (chk != PULSAR_OK || Tq == 0) return chk;
  const size_t need = pulsar_phase2_query_workspace_bytes(n_shards, Tq, S, G, Hq, Hkv, d);
  if (need > (size_t)PULSAR_STATIC_SCRATCH_BYTES) return PULSAR_ETOOLARGE;
  void* ws = nullptr;
  const int st = scratch_of_current_device(&ws);
  if (st != PULSAR_OK) return st;
  return pulsar_phase2_query(q, Kg, Vg, G, K, V, n_shards, Tq, S, Hq, Hkv, d, softmax_scale, o,
                             lse, ws, (size_t)PULSAR_STATIC_SCRATCH_BYTES, stream);
}

}  // extern "C"
