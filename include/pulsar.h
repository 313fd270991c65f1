/*
 * pulsar.h -- C ABI of the MI355X (gfx950) library for Pulsar Attention's
 * Phase-1 statistical context encoding and Phase-2 query attention.
 *
 * Paper: "Dropping the Anchor: Statistical Context Summarization for
 * Distributed Systems via Pulsar Attention" (arXiv 2607.20457).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every pointer argument is a device pointer (memory from hipMalloc or a
 *   PyTorch CUDA/HIP tensor) unless stated otherwise.  The caller owns all
 *   buffers; the library allocates no device memory.
 * - `stream` is a hipStream_t passed as void*; NULL is the default stream.
 *   Every call is asynchronous on that stream.  The return value reports
 *   host-side argument validation and launch errors only; a fault during
 *   execution surfaces at the caller's next synchronisation.
 * - Tensors are dense and row-major.  Per-token tensors are laid out
 *   [batch, tokens, heads, head_dim].  Element offsets are computed in 64 bits.
 * - bf16 tensors are passed as raw 16-bit storage (IEEE bfloat16).
 * - Return codes are pulsar_status values; 0 is success.
 * - The library keeps no mutable global state, apart from the static scratch
 *   of pulsar_phase2_query_noalloc (see there) and the work counters of the
 *   causal attention launches (pulsar_phase1_attn): a slot of 128 bytes per
 *   (device, stream) for the first 64 streams of a device, in static device
 *   memory, zero between launches.  Launches on one stream never overlap;
 *   launches on other streams use other slots, and a launch captured into a
 *   graph, or on a stream beyond the slots, uses none (one workgroup per row
 *   tile).  Calls on different streams may run concurrently as long as their
 *   output buffers do not overlap.  A slot belongs to the stream handle: let
 *   a stream's pulsar_phase1_attn launches finish (hipStreamSynchronize)
 *   before destroying it, since a stream created later may get the same
 *   handle and with it the slot.
 */
#ifndef PULSAR_H_
#define PULSAR_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PULSAR_OK = 0,
  PULSAR_EINVAL = -1,        /* an argument is out of range or a required pointer is NULL */
  PULSAR_EUNSUPPORTED = -2,  /* valid by the paper's definition but outside what this library runs */
  PULSAR_EHIP = -3,          /* the HIP runtime reported an error at launch */
  PULSAR_EWORKSPACE = -4,    /* the workspace is NULL or smaller than the size query returned */
  PULSAR_ETOOLARGE = -5      /* the no-allocation call's partials exceed its static scratch */
} pulsar_status;

typedef enum {
  /* Input_i = [S_sink || Sigma_0 || ... || Sigma_{i-1} || B_i] (Eq. 3) */
  PULSAR_PREFIX_SUMMARY = 0,
  /* Star Attention anchor baseline: Input_i = [B_0 || B_i] (Section 2) */
  PULSAR_PREFIX_ANCHOR = 1,
  /* Even-Spaced baseline (Appendix "Even-Spaced"): Eq. 3 with Sigma_j the
     sigma = topk * chunk positions j*Lb + floor(r (Lb - 1) / (sigma - 1)),
     r = 0 .. sigma - 1 (position j*Lb alone when sigma = 1); no sel_chunks */
  PULSAR_PREFIX_EVEN = 2
} pulsar_prefix_mode;

typedef enum { PULSAR_OUT_F32 = 0, PULSAR_OUT_BF16 = 1 } pulsar_out_dtype;

/* Rotary position ids of an assembled Phase-1 input (Appendix "RoPE Position
   ID Assignment"). */
typedef enum {
  PULSAR_POS_SPARSE = 0,      /* every row keeps its global position (the paper's default) */
  PULSAR_POS_CONTIGUOUS = 1,  /* block i's input renumbered 0 .. n_i - 1 */
  PULSAR_POS_NONE = 2         /* no rotation (values) */
} pulsar_pos_mode;

/* Chunk scorers (Appendix "Scoring Heuristic Details"). */
typedef enum {
  PULSAR_SCORE_MAXIDF = 0,  /* max over the chunk of IDF (Eq. maxidf) */
  PULSAR_SCORE_TFIDF = 1,   /* mean over the chunk of IDF (Eq. tfidf) */
  PULSAR_SCORE_BM25 = 2,    /* BM25 with k1 = 1.2, b = 0.75 (Eq. bm25) */
  PULSAR_SCORE_ENTROPY = 3  /* distinct tokens / chunk length (Eq. entropy) */
} pulsar_scorer;

/* Human-readable name of a status code (static storage; never NULL). */
const char* pulsar_status_string(int status);

/* Library ABI version (increases on any signature change). */
int pulsar_version(void);

/*
 * Max-IDF summaries (Section 3.1 "Summary generation", Eq. 2; Appendix
 * "Corpus-Level IDF Table", Eq. idf, and "Max-IDF", Eq. maxidf; the summary
 * step of Algorithm 1).
 *
 * For each of `batch` sequences of `L` token ids, split into `num_blocks`
 * contiguous blocks of Lb = L / num_blocks tokens:
 *   df(t)   = number of blocks of that sequence containing t;
 *   IDF(t)  = ln(num_blocks / max(df(t), 1));
 *   each block is cut into Lb / chunk non-overlapping chunks of `chunk`
 *   tokens; a chunk's score is the largest IDF among its tokens;
 *   the `topk` best chunks of each block (best = higher score, then lower
 *   chunk index) are written in ascending chunk-index order.
 * Ranking uses the per-chunk minimum df, which orders chunks exactly as the
 * maximum IDF does because the logarithm is strictly decreasing.
 *
 * ids         int32 [batch, L], each in [0, vocab); 16-byte aligned.
 *             Ids outside that range are the caller's error: the kernel
 *             never reads or writes outside its tables because of them, and
 *             the result is unspecified.
 * sel_chunks  out int32 [batch, num_blocks, topk], chunk indices within the
 *             block, ascending.
 * chunk_mindf out int32 [batch, num_blocks, Lb / chunk], nullable: the
 *             minimum df of each chunk (IDF of the chunk score = ln(N/mindf)).
 * idf         out float [batch, vocab], nullable: IDF(t) for every id.
 * A context of no tokens (L == 0, so topk must be 0) has no chunks: nothing
 * is read and only idf, when given, is written (ln(num_blocks) everywhere).
 * workspace   device buffer of at least pulsar_maxidf_workspace_bytes(...)
 *             bytes, 16-byte aligned, contents on entry irrelevant; or NULL.
 *             With it, a small batch runs in three launches split over the
 *             blocks and the vocabulary; with NULL (or a size query of 0) one
 *             workgroup takes each sequence.  The results are identical.
 * EWORKSPACE: a workspace smaller than the size query or misaligned.
 *
 * EINVAL: batch < 0, L < 0, num_blocks < 1, L % num_blocks != 0,
 *         Lb % chunk != 0, chunk < 1, topk < 0 or topk > Lb / chunk,
 *         vocab < 1, a NULL ids/sel_chunks pointer when batch*L > 0 (resp.
 *         batch*num_blocks*topk > 0), misaligned ids.
 * EUNSUPPORTED: num_blocks > 255, chunk not a power of two in [4, 256],
 *         or vocab/L/chunk such that the per-sequence df table and chunk
 *         scores do not fit in one compute unit's 160 KB local data share
 *         (vocab up to about 145,000 at chunk 32 and L = 128K).
 */
int pulsar_maxidf_summaries(const int32_t* ids, int batch, int64_t L, int num_blocks,
                            int chunk, int topk, int vocab, int32_t* sel_chunks,
                            int32_t* chunk_mindf, float* idf, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * Device workspace, in bytes, with which pulsar_maxidf_summaries spreads a
 * small batch (up to 16 sequences, 2..255 blocks, vocab up to 1310720, at
 * most 16384 chunks per block) over many compute units: per sequence one
 * presence bitmap of ceil(vocab / 32) words per block and a df table of
 * 32 ceil(vocab / 32) bytes (a byte per id, or a nibble per id when
 * num_blocks <= 16).  0 when the shapes take the one-workgroup-per-sequence
 * kernels.  Host-only.
 */
size_t pulsar_maxidf_workspace_bytes(int batch, int64_t L, int num_blocks, int chunk, int vocab);

/*
 * Chunk summaries under any of the four scorers (Appendix "Scoring Heuristic
 * Details": Corpus-Level IDF Table, TF-IDF, BM25, Entropy, Max-IDF).
 *
 * Blocks, df, IDF and chunks as for pulsar_maxidf_summaries.  For a chunk C
 * of m tokens (tf(t) = occurrences of t in C):
 *   MAXIDF   max over C of IDF(t);
 *   TFIDF    (1/m) * sum over the positions of C of IDF(t);
 *   BM25     sum over the distinct t of C of IDF_BM25(t) tf(t) (k1 + 1) /
 *            (tf(t) + k1 D), IDF_BM25(t) = ln((N - df(t) + 0.5) /
 *            (df(t) + 0.5) + 1), k1 = 1.2, b = 0.75, D = 1 - b + b m /
 *            l_bar = 1 (all chunks have the mean length l_bar = m);
 *   ENTROPY  (number of distinct tokens of C) / m.
 * A score is computed in fp64 and rounded once to fp32, as the paper scores
 * from an fp32 IDF table; the `topk` best chunks of each block (higher fp32
 * score, then lower chunk index) are written in ascending chunk order.
 * The chunk's tf comes from comparing each position with the whole chunk, so
 * BM25 and ENTROPY cost O(m) per token.
 *
 * ids, sel_chunks  as for pulsar_maxidf_summaries.
 * chunk_scores     out float [batch, num_blocks, Lb / chunk], nullable.
 * scorer           a pulsar_scorer.
 * workspace        device buffer of at least pulsar_chunk_workspace_bytes(...)
 *                  bytes, 16-byte aligned, contents on entry irrelevant; or
 *                  NULL.  With it, a small batch runs split over the blocks
 *                  and the vocabulary (the Max-IDF split path's presence and
 *                  df launches, then one workgroup per block); with NULL (or
 *                  a size query of 0) one workgroup takes each sequence.  The
 *                  scores agree bit for bit except where an fp64 sum taken
 *                  in another order rounds to the other side of an fp32
 *                  midpoint (one ulp), and the selections follow the scores.
 *
 * EINVAL: as for pulsar_maxidf_summaries, or an unknown scorer.
 * EUNSUPPORTED: num_blocks > 16, chunk not a power of two in [4, 256], or
 *         the df table, chunk keys and (BM25, ENTROPY) a 16 KB staging area
 *         do not fit in 160 KB of local data share (vocab up to about
 *         130,000 at chunk 32 and L = 128K for BM25 and ENTROPY).
 * EWORKSPACE: a workspace smaller than the size query or misaligned.
 */
int pulsar_chunk_summaries(const int32_t* ids, int batch, int64_t L, int num_blocks, int chunk,
                           int topk, int vocab, int scorer, int32_t* sel_chunks,
                           float* chunk_scores, void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * Device workspace, in bytes, with which pulsar_chunk_summaries spreads a
 * small batch over many compute units (the layout of
 * pulsar_maxidf_workspace_bytes, for shapes whose score workgroup also fits
 * its df table, chunk keys and staging in local data share); 0 when the
 * shapes take one workgroup per sequence.  Host-only.
 */
size_t pulsar_chunk_workspace_bytes(int batch, int64_t L, int num_blocks, int chunk, int vocab,
                                    int scorer);

/*
 * Number of rows n_i of block i's Phase-1 input (Eq. 3; Appendix
 * "Block-to-Host Scalability Analysis"):
 *   block 0: Lb;  summary and Even-Spaced modes: Lb + sink + block_idx *
 *   topk * chunk;  anchor mode (block_idx > 0): 2 * Lb.
 * Returns n_i >= 0, or a negative pulsar_status on invalid arguments
 * (L % num_blocks != 0, block_idx outside [0, num_blocks), sink > Lb,
 * topk * chunk > Lb, negative sizes, unknown mode).  Host-only; no GPU call.
 */
int64_t pulsar_phase1_len(int64_t L, int num_blocks, int block_idx, int sink, int chunk,
                          int topk, int prefix_mode);

/*
 * Row -> global position map of block i's Phase-1 input (Eq. 3 with sparse
 * position ids, Section 3.1 "Causal Assembly"; Appendix "RoPE Position ID
 * Assignment").  Rows [0, sink) are positions 0..sink-1; then for every
 * earlier block j < i and every selected chunk c of Sigma_j (in the order of
 * sel_chunks) the m positions j*Lb + c*m + r; then block i's own positions
 * i*Lb + r.  Block 0 is [B_0] alone; anchor mode is [B_0 || B_i]; the
 * Even-Spaced mode replaces each Sigma_j by its sigma = topk * chunk evenly
 * spaced positions (see PULSAR_PREFIX_EVEN).
 *
 * sel_chunks  int32 [batch, num_blocks, topk] (as written by
 *             pulsar_maxidf_summaries or pulsar_chunk_summaries); only
 *             blocks < block_idx are read; may be NULL in the anchor and
 *             Even-Spaced modes, when block_idx == 0 or topk == 0.
 *             Chunk indices must lie in [0, Lb / chunk).
 * pos         out int32 [batch, n_i].
 * Errors: as pulsar_phase1_len, plus EINVAL for NULL pointers, batch < 0,
 *         or L >= 2^31.
 */
int pulsar_phase1_positions(const int32_t* sel_chunks, int batch, int64_t L, int num_blocks,
                            int block_idx, int sink, int chunk, int topk, int prefix_mode,
                            int32_t* pos, void* stream);

/*
 * Block i's assembled Phase-1 input materialised with rotary position
 * embedding (Eq. 3; Appendix "RoPE Position ID Assignment").
 *
 * Row r of X_out is the row of X at the global position of assembled row r
 * (the map of pulsar_phase1_positions), rotated in the rotate-half form of
 * pulsar_rope by
 *   PULSAR_POS_SPARSE      its global position (the same rows as rotating X
 *                          once with pulsar_rope and gathering),
 *   PULSAR_POS_CONTIGUOUS  r: the input renumbered 0 .. n_i - 1,
 *   PULSAR_POS_NONE        nothing (a plain gather, for V).
 * Contiguous mode changes a row's rotation with the block whose input it
 * enters, so each block's Q and K are materialised this way; attention over
 * them is pulsar_phase1_attn on X_out with num_blocks = 1, block_idx = 0 and
 * L = n_i (the identity map), whose last Lb rows of K/V are the retained
 * KV(B_i).  Phase-2 tokens then take positions from max_i n_i on
 * (pulsar_rope with pos = NULL and pos_offset = max_i n_i + the number of
 * earlier Phase-2 tokens).
 *
 * X         bf16 [batch, L, H, d], 16-byte aligned, not modified.
 * sel_chunks as for pulsar_phase1_positions.
 * inv_freq  HOST pointer to d/2 frequencies, or NULL for base^(-2i/d)
 *           (ignored with PULSAR_POS_NONE).
 * X_out     out bf16 [batch, n_i, H, d], 16-byte aligned.
 * EINVAL: as pulsar_phase1_len, batch < 0, H < 1, unknown pos_mode, NULL or
 *         misaligned X / X_out when there is work, NULL sel_chunks when
 *         needed, odd d, a non-finite table entry or base, L >= 2^31.
 * EUNSUPPORTED: d not in {64, 128}; n_i >= 2^24.
 */
int pulsar_phase1_gather(const void* X, int batch, int64_t L, int H, int d, int num_blocks,
                         int block_idx, int sink, int chunk, int topk, const int32_t* sel_chunks,
                         int prefix_mode, int pos_mode, const float* inv_freq, double base,
                         void* X_out, void* stream);

/*
 * Phase-1 prefixed-block causal attention (Algorithm 1, forward pass of
 * Input_i; Eq. 1 with an index-causal mask over the assembled rows; KV
 * discard per Appendix "KV Cache Discard").
 *
 * Every row r of Input_i (n_i rows, order of Eq. 3, see
 * pulsar_phase1_positions) is a query row and attends to rows 0..r of
 * Input_i.  The query/key/value of a row are those of the token at its
 * global position; the assembly is fused into the kernel's loads and never
 * materialised.  Query head h reads KV head h / (Hq / Hkv).
 *
 * Q           bf16 [batch, L, Hq, d];  K, V  bf16 [batch, L, Hkv, d].
 * sel_chunks  int32 [batch, num_blocks, topk]; nullable as for
 *             pulsar_phase1_positions.
 * softmax_scale  multiplies q.k (the paper's 1/sqrt(d)).
 * O           out [batch, n_i, Hq, d], float32 or bf16 per o_dtype.
 * lse         out float32 [batch, Hq, n_i], nullable: ln sum_c exp(s_rc).
 * K_keep, V_keep  out bf16 [batch, Lb, Hkv, d], nullable (both or none):
 *             the retained KV(B_i) rows, i.e. the last Lb rows of Input_i.
 *
 * EINVAL: shape/size errors as pulsar_phase1_len, batch < 0, Hq % Hkv != 0,
 *         NULL Q/K/V/O, softmax_scale not finite and > 0, only one of
 *         K_keep/V_keep given, L >= 2^31.
 * EUNSUPPORTED: d not in {64, 128}; Hq / Hkv not 1, 2 or a multiple of 4.
 */
int pulsar_phase1_attn(const void* Q, const void* K, const void* V, int batch, int64_t L,
                       int Hq, int Hkv, int d, int num_blocks, int block_idx, int sink,
                       int chunk, int topk, const int32_t* sel_chunks, int prefix_mode,
                       float softmax_scale, void* O, int o_dtype, float* lse, void* K_keep,
                       void* V_keep, void* stream);

/*
 * Device workspace, in bytes, that pulsar_phase2_partial needs for these
 * shapes (0 when none is needed).  Host-only.
 */
size_t pulsar_phase2_workspace_bytes(int n_shards, int Tq, int64_t S, int Hq, int Hkv, int d);

/*
 * Phase-2 per-shard partial attention (Algorithm 1, Phase 2:
 * (A_h, l_h) <- FlashAttn(q, KV_h) for every host h; Appendix "Phase 2
 * Distributed Softmax Merge").  One launch computes all n_shards shards, in
 * place of n_shards hosts.
 *
 * For each shard h: o_h = softmax(q K_h^T * scale) V_h and
 * l_h = ln sum_c exp(q . k_c * scale), with no mask.
 *
 * q           bf16 [Tq, Hq, d].
 * K, V        bf16 [n_shards, S, Hkv, d] (shard h is rows [h*S, (h+1)*S)).
 * o_parts     out float32 [n_shards, Tq, Hq, d].
 * lse_parts   out float32 [n_shards, Hq, Tq].
 * workspace   device buffer of at least pulsar_phase2_workspace_bytes(...)
 *             bytes (may be NULL when that is 0).  Its contents on entry
 *             do not matter.
 * An empty shard (S == 0) gives lse = -inf and o = 0.
 *
 * EINVAL: negative sizes, Hq % Hkv != 0, NULL required pointers, scale not
 *         finite and > 0.  EWORKSPACE: workspace too small.
 * EUNSUPPORTED: d not in {64, 128}; Hq / Hkv not 1, 2 or a multiple of 4.
 */
int pulsar_phase2_partial(const void* q, const void* K, const void* V, int n_shards, int Tq,
                          int64_t S, int Hq, int Hkv, int d, float softmax_scale,
                          float* o_parts, float* lse_parts, void* workspace,
                          size_t workspace_bytes, void* stream);

/*
 * Online-softmax merge of H partials (Algorithm 1, Phase 2 merge; Appendix
 * "Phase 2 Distributed Softmax Merge", Eqs. lse-merge and out-merge).
 * Produces l = ln sum_h exp(l_h) and o = sum_h exp(l_h - l) o_h, which is
 * what folding Eq. lse-merge / Eq. out-merge over h gives in exact
 * arithmetic; partials with l_h = -inf contribute nothing, and if every
 * l_h is -inf the result is l = -inf, o = 0.
 *
 * o_parts     float32 [H, Tq, Hq, d];  lse_parts float32 [H, Hq, Tq].
 * o           out float32 [Tq, Hq, d]; lse out float32 [Hq, Tq] (nullable).
 * EINVAL: H < 1, negative sizes, NULL required pointers, d % 4 != 0.
 */
int pulsar_lse_merge(const float* o_parts, const float* lse_parts, int H, int Tq, int Hq,
                     int d, float* o, float* lse, void* stream);

/*
 * Phase-2 attention of new tokens (Algorithm 1, Phase 2: the query encoding
 * and every generation step).  Every query and generated token's KV is
 * appended to one designated generation shard; a new token attends, without
 * a mask, to all retained shards (KV_h after Phase 1) and to the appended
 * rows before it, and to itself.  Computed as the shard partials (as in
 * pulsar_phase2_partial), a partial over the G earlier appended rows, an
 * index-causal partial over the Tq new tokens' own rows, and one
 * online-softmax merge (Appendix "Phase 2 Distributed Softmax Merge").
 * With few query rows per KV head (Tq * Hq / Hkv <= 32, e.g. a decode
 * step) one launch computes every key range of the shards and of the
 * generation shard (token t limited to rows up to G + t) as its own
 * partial, and one merge follows.
 *
 * q         bf16 [Tq, Hq, d]: the new tokens' queries.
 * Kg, Vg    bf16 [G + Tq, Hkv, d]: the generation shard's appended rows, the
 *           G earlier tokens first, then the Tq new tokens' own keys/values.
 * K, V      bf16 [n_shards, S, Hkv, d]: the retained shards (nullable when
 *           n_shards == 0 or S == 0).
 * o         out float32 [Tq, Hq, d];  lse out float32 [Hq, Tq], nullable.
 * workspace device buffer of at least pulsar_phase2_query_workspace_bytes
 *           bytes, 16-byte aligned; contents on entry do not matter.
 * Query encoding: G = 0, Tq = query length.  Decode step: Tq = 1, G = the
 * number of query and generated tokens before it.
 *
 * EINVAL: negative sizes, Hq % Hkv != 0, NULL required pointers, misaligned
 *         buffers, scale not finite and > 0.  EWORKSPACE: workspace NULL,
 *         misaligned or too small.
 * EUNSUPPORTED: d not in {64, 128}; Hq / Hkv not 1, 2 or a multiple of 4;
 *         one shard's or the generation shard's K at 2 GiB or more.
 */
size_t pulsar_phase2_query_workspace_bytes(int n_shards, int Tq, int64_t S, int64_t G, int Hq,
                                           int Hkv, int d);
int pulsar_phase2_query(const void* q, const void* Kg, const void* Vg, int64_t G, const void* K,
                        const void* V, int n_shards, int Tq, int64_t S, int Hq, int Hkv, int d,
                        float softmax_scale, float* o, float* lse, void* workspace,
                        size_t workspace_bytes, void* stream);

/*
 * Phase-2 attention of new tokens without any allocation, for callers that
 * cannot allocate device memory or pass a workspace: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.
 *
 * Arguments, results and errors are those of pulsar_phase2_query without the
 * workspace.  The partials live in a static device array of
 * PULSAR_STATIC_SCRATCH_BYTES bytes, one per GPU, held from the library's
 * first use on that GPU until the process ends; its address is looked up
 * once per device on the first call made with that device current.  The
 * call allocates nothing (no hipMalloc, no library allocation).
 *
 * ETOOLARGE: pulsar_phase2_query_workspace_bytes(...) for these shapes
 *   exceeds PULSAR_STATIC_SCRATCH_BYTES (about 33 partials of 64 tokens x 32
 *   heads x 128 fit, e.g. a 64-token query encoding over 16 shards).
 * Every call on one GPU uses that GPU's one array: calls that overlap in time
 * on the same GPU (different streams, or host threads without ordering) race
 * and give undefined results.  Calls ordered on one stream are safe; nothing
 * in the array needs to start at zero.
 */
#define PULSAR_STATIC_SCRATCH_BYTES (64u << 20)
int pulsar_phase2_query_noalloc(const void* q, const void* Kg, const void* Vg, int64_t G,
                                const void* K, const void* V, int n_shards, int Tq, int64_t S,
                                int Hq, int Hkv, int d, float softmax_scale, float* o, float* lse,
                                void* stream);

/*
 * Rotary position embedding of query or key rows at given positions
 * (Appendix "RoPE Position ID Assignment").  In the paper's sparse mode every
 * token keeps its global position id, so rotating a layer's Q and K of the
 * whole context once, by position, gives every block's Phase-1 input (and
 * the retained KV) its rotated rows; pulsar_phase1_attn then reads them.
 *
 * Rotate-half form: for a head vector x of width d, pair i < d/2 is
 * (x_i, x_{i+d/2}) and becomes
 *   (x_i cos(p w_i) - x_{i+d/2} sin(p w_i),  x_{i+d/2} cos(p w_i) + x_i sin(p w_i))
 * for the row's position p.  The angle is formed in fp64 and reduced to
 * [-pi, pi]; the rotation is evaluated in fp32 and rounded once to bf16.
 *
 * X         bf16 [batch, n_rows, H, d], 16-byte aligned, rotated in place.
 * pos       int32 [batch, n_rows]: the rows' positions; NULL means the row
 *           index within its sequence.  pos_offset is added to every
 *           position (for example the first position of Phase-2 queries).
 * inv_freq  HOST pointer to d/2 floats, the frequencies w_i (a model's
 *           scaled table); NULL means w_i = base^(-2i/d).
 *
 * EINVAL: negative sizes, NULL or misaligned X when there is work, odd d,
 *         a non-finite table entry, or (without a table) base not finite
 *         and > 0.  EUNSUPPORTED: d not in {64, 128}.
 */
int pulsar_rope(void* X, int batch, int64_t n_rows, int H, int d, const int32_t* pos,
                int64_t pos_offset, const float* inv_freq, double base, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PULSAR_H_ */
