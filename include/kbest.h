/*
 * kbest.h -- C ABI of the MI355X (gfx950) output-layer library.
 *
 * One beam-search decode step of a neural MT output layer, as described in
 * Hoang et al., "Fast Neural Machine Translation Implementation" (WNMT 2018):
 *
 *   Section 2.2, steps 1-4:  p = w x  ->  p = p + b  ->  softmax  ->  k-best;
 *   Algorithm 4:             bias, softmax statistics and best-class search
 *                            fused into one pass over the scores;
 *   Algorithm 6:             the vocabulary is sharded, each shard reduced in
 *                            parallel, then the shard results are merged;
 *   Section 2.1, Alg. 2:     finished hypotheses are removed from the batch
 *                            after every step (mini-batching).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every buffer argument is device memory owned by the caller (hipMalloc'd
 *    or a framework tensor on the current device).  The library never
 *    allocates, frees or synchronises (KB_DEBUG below aside), and keeps no
 *    mutable global state; only the text returned by kb_last_error() is per
 *    thread.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream).
 *    Inputs must stay alive, and outputs must not be read, until the caller
 *    has synchronised with that stream.
 *  - Every function returns a kb_status and never aborts.  On any error the
 *    outputs are unspecified and nothing has been enqueued, except for
 *    KB_ERR_HIP, which reports a failed launch.
 *  - Inputs must be finite.  Non-finite inputs give unspecified results but
 *    no fault.
 *  - Device-resident index arrays (sentence offsets, entry sentence ids) are
 *    trusted.  With the environment variable KB_DEBUG=1 at call time, the
 *    calls that take them first run a validation kernel on `stream`, wait
 *    for it (the one case in which the library synchronises) and return
 *    KB_ERR_INVALID_ARG, with nothing else enqueued, if the contents break
 *    the stated preconditions.  The verdict word is written into the first
 *    int32 of an output of the call (out_token, kept_count), which the call
 *    overwrites when it goes ahead.
 *  - The projection's tile is chosen by a cost model (kb_kbest_plan reports
 *    the choice).  With the environment variable KB_TILE=<rows>x<words> at
 *    call time (e.g. 32x256) a step not taken by the few-row kernel uses that
 *    tile instead where its path has it: 128x256, 256x128, 32x512, 32x256
 *    or 32x128 on every path, 64x128 on the DMA pipeline, and 256x256 on the
 *    bf16 DMA pipeline with V >= 256.  Other values are ignored.  It exists to measure the
 *    model (paper_1805_09863_amd/tune_planner.py); the workspace size follows
 *    it, so size the workspace with the same setting.
 *  - Size limits (KB_ERR_UNSUPPORTED beyond them): N * V <= INT_MAX (a
 *    sentence's flat candidate index row * V + word is an int32), N * H
 *    elements of h below 4 GiB, N * k and S * k within int32.
 */
#ifndef KBEST_H
#define KBEST_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KB_ABI_VERSION 2
#define KB_MAX_K 16 /* largest k (beam width of the output) supported */

typedef enum kb_status {
  KB_OK = 0,
  KB_ERR_INVALID_ARG = 1, /* null pointer, bad size, k out of range, ... */
  KB_ERR_UNSUPPORTED = 2, /* a valid request the library does not handle */
  KB_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required  */
  KB_ERR_HIP = 4          /* a HIP launch failed; see kb_last_error()     */
} kb_status;

/* Storage type of h and W.  Bias, scores and all accumulation are float32. */
typedef enum kb_dtype {
  KB_F32 = 0,  /* float32 h and W; float32 products on the matrix cores      */
  KB_BF16 = 1  /* bfloat16 h and W (the half-precision GEMM of Section 2.3);  */
               /* exact bf16 x bf16 products, float32 accumulation           */
} kb_dtype;

/* KB_ABI_VERSION of the loaded library. */
int kb_abi_version(void);

/* Static text for a kb_status value. */
const char* kb_status_string(kb_status status);

/* Detail of the last failure on the calling thread ("" if none). */
const char* kb_last_error(void);

/*
 * Workspace bytes kb_kbest_step needs for this shape (0 when N == 0).
 * Depends only on (dtype, N, H, V, k, S); the same shape always gives the
 * same size.
 */
size_t kb_kbest_workspace_bytes(int dtype, int N, int H, int V, int k, int S);

/*
 * The projection plan kb_kbest_step (and kb_argmax_step, kb_shard_partials)
 * would choose for this shape when h, W and b have these addresses: which
 * kernel and tile (Section 2.2's fused pass, Algorithm 4), and how the
 * vocabulary is cut into splits (Algorithm 6).  Only the addresses'
 * alignment matters: nothing is read through them and no device call is
 * made, so any values will do (e.g. multiples of 16 for aligned operands).
 * For tests, tuning and capacity planning.
 *
 *   plan_out  KB_PLAN_FIELDS int32, written on KB_OK (all 0 when N == 0):
 *     [KB_PLAN_KERNEL]           one of KB_KERNEL_* below
 *     [KB_PLAN_TILE_ROWS]        rows per tile (KB_KERNEL_FEW: rows it holds)
 *     [KB_PLAN_TILE_WORDS]       words per tile (KB_KERNEL_FEW: per chunk)
 *     [KB_PLAN_ROW_TILES]        ceil(N / rows per tile)
 *     [KB_PLAN_SPLITS]           P, each split a run of whole tiles
 *     [KB_PLAN_TILES_PER_SPLIT]  tiles in each split (the last may be short)
 * Errors: the shape checks of kb_kbest_step (KB_ERR_INVALID_ARG,
 * KB_ERR_UNSUPPORTED); KB_ERR_INVALID_ARG for a null plan_out or for h, W or
 * b not aligned to their element size.
 */
#define KB_KERNEL_FEW 0  /* vector ALUs, W streamed once (a few rows)          */
#define KB_KERNEL_WIDE 1 /* 256 x 256 tiles, matrix cores, LDS DMA pipeline   */
#define KB_KERNEL_DMA 2  /* other tiles on the matrix cores, LDS DMA pipeline */
#define KB_KERNEL_REG 3  /* matrix cores, operands staged through registers  */
#define KB_PLAN_KERNEL 0
#define KB_PLAN_TILE_ROWS 1
#define KB_PLAN_TILE_WORDS 2
#define KB_PLAN_ROW_TILES 3
#define KB_PLAN_SPLITS 4
#define KB_PLAN_TILES_PER_SPLIT 5
#define KB_PLAN_FIELDS 6
kb_status kb_kbest_plan(int dtype, int N, int H, int V, int k, const void* h, const void* W, const float* b,
                        int32_t* plan_out);

/*
 * kb_kbest_step -- one decode step of the output layer with the beam k-best.
 *
 * Computes, for every live hypothesis row n (Section 2.2 steps 1-3):
 *     x[n, j]   = sum_i h[n, i] * W[i, j] + b[j]            (j < V)
 *     LSE[n]    = log sum_j exp(x[n, j])
 *     cand(n,j) = prev_score[n] + x[n, j] - LSE[n]         (cumulative log-prob)
 * and, for every sentence s owning rows sent_offsets[s] .. sent_offsets[s+1]-1,
 * the k best candidates over all of its rows and all words (step 4, extended
 * from the 1-best scan of Algorithms 3-5 to k-best across the beam), sorted
 * by descending score; equal scores keep the lower flat index
 * (row - sent_offsets[s]) * V + j, i.e. the lower parent row, then the lower
 * word -- the first-index-wins rule of the paper's strict '>' scans.
 *
 * The N x V scores are never written to memory: the projection's epilogue
 * keeps, per row and vocabulary shard, the softmax statistics (Algorithm 4's
 * running max and rescaled sum) and the k best (score, word) pairs, which a
 * second kernel merges across shards (Algorithm 6) and across each
 * sentence's rows.
 *
 * Arguments
 *   dtype         KB_F32 or KB_BF16: element type of h and W.
 *   N, H, V       rows (live hypotheses), state size, vocabulary size.
 *                 N >= S, H >= 1, V >= 1.  N == S == 0 is a no-op.
 *   k             outputs per sentence, 1 <= k <= min(KB_MAX_K, V).
 *   S             sentences (beams) in the batch.
 *   h             N x H row-major (H contiguous), element type `dtype`.
 *   W             H x V row-major (V contiguous), element type `dtype`.
 *   b             V float32 bias.
 *   prev_score    N float32 cumulative log-probability of each row.
 *   sent_offsets  S+1 int32 (the beam map): 0 = off[0] <= off[1] <= ... <=
 *                 off[S] <= N; sentence s owns rows off[s] .. off[s+1] - 1.
 *                 A sentence with no rows gets k entries with token and
 *                 parent -1 and score -inf; rows from off[S] on are projected
 *                 but belong to no sentence (a step sized by an upper bound,
 *                 see kb_compact_beams).  Device contents are trusted
 *                 (checked only under KB_DEBUG=1).
 *   out_token     S x k int32: word index in [0, V).
 *   out_parent    S x k int32: global row index of the parent hypothesis.
 *   out_score     S x k float32: cumulative log-probability, descending.
 *   out_row_lse   nullable; N float32 log-sum-exp of each row of a sentence
 *                 (rows from off[S] on are not written).
 *   workspace     device scratch of at least kb_kbest_workspace_bytes(...)
 *                 bytes, 256-byte aligned; contents need no initialisation
 *                 and are overwritten.
 *   stream        hipStream_t.
 * h and W must be aligned to their element size; 16-byte alignment with H
 * and V multiples of 8 (bf16) or 4 (f32) enables vector loads.
 */
kb_status kb_kbest_step(int dtype, int N, int H, int V, int k, int S,
                  const void* h, const void* W, const float* b,
                  const float* prev_score, const int32_t* sent_offsets,
                  int32_t* out_token, int32_t* out_parent, float* out_score,
                  float* out_row_lse,
                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * kb_kbest_step_events -- kb_kbest_step that also records two HIP events
 * (hipEvent_t, both nullable) on `stream` immediately before and after the
 * fused projection kernel, so a caller can time that kernel alone.
 */
kb_status kb_kbest_step_events(int dtype, int N, int H, int V, int k, int S,
                         const void* h, const void* W, const float* b,
                         const float* prev_score, const int32_t* sent_offsets,
                         int32_t* out_token, int32_t* out_parent, float* out_score,
                         float* out_row_lse,
                         void* workspace, size_t workspace_bytes, void* stream,
                         void* proj_begin_event, void* proj_end_event);

/*
 * kb_kbest_step_noalloc -- kb_kbest_step for callers that cannot allocate
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): no workspace argument.  The projection's partials and shared
 * row thresholds go to a fixed array of kb_kbest_step_scratch_max() bytes
 * (16 MiB) in the library's device memory, one per GPU, held from the
 * library's load on that GPU until the process ends.  The call allocates and
 * frees nothing; its first call on a device looks up that device's array.
 *   Arguments, results and errors as kb_kbest_step.  A shape whose
 *   kb_kbest_workspace_bytes exceeds the array returns KB_ERR_UNSUPPORTED
 *   (the V = 90,000, N = 3,072, k = 12 step needs 6.9 MB; N = 4,096 with
 *   k = 16 needs 9.2 MB).
 * Every call on a GPU shares that GPU's array and leaves its contents behind
 * (the thresholds are cleared by a kernel at the start of each call): calls
 * that overlap on one GPU, on different streams or host threads, race and
 * give undefined results.  Calls on one stream are ordered and safe.
 */
size_t kb_kbest_step_scratch_max(void);
kb_status kb_kbest_step_noalloc(int dtype, int N, int H, int V, int k, int S,
                                const void* h, const void* W, const float* b,
                                const float* prev_score, const int32_t* sent_offsets,
                                int32_t* out_token, int32_t* out_parent, float* out_score,
                                float* out_row_lse, void* stream);

/*
 * kb_argmax_step -- greedy decoding (beam 1): the best word of every row,
 * without any softmax (Algorithm 5: argmax of p = W h + b; Algorithm 6: the
 * vocabulary is sharded, each shard's (max, best) found in parallel, then
 * reduced).
 *   h, W, b           as for kb_kbest_step (N rows; no sentences, no prev).
 *   out_token         N int32: argmax_j (h[n] . W[:, j] + b[j]); among equal
 *                     maxima the lowest j (the strict '>' scans of the paper).
 *   out_logit         N float32: that maximum, h[n] . W[:, j] + b[j] (a raw
 *                     score, not a probability).
 *   workspace         at least kb_argmax_workspace_bytes(dtype, N, H, V)
 *                     bytes, 256-byte aligned, caller-owned scratch.
 * N == 0 is a no-op.  1 <= H, 1 <= V.  Errors and alignment as for
 * kb_kbest_step.  Scores accumulate in float32 (bf16 products are exact), so
 * words whose scores differ by less than the accumulation error may swap.
 */
size_t kb_argmax_workspace_bytes(int dtype, int N, int H, int V);
kb_status kb_argmax_step(int dtype, int N, int H, int V, const void* h, const void* W, const float* b,
                   int32_t* out_token, float* out_logit, void* workspace, size_t workspace_bytes,
                   void* stream);

/*
 * kb_kbest_step_unfused -- the same step as kb_kbest_step computed by the
 * unfused baseline the paper compares against (Section 3, the breakdown into
 * multiplication, add bias, softmax and k-best extraction): every stage is a
 * kernel of its own and the N x V scores are stored in the workspace between
 * stages.
 *   mode 0   Algorithm 3: p = W h; AddBias; Softmax in three passes (max,
 *            sum, normalise, in place); Find-Best extended to the k best of
 *            every row (on probabilities); beam merge.
 *   mode 1   Algorithm 4 over the stored scores: p = W h; one fused pass per
 *            row (bias, running max and sum, k best); beam merge.
 * Arguments and results are those of kb_kbest_step (same tie rules; scores
 * agree within float32 rounding).  Supported shapes: bf16, H % 128 == 0,
 * V % 8 == 0, V >= 256, h, W, b 16-byte aligned (else KB_ERR_UNSUPPORTED /
 * KB_ERR_INVALID_ARG).  The workspace (kb_unfused_workspace_bytes; about
 * N * V * 4 bytes) holds the scores.
 *   stage_events  nullable array of n_events hipEvent_t, recorded on the
 *                 stream at the stage boundaries: mode 0: before the
 *                 projection, after it, after AddBias, after Softmax, after
 *                 the k-best, after the merge (6); mode 1: before, after the
 *                 projection, after the fused pass, after the merge (4).
 *                 Events beyond n_events or NULL entries are skipped.
 */
size_t kb_unfused_workspace_bytes(int dtype, int N, int H, int V, int k, int S);
kb_status kb_kbest_step_unfused(int mode, int dtype, int N, int H, int V, int k, int S, const void* h,
                          const void* W, const float* b, const float* prev_score,
                          const int32_t* sent_offsets, int32_t* out_token, int32_t* out_parent,
                          float* out_score, float* out_row_lse, void* workspace,
                          size_t workspace_bytes, void* const* stage_events, int n_events,
                          void* stream);

/*
 * kb_compact_batch -- remove finished hypotheses from the batch (Section 2.1,
 * Algorithm 2: after each Decode, every hypothesis that produced EOS leaves
 * the batch; decoding stops when the batch is empty).
 *
 * The batch is a list of M entries (hypotheses), optionally tagged with the
 * sentence each belongs to.
 *   M                 entries, 0 <= M.
 *   alive_mask        M uint8, nonzero = the entry stays in the batch.
 *   keep_idx          M int32; the first *kept_count entries receive the
 *                     indices of the surviving entries in ascending order (a
 *                     stable compaction); the rest is left untouched.
 *   kept_count        device int32 scalar: number of surviving entries.
 *   entry_sentence    nullable, M int32: sentence id of every entry, >= 0 and
 *                     non-decreasing along the list (entries of a sentence
 *                     are contiguous).  Required by the two outputs below.
 *   new_sent_offsets  nullable, receives *new_S + 1 int32: for every
 *                     surviving sentence (one with a surviving entry), in
 *                     order, the position of its first surviving entry in
 *                     keep_idx, then *kept_count.  Needs room for one more
 *                     entry than entry_sentence has distinct ids.
 *   new_S             nullable, device int32 scalar: surviving sentences.
 *   workspace         kb_compact_workspace_bytes(M) bytes of device scratch
 *                     (NULL allowed when that is 0), 4-byte aligned.
 * M == 0 writes kept_count = 0 (new_S = 0, new_sent_offsets[0] = 0).
 * Integer work: results are exact.  KB_DEBUG=1 checks entry_sentence.
 */
size_t kb_compact_workspace_bytes(int M);
kb_status kb_compact_batch(int M, const uint8_t* alive_mask, int32_t* keep_idx,
                           int32_t* kept_count, const int32_t* entry_sentence,
                           int32_t* new_sent_offsets, int32_t* new_S,
                           void* workspace, size_t workspace_bytes, void* stream);

/*
 * kb_compact_beams -- kb_compact_batch for the S x k output of kb_kbest_step,
 * the shape a beam decoder compacts every step (Section 2.1, Algorithm 2).
 * Entry i = s*k + r is the r-th continuation of sentence s; the sentence ids
 * are implicit, no workspace is needed, and the surviving sentences' old
 * indices are reported as well.
 *   alive             S*k uint8, nonzero = the entry stays in the batch.
 *   keep_idx          S*k int32; the first *kept_count entries receive the
 *                     indices of the surviving entries in ascending order
 *                     (a stable compaction); the rest is left untouched.
 *   kept_count        device int32 scalar: number of surviving entries.
 *   new_sent_offsets  nullable, S+1 int32: the first *new_S + 1 entries are
 *                     the row offsets of the compacted batch (sentences with
 *                     no surviving entry are dropped); entries *new_S + 1 .. S
 *                     repeat *kept_count, so a step launched for more
 *                     sentences than survive (an upper bound known on the
 *                     host before the counts are) sees only empty sentences
 *                     past *new_S.
 *   kept_sentence     nullable, S int32: for each surviving sentence, its
 *                     index in the old batch.
 *   new_S             nullable, device int32 scalar: surviving sentences.
 * S == 0 writes kept_count = 0 (and new_S = 0, new_sent_offsets[0] = 0).
 * 1 <= k <= 1023; S*k must fit in int32.  Results are exact (integer work).
 */
kb_status kb_compact_beams(int S, int k, const uint8_t* alive, int32_t* keep_idx,
                           int32_t* kept_count, int32_t* new_sent_offsets,
                           int32_t* kept_sentence, int32_t* new_S, void* stream);

/*
 * kb_beam_finish -- per-hypothesis end of sentence after a step (Section 2.1,
 * Algorithm 2: every hypothesis that produced EOS leaves the batch; the
 * sentence's beam shrinks with it, and the sentence is done when its beam is
 * empty).  Run after kb_kbest_step(k) on the same S x k outputs, then
 * kb_compact_beams on `alive`.  One step t of T (0 <= t < T):
 *   token, parent, score   S x k outputs of kb_kbest_step (sorted per sentence).
 *   sent_id                S int32: original id (0..S0-1) of each live sentence.
 *   beam                   S int32, in/out: the sentence's beam size k_s <= k;
 *                          only its first k_s continuations are taken.  On
 *                          return, k_s minus the continuations that finished.
 *   prev_keep, prev_hist_base
 *                          the previous step's kb_compact_beams keep_idx and
 *                          that step's hist_base: row i of this step's batch
 *                          holds the hypothesis with history id
 *                          prev_hist_base + prev_keep[i]; NULL at the first
 *                          step (parents are the roots, history id -1).
 *   hist_base              where this step's S*k history entries go:
 *                          hist_token[hist_base + e] = token[e] and
 *                          hist_parent[hist_base + e] = the parent's history id.
 *   fin_*                  the finished store of each original sentence o,
 *                          k slots at o*k: fin_count[o] used slots (in/out),
 *                          fin_score (cumulative log-probability, EOS
 *                          included), fin_len (tokens, EOS included = t + 1),
 *                          fin_hist (history id of its last token).
 *   alive                  S*k uint8 out: 1 for taken continuations that did
 *                          not finish (the input of kb_compact_beams).
 * A taken continuation finishes if its token is `eos`, or at the last step
 * (t == T - 1) whatever it is.  Integer work except for copied scores: exact.
 */
kb_status kb_beam_finish(int S, int k, int t, int T, int eos, const int32_t* token, const int32_t* parent,
                   const float* score, const int32_t* sent_id, int32_t* beam, const int32_t* prev_keep,
                   int prev_hist_base, int hist_base, int32_t* hist_token, int32_t* hist_parent,
                   int32_t* fin_count, float* fin_score, int32_t* fin_len, int32_t* fin_hist,
                   uint8_t* alive, void* stream);

/*
 * kb_beam_backtrace -- the translation of every sentence: among its finished
 * hypotheses the one with the best length-normalised score
 * fin_score / fin_len^alpha (alpha = 0: raw scores; ties: the one finished
 * first), and its tokens, read back through the history.
 *   out_tokens  S0 x T int32: the tokens in order, EOS included, then -1.
 *   out_len     S0 int32 (0 for a sentence with nothing finished);
 *   out_score   S0 float32, the raw score;  out_norm  S0 float32, normalised.
 */
kb_status kb_beam_backtrace(int S0, int k, int T, float alpha, const int32_t* fin_count, const float* fin_score,
                      const int32_t* fin_len, const int32_t* fin_hist, const int32_t* hist_token,
                      const int32_t* hist_parent, int32_t* out_tokens, int32_t* out_len, float* out_score,
                      float* out_norm, void* stream);

/*
 * kb_gather_rows -- dst[i, :] = src[idx[i], :] for i < n, where
 * n = min(n_max, *n_dev) if n_dev is non-null, else n_max.  Rows are
 * row_bytes long (a multiple of 4); src, dst 4-byte aligned.  Moves the
 * per-hypothesis state of the surviving entries after compaction.
 * idx values must index valid rows of src (not checked).
 */
kb_status kb_gather_rows(int n_max, const int32_t* n_dev, const int32_t* idx,
                   const void* src, void* dst, size_t row_bytes, void* stream);

/*
 * Vocabulary shards -- one device's part of the step when the vocabulary is
 * split across devices (Section 2.2, Algorithm 6: every shard finds the best
 * of its own range, then one reduction over the shards' results).  Device g
 * holds W_g = W[:, base_g : base_g + V_g] (contiguous, H x V_g) and b_g, runs
 * kb_shard_partials into its slice of the combined partial arrays, the
 * arrays are exchanged (an all-gather of N * (8 + 8k) bytes per split), and
 * kb_merge_partials over all splits gives exactly kb_kbest_step's result.
 *
 * Partial layout, split-major with rows N apart (one split = one vocabulary
 * range of one shard):
 *   stats  P x N x 2 float32: per split and row the running max m and
 *          sum of exp(x - m) over the split's words (Algorithm 4's pair);
 *   lists  P x N x k x 2 int32: per split and row its k best (score bits,
 *          word) sorted by (score desc, word asc), words already global;
 *          entries past a split's words hold a score below every real one.
 *
 * kb_shard_splits -- *splits = the number of splits kb_shard_partials writes
 * for these operands (it depends on the shape and on the pointers' 16-byte
 * alignment, as the projection's plan does); 0 when N == 0.
 * kb_shard_workspace_bytes -- workspace kb_shard_partials needs (0 when N == 0).
 *
 * kb_shard_partials -- the fused projection over one shard:
 *   dtype, N, H, k   as kb_kbest_step (k <= V_shard);
 *   V_shard          the shard's words; word_base its first word's global
 *                    index (0 <= word_base, word_base + V_shard <= INT_MAX);
 *   h                N x H; W_shard H x V_shard row-major; b_shard V_shard;
 *   stats, lists     where this shard's *splits splits go (8-byte aligned),
 *                    normally the shard's slice of the combined arrays.
 *   Asynchronous on `stream`; the workspace is scratch (same rules as
 *   kb_kbest_step).
 *
 * kb_merge_partials -- the reduction over the shards and the beam merge:
 *   N, V, k, S       rows, the whole vocabulary's size, outputs per sentence,
 *                    sentences (k <= min(KB_MAX_K, V));
 *   P                total splits of all shards, 1 <= P <= 256;
 *   stats, lists     the combined partials (layout above);
 *   prev_score, sent_offsets, out_* as kb_kbest_step (out_row_lse nullable).
 *   Token, parent and score follow kb_kbest_step's order and tie rule.
 */
kb_status kb_shard_splits(int dtype, int N, int H, int V_shard, int k, const void* h,
                    const void* W_shard, const float* b_shard, int* splits);
size_t kb_shard_workspace_bytes(int dtype, int N, int H, int V_shard, int k);
kb_status kb_shard_partials(int dtype, int N, int H, int V_shard, int word_base, int k,
                      const void* h, const void* W_shard, const float* b_shard,
                      float* stats, int32_t* lists,
                      void* workspace, size_t workspace_bytes, void* stream);
kb_status kb_merge_partials(int N, int V, int k, int S, int P, const float* stats,
                      const int32_t* lists, const float* prev_score,
                      const int32_t* sent_offsets, int32_t* out_token,
                      int32_t* out_parent, float* out_score, float* out_row_lse,
                      void* stream);

#ifdef __cplusplus
} /* extern "C" */
#endif

#endif /* KBEST_H */
