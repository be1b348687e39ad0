/*
 * kbest_standin.h -- decoder stand-in of the synthetic decode loop.
 *
 * Not part of the output layer.  The paper's decoder (an RNN) produces the
 * state h of every live hypothesis before each output-layer step; the loop
 * that measures mini-batching (Section 2.1, Algorithm 2 against the constant
 * batch of Algorithm 1) replaces it by a seeded table of states and a drawn
 * length per sentence, at which all of the sentence's continuations end.
 * These calls keep that bookkeeping on the device, so a loop step needs no
 * host work beyond reading two counts.  Conventions (caller-owned device
 * buffers, stream ordering, kb_status returns, kb_last_error) are those of
 * kbest.h; the functions live in the same library.
 */
#ifndef KBEST_STANDIN_H
#define KBEST_STANDIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * kb_standin_alive -- alive[s*k + r] = (s < S_live && t < lengths[sid[s]] - 1)
 * ? 1 : 0 for s < S, r < k: the batch entries that stay after step t, when
 * sentence s (original id sid[s]) emits EOS on every continuation at step
 * lengths[sid[s]] - 1.  S_live = min(S, *S_dev), or S if S_dev is NULL: a
 * loop that sizes a step by an upper bound S on the sentence count passes the
 * exact count on the device, and the entries of sentences past it are 0 (sid
 * is not read for them).
 *   S_dev    NULL or one int32 on the device (e.g. kb_compact_beams's new_S).
 *   sid      S int32, original sentence ids (indices into lengths).
 *   lengths  int32 per original sentence.
 *   alive    S*k uint8 output, the input of kb_compact_beams.
 * S == 0 is a no-op.  0 <= S, 1 <= k, S*k fits in int32.
 */
kb_status kb_standin_alive(int S, const int32_t* S_dev, int k, int t, const int32_t* sid, const int32_t* lengths,
                     uint8_t* alive, void* stream);

/*
 * kb_standin_step -- the bookkeeping of one loop step after the output layer,
 * in one launch: the mask of kb_standin_alive, the compaction of
 * kb_compact_beams over it (the same scan: Section 2.1, Algorithm 2's removal
 * of finished hypotheses, stable), the gathers that carry the surviving
 * entries' scores and the surviving sentences' original ids to the next
 * step, and, if next_h is given, the gather of kb_standin_next_h for step
 * t + 1 (the surviving entries' next states).
 *   S, S_dev, k, t, sid, lengths   as kb_standin_alive (ids at or past
 *              min(S, *S_dev) are not used; see below).
 *   score      S*k float32, the step's scores (kb_kbest_step's out_score).
 *   keep_idx   S*k int32 out: the surviving entries in order (first counts[0]).
 *   counts     2 int32 out: [0] surviving entries, [1] surviving sentences.
 *   new_sent_offsets  S+1 int32 out: the next batch's offsets; entries past
 *              counts[1] repeat counts[0] (empty sentences), as kb_compact_beams.
 *   prev_next  S*k float32 out: prev_next[i] = score[keep_idx[i]], i < counts[0].
 *   sid_next   S int32 out: the original id of surviving sentence j, j < counts[1].
 *   alive      NULL or S*k uint8 out: the mask itself.
 *   counts_host  NULL or 3 int32 of pinned host memory (allocated pinned, so
 *              the device can write it): [0], [1] the counts again, then
 *              [2] = t + 1, each after a system-scope fence: a host that
 *              polls [2] for t + 1 (having set it to another value first)
 *              reads the counts without an event or a separate copy.
 *   table, T, next_h, row_bytes   NULL next_h: no state gather (table, T and
 *              row_bytes are not read).  Else as kb_standin_next_h with
 *              step t + 1, keep = keep_idx and n = counts[0]: row i of next_h
 *              (i < counts[0]) = table row ((sid[e/k] * T + t + 1) * k + e%k),
 *              e = keep_idx[i]; next_h holds S*k rows of row_bytes; requires
 *              t + 1 < T, row_bytes a positive multiple of 4, table and
 *              next_h 4-byte aligned.  Rows past counts[0] are not written.
 * Buffers are distinct, caller-owned device memory (counts_host aside).  S == 0 writes counts = 0
 * and new_sent_offsets[0] = 0.  1 <= k < 1024; S*k fits in int32.  sid[s]
 * may be read for every s < S, but an id is used (to index lengths) only
 * below min(S, *S_dev).  Workgroup 0 does the bookkeeping; with next_h the
 * other workgroups (one per 32 KB of states) each work the compaction out
 * again in their own LDS and gather their share of the states, so the whole
 * step is one launch while S*k + S + 1 int32 fit in 64 KB (two launches
 * above).  KB_ERR_INVALID_ARG for null required pointers or bad sizes.
 */
kb_status kb_standin_step(int S, const int32_t* S_dev, int k, int t, const int32_t* sid, const int32_t* lengths,
                          const float* score, int32_t* keep_idx, int32_t* counts, int32_t* new_sent_offsets,
                          float* prev_next, int32_t* sid_next, uint8_t* alive, int32_t* counts_host,
                          const void* table, int T, void* next_h, size_t row_bytes, void* stream);

/*
 * kb_standin_next_h -- the states of step t for the entries kept by
 * kb_compact_beams: for i < n = min(n_max, *n_dev) (n_max if n_dev is NULL),
 *   e = keep[i];  out[i, :] = table[(sid[e / k] * T + t) * k + e % k, :]
 * i.e. the table row of (original sentence sid[e / k], step t, beam slot
 * e % k); rows are row_bytes long (a positive multiple of 4).
 *   keep     kb_compact_beams's keep_idx (entries of the old S x k batch).
 *   sid      the OLD batch's original sentence ids (S_old int32).
 *   table    (S0 * T * k) rows; out at least n_max rows.  4-byte aligned.
 * 0 <= t < T; keep and sid must index valid entries (not checked).
 */
kb_status kb_standin_next_h(int n_max, const int32_t* n_dev, int k, int T, int t, const int32_t* keep,
                      const int32_t* sid, const void* table, void* out, size_t row_bytes, void* stream);

#ifdef __cplusplus
} /* extern "C" */
#endif

#endif /* KBEST_STANDIN_H */
