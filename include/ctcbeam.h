/*
 * ctcbeam - batched CTC beam search with n-gram LM shallow fusion and phrase
 * boosting on AMD MI355X (gfx950).  C ABI.
 *
 * The operation is the per-frame beam-search step of FlexCTC (arXiv
 * 2508.07315), Algorithm 1, with the hypothesis score of Eq. 1:
 *     s = log P_CTC + alpha * log P_LM + boost_w * P_PB + beta * N.
 * Input (Algorithm 1 "Input"; Sec. III-C): log-probabilities D [B, T, V+1]
 * and valid lengths L [B].  Output (Algorithm 1 "Output"; Sec. III-A, the
 * trie of hypotheses reconstructed on demand): the best hypothesis per
 * utterance, as collapsed token ids and its score.
 *
 * Conventions for every entry point:
 *   - labels 0..V-1 are tokens and label V is blank, so a frame row holds
 *     W = V+1 fp32 values; rows are contiguous, utterances are [T, W] blocks;
 *   - LM ids are 0..V-1 (tokens), V (</s>) and V+1 (<s>);
 *   - return codes: 0 OK, 1 invalid argument, 2 unsupported (a size above a
 *     documented limit), 3 out of memory, 4 HIP runtime error;
 *     ctcbeam_last_error() describes the last non-zero return of the calling
 *     thread.  On any error nothing is launched and no output is written.
 *
 * Reading of the paper's open points (fixed here; the CPU test oracle follows
 * the same reading):
 *   - the repeat mask compares a label with the beam's previous *frame*
 *     label, blank included; the first frame's previous label is blank;
 *   - a candidate's score is formed in fp32, in this order:
 *       x = s_k + D[t][c]; if c is neither blank nor a repeat:
 *       x = x + beta; x = x + fl(alpha * LM); x = x + fl(boost_w * BT);
 *   - TopK keeps the K best by (score descending, flat index k*W + c
 *     ascending); candidates at -inf are never kept as live beams;
 *   - pruning: a kept score below (best kept score - theta) becomes -inf;
 *   - recombination keeps the first (best) of the beams that share the
 *     collapsed transcript and whether they end in blank; the others become
 *     -inf in place (max, not log-sum-exp);
 *   - LM scores are natural-log ARPA backoff values, each entry converted
 *     once as fl(double(log10 value) * ln 10); a context's backoff chain is
 *     summed innermost (shortest context) first;
 *   - at the end, live beams get fl(alpha * LM(</s>)); the best beam is the
 *     highest score, lowest slot on ties; if every beam is dead the output is
 *     empty with score -inf.
 */
#ifndef CTCBEAM_H
#define CTCBEAM_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ctcbeam_lm ctcbeam_lm;
typedef struct ctcbeam_boost ctcbeam_boost;

/* Limits of the library (requests beyond them return 2). */
#define CTCBEAM_MAX_K 128       /* beam size (above 64: V <= 1024) */
#define CTCBEAM_MAX_V 4096      /* tokens (blank excluded) */
#define CTCBEAM_MAX_ORDER 8     /* n-gram order */

/*
 * Build a GPU-resident backoff n-gram LM (Sec. II "NGPU-LM": an n-gram model
 * laid out for batched full-vocabulary queries on the GPU; Sec. IV-A: built
 * from the same ARPA file as a CPU LM).
 *   order       : n-gram order, 1..CTCBEAM_MAX_ORDER
 *   vocab_size  : V, 1..CTCBEAM_MAX_V
 *   counts      : host [order]; counts[m-1] = number of m-grams
 *   ngram_ids   : host [order] pointers; ngram_ids[m-1] holds counts[m-1]*m
 *                 int32 ids, row-major (oldest word first)
 *   log10_prob  : host [order] pointers to counts[m-1] log10 probabilities
 *   log10_bow   : host [order] pointers to counts[m-1] log10 backoff weights,
 *                 or NULL (a whole order, or the array itself) for none
 *   out         : receives the handle
 * Requirements: every token and </s> has a unigram; <s> appears only first
 * and </s> only last in an n-gram; every n-gram's prefix (its context) is
 * itself an entry; no duplicates.  Input order is free.  The host arrays are
 * only read during the call.  The handle owns its device tables (hipMalloc'd
 * on the current device, immutable, usable from any stream) until
 * ctcbeam_lm_free.  Synchronous (copies to the device).
 * Returns 2 if a context's whole backoff chain holds more than 4096 explicit
 * continuations (the per-hypothesis staging limit).
 */
int ctcbeam_lm_build(int order, int vocab_size, const int64_t* counts,
                     const int32_t* const* ngram_ids, const float* const* log10_prob,
                     const float* const* log10_bow, ctcbeam_lm** out);

/* Same as ctcbeam_lm_build, reading an ARPA text file whose words are
 * "0".."V-1", "<s>" and "</s>" (n-grams with any other word are skipped). */
int ctcbeam_lm_build_arpa(const char* path, int vocab_size, ctcbeam_lm** out);

/* Host-only builds: the same tables without a device copy, for inspection
 * with ctcbeam_lm_tables (a decode with such a handle returns 1). */
int ctcbeam_lm_build_arpa_host(const char* path, int vocab_size, ctcbeam_lm** out);
int ctcbeam_lm_build_host(int order, int vocab_size, const int64_t* counts,
                          const int32_t* const* ngram_ids, const float* const* log10_prob,
                          const float* const* log10_bow, ctcbeam_lm** out);

void ctcbeam_lm_free(ctcbeam_lm* lm);

/*
 * Build a phrase-boosting tree (Sec. III-B: a phrase prefix tree with
 * Aho-Corasick failure links on the NGPU-LM layout; boosting spread over the
 * tree by depth).  Scores per token read: +1 for each token that extends a
 * phrase prefix; on a mismatch the pending (not yet completed) tokens are
 * rolled back; a completed phrase stays banked and matching restarts at the
 * root.  Precisely, with pot(n) = |n| - (longest whole phrase that is a
 * prefix of n) and f(n) = the longest suffix u of n, |u| < |n| and
 * |u| <= pot(n), that is a prefix of some phrase (empty if none):
 *   step(q, c) = +1 into q.c if q.c is a prefix; 0 at the root otherwise;
 *                else (pot(f(q)) - pot(q)) + step(f(q), c).
 *   vocab_size : V
 *   n_phrases  : number of phrases (>= 0)
 *   offsets    : host [n_phrases+1], non-decreasing; phrase p is
 *                tokens[offsets[p] .. offsets[p+1]); empty phrases are ignored
 *   tokens     : host token ids in 0..V-1
 * Limits (return 2 beyond them): at most 2^20-1 tree nodes, phrase length at
 * most 62.
 * Ownership and synchrony as for ctcbeam_lm_build.
 */
int ctcbeam_boost_build(int vocab_size, int n_phrases, const int32_t* offsets,
                        const int32_t* tokens, ctcbeam_boost** out);
int ctcbeam_boost_build_host(int vocab_size, int n_phrases, const int32_t* offsets,
                             const int32_t* tokens, ctcbeam_boost** out);
void ctcbeam_boost_free(ctcbeam_boost* boost);

/* Device workspace needed by a decode of this shape, in bytes: a 256-byte
 * header (the batch size, for ctcbeam_query_status), a status word per
 * utterance and the back-pointers [B, T, K] int32. */
size_t ctcbeam_workspace_bytes(int B, int T, int K);

/*
 * Batched beam search over all frames (Algorithm 1 from initialisation to
 * LM.Final), one kernel launch on `stream`, no host synchronisation and no
 * allocation.
 *   logprobs     : device fp32 [B, T, V+1] (blank = V); only frames t < L_b
 *                  of utterance b are read
 *   lengths      : device int32 [B]; values outside [0, T] are clamped and
 *                  flagged (ctcbeam_query_status)
 *   B, T, V, K   : batch, padded frames, tokens, beam size (1..CTCBEAM_MAX_K;
 *                  beams above 64 need V <= 1024, else 2)
 *   alpha, beta, boost_w : weights of Eq. 1 (alpha ignored without an LM,
 *                  boost_w ignored without a boosting tree)
 *   lm, boost    : handles built on the current device, or NULL
 *   workspace    : device buffer of ctcbeam_workspace_bytes(B, T, K) bytes,
 *                  caller-owned, contents need no initialisation; it holds
 *                  the batch size, a status word per utterance and the
 *                  per-frame back-pointers
 *   out_tokens   : device int32 [B, T]: best transcript, -1 padded
 *   out_lengths  : device int32 [B] (may be NULL): transcript lengths
 *   out_scores   : device fp32 [B]: best score
 * The call only enqueues work.  Concurrent calls need distinct workspaces.
 */
int ctcbeam_decode(const float* logprobs, const int32_t* lengths, int B, int T, int V, int K,
                   float alpha, float beta, float boost_w, const ctcbeam_lm* lm,
                   const ctcbeam_boost* boost, void* workspace, size_t workspace_bytes,
                   int32_t* out_tokens, int32_t* out_lengths, float* out_scores,
                   hipStream_t stream);

/* Variant flags (ctcbeam_opts.flags) for points Sec. III-C leaves open. */
#define CTCBEAM_FLAG_LOGSUMEXP 1       /* recombination merges duplicate hypotheses
                                          by log-sum-exp (summed probability of
                                          their alignments) instead of max: the
                                          lower slot takes lse(own, other) for each
                                          later duplicate in slot order, with a
                                          fixed fp32 exp / log1p (Cody-Waite
                                          reduction + degree-7 Taylor polynomial;
                                          atanh series) */
#define CTCBEAM_FLAG_BOOST_ROLLBACK 2  /* after LM.Final, live hypotheses get
                                          fl(boost_w * -pending), taking back the
                                          boosting of an unfinished phrase */
#define CTCBEAM_FLAG_NO_ROW_CACHE 4    /* performance only, identical results:
                                          refill the per-token LM rows of every
                                          beam every frame instead of keeping
                                          one row per LM state across frames
                                          (rows are reused with an LM of at
                                          most 2^23 states, no boosting, and
                                          V of 513..1024 with K <= 8, up to
                                          2048 with K <= 4, up to 4096 with
                                          K <= 2) */
#define CTCBEAM_FLAG_REPEAT_SCORE 8    /* Sec. III-C's alternative of scoring
                                          repeated emissions at every
                                          occurrence: a frame that repeats the
                                          beam's last frame label (a token)
                                          adds again the fl(alpha * LM) and
                                          fl(boost_w * BT) terms that token got
                                          when it was emitted (no beta; the LM
                                          and boosting states do not move).
                                          Beam, N-best and greedy paths. */

typedef struct ctcbeam_opts {
  float prune_theta;   /* Algorithm 1 threshold theta; +inf disables pruning */
  int64_t* stats;      /* device int64 [B, 8] or NULL: per-utterance counts of
                          frames, live beam-frames, LM chain states, LM arcs,
                          boosting chain nodes, boosting arcs, emitting winners */
  int flags;           /* CTCBEAM_FLAG_* bits; unknown bits return 1 */
  int reserved[3];
} ctcbeam_opts;

/* ctcbeam_decode with options (opts may be NULL: theta = +inf, no stats). */
int ctcbeam_decode_ex(const float* logprobs, const int32_t* lengths, int B, int T, int V,
                      int K, float alpha, float beta, float boost_w, const ctcbeam_lm* lm,
                      const ctcbeam_boost* boost, void* workspace, size_t workspace_bytes,
                      int32_t* out_tokens, int32_t* out_lengths, float* out_scores,
                      hipStream_t stream, const ctcbeam_opts* opts);

/*
 * N-best output (Algorithm 1 keeps K hypotheses per utterance in the batch;
 * Sec. III-A: any of them can be read back from the hypothesis trie): the
 * same search as ctcbeam_decode_ex, returning every beam slot's final
 * hypothesis after LM.Final instead of the best one only.
 *   nbest_tokens  : device int32 [B, K, T]; row r of utterance b holds the
 *                   collapsed transcript of the r-th best slot, -1 padded
 *   nbest_lengths : device int32 [B, K]; 0 for a dead slot
 *   nbest_scores  : device fp32 [B, K]; descending, ties in slot order;
 *                   -inf for a dead slot (dead slots sort last)
 * Row 0 equals ctcbeam_decode_ex's output.  Rows are not deduplicated beyond
 * the recombination of Algorithm 1 (two slots can hold the same transcript,
 * one ending in blank and one not).  Workspace, stream, opts, ownership and
 * errors as for ctcbeam_decode_ex; all three outputs are required.
 */
int ctcbeam_decode_nbest(const float* logprobs, const int32_t* lengths, int B, int T, int V,
                         int K, float alpha, float beta, float boost_w, const ctcbeam_lm* lm,
                         const ctcbeam_boost* boost, void* workspace, size_t workspace_bytes,
                         int32_t* nbest_tokens, int32_t* nbest_lengths, float* nbest_scores,
                         hipStream_t stream, const ctcbeam_opts* opts);

/*
 * Greedy decoding with LM shallow fusion and phrase boosting: Algorithm 1
 * with a single hypothesis (the greedy rows with LM / PB customisation of
 * Table II, Sec. V-A).  At every frame the hypothesis takes the label
 * with the best Eq. 1 score (same fp32 fold and tie order as the beam search;
 * pruning and recombination have no effect with one hypothesis), then
 * LM.Final.  Results equal ctcbeam_decode_ex with K = 1.
 *   logprobs, lengths, B, T, V, alpha, beta, boost_w, lm, boost, out_* :
 *                  as for ctcbeam_decode (out_lengths may be NULL)
 *   workspace    : device buffer of at least ctcbeam_workspace_bytes(B, 0, 1)
 *                  bytes (only the header and the per-utterance status words
 *                  are used; a workspace sized for a beam decode of the same
 *                  B fits)
 *   opts         : may be NULL; prune_theta and CTCBEAM_FLAG_LOGSUMEXP are
 *                  ignored (no effect with one hypothesis); stats, when given,
 *                  receives per utterance {frames, live frames, LM chain
 *                  states read, LM arcs read, boosting chain nodes, boosting
 *                  arcs, emitted tokens, state refills}
 * One kernel launch on `stream`, one wave per utterance, no allocation.
 * Errors as for ctcbeam_decode_ex.
 */
int ctcbeam_greedy_decode(const float* logprobs, const int32_t* lengths, int B, int T, int V,
                          float alpha, float beta, float boost_w, const ctcbeam_lm* lm,
                          const ctcbeam_boost* boost, void* workspace, size_t workspace_bytes,
                          int32_t* out_tokens, int32_t* out_lengths, float* out_scores,
                          hipStream_t stream, const ctcbeam_opts* opts);

/*
 * For callers that cannot allocate device memory (code under stream capture,
 * tight serving loops, harnesses that forbid hipMalloc): ctcbeam_decode_ex
 * without a workspace argument.  The workspace lives in a fixed device array
 * of CTCBEAM_NOALLOC_MAX_WORKSPACE bytes that the library holds on each device
 * it runs on until the process ends; the call allocates nothing.  Requests
 * whose ctcbeam_workspace_bytes(B, T, K) exceeds that size return 2.
 * Every call on one device shares that device's array: calls that overlap on
 * one device race (serialise them, e.g. on one stream).  Status bits of these
 * decodes are not readable through ctcbeam_query_status.  All other
 * arguments, results and errors as for ctcbeam_decode_ex.
 */
#define CTCBEAM_NOALLOC_MAX_WORKSPACE (16u << 20)
int ctcbeam_decode_noalloc(const float* logprobs, const int32_t* lengths, int B, int T, int V, int K,
                           float alpha, float beta, float boost_w, const ctcbeam_lm* lm,
                           const ctcbeam_boost* boost, int32_t* out_tokens, int32_t* out_lengths,
                           float* out_scores, hipStream_t stream, const ctcbeam_opts* opts);

/* Status bits of the last decode that used `workspace`, ORed over its
 * utterances: bit 0 = a length was clamped, bit 1 = internal traceback
 * mismatch, bit 2 = internal staging overflow.  Debug aid; synchronises
 * `stream`, which must be the stream that decode was enqueued on (or one
 * ordered after it).  The decode records its batch size in the workspace
 * header, so the workspace alone identifies the utterances.  Returns 1 if the
 * workspace holds no decode record (never passed to a decode). */
int ctcbeam_query_status(const void* workspace, hipStream_t stream, uint32_t* bits);

/* Thread-local message for the last non-zero return of this thread. */
const char* ctcbeam_last_error(void);

/* Read-only views of a handle's host tables (for inspection and tests).
 * LM: states [n_states * nlev] records {arc_begin, arc_count | exists<<31,
 * backoff(ln, as float bits)}; arcs [n_arcs] {ln prob (float bits), target
 * state, token}; unigram [V+1] ln probabilities (index V = </s>).  State c is
 * the unigram context of token c, state V is <s>. */
typedef struct ctcbeam_lm_view {
  int order, vocab_size, nlev;
  int64_t n_states, n_arcs;
  const uint32_t* states;
  const uint32_t* arcs;
  const float* unigram;
} ctcbeam_lm_view;
int ctcbeam_lm_tables(const ctcbeam_lm* lm, ctcbeam_lm_view* view);

/* Boosting: nodes [n_nodes] {list_begin, list_count, pot | chain_nodes<<8,
 * chain_arcs}; list [n_list] {token, key}; root_key [V]; key = 0 (none) or
 * (depth+1)<<26 | (pot+1)<<20 | child node of the tree state that owns the
 * continuation. */
typedef struct ctcbeam_boost_view {
  int vocab_size;
  int64_t n_nodes, n_list;
  const uint32_t* nodes;
  const uint32_t* list;
  const uint32_t* root_key;
} ctcbeam_boost_view;
int ctcbeam_boost_tables(const ctcbeam_boost* boost, ctcbeam_boost_view* view);

#ifdef __cplusplus
}
#endif

#endif /* CTCBEAM_H */
