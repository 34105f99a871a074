/*
 * ngpu_lm.h -- C ABI of the MI355X batched backoff n-gram language model.
 *
 * The library answers the query of Section 2.2 of the NGPU-LM paper
 * (arXiv 2505.22857): for a batch of B language-model states it returns the
 * score of every vocabulary token and the state reached after it,
 *     state[B] -> (scores[B, V], next_state[B, V]),
 * by walking the backoff chain of each state (Algorithm 1), and it fuses that
 * query into one greedy shallow-fusion decoding step (Section 2.3).
 *
 * Conventions shared by every call:
 *   - Weights are natural logarithms in fp32 (the paper stores "logarithms"
 *     without a base; an ARPA log10 value must be multiplied by ln 10 before it
 *     is passed in).  Scores are natural-log fp32.
 *   - A state is a context: the empty context (state 0) or a listed n-gram of
 *     order 1..N-1 (Section 2.1; highest-order n-grams have no state).  State ids
 *     are canonical: 0 is the empty context, then contexts ordered by
 *     (order ascending, token tuple lexicographically ascending) -- the order of
 *     arcs sorted by (from_state, token), Section 2.2.
 *   - Device memory is always owned by the caller.  The library never
 *     allocates device memory and never synchronises a stream except in
 *     ngpu_lm_check_states.  Calls taking `hip_stream` enqueue work on that
 *     hipStream_t (NULL = the null stream) and return once it is enqueued.
 *   - Queries launch on the current device, which must be the device whose
 *     memory holds the uploaded image (NGPU_E_INVALID_ARG otherwise).
 *   - Every call returns NGPU_OK (0) or a negative NGPU_E_* code and then sets a
 *     thread-local message readable with ngpu_lm_last_error().  No call throws.
 *   - A handle may be used from several threads for queries; build, upload and
 *     free must not race with other calls on the same handle.
 */
#ifndef NGPU_LM_H
#define NGPU_LM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define NGPU_LM_MAX_ORDER 10      /* the paper's models go up to order 10 */
#define NGPU_LM_MAX_VOCAB 8192    /* a V-wide score/state row (8 bytes per token) must fit in 64 KiB of LDS */
/* Most states a model may have: the kernels keep a state id in 30 bits of a
 * 32-bit word (the two high bits flag how a row slot was filled).  A larger
 * model is rejected with NGPU_E_TOO_LARGE. */
#define NGPU_LM_MAX_STATES ((int64_t)1 << 30)
/* Most hypotheses (or utterances) per call: the launch grid, 64 work-items per
 * hypothesis, must fit a 32-bit dispatch size.  Larger batches return
 * NGPU_E_INVALID_ARG; split them into several calls. */
#define NGPU_LM_MAX_BATCH ((int64_t)(1 << 26) - 256)

enum ngpu_status {
    NGPU_OK = 0,
    NGPU_E_INVALID_ARG = -1,      /* null pointer, bad size, misaligned buffer, bad mode */
    NGPU_E_TOKEN_RANGE = -2,      /* a token outside [0, V) */
    NGPU_E_ORDER_RANGE = -3,      /* an order outside [1, max_order] or max_order outside [1, 10] */
    NGPU_E_DUPLICATE_NGRAM = -4,  /* the same token tuple listed twice */
    NGPU_E_MISSING_PREFIX = -5,   /* an n-gram whose context (all but the last token) is not listed */
    NGPU_E_MISSING_SUFFIX = -6,   /* an n-gram whose suffix (all but the first token) is not listed */
    NGPU_E_MISSING_UNIGRAM = -7,  /* a token with no unigram and no <unk> weight given */
    NGPU_E_NOT_UPLOADED = -8,     /* a query before ngpu_lm_upload */
    NGPU_E_HIP = -9,              /* a HIP runtime error (message has the HIP error string) */
    NGPU_E_NONFINITE = -10,       /* a NaN/inf weight */
    NGPU_E_TOO_LARGE = -11,       /* vocabulary, order or count beyond the library's limits */
    NGPU_E_BAD_STATE = -12,       /* ngpu_lm_check_states found out-of-range input states */
    NGPU_E_NO_MEMORY = -13        /* host allocation failed */
};

typedef struct ngpu_lm ngpu_lm;   /* opaque; owns host arrays only */

/* An n-gram list, the array form of an ARPA file (Section 2.1).  Row i is the
 * n-gram tokens[i*max_order .. i*max_order + order[i] - 1] (context first,
 * predicted token last; the remaining entries of the row are ignored), with
 * log-probability logprob[i] and backoff weight backoff[i] (0 when the ARPA
 * line has none; ignored for order max_order).  Rows may come in any order.
 * The list must be closed: every n-gram of order k >= 2 needs its first k-1
 * tokens and its last k-1 tokens listed as n-grams too (KenLM output is). */
typedef struct {
    int64_t num_ngrams;
    int32_t max_order;            /* N, 1..NGPU_LM_MAX_ORDER */
    const int32_t *order;         /* [num_ngrams] */
    const int32_t *tokens;        /* [num_ngrams * max_order] */
    const float *logprob;         /* [num_ngrams] natural log */
    const float *backoff;         /* [num_ngrams] natural log */
} ngpu_ngram_list;

typedef struct {
    int64_t num_states;           /* S: 1 + number of n-grams of order < N */
    int64_t num_arcs;             /* arcs out of non-empty contexts (n-grams of order >= 2) */
    int32_t max_order;
    int32_t vocab_size;
    int64_t device_bytes;         /* size of the device image */
} ngpu_lm_info_t;

/* Build flag: the list also holds the sentence markers of an ARPA model, as
 * token V (<s>) and token V + 1 (</s>).  <s> may only open an n-gram and is
 * never scored (its unigram weight is ignored); the state of the context <s>
 * is the start state (ngpu_lm_start_state).  </s> may only close an n-gram;
 * n-grams ending in </s> are not arcs but give each state its final weight,
 * the </s> score folded through the backoff chain at build time (Section 2.3,
 * AED; ngpu_lm_final_weights, NGPU_FUSION_AED).  Both need a unigram (or, for
 * </s>, an <unk> weight). */
#define NGPU_BUILD_BOS_EOS 1u

/* Build flag: close a list that is not closed (a pruned ARPA model) instead of
 * rejecting it.  Every missing prefix and suffix of a listed n-gram (for an
 * n-gram ending in </s>, its prefix) is inserted with backoff weight 0 and the
 * weight the backoff rule of Section 2.1 gives it on the list without it; for
 * an inserted c + v of order >= 2 that is B(c) + W(c[1:] + v) in one fp32 add
 * (B(c) = 0 when c is inserted too), for an inserted unigram the <unk> weight
 * (NGPU_E_MISSING_UNIGRAM without one).  The score of every token after every
 * history is unchanged; the inserted contexts become states, so the state walk
 * reaches the longest listed context of a history as the backoff rule does. */
#define NGPU_BUILD_REPAIR_CLOSURE 2u

/* Build the trie from a closed n-gram list (Section 2.2): states numbered
 * canonically, arcs sorted by (from_state, token) with one contiguous range per
 * state, a dense row over all V tokens for the empty context (a token without a
 * unigram gets unk_logprob and leads to state 0; pass NaN when every token has
 * a unigram), and per state its backoff weight and backoff state (its context
 * minus the first token).  An arc of order < N leads to the state of its own
 * n-gram, an arc of order N to the state of its last N-1 tokens.  The image
 * stores this as one record per state holding its whole backoff chain (arc
 * ranges and the backoff weights already summed in Algorithm 1's order) and a
 * dense V-wide row per order-1 context (layout in csrc/trie.h).
 * vocab_size: 1..NGPU_LM_MAX_VOCAB; additionally ceil(log2 V') * N <= 128 with
 * V' = V (V + 2 with NGPU_BUILD_BOS_EOS), and at most NGPU_LM_MAX_STATES
 * states (NGPU_E_TOO_LARGE otherwise).
 * flags: NGPU_BUILD_BOS_EOS and/or NGPU_BUILD_REPAIR_CLOSURE (else
 * NGPU_E_MISSING_PREFIX / NGPU_E_MISSING_SUFFIX for a list that is not closed).
 * The list is read only during the call.
 * On success *out holds a new handle (free with ngpu_lm_free). */
int ngpu_lm_build(const ngpu_ngram_list *list, int32_t vocab_size, float unk_logprob,
                  uint32_t flags, ngpu_lm **out);

void ngpu_lm_free(ngpu_lm *lm);

int ngpu_lm_info(const ngpu_lm *lm, ngpu_lm_info_t *out);

/* Context tuple of a state: writes its order to *order_out (0 for state 0) and
 * its tokens to tokens_out[0 .. order-1] (capacity max_order - 1). */
int ngpu_lm_state_context(const ngpu_lm *lm, int64_t state, int32_t *tokens_out, int32_t *order_out);

/* The state decoding starts from: the context <s> for a model built with
 * NGPU_BUILD_BOS_EOS (and order >= 2), else the empty context 0. */
int ngpu_lm_start_state(const ngpu_lm *lm, int64_t *state);

/* Final weight of each state d_states[b] into d_final[b] (fp32): the </s>
 * score of the state (Section 2.3, AED), precomputed per state at build time
 * by the same fp32 fold as a query.  Needs NGPU_BUILD_BOS_EOS
 * (NGPU_E_INVALID_ARG otherwise).  Out-of-range states give NaN and are
 * counted for ngpu_lm_check_states.  Asynchronous on hip_stream. */
int ngpu_lm_final_weights(const ngpu_lm *lm, const int32_t *d_states, int64_t B, float *d_final,
                          void *hip_stream);

/* Bytes of device memory the trie image needs (also in ngpu_lm_info). */
size_t ngpu_lm_device_bytes(const ngpu_lm *lm);

/* Copy the trie image into dev_buf (caller-owned device memory of at least
 * ngpu_lm_device_bytes bytes, 256-byte aligned) with one asynchronous copy on
 * hip_stream, and remember dev_buf for later queries.  The host image stays
 * alive in the handle, so the copy needs no synchronisation by the caller
 * beyond stream order.  dev_buf must stay valid while queries are in flight.
 * Uploading again (e.g. to another buffer) replaces the remembered pointer. */
int ngpu_lm_upload(ngpu_lm *lm, void *dev_buf, size_t dev_bytes, void *hip_stream);

/* Batched full-vocabulary query (Algorithm 1, batched): for each b < B,
 * row b of d_scores ([B, V] fp32, row-major) and d_next ([B, V] int32) get the
 * score and the next state of every token v from state d_states[b].
 * The score is the fp32 left fold of Algorithm 1: an accumulator starting at 0
 * gains the backoff weight of each state left on the way down, and the first
 * level holding v adds its weight once.  Device pointers; d_scores and d_next
 * must not overlap.  States must lie in [0, num_states): an out-of-range state
 * yields a row of NaN scores and -1 next states and is counted for
 * ngpu_lm_check_states.  B = 0 is a no-op.  Asynchronous on hip_stream. */
int ngpu_lm_advance(const ngpu_lm *lm, const int32_t *d_states, int64_t B, float *d_scores,
                    int32_t *d_next, void *hip_stream);

enum ngpu_fusion_mode {
    NGPU_FUSION_PLAIN = 0,        /* argmax_v fma(lambda, lm[v], asr[v]) over v < V, then advance */
    NGPU_FUSION_CTC = 1,          /* blank / repeat / other groups (Section 2.3, CTC) */
    NGPU_FUSION_TRANSDUCER = 2,   /* two-stage selection (Section 2.3, transducers) */
    NGPU_FUSION_AED = 3           /* class V is <eos>, scored with the state's final weight (Section 2.3, AED) */
};

/* One greedy shallow-fusion step (Section 2.3) for B hypotheses.
 * d_asr: [B, asr_ld] fp32 ASR log-probabilities; row b holds classes 0..V-1
 *   (tokens) and, for CTC and transducer modes, class V = blank (AED: <eos>);
 *   asr_ld >= V (PLAIN) or >= V + 1.  Blank is always the last class, so no
 *   blank index is passed.
 * lambda: LM weight; the fused score of token v is fmaf(lambda, lm[v], asr[v])
 *   (single rounding), lm[v] being the advance score.
 * PLAIN: label = argmax over v < V of the fused score; state <- next[label].
 * CTC: a = argmax over all V + 1 classes of the raw ASR score.  If a is blank
 *   or equals d_prev[b] (a repeat, collapsed by CTC and not rescored), label = a
 *   and the state stays.  Otherwise label = argmax over v < V, v != d_prev[b]
 *   of the fused score, and state <- next[label].  Then d_prev[b] = label.
 * TRANSDUCER: a = raw argmax over V + 1 classes; blank stays blank with no state
 *   change; otherwise label = fused argmax over v < V and the state advances.
 * AED (model built with NGPU_BUILD_BOS_EOS): class V is <eos>; label = argmax
 *   over v <= V of the fused score, <eos> using the state's final weight as its
 *   LM score; <eos> leaves the state unchanged, a token advances it.
 * Ties go to the lowest index (-0 equals +0).  ASR scores may be -inf: a
 * candidate set entirely at -inf yields its first candidate, as a strict '>'
 * scan from index 0 does; NaN is not supported.  In/out: d_states[B] (int32), d_prev[B] (CTC
 * only; may be NULL otherwise).  Out: d_tokens[B] (int32 label, V = blank).
 * Out-of-range states give label -1, leave the state unchanged and are counted
 * for ngpu_lm_check_states.  Asynchronous on hip_stream. */
int ngpu_lm_fused_greedy_step(const ngpu_lm *lm, const float *d_asr, int64_t B, int64_t asr_ld,
                              int32_t mode, float lambda, int32_t *d_states, int32_t *d_prev,
                              int32_t *d_tokens, void *hip_stream);

#define NGPU_LM_MAX_TOPK 256

/* The k best tokens of the fused score fmaf(lambda, lm[v], asr[v]) over
 * v < V for each hypothesis -- the expansion step of a beam search with the
 * LM fused over the full vocabulary (Section 2.3: full-vocabulary scoring
 * before selection; the paper applies it to AED beam search).  Row b of the
 * outputs ([B, k] each, row-major) lists the k best in descending order of
 * the fused score, ties to the lower token index: d_tokens (int32), d_scores
 * (fp32 fused scores), d_next (int32 state after that token); when fewer
 * than k tokens score above -inf, the rest follow in index order (as a strict
 * '>' selection gives).  States are read only.
 * 1 <= k <= min(V, NGPU_LM_MAX_TOPK); cost per hypothesis: one pass over the V
 * tokens, then for V <= 1024 a selection whose cost hardly grows with k (a
 * binary search for the k-th value, then ranking the k taken tokens), for
 * larger V per selected token one wavefront reduction and a rescan of the
 * V / 64 tokens of one lane.  An out-of-range state gives a
 * row of -1 tokens, NaN scores and -1 states and is counted for
 * ngpu_lm_check_states.  Asynchronous. */
int ngpu_lm_fused_topk(const ngpu_lm *lm, const float *d_asr, int64_t B, int64_t asr_ld, float lambda, int32_t k,
                       const int32_t *d_states, int32_t *d_tokens, float *d_scores, int32_t *d_next,
                       void *hip_stream);

/* A whole greedy decode (Section 2.3) in one launch: for each utterance b,
 * frames t = 0 .. len_b - 1 run the rule of ngpu_lm_fused_greedy_step on the
 * ASR row d_asr + b * stride_b + t * stride_t (strides in floats; the row holds
 * classes 0..V-1 and, for CTC and transducer, blank = V), carrying the state
 * and the previous label from frame to frame.
 * d_lengths: [B] int32 frame counts (clamped to [0, T]) or NULL for T.
 * In/out: d_states[B] (start states; final states on return), d_prev[B] (CTC:
 *   the label before frame 0, blank = V for a new utterance; the last label on
 *   return; may be NULL otherwise).  Passing the returned states and labels
 *   back continues a decode exactly where it stopped.
 * Out: d_labels[B, T] int32 (row b at d_labels + b * T): the label of each
 *   frame, -1 past the utterance's length; d_label_states[B, T] (or NULL): the
 *   state after each frame.  An out-of-range start state gives a row of -1 and
 *   is counted for ngpu_lm_check_states.  Asynchronous on hip_stream. */
int ngpu_lm_fused_greedy_decode(const ngpu_lm *lm, const float *d_asr, int64_t B, int64_t T, int64_t stride_b,
                                int64_t stride_t, const int32_t *d_lengths, int32_t mode, float lambda,
                                int32_t *d_states, int32_t *d_prev, int32_t *d_labels, int32_t *d_label_states,
                                void *hip_stream);

/* Synchronises hip_stream, then reports (and clears) how many out-of-range
 * input states the queries enqueued since the last check met.  Returns
 * NGPU_E_BAD_STATE when the count is non-zero. */
int ngpu_lm_check_states(const ngpu_lm *lm, void *hip_stream, int64_t *bad_count);

/* The same check without the count: synchronises hip_stream and returns
 * NGPU_E_BAD_STATE (clearing the count) when queries enqueued since the last
 * check met out-of-range input states, else NGPU_OK.  Every query kernel
 * performs the range check itself (one compare per hypothesis), so no build
 * flag enables it. */
int ngpu_lm_sync_check(const ngpu_lm *lm, void *hip_stream);

/* Algorithmic memory traffic of ngpu_lm_advance on host-side states h_states[B]:
 *   *hbm_bytes   = 8V (output row) + the state's chain record (16 bytes per
 *                  order, 16 for state 0) + 12 bytes per arc of each state of
 *                  order >= 2 on its backoff chain,
 *   *total_bytes = *hbm_bytes + 8V (the dense row of the order-1 ancestor, or
 *                  of the empty context),
 * summed over the batch.  The dense rows are shared by all hypotheses and
 * mostly served from the caches, hence the two figures.  Host-only. */
int ngpu_lm_query_bytes(const ngpu_lm *lm, const int32_t *h_states, int64_t B,
                        int64_t *hbm_bytes, int64_t *total_bytes);

/* Read-only view of the host copy of the trie image (the bytes that
 * ngpu_lm_upload copies), valid until ngpu_lm_free.  Its layout belongs to this
 * library build; it is exposed for saving an image and for white-box tests. */
int ngpu_lm_host_image(const ngpu_lm *lm, const void **data, size_t *bytes);

/* ARPA text (Section 2.1: "W context token B" lines, base-10 logarithms, as
 * KenLM writes them) parsed into an n-gram list for ngpu_lm_build.
 * vocab[0..V-1]: the scored vocabulary as words (NUL-terminated, distinct,
 * without <unk>, <s>, </s>); every other word of the file is an error
 * (NGPU_E_TOKEN_RANGE).  Weights become natural logarithms: x * ln 10 in
 * double, rounded once to fp32.  The <unk> unigram's weight is returned as
 * the <unk> weight; longer n-grams containing <unk> are dropped.  With
 * NGPU_BUILD_BOS_EOS, <s> and </s> become tokens V and V + 1; without it,
 * n-grams containing them are dropped (a closed file stays closed either
 * way).  The header's n-gram counts must match the file.  text need not be
 * NUL-terminated; it is read only during the call.  On success *out owns the
 * list (free with ngpu_arpa_free). */
typedef struct ngpu_arpa ngpu_arpa;
int ngpu_arpa_parse(const char *text, size_t len, const char *const *vocab, int32_t V, uint32_t flags,
                    ngpu_arpa **out);

/* The parsed list (arrays owned by a, valid until ngpu_arpa_free) and the
 * <unk> weight (NaN when the file has no <unk> unigram). */
int ngpu_arpa_list(const ngpu_arpa *a, ngpu_ngram_list *list, float *unk_logprob);

void ngpu_arpa_free(ngpu_arpa *a);

/* Message of the last failing call on this thread ("" if none). */
const char *ngpu_lm_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* NGPU_LM_H */
