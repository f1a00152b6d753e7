/*
 * fusion.h - C ABI of the MI355X shallow-fusion decode step.
 *
 * At every decode step of a streaming Transducer, each live hypothesis
 * scores the whole vocabulary with Eq. (1) of the paper (Sec. III-C):
 *
 *   score(y) = log p_AM(y|x) + lambda * log p_LM(y) + beta * boost(y)
 *
 * with one backoff n-gram LM over sub-word tokens (the alpha_i of Eq. (1),
 * written lambda here) and a phrase-boosting tree built from a user word list
 * (weight beta).  The step then selects the greedy token (Sec. III: greedy
 * decoding emits the text) or the top-k, and advances the LM and phrase
 * states.  The blank symbol never receives LM or boost terms.
 *
 * Token space.  ASR ids 0..V-1; blank_id is one of them and never occurs in
 * the LM or in phrases.  The LM adds <s> = V and </s> = V+1.  LM tables are
 * natural-log (the paper does not fix a base).
 *
 * Canonical state ids (part of the contract, reproduced independently by
 * the test oracle):
 *   LM: the state of a history is its longest suffix of at most N-1 tokens
 *       that is an n-gram of the model.  A one-token context w has id w; a
 *       k-token context (2 <= k <= N-1) has id off_k + its lexicographic rank
 *       among the order-k n-grams, with off_2 = V+2, off_{k+1} = off_k + n_k.
 *       The start state is <s> (id V).  Order-N n-grams are never states.
 *   Phrases: a state is a prefix of some phrase; its id is its rank under
 *       (length, tokens); the empty prefix (root) is 0.
 *
 * Arithmetic (fp32, one rounding per operation, no fused multiply-add):
 *   lm(y|c)   = p*(c y) if (c y) is an n-gram, else lm(y|c[1:]) + bo(c)
 *               (bo(c) = 0 when c is not an n-gram), lm(y|empty) = p*(y)
 *   boost(y|q) = E(q') - phi(q), q' = the phrase state after y,
 *               phi(n) = 0 for a complete phrase else depth(n) * token_score,
 *               E(n) = phi(n) + out(n), out(n) = completion bonuses of the
 *               phrases that are suffixes of n, added shortest first
 *   key(y)    = (x_y + lambda * lm(y)) + beta * boost(y);  key(blank) = x_blank
 *   fused(y)  = key(y) - lse(x),  lse = log sum exp over the row
 * Selection, ties to the lowest id:
 *   FUSION_BLANK_AM (k = 1): blank if the raw-logit argmax is blank, else the
 *     argmax of key over the non-blank tokens;
 *   FUSION_BLANK_COMPETE: the top-k of key over all tokens.
 *
 * Errors.  Every call returns FUSION_OK (0) or a negative code and never
 * aborts; fusion_last_error() describes the last failure of the calling
 * thread.  A kernel that meets a state id out of range emits blank with
 * unchanged states for that hypothesis and sets a device status word, read
 * and cleared by fusion_device_status().
 */
#ifndef MI355X_FUSION_H
#define MI355X_FUSION_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  FUSION_OK = 0,
  FUSION_E_ARG = -1,         /* null pointer, size out of range, handle/size mismatch */
  FUSION_E_NOMEM = -2,       /* host or device allocation failed */
  FUSION_E_HIP = -3,         /* a HIP runtime call failed */
  FUSION_E_LM_FORMAT = -4,   /* malformed n-gram tables */
  FUSION_E_PHRASES = -5,     /* malformed phrase list */
  FUSION_E_UNSUPPORTED = -6  /* valid request outside this build's limits */
};

enum {
  FUSION_BLANK_AM = 0,      /* greedy default: acoustic argmax decides blank vs. emit */
  FUSION_BLANK_COMPETE = 1  /* blank (key x_blank) competes with the fused keys */
};

/* status bits reported by fusion_device_status */
enum { FUSION_STATUS_BAD_LM_STATE = 1, FUSION_STATUS_BAD_BOOST_STATE = 2,
       FUSION_STATUS_SYNC_TIMEOUT = 4 /* a beam stream's workgroups failed to meet (results invalid) */ };

/* limits of this build */
#define FUSION_MAX_ORDER 6   /* n-gram order N (the per-level registers of the fusion kernel are sized for it) */
#define FUSION_MAX_VOCAB 8190
#define FUSION_MAX_K 8
#define FUSION_MAX_BEAM 32
#define FUSION_MAX_LMS 2     /* LMs per fusion_step_lms / fusion_run_lms call (2 needs V <= 4096) */

/* flags of fusion_run_lms */
#define FUSION_RUN_RECOMBINE 1 /* beam: merge candidates that reach the same history */

typedef struct NgramTables NgramTables; /* opaque, device resident, immutable after load */
typedef struct BoostTrie BoostTrie;     /* opaque, device resident, immutable after build */

/*
 * ngram_load - build the device-resident n-gram tables (the LM term of Eq. (1)).
 *   order    N, 2..FUSION_MAX_ORDER
 *   vocab    V (ASR ids 0..V-1), 2..FUSION_MAX_VOCAB; blank_id in [0, V)
 *   count    [N] host: number of n-grams of each order (count[k-1] for order k)
 *   tokens   [N] host pointers: order k holds count[k-1] rows of k int32 ids,
 *            oldest first, any row order; ids in [0, V+2), never blank_id
 *   logp     [N] host pointers: natural-log probability per row (finite)
 *   backoff  [N] host pointers or NULL: natural-log backoff per row (finite);
 *            backoff[N-1] is ignored; a NULL array means 0
 *   stream   HIP stream for the uploads
 * Requirements (FUSION_E_LM_FORMAT otherwise): no duplicate rows; every
 * non-blank id and <s> has a unigram; every row of order k >= 2 has its
 * (k-1)-token prefix and suffix in the model.  Inputs are copied: the
 * caller may free them when the call returns (it synchronizes the stream).
 * On success *out owns its device memory until ngram_free().
 * Contexts of two or more tokens with more than 1024 / (N - 2) successors get
 * a pre-resolved LM row on the device (so that the remaining successors of
 * any state fit one memory round trip); the environment variable
 * FUSION_CONTEXT_ROW_MIN_ARCS, read at each call, replaces that threshold.
 * Results do not depend on it.
 */
int ngram_load(int32_t order, int32_t vocab, int32_t blank_id, const int64_t *count,
               const int32_t *const *tokens, const float *const *logp,
               const float *const *backoff, hipStream_t stream, NgramTables **out);
/* the id of the <s> start state (= V) */
int ngram_bos_state(const NgramTables *lm, int32_t *state);
/* number of LM state ids (V+2 + n_2 + ... + n_{N-1}) and device bytes held */
int ngram_info(const NgramTables *lm, int64_t *n_states, int64_t *device_bytes);
void ngram_free(NgramTables *lm);

/*
 * boost_build - build the device-resident phrase-boosting tree (the boost
 * term of Eq. (1)) from a user word list in CSR form.
 *   vocab, blank_id  as for ngram_load
 *   n_phrases        >= 0 (0 gives a tree whose boost is 0 everywhere)
 *   tokens, offsets  host: phrase i = tokens[offsets[i] .. offsets[i+1]);
 *                    offsets has n_phrases+1 entries, offsets[0] = 0
 *   completion       host [n_phrases] or NULL: bonus banked when phrase i
 *                    completes; NULL means token_score * length
 *   token_score      credit per matched token of a partial match
 * Phrases must be non-empty, at most 255 tokens, with ids in [0, V) other
 * than blank_id (FUSION_E_PHRASES otherwise).  A repeated phrase keeps the
 * bonus of its first occurrence.  Inputs are copied; the call synchronizes
 * the stream.  On success *out owns its device memory until boost_free().
 */
int boost_build(int32_t vocab, int32_t blank_id, int32_t n_phrases, const int32_t *tokens,
                const int64_t *offsets, const float *completion, float token_score,
                hipStream_t stream, BoostTrie **out);
int boost_info(const BoostTrie *t, int32_t *n_nodes, int32_t *max_depth, int64_t *device_bytes);
void boost_free(BoostTrie *t);

/*
 * fusion_step - one decode step for H independent hypotheses: Eq. (1) of
 * Sec. III-C over the full vocabulary of each hypothesis (the acoustic term
 * is the log-softmax of the joint output, Sec. III), then the greedy token of
 * Sec. III or the top-k, and the LM / phrase state after each selected token.
 *   lm, trie     handles (trie NULL: the beta term is 0)
 *   logits       device [H, V] fp32, row-major (joint output of this frame)
 *   lm_state     device [H] LM state ids;  boost_state device [H] phrase state ids
 *   H            0..2^24;  V must equal the handles' vocab.  H == 0 checks
 *                the scalar arguments and handles and returns FUSION_OK
 *                without reading or writing any buffer
 *   lambda, beta fusion weights of Eq. (1)
 *   k            1..FUSION_MAX_K candidates per hypothesis (k <= V)
 *   blank_mode   FUSION_BLANK_AM (requires k == 1) or FUSION_BLANK_COMPETE
 *   fused        device [H, V] fp32 or NULL: fused(y) for every token
 *   tokens       device [H, k] selected ids, best first
 *   scores       device [H, k] fused score of each selected token
 *   next_lm      device [H, k] LM state after each selected token
 *   next_boost   device [H, k] phrase state after each selected token
 *   stream       all work is enqueued on this stream; the call does not sync
 * All device buffers belong to the caller.  A blank selection leaves both
 * states unchanged.  Unused candidate slots (k > number of candidates) get
 * token -1.
 */
int fusion_step(const NgramTables *lm, const BoostTrie *trie, const float *logits,
                const int32_t *lm_state, const int32_t *boost_state, int32_t H, int32_t V,
                float lambda, float beta, int32_t blank_id, int32_t k, int32_t blank_mode,
                float *fused, int32_t *tokens, float *scores, int32_t *next_lm,
                int32_t *next_boost, hipStream_t stream);

/*
 * fusion_run - T consecutive frames for S streams of B hypotheses
 * (H = S * B, hypothesis h = s * B + b), in one launch: the frame loop of the
 * streaming decoder (Sec. III, greedy decoding; Sec. IV-A, 80 ms frames fed
 * in look-ahead chunks, e.g. 13 frames for 1040 ms), each frame one
 * fusion_step of Eq. (1) with the states carried from frame to frame.  The
 * beam (B > 1) is not in the paper, which decodes greedily: it extends the
 * same step to k candidates per hypothesis.
 *   logits       device [T, H, V] fp32
 *   B == 1       greedy: k must be 1; hyp_score and parents may be NULL
 *   B > 1        frame-synchronous beam (one symbol per frame): every live
 *                hypothesis proposes its top-k (FUSION_BLANK_COMPETE
 *                required); each stream keeps the best B of the B*k
 *                candidates by (hyp_score + fused desc, parent asc, rank
 *                asc); slots left without a candidate are dead
 *                (hyp_score -inf, token and parent -1) and propose nothing
 *   lm_state, boost_state  device [H], in: initial states, out: final states
 *   hyp_score    device [H] fp64, in/out running scores (B > 1); start a
 *                stream with {0, -inf, ...} for a single live hypothesis
 *   tokens       device [T, H]: token chosen for each slot at each frame
 *   parents      device [T, H] (B > 1): slot of the previous frame it extends
 *   fused        device [T, H, V] fp32 or NULL (slots of dead hypotheses untouched)
 *   traffic      device [2] int64 or NULL: adds the algorithmic bytes of the
 *                launch (logits rows, per LM level the smaller of its arc list
 *                and a dense row, phrase rows, outputs) and the number of
 *                hypothesis-steps processed
 * States carry across calls, so a stream can be decoded chunk by chunk with
 * the same result as one call over all frames.  T == 0 or S == 0 checks the
 * scalar arguments and handles and returns FUSION_OK without reading or
 * writing any buffer (logits and outputs may then be NULL).
 */
int fusion_run(const NgramTables *lm, const BoostTrie *trie, const float *logits, int32_t T,
               int32_t S, int32_t B, int32_t V, int32_t k, float lambda, float beta,
               int32_t blank_id, int32_t blank_mode, int32_t *lm_state, int32_t *boost_state,
               double *hyp_score, int32_t *tokens, int32_t *parents, float *fused,
               int64_t *traffic, hipStream_t stream);

/*
 * fusion_step_lms / fusion_run_lms - fusion_step / fusion_run with several
 * n-gram LMs, the sum over i of alpha_i * log p_LM,i(y) in Eq. (1) (Sec. III-C):
 * each LM has its own weight and its own state, advanced by the same tokens.
 *   lms, alphas  host arrays of n_lm handles and weights, 1 <= n_lm <= FUSION_MAX_LMS;
 *                every LM must have the call's vocab and blank_id (orders may differ)
 *   lm_state     device [n_lm, H] state ids (LM i's state of hypothesis h at
 *                i * H + h); fusion_run_lms writes the final states back there
 *   next_lm      (step) device [n_lm, H, k]: LM i's state after each selection
 *   flags        (run) 0 or FUSION_RUN_RECOMBINE: beam recombination.  Candidates
 *                that reach the same history (the slot's initial states and the
 *                tokens emitted since, compared as a 48-bit hash) merge into the
 *                first of them in candidate order (parent asc, rank asc), whose
 *                total becomes the log-sum of theirs (fp64, folded in that
 *                order); the others leave the ranking.  Ignored for B == 1.
 *   hist         (run) device [H] uint64 or NULL, used only with
 *                FUSION_RUN_RECOMBINE: in, each slot's history hash carried
 *                from the previous call of the same streams (0 at the start of
 *                a stream: the history then begins at the slot's initial
 *                states); out, the hash after the last frame.  Passing the same
 *                buffer to consecutive calls makes a chunked recombining beam
 *                equal to one call over all frames.  With NULL every call
 *                starts each slot's history at its initial states, so slots
 *                whose states agree at a call boundary can merge although
 *                their earlier tokens differ.
 * Every other argument is as in fusion_step / fusion_run (beta is the boost
 * weight).  Keys are fp32 with one rounding per operation, the LM terms added
 * in the order of lms: key = (...((x + a_1 lm_1) + a_2 lm_2)...) + beta boost.
 * With n_lm == 1 the calls are fusion_step / fusion_run with lambda = alphas[0].
 * Two LMs with V > 4096 return FUSION_E_UNSUPPORTED (LDS).
 */
int fusion_step_lms(const NgramTables *const *lms, const float *alphas, int32_t n_lm,
                    const BoostTrie *trie, const float *logits, const int32_t *lm_state,
                    const int32_t *boost_state, int32_t H, int32_t V, float beta, int32_t blank_id,
                    int32_t k, int32_t blank_mode, float *fused, int32_t *tokens, float *scores,
                    int32_t *next_lm, int32_t *next_boost, hipStream_t stream);
int fusion_run_lms(const NgramTables *const *lms, const float *alphas, int32_t n_lm,
                   const BoostTrie *trie, const float *logits, int32_t T, int32_t S, int32_t B,
                   int32_t V, int32_t k, float beta, int32_t blank_id, int32_t blank_mode,
                   int32_t *lm_state, int32_t *boost_state, double *hyp_score, int32_t *tokens,
                   int32_t *parents, float *fused, int64_t *traffic, int32_t flags, uint64_t *hist,
                   hipStream_t stream);

/*
 * fusion_run_lms_noalloc - fusion_run_lms for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments, results and errors as
 * fusion_run_lms; it calls no hipMalloc / hipFree / allocating routine.  The
 * beam's exchange records (B > 1) live in a library-owned static device array
 * of FUSION_NOALLOC_SCRATCH_BYTES on each GPU, held until the process ends;
 * streams that do not fit in it at once run in further launches.  One
 * stream's records (2 * B * k * (3 + n_lm + recombine) 8-byte words) must fit
 * (FUSION_E_UNSUPPORTED otherwise; every size within this build's limits
 * does).  Every call on a GPU shares that GPU's array and leaves the last
 * call's records in it (each launch clears what it uses first): calls that
 * overlap on one GPU, on different streams or threads, race and must not be
 * made.  Greedy calls (B == 1) use no scratch at all.
 */
#define FUSION_NOALLOC_SCRATCH_BYTES (1 << 20)
int fusion_run_lms_noalloc(const NgramTables *const *lms, const float *alphas, int32_t n_lm,
                           const BoostTrie *trie, const float *logits, int32_t T, int32_t S, int32_t B,
                           int32_t V, int32_t k, float beta, int32_t blank_id, int32_t blank_mode,
                           int32_t *lm_state, int32_t *boost_state, double *hyp_score, int32_t *tokens,
                           int32_t *parents, float *fused, int64_t *traffic, int32_t flags, uint64_t *hist,
                           hipStream_t stream);

/*
 * fusion_end_scores - end-of-stream scoring: the LM terms of Eq. (1) for the
 * end-of-sentence token </s>, added when a stream ends so that its hypotheses
 * are compared as complete sentences.
 *   lms, alphas, n_lm  as in fusion_run_lms (every LM must contain </s>:
 *                      FUSION_E_UNSUPPORTED otherwise)
 *   lm_state     device [n_lm, H] final LM state ids (as fusion_run_lms leaves them)
 *   hyp_score    device [H] fp64 or NULL: in/out, hyp_score[h] += t_1, += t_2, ...
 *                with t_i = fl32(alphas[i] * lm_i(</s> | state)) in LM order;
 *                -inf (dead) stays -inf
 *   end_term     device [H] fp64 or NULL: out, (0 + t_1) + t_2 ...
 * lm_i(</s> | state) is the backoff recursion of fusion_step in fp32.  At
 * least one of hyp_score / end_term must be given.  A state that is blank,
 * </s> or out of range adds nothing for that LM and sets
 * FUSION_STATUS_BAD_LM_STATE (fusion_device_status).  Only enqueues work.
 */
int fusion_end_scores(const NgramTables *const *lms, const float *alphas, int32_t n_lm,
                      const int32_t *lm_state, int32_t H, double *hyp_score, double *end_term,
                      hipStream_t stream);

/*
 * joint_project - output projection of the Transducer joint network (the
 * network whose log-softmax is the acoustic term of Eq. (1), Sec. III-C),
 * for M hypothesis-frames at once, on the matrix cores:
 *     out[m, n] = sum_k A[m, k] * W[n, k] + bias[n]
 *   A      device [M, K] bf16 (raw 16-bit patterns), row-major: joint hidden states
 *   W      device [N, K] bf16, row-major (a linear layer's weight, N = vocabulary)
 *   bias   device [N] fp32 or NULL
 *   out    device [M, N] fp32, row-major: the logits fusion_step / fusion_run read
 * Products are exact in fp32; the K products of an output are summed in fp32
 * in an unspecified order, then the bias is added.  M >= 0 (0 does nothing),
 * N >= 1, K >= 8 with K % 8 == 0 (FUSION_E_UNSUPPORTED otherwise), A and W
 * 16-byte aligned, each operand under 2 GiB (split larger calls along M).
 * All buffers belong to the caller; the call only enqueues work on `stream`.
 */
int joint_project(const uint16_t *A, const uint16_t *W, const float *bias, int32_t M, int32_t N,
                  int32_t K, float *out, hipStream_t stream);

/*
 * fusion_run_projected - the frame loop with the joint output projection as its
 * producer (the joint network's output layer feeds the acoustic term of Eq. (1),
 * Sec. III): frames are taken in chunks of `chunk` frames (the last may be
 * shorter); for each chunk, joint_project turns the chunk's joint hidden states
 * into logits [chunk, H, V] in the caller's workspace, and the chunk's frames
 * are decoded by fusion_run_lms (states, scores and history hashes carried to
 * the next chunk), all enqueued on `stream`.  chunk = 1 is the per-frame
 * producer; a streaming recogniser passes the frames of one encoder chunk.
 *   A        device [T, H, K] bf16: joint hidden states, frame-major
 *   W, bias  device [V, K] bf16 and [V] fp32 or NULL, as in joint_project
 *   logits   device [chunk, H, V] fp32 workspace (holds the last chunk's
 *            logits on return, at its first rows)
 *   chunk    frames per projection, 1 <= chunk (larger than T acts as T)
 * Every other argument is as in fusion_run_lms (no fused rows, no traffic
 * count).  The results equal joint_project over all T * H rows followed by one
 * fusion_run_lms over the T frames, bit for bit, for every chunk size.  With a
 * beam the exchange records live through all chunks (allocated once per call,
 * stream-ordered), and the frames of every chunk after the first are numbered
 * on from the previous chunk's, so the records need no reset between chunks.
 */
int fusion_run_projected(const NgramTables *const *lms, const float *alphas, int32_t n_lm, const BoostTrie *trie,
                         const uint16_t *A, const uint16_t *W, const float *bias, int32_t K, float *logits,
                         int32_t chunk, int32_t T, int32_t S, int32_t B, int32_t V, int32_t k, float beta, int32_t blank_id,
                         int32_t blank_mode, int32_t *lm_state, int32_t *boost_state, double *hyp_score,
                         int32_t *tokens, int32_t *parents, int32_t flags, uint64_t *hist, hipStream_t stream);

/* description of the calling thread's last failure (library-owned string) */
const char *fusion_last_error(void);
/* synchronizes `stream`, returns the device status bits in *code and clears them */
int fusion_device_status(hipStream_t stream, int32_t *code);

#ifdef __cplusplus
}
#endif

#endif /* MI355X_FUSION_H */
