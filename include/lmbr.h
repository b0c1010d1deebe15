/*
 * lmbr.h -- C ABI of the batched NMT beam decoder with LMBR n-gram posteriors
 * for AMD Instinct MI355X (gfx950).
 *
 * The operations follow Iglesias et al., "Accelerating NMT Batched Beam
 * Decoding with LMBR Posteriors for Deployment" (NAACL-HLT 2018):
 *   - Eq. 1: per-step NMT log-probabilities (softmax over V logits),
 *   - Eq. 2: the LMBR term L = theta0 + sum_{n=1..4} theta_n P(n-gram ending in y),
 *   - Algorithm 1 (DecodeNMT): per-step scoring, TopB, realignment by
 *     backpointer, EOS push/mask, and the final traceback,
 *   - Section 3.1: sentence batching (B sentences x K beams per step).
 * Notation: this library's B = sentences and K = beams per sentence (the
 * paper's N and B).
 *
 * Conventions for every entry point:
 *   - Return value: LMBR_OK (0) or a negative LMBR_E_* code.  On error a
 *     message is available from lmbr_last_error(ctx) (or lmbr_last_error(NULL)
 *     for failures of lmbr_create); arguments are validated on the host before
 *     any launch, and an invalid call changes no state.
 *   - Faults found by the kernels themselves (non-finite logits, a corrupt
 *     table) never stop a kernel: they set bits of a device flag of the
 *     context (LMBR_DEV_*), which lmbr_decode reads at its end and
 *     lmbr_device_status on request; both then return LMBR_E_DEVICE.
 *   - Device pointers are owned by the caller unless stated otherwise and must
 *     stay valid until the work enqueued on `stream` has completed.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *     stream) unless stated otherwise.  Calls on one context must not overlap
 *     in time on different streams: the context's workspace is shared.
 *   - Index layout: slot (sentence s, beam k) is row s*K + k everywhere.
 *   - Tokens are int32 in [0, V); EOS is config.eos_id.
 *   - Scores are float64; a dead slot has score -infinity.
 */
#ifndef LMBR_H
#define LMBR_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  LMBR_OK = 0,
  LMBR_E_INVALID = -1,   /* bad argument (null pointer, out-of-range size or value) */
  LMBR_E_CAPACITY = -2,  /* a documented size limit is exceeded */
  LMBR_E_HIP = -3,       /* a HIP runtime call failed (device missing, out of memory, ...) */
  LMBR_E_STATE = -4,     /* call out of order (no projection set, history full, ...) */
  LMBR_E_DEVICE = -5,    /* the kernels flagged a data fault (LMBR_DEV_* bits below) */
};

/* Device fault bits (see lmbr_device_status).  The kernels set them and finish
 * normally; the results of the steps involved are then unspecified. */
enum {
  LMBR_DEV_NONFINITE = 1,  /* a live row's log-softmax normaliser is not finite (a NaN or
                              +inf logit, from the caller's logits or bias), or a selected
                              score is NaN */
  LMBR_DEV_TABLE = 2,      /* a context probe found no empty slot in a full pass over a
                              sentence's hash, or a successor range lies outside its table */
};

#define LMBR_MAX_K 16           /* beams per sentence */
#define LMBR_MAX_V 262144       /* vocabulary size limit (tokens are < 2^21 in packed contexts) */
#define LMBR_MAX_ORDER 4        /* n-gram orders 1..4 (Eq. 2) */

typedef struct lmbr_ctx lmbr_ctx;

/* Problem configuration (Algorithm 1 with sentence batching, Eq. 2). */
typedef struct {
  int32_t B;            /* sentences decoded together, >= 1 */
  int32_t K;            /* beams per sentence, 1..LMBR_MAX_K */
  int32_t V;            /* vocabulary size, 2..LMBR_MAX_V */
  int32_t H;            /* decoder hidden size, a positive multiple of 64 */
  int32_t T_max;        /* capacity of the step history (max decode length), >= 1 */
  int32_t eos_id;       /* end-of-sentence token, in [0, V) */
  float   lambda;       /* weight of the LMBR term: score = log P_NMT + lambda * L */
  float   theta[5];     /* theta0..theta4 of Eq. 2 */
  float   load_factor;  /* context hash load factor, in (0, 0.9]; 0 selects 0.5 */
} lmbr_config;

/* Per-sentence decode record, kept on the device for the decode options:
 *   best_final  the best finished value so far (score, or score per word under
 *               length_norm; -inf: none), for early pruning;
 *   backup_*    the fallback hypothesis of LMBR_FINISH_EOS_BACKUP: the best EOS
 *               candidate of a live slot that did not survive TopB, over all
 *               steps so far (backup_step = 0: none yet).  It ends the
 *               hypothesis of slot backup_slot at 1-based step backup_step - 1
 *               with EOS, at cumulative score backup_score. */
typedef struct {
  double  best_final;
  double  backup_score;
  int32_t backup_step;
  int32_t backup_slot;
} lmbr_sentence_record;

/*
 * Beam state (the paper's q, b, y and the per-hypothesis histories), held in
 * caller-owned device buffers.  Sizes with M = B*K:
 *   q      double  [M]           running score q_{t}; -inf marks a dead slot
 *   ctx    uint64  [M]           last <= 3 words: (word+1) in 21-bit fields, newest lowest
 *   hhash  uint64  [M]           rolling hash of the whole history (state of the built-in
 *                                stand-in model; hh <- SplitMix64(hh ^ (word+1)))
 *   len    int32   [M]           number of words in the history
 *   ranges int32   [M*3*2]       for orders n = 2..4: (offset, count) of the successor
 *                                list of the slot's (n-1)-word context, for the next step
 *                                (tables of the dense layout: the slot's row of L in the
 *                                first field, 0 elsewhere)
 *   bp     int32   [T_max*M]     backpointers b_t: parent slot k of slot j at step t
 *   tok    int32   [T_max*M]     words y_t
 *   qhist  double  [T_max*M]     score of slot j at step t before EOS masking (-inf for a
 *                                slot early pruning dropped); an entry with tok == eos and
 *                                a finite score is a member of F
 *   sent   lmbr_sentence_record [B]  per-sentence record of the decode options (required
 *                                with LMBR_FINISH_EOS_BACKUP or early pruning; else may be NULL)
 *   t      host int              steps done so far (advanced by lmbr_beam_step)
 * Step t (0-based) writes row t of bp/tok/qhist.  The struct may be copied and
 * the buffers snapshotted between calls; restoring them resumes the decode.
 */
typedef struct {
  double   *q;
  uint64_t *ctx;
  uint64_t *hhash;
  int32_t  *len;
  int32_t  *ranges;
  int32_t  *bp;
  int32_t  *tok;
  double   *qhist;
  lmbr_sentence_record *sent;
  int32_t   t;
} lmbr_beam_state;

/* Message for the last failure on ctx (or of lmbr_create when ctx is NULL).
 * The string is owned by the library and valid until the next call on ctx. */
const char *lmbr_last_error(const lmbr_ctx *ctx);

/* Bytes of device workspace a context for cfg needs (the state of the step
 * path: per-strip partials, decoder-state staging, the two-pass step's logits
 * fp32 [M, ceil(V / 64) * 64], the tables' descriptors and the empty table,
 * per-sentence option arrays, the traceback staging of lmbr_decode and the
 * device fault flag), or 0 when cfg is invalid (lmbr_create says why). */
size_t lmbr_workspace_bytes(const lmbr_config *cfg);

/* Create a context on the current HIP device.  Validates cfg.
 *   workspace  caller-owned device memory of at least
 *              lmbr_workspace_bytes(cfg) bytes, 256-byte aligned, used by the
 *              context until lmbr_destroy (and not freed by it); or NULL, in
 *              which case the context allocates its workspace with hipMalloc
 *              here.  Either way no call on the step path allocates.
 *   bytes      size of workspace (ignored when it is NULL).
 * Posterior tables (sized by the n-grams given later) are allocated by
 * lmbr_load_posteriors, and the [H, V] repack by lmbr_set_projection, outside
 * the step path.  *out receives the context; free it with lmbr_destroy. */
int32_t lmbr_create(const lmbr_config *cfg, void *workspace, size_t bytes, lmbr_ctx **out);

/* Release the context and every device buffer it allocated (synchronises the
 * device); a caller-provided workspace is left to the caller. */
void lmbr_destroy(lmbr_ctx *ctx);

/* Bytes of device memory the context uses (workspace plus loaded tables). */
size_t lmbr_device_bytes(const lmbr_ctx *ctx);

/* Waits for `stream`, then reads and clears the context's device fault flag.
 * Returns LMBR_OK when no kernel flagged a fault since the last read, else
 * LMBR_E_DEVICE with the LMBR_DEV_* bits in *bits (if not NULL) and named by
 * lmbr_last_error. */
int32_t lmbr_device_status(lmbr_ctx *ctx, int32_t *bits, hipStream_t stream);

/* Set the output projection of the model (the last layer of f_NMT in
 * Algorithm 1, whose B x V output feeds Eq. 1's softmax).
 *   w      bf16 bit patterns.  layout 0: [V, H] row-major, referenced (not copied;
 *          must outlive the context's use).  layout 1: [H, V] row-major, repacked
 *          once into a context-owned [V, H] copy on `stream`.
 *   bias   fp32 [V] or NULL (zero), referenced. */
int32_t lmbr_set_projection(lmbr_ctx *ctx, const uint16_t *w, int32_t layout,
                            const float *bias, hipStream_t stream);

/* Load the n-gram posteriors of one sentence (Eq. 2's P_LMBR over the
 * sentence's evidence space; Section 2: the sparse part of L is prepared on
 * the CPU and uploaded).  All arrays are HOST memory:
 *   order  int32 [n], each in 1..4
 *   tokens int32 [n*4], row i holds the n-gram's words oldest first in its
 *          first order[i] entries (the rest are ignored); words in [0, V)
 *   post   fp32  [n], each in (0, 1]
 * Builds, on the host, a linear-probing hash of the (n-1)-word contexts
 * (capacity a power of two >= contexts / load_factor; slot = SplitMix64(key)
 * & (capacity-1)) and per-context successor lists sorted by word, and uploads
 * them to context-owned device memory.  n may be 0 (empty table: L = theta0).
 * Duplicate n-grams, out-of-range orders, words or posteriors return
 * LMBR_E_INVALID.  Synchronous: returns after the upload (ordered after the
 * work already on `stream`) has finished. */
int32_t lmbr_load_posteriors(lmbr_ctx *ctx, int32_t sentence, int64_t n,
                             const int32_t *order, const int32_t *tokens,
                             const float *post, hipStream_t stream);

/* For callers that own all device memory (Section 2's table upload without
 * an allocation in the library): lmbr_table_bytes builds the sentence's table
 * on the host, as lmbr_load_posteriors does, and returns the device bytes it
 * takes under the context's current layout (lmbr_set_lmbr_layout), or 0 with
 * lmbr_last_error for invalid arguments; it touches no device.
 * lmbr_load_posteriors_into then builds and uploads it into table_mem, caller-
 * owned device memory of at least that many bytes, 256-byte aligned, which the
 * context reads until the sentence is loaded again or the context is
 * destroyed (it never frees it).  Same arguments, checks and ordering as
 * lmbr_load_posteriors; LMBR_E_CAPACITY when bytes is too small (nothing is
 * changed).  If table_mem is the sentence's current table memory and the
 * upload fails, that sentence's table is undefined until it is loaded again. */
size_t lmbr_table_bytes(lmbr_ctx *ctx, int64_t n, const int32_t *order, const int32_t *tokens,
                        const float *post);
int32_t lmbr_load_posteriors_into(lmbr_ctx *ctx, int32_t sentence, int64_t n,
                                  const int32_t *order, const int32_t *tokens, const float *post,
                                  void *table_mem, size_t bytes, hipStream_t stream);

/* How L is held for the tables loaded from now on (each sentence keeps the
 * layout it was loaded with):
 *   LMBR_L_SPARSE (default): the history-free part of L as one dense row per
 *     sentence plus successor lists of the order 2..4 histories, found by a
 *     hash probe per hypothesis and order and added on the fly;
 *   LMBR_L_DENSE: the paper's arrangement (Section 2; Algorithm 1 adds
 *     GetMatrixByRows(L, h) to the scores): one dense fp32 row of lambda * L
 *     per history of the evidence space (lmbr_table_dense, then lambda *
 *     theta0 added on the device), each hypothesis reading the row of its
 *     longest history in the table.  For small evidence spaces: a sentence
 *     whose rows would exceed 2 GiB is refused with LMBR_E_CAPACITY by
 *     lmbr_load_posteriors.
 * The state's ranges then hold, per slot, the row of L in the first field.
 * LMBR_E_INVALID for another value. */
enum { LMBR_L_SPARSE = 0, LMBR_L_DENSE = 1 };
int32_t lmbr_set_lmbr_layout(lmbr_ctx *ctx, int32_t layout);

/* Reset `st` to the start of Algorithm 1: q = (0, -inf, ..., -inf) per
 * sentence (only beam 0 is live), empty histories, t = 0, and the built-in
 * model's history hash hh_0(s) = SplitMix64(SplitMix64(seed + 0x48) ^ s). */
int32_t lmbr_state_init(lmbr_ctx *ctx, lmbr_beam_state *st, uint64_t seed, hipStream_t stream);

/* Recompute st->ranges from st->ctx and st->len (after the caller has written
 * q/ctx/len itself, e.g. to resume from a snapshot). */
int32_t lmbr_state_probe(lmbr_ctx *ctx, lmbr_beam_state *st, hipStream_t stream);

/* The built-in stand-in for f_NMT's decoder state: hidden[m, i] =
 * bf16(IrwinHall(SplitMix64(hh[m] + i))) for every slot, bf16 bits [M, H]. */
int32_t lmbr_synth_hidden(lmbr_ctx *ctx, const lmbr_beam_state *st, uint16_t *hidden,
                          hipStream_t stream);

/* Projection alone (the model's output layer): logits[m, v] =
 * sum_i hidden[m, i] * W[v, i] + bias[v], bf16 inputs, fp32 accumulation and
 * output.  hidden bf16 [M, H]; logits fp32 with row stride ld >= V. */
int32_t lmbr_project(lmbr_ctx *ctx, const uint16_t *hidden, float *logits, int64_t ld,
                     hipStream_t stream);

/* The route of a step from decoder states (lmbr_beam_step, lmbr_score,
 * lmbr_decode); both score the same fp32 logits under the same total order:
 *   LMBR_STEP_TWO_PASS (default): the projection writes the logits into a
 *     context-owned workspace fp32 [M, ceil(V / 64) * 64], then the score pass
 *     reads them once (the work of lmbr_project followed by lmbr_score_logits);
 *   LMBR_STEP_FUSED: one kernel projects and scores each tile while it is on
 *     chip; the logits never reach memory.
 * Applies to later steps of the context.  LMBR_E_INVALID for another value
 * (nothing changes). */
enum { LMBR_STEP_TWO_PASS = 0, LMBR_STEP_FUSED = 1 };
int32_t lmbr_set_step_path(lmbr_ctx *ctx, int32_t path);

/* Rows the last step from decoder states projected (waits for `stream`):
 * on LMBR_STEP_TWO_PASS only the live slots (finite running score) are
 * projected -- the dead ones are never read by the score pass -- so this is
 * their number; on LMBR_STEP_FUSED it is M, the fused kernel compacting live
 * rows itself by whole 256-row blocks.  Before any step: M. */
int32_t lmbr_projected_rows(lmbr_ctx *ctx, int32_t *rows, hipStream_t stream);

/* One step of Algorithm 1 for all B sentences (the loop body: scoring, the
 * LMBR add, TopB per sentence, realignment, EOS push and mask), by the
 * context's step path:
 *   hidden    bf16 [M, H] decoder states of the current slots
 *   eos_bias  fp32 [B] added to the EOS logit of every slot of sentence s before
 *             the log-softmax (a constraint on P_t before TopB), or NULL
 *   parent_out, token_out int32 [M] and score_out double [M]: optional copies
 *             (NULL to skip) of the new b_t, y_t and pre-mask scores, which are
 *             also written to row st->t of the history.
 * Advances st->t; LMBR_E_STATE when st->t == T_max or no projection is set. */
int32_t lmbr_beam_step(lmbr_ctx *ctx, lmbr_beam_state *st, const uint16_t *hidden,
                       const float *eos_bias, int32_t *parent_out, int32_t *token_out,
                       double *score_out, hipStream_t stream);

/* The same step from precomputed logits (fp32 [M, V] with row stride ld,
 * ld >= V, ld % 4 == 0, 16-byte aligned): for models that produce P_t's
 * logits themselves.  No projection is needed. */
int32_t lmbr_beam_step_logits(lmbr_ctx *ctx, lmbr_beam_state *st, const float *logits,
                              int64_t ld, const float *eos_bias, int32_t *parent_out,
                              int32_t *token_out, double *score_out, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the step of
 * lmbr_beam_step_logits, same arguments and results bit for bit, with the
 * score pass's per-(row, strip) partials and EOS column kept in the library's
 * static device scratch of LMBR_STATIC_SCRATCH_BYTES instead of the context's
 * workspace.  It allocates nothing.  The scratch is one array per GPU, taken
 * by lmbr_create and held until the process ends; calls that overlap on one
 * GPU (any context, any stream) race on it, and each call keeps its contents
 * only until the next.  LMBR_E_CAPACITY, with nothing launched, when the
 * configuration needs more than the scratch holds
 * (lmbr_static_scratch_bytes(cfg) > LMBR_STATIC_SCRATCH_BYTES). */
#define LMBR_STATIC_SCRATCH_BYTES 4194304u
size_t lmbr_static_scratch_bytes(const lmbr_config *cfg);
int32_t lmbr_beam_step_logits_static(lmbr_ctx *ctx, lmbr_beam_state *st, const float *logits,
                                     int64_t ld, const float *eos_bias, int32_t *parent_out,
                                     int32_t *token_out, double *score_out, hipStream_t stream);

/* The two halves of a step, for callers that schedule or time them apart
 * (lmbr_beam_step = lmbr_score + lmbr_select; lmbr_beam_step_logits =
 * lmbr_score_logits + lmbr_select).
 *
 * lmbr_score: the scoring half from decoder states (arguments as for
 * lmbr_beam_step, by the context's step path): the projection, the log-softmax
 * partials, the LMBR add and the per-row partial top-K.  The partial results
 * stay in the context's workspace until the next lmbr_select on the same
 * stream.  LMBR_E_STATE when no projection is set or st->t == T_max.
 * lmbr_score_logits: the same from precomputed logits (as for
 * lmbr_beam_step_logits).
 * lmbr_select: TopB per sentence over the partials of the last score call,
 * realignment, EOS push and mask, history writes and the next step's context
 * probes; outputs as for lmbr_beam_step; advances st->t.  LMBR_E_STATE
 * without a preceding score call (each score call is consumed by one select). */
int32_t lmbr_score(lmbr_ctx *ctx, const lmbr_beam_state *st, const uint16_t *hidden,
                   const float *eos_bias, hipStream_t stream);
int32_t lmbr_score_logits(lmbr_ctx *ctx, const lmbr_beam_state *st, const float *logits,
                          int64_t ld, const float *eos_bias, hipStream_t stream);
int32_t lmbr_select(lmbr_ctx *ctx, lmbr_beam_state *st, int32_t *parent_out, int32_t *token_out,
                    double *score_out, hipStream_t stream);

/* ---- decode options (Sections 3 and 3.1) --------------------------------
 * Each applies to every later step and traceback of the context until it is
 * set again; set them before lmbr_state_init.  Defaults: no length
 * normalisation, finish = LMBR_FINISH_AT_T, T_s = T_max, no constraint.
 *
 * length_norm = 1: GetBestHypothesis ranks finished hypotheses by score per
 *   word (score / t for a hypothesis of t words, EOS counted) instead of by
 *   score; ties as before (earlier step, then lower slot).
 * finish = LMBR_FINISH_AT_T: the slots still live after a sentence's last
 *   step are finished hypotheses (F also holds them).
 * finish = LMBR_FINISH_EOS_BACKUP: only EOS hypotheses finish; every step
 *   also keeps, per sentence, the best EOS candidate of a live slot that TopB
 *   did not keep (in st->sent, which lmbr_state_init resets), and when F is
 *   empty at the end GetBestHypothesis returns that one.
 * early_prune = 1 (Section 4.3's early pruning): per sentence the best finished
 *   value so far (score, or score per word) is tracked in st->sent; after each
 *   step's EOS push, a live slot whose value falls below it minus prune_width
 *   (>= 0, natural-log score units; the paper's width 0.01 read as a
 *   probability ratio is ln 100) is dropped: neither expanded nor finished.
 *   Its history entry then reads -inf (score_out still reports its score).
 * Returns LMBR_E_INVALID for a NULL opt or a value outside these. */
enum { LMBR_FINISH_AT_T = 0, LMBR_FINISH_EOS_BACKUP = 1 };
typedef struct {
  int32_t length_norm;  /* 0 or 1 */
  int32_t finish;       /* LMBR_FINISH_* */
  int32_t early_prune;  /* 0 or 1 */
  double  prune_width;  /* >= 0 when early_prune = 1 */
} lmbr_decode_options;
int32_t lmbr_set_decode_options(lmbr_ctx *ctx, const lmbr_decode_options *opt);

/* Per-sentence decode lengths T_s: steps host int32 [B], each in
 * [1, T_max], copied (synchronously) into the context; NULL restores T_s =
 * T_max.  The step that reaches T_s ends every slot of sentence s (under
 * LMBR_FINISH_AT_T the live ones join F at that step); later steps leave the
 * sentence's slots dead, and GetBestHypothesis looks at steps <= T_s only.
 * LMBR_E_INVALID for a value outside [1, T_max]. */
int32_t lmbr_set_sentence_steps(lmbr_ctx *ctx, const int32_t *steps);

/* A constraint on the output words: allowed is device uint32 [B, ceil(V/32)]
 * (bit v % 32 of word v / 32 of row s set = word v may follow any
 * hypothesis of sentence s), caller-owned and read by every later step until
 * replaced; NULL removes the constraint.  Disallowed words stay in the
 * log-softmax normaliser and leave the candidates before TopB (score -inf);
 * when fewer than K candidates remain, the surplus slots are dead.  Bits at
 * v >= V are ignored.  LMBR_E_INVALID for a pointer not 4-byte aligned. */
int32_t lmbr_set_constraints(lmbr_ctx *ctx, const uint32_t *allowed);

/* GetBestHypothesis (Algorithm 1's return): per sentence, the best member of
 * F = {EOS entries of the history} U {slots still live after the last step},
 * ordered by score (by score per word under length_norm), then earlier step,
 * then lower slot, traced back through bp/tok; with LMBR_FINISH_EOS_BACKUP
 * and F empty, the sentence's backup EOS candidate (step_out/slot_out then
 * name its EOS step and parent slot).  tokens_out int32 [B, T_max] (padded with -1; EOS included when the
 * hypothesis ended on it), len_out int32 [B], score_out double [B] (-inf and
 * length 0 when F is empty), step_out/slot_out int32 [B] or NULL. */
int32_t lmbr_traceback(lmbr_ctx *ctx, const lmbr_beam_state *st, int32_t *tokens_out,
                       int32_t *len_out, double *score_out, int32_t *step_out,
                       int32_t *slot_out, hipStream_t stream);

/* The model's side of a decode step (f_NMT's decoder state in Algorithm 1):
 * called on the host once per step, before the step, with the step index t
 * (0-based, = st->t), the state (device buffers; at t > 0, row t - 1 of st->bp
 * and st->tok holds the previous step's backpointers and words, with which the
 * model realigns its own state, e.g. by lmbr_gather_rows) and a device buffer
 * to fill with the bf16 decoder states [M, H] of the current slots, all on
 * `stream`.  Returns 0, or any other value to stop the decode (lmbr_decode
 * then returns that value). */
typedef int32_t (*lmbr_state_fn)(void *user, int32_t t, const lmbr_beam_state *st,
                                 uint16_t *hidden_out, hipStream_t stream);

/* DecodeNMT (Algorithm 1): T steps from the current state, each the model's
 * decoder states (state_fn, or with state_fn NULL the built-in stand-in
 * lmbr_synth_hidden) then lmbr_beam_step, then GetBestHypothesis
 * (lmbr_traceback) into the context's staging buffers and one device-to-host
 * copy of the results:
 *   eos_bias   device fp32 [T, B] (row = step of this call) or NULL
 *   tokens_out HOST int32 [B, T_max], len_out HOST int32 [B], score_out HOST
 *              double [B]: as in lmbr_traceback.
 * Synchronous: waits for `stream` once at the end, then reads the device
 * fault flag (LMBR_E_DEVICE when set; the outputs are still written).
 * Requires st->t + T <= T_max.  With state_fn NULL the T steps are captured
 * into a HIP graph on a context-owned stream at the first call and replayed
 * by later calls with the same T, starting step, state buffers, eos_bias
 * pointer, projection and options (contents behind those pointers are read
 * when the graph runs); the context keeps the graphs of its last four such
 * keys.  Results are bit-identical to launching the steps one by one.  With a state_fn the steps are launched one by one, so the model
 * may do anything stream-ordered.  Not for use under stream capture (use
 * lmbr_beam_step and lmbr_traceback there).  Calls that overlap on one
 * context race. */
int32_t lmbr_decode(lmbr_ctx *ctx, lmbr_beam_state *st, int32_t T, lmbr_state_fn state_fn,
                    void *user, const float *eos_bias, int32_t *tokens_out, int32_t *len_out,
                    double *score_out, hipStream_t stream);

/* GetMatrixByRows (Algorithm 1): dst row i = src row rows[i], for i < n;
 * rows int32 [n] on the device, each row row_bytes long (a multiple of 4).
 * Realigns a caller's model state with the survivors of a step (b_t). */
int32_t lmbr_gather_rows(void *dst, const void *src, const int32_t *rows, int32_t n,
                         size_t row_bytes, hipStream_t stream);

/* ---- host-only helpers (no device needed) ------------------------------- */

/* The host image of one sentence's posterior table, as lmbr_load_posteriors
 * builds it.  Arrays are owned by the library; free with lmbr_table_free. */
typedef struct {
  int64_t   n_slots;      /* hash capacity (power of two) */
  int64_t   n_entries;    /* successor entries */
  uint64_t *slot_key;     /* [n_slots] packed context, UINT64_MAX = empty slot */
  uint32_t *slot_off;     /* [n_slots] first entry of the context's successors */
  uint32_t *slot_cnt;     /* [n_slots] number of successors */
  int32_t  *entry_tok;    /* [n_entries] successor word, ascending within a context */
  float    *entry_post;   /* [n_entries] posterior of (context, word) */
  uint32_t  uni_off;      /* successors of the empty context (unigrams) */
  uint32_t  uni_cnt;
} lmbr_table_image;

int32_t lmbr_table_build(int32_t V, int64_t n, const int32_t *order, const int32_t *tokens,
                         const float *post, float load_factor, lmbr_table_image *out,
                         char *err, size_t err_len);
void lmbr_table_free(lmbr_table_image *img);

/* Sentence batching for a corpus (Sections 3.1 and 4.5: batches of sentences
 * of similar length finish together, so a batch runs fewer steps and holds
 * fewer dead rows): order_out [n] lists the sentences batch after batch, B
 * per batch (the last may be short) -- by decreasing length (stable) when
 * sorted != 0, else in corpus order -- and batch_steps_out [ceil(n / B)] the
 * decode length of each batch (its longest sentence; lengths are the
 * per-sentence T_s of lmbr_set_sentence_steps, each >= 1).  LMBR_E_INVALID
 * for a bad argument. */
int32_t lmbr_plan_batches(int64_t n, const int32_t *lengths, int32_t B, int32_t sorted,
                          int64_t *order_out, int32_t *batch_steps_out);

/* Section 2's dense arrangement of L for a table image: one row per n-gram
 * history of the evidence space -- row 0 the empty history, then every
 * occupied slot in slot order -- holding the sparse part of lambda * L(h, y)
 * for every word y: lambda * sum_{n=1..l+1} theta_n P_LMBR(last n-1 words of
 * h, y) for a history h of l words (computed in fp64, stored fp32; 0 where no
 * n-gram applies).  The constant lambda * theta0 is NOT included (the paper
 * adds it on the GPU after the upload).  A hypothesis takes the row of the
 * longest suffix of its last three words that is a history of the table
 * (every n-gram with a longer context has posterior 0).
 *   rows_out      [lmbr_table_history_count(img) + 1, ld] floats, ld >= V
 *                 (columns >= V are 0)
 *   slot_row_out  [img->n_slots]: each slot's row, UINT32_MAX for empty slots
 * lmbr_table_history_count gives the number of occupied slots (the histories
 * other than the empty one).
 * Returns LMBR_E_INVALID for NULL arguments or ld < V. */
int64_t lmbr_table_history_count(const lmbr_table_image *img);
int32_t lmbr_table_dense(const lmbr_table_image *img, int32_t V, int64_t ld, float lambda,
                         const float *theta, float *rows_out, uint32_t *slot_row_out);

#ifdef __cplusplus
}
#endif
#endif /* LMBR_H */
