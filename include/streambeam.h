/*
 * streambeam -- streaming variable-width batched beam search on MI355X (gfx950).
 *
 * C ABI of the decoding library. It implements the per-timestep batched
 * beam-search step of Var-Stream (Yang et al., "A Streaming Approach For
 * Efficient Batched Beam Search", EMNLP 2020, Sec. 3 and Alg. 1) and its
 * settings Fixed and Var-Batch, on a synthetic Elman decoder
 *     h = tanh(W_h h_prev + E[y]),  z = W_out h,  z[0] += beta (t - L_x),
 *     log-probabilities = z - logsumexp(z)      (the decoder D of Sec. 2).
 * The calls follow Alg. 1's problem statement Decode(X, E, D, n, eps, k, H):
 * create a decoder with (k, n, eps, H), submit inputs, step, collect the
 * finalized hypotheses Y.
 *
 * Conventions for every entry point:
 *  - Device pointers are HIP device addresses on the current device; host
 *    pointers are ordinary process memory. The header needs no HIP headers:
 *    streams are passed as void* (a hipStream_t, or NULL for the default
 *    stream).
 *  - The caller owns all device memory (weights, the workspace, h0 staging);
 *    it must outlive the decoder. The library never allocates or frees device
 *    memory; it owns a small host-side object, pinned host staging for the
 *    per-input lengths (8 bytes per queue entry) and a few HIP events. The
 *    one exception is sb_create_noalloc, whose decoders use a static device
 *    array of the library in place of a caller workspace.
 *  - All device work is ordered on the decoder's stream.
 *  - No call aborts or throws across the ABI. Errors return an sb_status;
 *    sb_last_error() gives the text of the decoder's last failure.
 *  - A decoder is not thread-safe; distinct decoders are independent.
 */
#ifndef STREAMBEAM_H
#define STREAMBEAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SB_OK = 0,
  SB_E_INVALID_ARG = 1,   /* a pointer, size or parameter is out of range       */
  SB_E_WORKSPACE = 2,     /* workspace missing, misaligned or too small          */
  SB_E_STATE = 3,         /* call not valid in the decoder's current state       */
  SB_E_QUEUE_FULL = 4,    /* submit would exceed params.max_inputs                */
  SB_E_TRUNCATED = 5,     /* collect buffers full; the rest stays pending        */
  SB_E_HIP = 6,           /* a HIP runtime call failed (text in sb_last_error)   */
  SB_E_UNSUPPORTED = 7    /* shape or option the library does not implement      */
} sb_status;

/* Schedulers of Sec. 3 / Alg. 1. Fixed = fixed-width search with the
 * paper's own finalization rule (App. A.1: eps = 0, no pruning); Var-Batch =
 * variable-width search, refill only when the batch is empty (eps = 0);
 * Var-Stream = refill when at most eps*n beams remain, expand only the beams
 * with the fewest steps taken; Var-Str-FIFO (App. A, alternative method
 * analysis) = Var-Stream's refill, but every live beam is expanded at each
 * timestep (the batch capacity n taken from the beam with the most steps
 * down; at most n beams are live). All four return the same outputs for
 * the same parameters (eps, delta, M as forced below). */
typedef enum {
  SB_FIXED = 0, SB_VAR_BATCH = 1, SB_VAR_STREAM = 2, SB_VAR_FIFO = 3, SB_FIXED_STREAM = 4, SB_VAR_CAP = 5
} sb_sched;
/* SB_FIXED_STREAM (App. A.1, Table 3): fixed-width search (delta=+inf, M=k)
 * with Var-Stream's refill and selection; its outputs equal SB_FIXED's.
 * SB_VAR_CAP (Sec. 3, last paragraph; Sec. 4.2, 4.3): capacity-constrained
 * Var-Stream. Up to params.pool >= n beams are cached; the refill test and
 * amount use the pool size (refill when live <= eps*pool, up to pool beams);
 * each timestep takes the live beams in order of (steps taken, admission)
 * while their active candidates total at most n*k rows, stopping at the
 * first beam that would exceed that limit. Outputs equal Var-Batch's. */

/* Finalization rule (App. A.1, implementation differences to Fairseq).
 * SB_RULE_PAPER: terminated candidates stay on the beam through no-op
 * expansions, are output once nothing active ranks above them, and may be
 * displaced meanwhile; Y[i] is the final beam in rank order.
 * SB_RULE_FAIRSEQ: a terminated candidate entering the best k expansions is
 * output at once; the beam keeps the k best active expansions; the input
 * finishes with k outputs, Y[i] in the order they were finalized. Fixed
 * width: delta and M are not applied. Needs k <= 15. */
typedef enum { SB_RULE_PAPER = 0, SB_RULE_FAIRSEQ = 1 } sb_rule;

/* Storage type of weights, h0 and decoder states. SB_F32: fp32 everywhere
 * (MFMA fp32, fp32 accumulation). SB_BF16: bf16 weights and states; the
 * projection accumulates in fp32; the recurrence pre-activation is the
 * exact sum of the bf16 products (integer digit products, d a multiple of
 * 256 up to 2048; otherwise, or when W_h has many values far below its
 * rows' largest, an fp64 sum), rounded once to fp64, so that the rounded
 * bf16 state is reproducible. h0 values must be finite. */
typedef enum { SB_F32 = 0, SB_BF16 = 1 } sb_dtype;

/* Status of a finalized hypothesis. */
enum { SB_HYP_EOS = 2, SB_HYP_MAXLEN = 3 };

/* Search parameters (Alg. 1 inputs n, eps, k, H; Sec. 4 heuristics). */
typedef struct {
  int32_t k;             /* beam width, 1..16                                      */
  int32_t n;             /* batch size: beams resident at once, >= 1               */
  double  eps;           /* refill threshold in [0,1): refill when live <= eps*n   */
  double  delta;         /* relative threshold (nats): drop y if score(y) <
                            score(best) - delta; +inf disables (Sec. 4, App. A.3) */
  int32_t max_per_node;  /* M: max kept expansions per parent per step, 1..k      */
  int32_t sched;         /* sb_sched; SB_FIXED forces eps=0, delta=+inf, M=k;
                            SB_FIXED_STREAM forces delta=+inf, M=k;
                            SB_VAR_BATCH forces eps=0                             */
  int32_t max_len_cap;   /* upper bound on every input's max_len, 1..4096         */
  int32_t max_inputs;    /* queue capacity (inputs per decoder lifetime/reset)    */
  int32_t finalize_rule; /* sb_rule; SB_RULE_FAIRSEQ forces delta=+inf, M=k       */
  int32_t pool;          /* beams cached at once: 0 means n; with SB_VAR_CAP any
                            value in [n, 4096], else it must be 0 or n. Beam and
                            candidate storage scale with it, row buffers with
                            n*k                                                   */
} sb_params;

/* Synthetic decoder D (Sec. 2). Token 0 is EOS and also the start symbol.
 * Device arrays, row-major, element type per `dtype` (float or bf16 bits):
 *   W_h   [d][d]     h = tanh(W_h h_prev + E[y])
 *   E     [vocab][d] token embeddings
 *   W_out [vocab][d] z[v] = sum_j W_out[v][j] h[j]
 *   W_kv  [kv_layers][2][d][d] (bf16 only, or NULL): each expansion appends
 *         the rows bf16(h . W_kv[l][j]) to the candidate's KV-like state.
 * With attn = 1 (length-dependent step, App. A.2 and Fig. 2: decoder
 * self-attention) the projection reads x instead of h:
 *   a_l = sum_s softmax_s(K_l[s] . h / sqrt(d)) V_l[s] over the candidate's
 *         KV rows s = 0 .. t-1, the row of this step included (K_l, V_l =
 *         planes j = 0, 1 of layer l);
 *   x   = bf16(h + (1/L) sum_l a_l), computed in fp64 and rounded once.
 * The recurrence keeps reading h. */
typedef struct {
  int32_t vocab;         /* |V| >= 2                                               */
  int32_t d;             /* state size in [64, 4096], a multiple of 64 (fp32) or
                            of 128 (bf16)                                        */
  int32_t dtype;         /* sb_dtype                                               */
  float   eos_beta;      /* EOS bias slope beta                                    */
  const void *W_h, *E, *W_out;
  int32_t kv_layers;     /* 0, or 1..8 with dtype SB_BF16                          */
  const void *W_kv;
  int32_t attn;          /* 0, or 1: attention read-out (needs kv_layers > 0 and
                            d in {256, 512, 1024, 2048})                          */
} sb_model;

/* One finalized hypothesis y_ij of Y[i] (Alg. 1 output). */
typedef struct {
  int64_t input;         /* id of its input given to sb_submit (its queue position,
                            in submission order, when no ids were given)         */
  int32_t rank;          /* position in Y[i]: rank order (0 = best) under the
                            paper's rule, finalization order under Fairseq's      */
  int32_t length;        /* number of tokens, EOS included when present            */
  int32_t status;        /* SB_HYP_EOS or SB_HYP_MAXLEN                             */
  int32_t finalize_step; /* global timestep at which its beam finished            */
  double  score;         /* cumulative natural-log probability                     */
  int64_t tok_offset;    /* offset of its tokens in the collect token buffer       */
} sb_hyp;

/* Counters of Table 5's columns: timesteps, candidate expansions (decoder
 * evaluations of one active candidate), plus no-op expansions of terminated
 * candidates, refills, admitted inputs, finalized hypotheses, finished inputs,
 * the output positions t of the expansions summed (an attention step reads t
 * KV rows per layer and plane), and the (row, 128-token tile) pairs whose
 * logits the row merge recomputed because the projection's short per-tile
 * list could not rule out more of the row's best k there. */
typedef struct {
  int64_t timesteps, expansions, noops, refills, admitted, hyps, finished, positions, tile_recomputes;
} sb_stats_t;

typedef struct sb_decoder sb_decoder;

/* Bytes of device workspace a decoder with this model/params needs (0 if the
 * arguments are invalid). Host-only arithmetic: needs no GPU. */
size_t sb_workspace_bytes(const sb_model *model, const sb_params *params);

/* Check model/params without touching the GPU. Returns SB_OK or the error
 * sb_create would return for them. */
sb_status sb_validate(const sb_model *model, const sb_params *params);

/* Create a decoder over a caller-owned device workspace of `bytes` bytes
 * (>= sb_workspace_bytes, 256-byte aligned). The workspace is initialised on
 * `stream`; the weights are read, never written. The KV path keeps a
 * transposed copy of W_kv in the workspace. */
sb_status sb_create(const sb_model *model, const sb_params *params, void *workspace,
                    size_t bytes, void *stream, sb_decoder **out);

/* Largest workspace (bytes) a decoder made by sb_create_noalloc can use. */
#define SB_NOALLOC_SCRATCH_BYTES (64u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): sb_create
 * without a caller workspace. The decoder uses the library's static scratch,
 * a device array of SB_NOALLOC_SCRATCH_BYTES that each GPU the library runs
 * on holds until the process ends, and static host storage for the decoder
 * object; the call makes no device or pinned-host allocation (no hipMalloc,
 * hipHostMalloc, hipFree, event or stream creation).
 *  - Shapes whose workspace (sb_workspace_bytes) exceeds the scratch return
 *    SB_E_WORKSPACE; sb_last_error(NULL) gives the sizes.
 *  - One such decoder per GPU at a time: while one is alive (until
 *    sb_destroy), another call on the same GPU returns SB_E_STATE. The
 *    scratch keeps the last decoder's contents; sb_create_noalloc
 *    initialises everything the search reads.
 *  - Otherwise the decoder behaves as one from sb_create, with two
 *    differences: sb_submit waits for its length copies before returning
 *    (there is no pinned staging), and the first sb_run creates the two
 *    events it polls with.
 * The weights are read, never written, and must outlive the decoder. */
sb_status sb_create_noalloc(const sb_model *model, const sb_params *params, void *stream, sb_decoder **out);

/* Append `count` inputs to the queue (Alg. 1's X, in index order).
 * ids: host [count] caller ids echoed in sb_hyp.input, or NULL for the
 * queue positions. h0: device [count][d] (dtype of the model), the
 * encodings e_i = E(x_i), copied asynchronously on the stream (the caller
 * may reuse it once the stream has passed this point). L_x, max_len: host
 * [count], copied before return; 1 <= max_len[i] <= max_len_cap. */
sb_status sb_submit(sb_decoder *dec, int32_t count, const int64_t *ids, const void *h0, const int32_t *L_x,
                    const int32_t *max_len);

/* Enqueue one timestep of Alg. 1's loop (refill, select, expand, update,
 * finalize). If `done` is non-NULL, synchronizes and stores 1 when no input
 * is pending and no beam is live, else 0. With done == NULL nothing waits. */
sb_status sb_step(sb_decoder *dec, int32_t *done);

/* Step until every submitted input is finished, then rebuild the tokens of
 * every finished hypothesis in device memory; returns after the stream has
 * completed the work. Steps run as a captured HIP graph of 8 timesteps,
 * replayed on the decoder's stream (captured on first use; the library keeps
 * a private capture stream). Timesteps past completion are no-ops. */
sb_status sb_run(sb_decoder *dec);

/* Copy finalized hypotheses to the host, in input order then rank order,
 * starting at the first not-yet-collected input and stopping at the first
 * unfinished one. Token ids of hypothesis h are tokens[h.tok_offset ..
 * h.tok_offset + h.length). Returns SB_E_TRUNCATED (with everything that fit)
 * when a buffer is too small; the rest stays pending for the next call.
 * Synchronizes the stream. */
sb_status sb_collect(sb_decoder *dec, sb_hyp *hyps, int64_t hyp_cap, int32_t *tokens,
                     int64_t tok_cap, int64_t *n_hyps, int64_t *n_tokens);

/* Counters since create/reset. Synchronizes the stream. */
sb_status sb_stats(sb_decoder *dec, sb_stats_t *out);

/* Timesteps by number of rows (active candidates) expanded: counts[b] is the
 * number of timesteps with b*w <= rows < (b+1)*w, w = *bucket_width (the last
 * bucket also takes everything above). counts: host [64]. Synchronizes. */
sb_status sb_rows_histogram(sb_decoder *dec, int64_t *counts, int32_t *bucket_width);

/* Forget all inputs, beams, outputs and counters (the queue restarts at
 * position 0). Asynchronous on the stream. */
sb_status sb_reset(sb_decoder *dec);

/* Enable (1) or disable (0) timing of the vocabulary-projection kernel:
 * sb_run then launches the step kernels one by one (instead of replaying the
 * step graph) and brackets every projection launch with a pair of HIP events
 * recorded on the decoder's stream. */
sb_status sb_set_timing(sb_decoder *dec, int32_t enable);

/* Sum of the timed projection-kernel durations (ms) and the number of timed
 * launches since timing was enabled. Synchronizes the stream. */
sb_status sb_timing(sb_decoder *dec, double *proj_ms, int64_t *proj_launches);

sb_status sb_destroy(sb_decoder *dec);
/* Text of the decoder's last failure; with dec == NULL, of the calling
 * thread's last failed sb_create_noalloc. */
const char *sb_last_error(const sb_decoder *dec);
const char *sb_status_string(sb_status s);

/* ------------------------------------------------------------------------
 * Test support. Not part of the decoding interface: these calls expose one
 * decoder step and one candidate slot so that tests can compare them with
 * the oracle. They synchronize the stream and may reset the decoder.
 * ------------------------------------------------------------------------ */

/* Run one decoder step (recurrence, projection, row merge) on R explicit
 * rows, outside any search. Valid only on a decoder with no live beams
 * (after create/reset/run); it leaves the decoder reset.
 * h_prev: device [R][d] (model dtype); y, t, L_x: host [R] (last token,
 * 1-based emitted position, input length); R <= n*k. Outputs: h_out device
 * [R][d] (model dtype), lse host [R], top_lp host [R][k] (log-probabilities
 * of the row's best k tokens, best first), top_tok host [R][k].
 * SB_E_UNSUPPORTED on a model with attn = 1 (its step needs KV history). */
sb_status sb_debug_expand(sb_decoder *dec, int32_t R, const void *h_prev, const int32_t *y,
                          const int32_t *t, const int32_t *L_x, void *h_out, double *lse,
                          double *top_lp, int32_t *top_tok);

/* View of the candidate slot (beam, rank) after the last step: status,
 * score, input id, steps taken, its tokens so far (up to tok_cap; n_tokens
 * gets the count) and, with a KV state, its KV rows [layers][2][steps][d] as
 * bf16 bits (up to kv_cap elements; kv may be NULL). */
sb_status sb_debug_slot(sb_decoder *dec, int32_t beam, int32_t rank, int32_t *status,
                        double *score, int64_t *input, int32_t *steps, int32_t *tokens,
                        int32_t tok_cap, int32_t *n_tokens, uint16_t *kv, int64_t kv_cap);

#ifdef __cplusplus
}
#endif
#endif /* STREAMBEAM_H */
