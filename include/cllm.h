/*
 * cllm.h -- C ABI of libcllm.so: the Jacobi-decoding iteration of CLLMs
 * ("CLLMs: Consistency Large Language Models", arXiv 2403.00835) on one AMD MI355X (gfx950).
 *
 * The library runs a LLaMA-style causal decoder (pre-norm RMSNorm, rotate-half RoPE,
 * multi-head attention, SwiGLU FFN, untied LM head, no biases) with hand-written HIP
 * kernels and decodes greedily, either autoregressively (eq. ar_decoding) or by Jacobi
 * iteration with a KV cache (Section 3.1, eq. jacobi_decoding, and the appendix algorithm
 * "Jacobi Decoding with KV Cache").
 *
 * Conventions for every call:
 *   - Token arrays are HOST int32 arrays owned by the caller; they are read or written only
 *     during the call. Ids must lie in [0, vocab).
 *   - The library owns its device memory (weights, KV cache, workspace) and releases it in
 *     cllm_model_free, except an iteration workspace the caller hands over in
 *     cllm_runtime_opts.workspace (e.g. a PyTorch tensor), which stays the caller's.
 *   - Work is queued on the stream given at creation (a hipStream_t; NULL = the default
 *     stream). cllm_prefill, cllm_jacobi_step, cllm_jacobi_decode and cllm_ar_decode return
 *     after the device work has completed.
 *   - Every call returns a cllm_status and never aborts. A failed argument check leaves the
 *     state unchanged. A device error is sticky: every later call on the context returns
 *     CLLM_ERR_DEVICE. cllm_last_error gives a message.
 *   - A context is not thread-safe; use one host thread per context.
 */
#ifndef CLLM_H
#define CLLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum cllm_status {
    CLLM_OK = 0,
    CLLM_ERR_ARG = 1,      /* bad argument: NULL pointer, id out of range, bad size */
    CLLM_ERR_STATE = 2,    /* call not valid in the current state (e.g. step before prefill) */
    CLLM_ERR_CAPACITY = 3, /* would exceed max_ctx, max_block or max_new */
    CLLM_ERR_OOM = 4,      /* device or host allocation failed */
    CLLM_ERR_IO = 5,       /* weight file could not be read */
    CLLM_ERR_FORMAT = 6,   /* weight file header or size is wrong */
    CLLM_ERR_DEVICE = 7,   /* a HIP call failed; the context is unusable */
    CLLM_ERR_NUMERIC = 8   /* a logit was NaN; the sequence stops, and the slot's next prefill
                              clears its key and value caches before it runs */
} cllm_status;

#define CLLM_DTYPE_F32 0
#define CLLM_DTYPE_BF16 1

/* Decoder shape. head_dim must be even; n_heads * head_dim == d_model.
 * dtype CLLM_DTYPE_BF16: bf16 weights and a bf16 KV cache; every other value (residual stream,
 * norm outputs, queries, attention probabilities, FFN hidden) keeps ~fp32 precision (matrix
 * products take it as two bf16 planes, hi + lo) with fp32 accumulation and softmax.
 * CLLM_DTYPE_F32: fp32 everywhere. */
typedef struct cllm_config {
    int32_t n_layers, d_model, n_heads, head_dim, ffn_dim, vocab;
    float rms_eps, rope_base;
    int32_t dtype;
} cllm_config;

/* Capacity of a context. max_ctx bounds prompt + generated tokens + one block, per sequence;
 * max_block (1..64) bounds the Jacobi block length n; max_new bounds tokens per decode;
 * max_batch (1..64; 0 means 1) is the number of sequence slots. Each slot is an independent
 * sequence with its own KV cache and state; every call taking `seq` addresses slot seq in
 * [0, max_batch). A batched iteration runs up to max_batch blocks of up to max_block rows.
 * prefill_chunk: prompt rows per forward pass of cllm_prefill, and of the shared passes into
 * which a batched decode packs its prompts (0 means 512; rounded up to a multiple of 64, at most
 * 4096, and to no more than max_ctx rounded up to 64). A prompt is processed in chunks of that
 * many rows; a row's values do not depend on the chunk size (every
 * reduction has an order fixed by the model shape), so the size changes speed and activation
 * memory only (about 200 KiB per row at the LLaMA-2-7B shape).
 * workspace, workspace_bytes: optional caller-owned device memory of the context's GPU (for
 * example a PyTorch tensor on that device), 256-byte aligned, of at least cllm_workspace_bytes()
 * bytes, or NULL (0 bytes) for library-allocated memory. When given, the context's iteration
 * workspace (activation operands, split and attention partials, argmax partials, control blocks,
 * the row table, token staging and decode outputs: every buffer made at creation except the
 * weights, the RoPE tables and the KV cache) is carved from it and zeroed at creation; the
 * library never frees it, and the caller keeps it alive and leaves it untouched until
 * cllm_model_free returns. Buffers made on demand later (debug logits, trajectory records, the
 * loss head's workspace) are still the library's. Errors of cllm_model_create: ERR_ARG (not
 * device memory of that GPU, misaligned, or bytes without a pointer), ERR_CAPACITY (too small). */
typedef struct cllm_runtime_opts {
    int32_t max_ctx, max_block, max_new;
    int32_t device;  /* HIP device ordinal */
    void *stream;    /* hipStream_t or NULL */
    int32_t max_batch;
    int32_t prefill_chunk;
    void *workspace;        /* caller-owned device buffer, or NULL */
    size_t workspace_bytes;
} cllm_runtime_opts;

/* Bytes of the iteration workspace of a context created with cfg and opts (their workspace
 * fields are ignored): the least workspace_bytes that cllm_model_create accepts with a caller
 * workspace. No device call. Errors: ERR_ARG (as cllm_model_create's checks), ERR_OOM. */
cllm_status cllm_workspace_bytes(const cllm_config *cfg, const cllm_runtime_opts *opts, size_t *bytes);

/* Guess provider of the decode (reading of the paper's random initial n-token sequence).
 * policy CLLM_GUESS_UNIFORM: uniform ids. CLLM_GUESS_STREAM: stream[t], corrupted with rate p,
 * initialises each block, then the model's own predictions iterate (the printed algorithm).
 * CLLM_GUESS_STREAM_REINJECT: after every iteration each unfixed position is re-drawn from
 * the corrupted stream (emulates a consistency-trained model).
 * block_policy CLLM_BLOCK_SHRINK: the state shrinks by the accepted length until the block of
 * n is fixed (the printed algorithm); CLLM_BLOCK_SLIDE: the state is always the next
 * min(n, remaining) positions.
 * A draw for output position t at draw index d is h = mix(mix(mix(mix(seed)^seq)^t)^d) with the
 * SplitMix64 output function mix; uniform ids are ((h >> 32) * vocab) >> 32; a stream id is
 * corrupted when (h >> 11) < thr53 and then replaced by
 * (stream[t] + 1 + (((mix(h) >> 32) * (vocab - 1)) >> 32)) mod vocab. d is 0 for the initial
 * guesses and, under REINJECT, the number of iterations done so far. */
#define CLLM_GUESS_UNIFORM 0
#define CLLM_GUESS_STREAM 1
#define CLLM_GUESS_STREAM_REINJECT 2
#define CLLM_BLOCK_SHRINK 0
#define CLLM_BLOCK_SLIDE 1
typedef struct cllm_guess_spec {
    int32_t policy, block_policy;
    const int32_t *stream; /* host, stream_len >= max_new ids; NULL for UNIFORM */
    int32_t stream_len;
    uint64_t thr53;        /* round(p * 2^53), p in [0, 1] */
    uint64_t seed;
} cllm_guess_spec;

typedef struct cllm_decode_stats {
    int64_t steps;            /* Jacobi iterations (forward passes after the prefill) */
    int64_t blocks;
    int64_t tokens;           /* tokens emitted (== max_new) */
    int64_t accept_hist[65];  /* accept_hist[a]: iterations that accepted a tokens */
    double prefill_ms;        /* device time of the prefill */
    double decode_ms;         /* device time of the iterations */
    int64_t rows;             /* block rows run through the decoder by the iterations (sum of m) */
    /* Device time per iteration (between consecutive iteration boundaries on the stream):
     * percentiles over the decode's iterations, and the median over the iterations that ran a
     * full block of n rows (the first iteration of each block). For a batched decode: over the
     * batched iterations, and the full-block figures equal the overall ones. */
    double iter_ms_p10, iter_ms_p50, iter_ms_p90, iter_ms_full_p50;
    double iter_ms_full_p10, iter_ms_full_p90; /* p10, p90 over the full-block iterations */
} cllm_decode_stats;

typedef struct cllm_ctx cllm_ctx;

/* Create a context with zero weights (set them with cllm_model_set_weights).
 * Errors: ERR_ARG (bad shape or options), ERR_OOM, ERR_DEVICE. */
cllm_status cllm_model_create(const cllm_config *cfg, const cllm_runtime_opts *opts, cllm_ctx **out);

/* Upload all weights from host arrays, in this order (n_tensors = 3 + 9 * n_layers):
 *   embed [vocab][d]; per layer: attn_norm [d], wq [d][d], wk [d][d], wv [d][d], wo [d][d],
 *   ffn_norm [d], w_gate [ffn][d], w_up [ffn][d], w_down [d][ffn]; final_norm [d];
 *   lm_head [vocab][d].
 * Matrices are row-major [out][in] (y = x W^T). Elements are bf16 bit patterns (uint16) for a
 * bf16 model and float for an f32 model; norm gains are always float. The library repacks the
 * matrices into its streaming layout on the device; the host arrays are not retained.
 * Resets every sequence. Errors: ERR_ARG, ERR_DEVICE. */
cllm_status cllm_model_set_weights(cllm_ctx *ctx, const void *const *tensors, int32_t n_tensors);

/* Create a context whose weights are seeded synthetic ones drawn on the GPU (no host arrays): in
 * the order of cllm_model_set_weights, tensor k comes from generator stream s_k: embed 1; layer
 * l's nine tensors 1000 (l + 1) + 0..8; final_norm 2; lm_head 3. Norm gains are 1.0; every
 * matrix element i is 0.02 x a standard normal deviate from the counter-based generator
 * key = mix(mix(seed) ^ s_k) (mix: the SplitMix64 output function of Steele, Lea and Flood,
 * OOPSLA 2014): the Box-Muller pair j = i / 2 takes b1 = mix(key ^ 2j), b2 = mix(key ^ (2j + 1)),
 * u1 = ((b1 >> 11) + 1) 2^-53, u2 = (b2 >> 11) 2^-53, r = sqrt(-2 ln u1), element 2j gets
 * r cos(2 pi u2) and element 2j + 1 gets r sin(2 pi u2), in double; scaled, rounded to fp32 and,
 * for a bf16 model, to bf16 (both nearest even). Errors: those of cllm_model_create, ERR_OOM,
 * ERR_DEVICE. */
cllm_status cllm_model_init_random(const cllm_config *cfg, uint64_t seed, const cllm_runtime_opts *opts,
                                   cllm_ctx **out);

/* Create a context from a weight file: a 64-byte header (magic "CLLMWTS1", int32 version 1,
 * then the cllm_config fields in order, zero padding) followed by the tensors of
 * cllm_model_set_weights in order, little-endian, no gaps.
 * Errors: ERR_IO, ERR_FORMAT, and those of cllm_model_create. */
cllm_status cllm_model_load(const char *path, const cllm_runtime_opts *opts, cllm_ctx **out);

void cllm_model_free(cllm_ctx *ctx);

/* Prefill (the algorithm's first forward): run the prompt through the decoder, fill the KV
 * cache of positions [0, len) and return the greedy first token y0 (the pending token).
 * Replaces any previous state of sequence slot seq.
 * Errors: ERR_ARG (seq, len < 1, ids), ERR_CAPACITY (len + 1 > max_ctx), ERR_NUMERIC, ERR_DEVICE. */
cllm_status cllm_prefill(cllm_ctx *ctx, int32_t seq, const int32_t *prompt, int32_t len, int32_t *first_token);

/* One Jacobi iteration (eq. jacobi_decoding with the cache). block_in[0..m) holds the pending
 * token followed by m-1 guesses for the next positions. On return block_out[i] is the greedy
 * prediction of the token after block_in[i] (argmax of row i, ties to the lowest id) and
 * accepted_len = a = 1 + the number of leading k >= 1 with block_in[k] == block_out[k-1]. The
 * KV of block_in[0..a) is committed (committed length L += a) and the pending token becomes
 * block_out[a-1]. Preconditions: prefilled; 1 <= m <= max_block; L + m <= max_ctx;
 * block_in[0] == pending. Errors: ERR_ARG, ERR_STATE, ERR_CAPACITY, ERR_NUMERIC, ERR_DEVICE. */
cllm_status cllm_jacobi_step(cllm_ctx *ctx, int32_t seq, const int32_t *block_in, int32_t m, int32_t *block_out,
                             int32_t *accepted_len);

/* Jacobi decoding of max_new tokens after a prefill of the prompt, in blocks of n
 * (1 <= n <= max_block), with the iteration loop resident on the device (no host round trip
 * per iteration): the appendix algorithm "Jacobi Decoding with KV Cache" (prefill, then per
 * block the iterations of eq. jacobi_decoding until the block reproduces itself, keeping the KV
 * of accepted tokens), applied to one n-token truncation after another as Section 3.2.1 decodes
 * long responses; Section 3.1 fixes the result, the greedy output of eq. ar_decoding. out_tokens receives max_new ids (y0 first). guess may be NULL (uniform
 * guesses, shrink). stats may be NULL. The output equals greedy AR decoding.
 * Errors: those of cllm_prefill, ERR_ARG (n, max_new, guess stream too short),
 * ERR_CAPACITY (len + max_new + n > max_ctx or max_new above the context's max_new). */
cllm_status cllm_jacobi_decode(cllm_ctx *ctx, int32_t seq, const int32_t *prompt, int32_t len, int32_t n,
                               int32_t max_new, const cllm_guess_spec *guess, int32_t *out_tokens,
                               cllm_decode_stats *stats);

/* Greedy AR decoding of max_new tokens (eq. ar_decoding): one forward per token, on the same
 * kernels as the Jacobi iteration with a block of one token. stats may be NULL. */
cllm_status cllm_ar_decode(cllm_ctx *ctx, int32_t seq, const int32_t *prompt, int32_t len, int32_t max_new,
                           int32_t *out_tokens, cllm_decode_stats *stats);

/* Batched Jacobi iteration (the batched ragged variant of the iteration; the paper generates
 * its Jacobi trajectories at batch size 16, appendix "Computation cost for CLLMs training"): one
 * forward pass over the blocks of B sequence slots at once, each against its own cache, each
 * entry one iteration of eq. jacobi_decoding with the cache (Section 3.1). Entry b is slot
 * seq_ids[b] (distinct, prefilled) with block blocks_in[b * max_block + i], i < m[b]
 * (1 <= m[b] <= max_block, blocks_in[b * max_block] == the slot's pending token). Outputs as
 * cllm_jacobi_step, per entry: blocks_out[b * max_block + i] and accepted[b]. Every row is
 * computed exactly as cllm_jacobi_step computes it: the results of a sequence do not depend
 * on the other sequences of the batch. 1 <= B <= max_batch.
 * Errors: those of cllm_jacobi_step (the state is unchanged on an argument error). */
cllm_status cllm_jacobi_step_batch(cllm_ctx *ctx, int32_t B, const int32_t *seq_ids, const int32_t *blocks_in,
                                   const int32_t *m, int32_t *blocks_out, int32_t *accepted);

/* Batched Jacobi decoding (the appendix algorithm "Jacobi Decoding with KV Cache" for B sequences
 * at once, as the appendix "Computation cost for CLLMs training" generates trajectories at
 * batch size 16; each sequence's output is Section 3.1's greedy fixed point): prefill B prompts
 * (prompt b is prompts[off_b .. off_b + lens[b]), off_b = lens[0] + ... + lens[b-1]) into
 * slots seq_ids[b], then decode max_new tokens for
 * each in blocks of n, all sequences in one device-resident loop whose iterations run the
 * blocks of every unfinished sequence together (sequences finish at different iterations).
 * guesses: B specs (NULL = uniform guesses, shrink); a spec's draws use its slot id as `seq`.
 * out_tokens: B x max_new (row b = sequence b). stats: B entries (may be NULL): steps and the
 * accept histogram per sequence; prefill_ms and decode_ms are the batch's.
 * Output b equals greedy AR decoding of prompt b.
 * Errors: those of cllm_jacobi_decode, ERR_ARG (B, seq_ids). */
cllm_status cllm_jacobi_decode_batch(cllm_ctx *ctx, int32_t B, const int32_t *seq_ids, const int32_t *prompts,
                                     const int32_t *lens, int32_t n, int32_t max_new, const cllm_guess_spec *guesses,
                                     int32_t *out_tokens, cllm_decode_stats *stats);

/* Forget the state of a slot (it must be prefilled again). Errors: ERR_ARG. */
cllm_status cllm_reset(cllm_ctx *ctx, int32_t seq);

/* Debug: when enabled, every later cllm_jacobi_step / cllm_jacobi_step_batch also copies the
 * fp32 logits of its rows into host_buf (row-major rows x vocab, batch entries' rows in order),
 * and cllm_prefill copies those of the prompt's last 64-row tile (prompt rows
 * 64 floor((len - 1) / 64) .. len - 1) to host rows 0.., so the last prompt row's logits are
 * host row (len - 1) mod 64. host_floats: capacity of host_buf in floats, at least
 * max(64, max_batch * max_block) * vocab. The first enable allocates the context's device
 * logits buffer (row capacity x vocab floats; freed with the context).
 * Errors: ERR_ARG, ERR_OOM, ERR_DEVICE. */
cllm_status cllm_debug_logits(cllm_ctx *ctx, int32_t enable, float *host_buf, size_t host_floats);

/* Trajectory recording (the paper's profiling of Jacobi trajectories, Section 5: fast-forwarded
 * and stationary tokens). While enabled, every iteration of a decode call (cllm_jacobi_decode,
 * cllm_jacobi_decode_batch) writes one record per sequence into a device buffer of max_batch x
 * max_new records that the context allocates on the first enable (and frees with the context).
 * A record is CLLM_TRACE_STRIDE int32: [0] committed length L before the iteration, [1] output
 * position e of the block's first token (z[0] = out_tokens[e]), [2] first output position of
 * the current block (shrink policy; e for the slide policy), [3] rows m, [4] accepted length a,
 * [5 .. 5+m) the block tokens z, [5+64 .. 5+64+m) the predictions (row k predicts output
 * position e+k+1); other entries are unspecified. Errors: ERR_ARG, ERR_OOM. */
#define CLLM_TRACE_STRIDE (5 + 2 * 64)
cllm_status cllm_trace_enable(cllm_ctx *ctx, int32_t enable);

/* Copies up to cap records of the last decode of slot seq that ran with recording on into
 * records[cap * CLLM_TRACE_STRIDE] (caller-owned host memory); *n_records = the number that
 * decode wrote (0 if it ran without recording). Synchronous. Errors: ERR_ARG, ERR_DEVICE. */
cllm_status cllm_trace_read(cllm_ctx *ctx, int32_t seq, int32_t *records, int64_t cap, int64_t *n_records);

/* Counts over a recorded trajectory (host computation, no context): the fast-forward count of
 * an iteration is its accepted length (it includes the token that is right without fast
 * forwarding); output position q is stationary when, in some iteration t0 before the one that
 * accepts q, q lies past the next pending position (q >= e + a + 1) and its prediction equals
 * tokens[q] (the decode's output) in every iteration from t0 until q is accepted. windows =
 * blocks of the shrink policy (block_policy 0) or ceil(n_tokens / n) n-token windows of the
 * slide policy (1). Errors: ERR_ARG for null pointers, n outside [1, 64], an unknown policy
 * or records inconsistent with n_tokens. */
typedef struct {
    int64_t iterations;
    double fast_forward_mean;
    int64_t stationary;
    int64_t windows;
    double stationary_per_window;
} cllm_trace_stats;
cllm_status cllm_trace_count(const int32_t *records, int64_t n_records, const int32_t *tokens, int64_t n_tokens,
                             int32_t n, int32_t block_policy, cllm_trace_stats *out);

/* Jacobi trajectory collection with data augmentation (the paper's Algorithm 1, Section 3.2.1),
 * from the records of one decode with the shrink block policy and its output tokens (host
 * computation, no context). For every block (first output position b0, size nb <= n) the
 * trajectory holds the block's full state at each iteration (the tokens already fixed in the
 * block, then the iteration's block z) and finally the fixed point tokens[b0 .. b0+nb). State
 * number s (counted from 0 over the whole collection) goes to states[s*n ..] and, with false
 * tokens corrected at random, to augmented[s*n ..]: position i with a token different from the
 * fixed point's takes the fixed point's token when the top 53 bits of the SplitMix64 draw
 * mix(mix(mix(seed) ^ s) ^ i) are below rate * 2^53 (mix: SplitMix64's output function).
 * Entries past nb are -1; block_start[s] = b0. At most cap states are written (caller-owned
 * host arrays of cap*n, cap*n and cap int32); *n_states = the number the collection holds.
 * Errors: ERR_ARG for null pointers, n outside [1, 64], rate outside [0, 1], or records that
 * are not a shrink-policy trajectory of these tokens. */
cllm_status cllm_collect_states(const int32_t *records, int64_t n_records, const int32_t *tokens, int64_t n_tokens,
                                int32_t n, double rate, uint64_t seed, int32_t *states, int32_t *augmented,
                                int32_t *block_start, int64_t cap, int64_t *n_states);

/* CLLM training loss at the LM head (Section 3.2.2: global consistency loss with the forward
 * KL, eq. global_loss, plus omega times the AR loss, eq. ar_loss), forward then backward, on the
 * context's LM-head weights W [V][d]. Inputs are LM-head input rows (after the final RMSNorm),
 * fp32 host arrays: teacher[n_pairs][d] (conditioned on the fixed point y*; the stop-gradient
 * model, so no gradient flows through them), student[n_pairs][d] (conditioned on a trajectory
 * state y at the same positions), ar_rows[n_ar][d] with ar_targets[n_ar] in [0, V) (the target
 * model's generation). Per pair KL(softmax(W teacher) || softmax(W student)) -> row_kl[n_pairs];
 * per AR row -log softmax(W ar)[target] -> row_nll[n_ar]; *loss = sum row_kl + omega * sum
 * row_nll (sums; the expectation's normalisation is the caller's). Gradients of *loss:
 * d_student[n_pairs][d], d_ar[n_ar][d] and, when d_weight is not NULL, d_weight[V][d] (fp32,
 * through the student and AR rows). Logits and reductions in fp32 (the products as in the
 * decode: bf16 weights, activations in hi + lo bf16 planes), every sum in a fixed order.
 * Synchronous; the context keeps a workspace (grown on demand) until it is freed. Errors:
 * ERR_ARG (n_pairs + n_ar outside [1, 64], null arrays, target out of range), ERR_STATE (no
 * weights), ERR_OOM, ERR_DEVICE. */
cllm_status cllm_loss_head(cllm_ctx *ctx, const float *teacher, const float *student, int32_t n_pairs,
                           const float *ar_rows, const int32_t *ar_targets, int32_t n_ar, float omega, float *row_kl,
                           float *row_nll, float *d_student, float *d_ar, float *d_weight, double *loss);

/* cllm_loss_head on device arrays, for a training loop whose rows and gradients stay in HBM:
 * the same arguments, computation and results (bit for bit), but every array (rows, targets,
 * row_kl, row_nll, d_student, d_ar, d_weight, and loss, a device double) is memory the context's
 * GPU can access: its device memory, managed or pinned host memory; each is checked and anything
 * else is ERR_ARG. The work is enqueued on the context's stream and the call returns without
 * waiting: results are ready when that stream reaches this point; the caller keeps the inputs
 * alive and unmodified until then. loss may be NULL (no total). Sizes are not checked beyond the
 * row counts: each array must hold its rows. A target outside [0, V) cannot be checked on the
 * host here: that AR row's row_nll and gradient row, and every d_weight entry it reaches, are
 * NaN. Calls on one context share its workspace and must be ordered by its stream. The first
 * call after the weights are set also builds the LM head's transposed copy (Vp x d elements of
 * workspace, kept until the context is freed); a call with more rows than any before grows the
 * workspace, and freeing the old buffers waits for the device. Errors: ERR_ARG (n_pairs + n_ar
 * outside [1, 64], null or inaccessible arrays), ERR_STATE, ERR_OOM (workspace growth, the only
 * allocation), ERR_DEVICE. */
cllm_status cllm_loss_head_device(cllm_ctx *ctx, const float *teacher, const float *student, int32_t n_pairs,
                                  const float *ar_rows, const int32_t *ar_targets, int32_t n_ar, float omega,
                                  float *row_kl, float *row_nll, float *d_student, float *d_ar, float *d_weight,
                                  double *loss);

/* LM-head input rows of an iteration over block[0..m) at the slot's committed length L, without
 * a commit: row k = RMSNorm(x_k) (.) g_final of the last layer's residual row (fp32; the rows
 * whose products with the LM head give the next-token logits after z[0..k]). These are the rows
 * the training loss of Section 3.2.2 takes: for a trajectory state y and its fixed point y* of
 * one n-token block, rows 0..n-2 over y are the student rows and over y* the teacher rows (and,
 * the fixed point being the greedy generation, also the AR rows with targets y*[1..n)). block[0]
 * may be any token (the loss conditions on each state as given). The KV rows L..L+m-1 are
 * written provisionally (as by a Jacobi step) and nothing else of the slot changes.
 * rows_out: caller-owned host array of m x d_model floats. Synchronous. Errors: ERR_ARG (m
 * outside [1, max_block], ids out of range, NULL), ERR_STATE (slot not prefilled),
 * ERR_CAPACITY (L + m > max_ctx), ERR_OOM, ERR_DEVICE. */
cllm_status cllm_hidden_rows(cllm_ctx *ctx, int32_t seq, const int32_t *block, int32_t m, float *rows_out);

/* cllm_hidden_rows without any allocation, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * arguments, kernels and results (bit for bit), but the staging rows live in a fixed device array
 * of the library (64 x 8192 floats = 2 MiB per GPU, held until the process ends) instead
 * of a context buffer grown by hipMalloc; the call makes no hipMalloc, hipFree or other
 * allocating call. Every call on one GPU, from any context, uses that GPU's one array: calls that
 * overlap on one GPU (two host threads, or contexts on different streams) race and must be
 * serialised by the caller. Errors: those of cllm_hidden_rows, ERR_CAPACITY (m x d_model above
 * the array), ERR_STATE (no array address for the context's device). */
cllm_status cllm_hidden_rows_noalloc(cllm_ctx *ctx, int32_t seq, const int32_t *block, int32_t m, float *rows_out);

/* Committed length L and pending token of a sequence slot. Errors: ERR_ARG, ERR_STATE. */
cllm_status cllm_seq_state(const cllm_ctx *ctx, int32_t seq, int32_t *committed_len, int32_t *pending);

/* Kernel timing for measurement: kernel_class selects one class of kernels (CLLM_KT_*
 * below); while enabled, launches of that class are bracketed by HIP events on the context's
 * stream. max_rows > 0 restricts timing to launches sized for that many rows (the kernels are
 * instantiated for 16, 32 or 64 rows per row tile: max_rows = n times the Jacobi iterations of
 * blocks of n when n <= 32); 0 times every launch. Launches of a prefill are never timed.
 * every >= 1 samples: one of every `every` eligible launches is timed (each bracket costs a
 * few microseconds of queue time; a stride coprime with the layer count rotates the sample over
 * the layers). cllm_timing_read returns the number of timed launches and their total device
 * time since the last enable, and clears them. kernel_class < 0 disables. The loss head's
 * launches (classes CLLM_KT_LOSS_*) are timed whatever max_rows. Errors: ERR_ARG for an unknown
 * class, max_rows outside [0, 64] or every < 1. */
#define CLLM_KT_GEMM_QKV 0
#define CLLM_KT_ATTN 1
#define CLLM_KT_GEMM_O 2
#define CLLM_KT_GEMM_GATE_UP 3
#define CLLM_KT_GEMM_DOWN 4
#define CLLM_KT_LM_HEAD 5
#define CLLM_KT_SCAN 6
#define CLLM_KT_ATTN_COMBINE 7
#define CLLM_KT_EMBED 8
#define CLLM_KT_LOSS_LOGITS 9   /* loss head: logits GEMM */
#define CLLM_KT_LOSS_ROWS 10    /* loss head: per-row losses and logit gradients */
#define CLLM_KT_LOSS_DH 11      /* loss head: gradient of the input rows */
#define CLLM_KT_LOSS_DW 12      /* loss head: gradient of the LM-head weight */
cllm_status cllm_timing_enable(cllm_ctx *ctx, int32_t kernel_class, int32_t max_rows, int32_t every);
cllm_status cllm_timing_read(cllm_ctx *ctx, int64_t *launches, double *total_ms);

/* Bytes of weights streamed by one forward pass (all matrices except the embedding), after
 * padding to the kernels' tiles. */
int64_t cllm_streamed_weight_bytes(const cllm_ctx *ctx);

const char *cllm_status_string(cllm_status s);
const char *cllm_last_error(const cllm_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* CLLM_H */
