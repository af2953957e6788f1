/*
 * pard.h -- C ABI of the PARD parallel-draft speculative-decode engine
 * (hand-written HIP kernels for AMD Instinct MI355X, gfx950).
 *
 * The engine runs one speculative-decoding step as the paper states it:
 *   - drafting stage (Sec. 2.2; Sec. 3.1 eq. 7): the draft model makes ONE
 *     forward pass over the tokens it has not yet seen followed by K-1 copies of
 *     a shared mask token (Sec. 4.3, shared mask id) and proposes K candidates;
 *   - verification stage (Sec. 2.2): the target model scores the pending token
 *     and the K candidates in one forward pass; greedy decoding (Sec. 2.1 eq. 2)
 *     keeps the longest prefix of candidates that equals the target's argmax,
 *     plus one bonus token, and rolls the KV caches back to the accepted length.
 * Weights are generated on the device from a seed (no checkpoints); see
 * pard_model_load.
 *
 * Conventions for every call
 *   - Return value: PARD_OK (0) or a negative pard_status.  On error nothing in
 *     the context has changed and pard_last_error() describes the problem.
 *     Validation of arguments, state and capacity happens on the host before
 *     any device work.  Nothing aborts, prints or allocates device memory.
 *     The one exception is PARD_ERR_RANGE: activations and the KV cache are
 *     held in fp16, and a call whose passes produced a value fp16 cannot hold
 *     (|x| >= 65520, or NaN) runs to its end and then returns PARD_ERR_RANGE;
 *     its outputs and the caches of its sequences are invalid (prefill them
 *     again).  Weights whose activations stay within fp16's range never see it.
 *   - Host pointers (prompt, prefix, cand, outputs) are owned by the caller and
 *     are only accessed during the call.  Granular calls return after their
 *     outputs are valid (one device->host copy and a stream synchronisation).
 *   - Device memory: the caller provides one arena (pard_arena_bytes bytes,
 *     256-byte aligned) that must outlive the context; the library carves
 *     weights, KV caches, activations and workspaces out of it and never
 *     frees it.  All device work is enqueued on the caller's HIP stream.
 *   - Token ids must lie in [0, vocab).  0 <= K <= max_k <= 32.
 *   - A context is not thread-safe.
 */
#ifndef PARD_H
#define PARD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PARD_OK = 0,
  PARD_ERR_ARG = -1,         /* bad argument (null pointer, id out of range, bad shape) */
  PARD_ERR_STATE = -2,       /* call not valid in the current state (e.g. before prefill) */
  PARD_ERR_CAPACITY = -3,    /* would exceed max_ctx / max_k / max_batch */
  PARD_ERR_NOMEM = -4,       /* arena smaller than pard_arena_bytes() */
  PARD_ERR_DEVICE = -5,      /* a HIP runtime call failed */
  PARD_ERR_UNSUPPORTED = -6, /* valid request the library does not implement */
  PARD_ERR_RANGE = -7        /* the call ran, but an activation exceeded fp16's range (see below) */
} pard_status;

enum { PARD_F32 = 0, PARD_BF16 = 1 };
enum { PARD_TARGET = 0, PARD_DRAFT = 1 };
/* Drafting of the fused loop: PARD's one parallel pass over the pending tokens
 * and K-1 mask tokens (Sec. 3.1, eq. 7), or vanilla speculative decoding's K
 * sequential one-token draft passes (Sec. 2.1, eq. 3; the baseline PARD is
 * compared with). */
enum { PARD_MODE_PARALLEL = 0, PARD_MODE_VANILLA = 1 };

/* Shape and initialisation of one Llama-family decoder (Sec. 4.1 names
 * LLaMA3 and Qwen2.5 members).  Weights are drawn N(0, init_std^2) with the
 * counter-based generator below and rounded to bf16; RMSNorm gains are 1.
 * The device keeps each bf16 weight in fp16 encoding for its fp16 matrix
 * cores (the same value when |w| >= 2^-14; smaller weights round to fp16
 * subnormals, within 2^-25).  Q/K/V biases stay fp32 holding the bf16 value.
 * Constraints: d_model % 32 == 0, head_dim in {64, 128},
 * n_heads % n_kv_heads == 0, vocab % 16 == 0, dtype == PARD_BF16, and every
 * weight matrix (rows padded to 16, columns to 32) below 2 GiB in its 2-byte
 * encoding (UNSUPPORTED otherwise: the kernels address a matrix with 32-bit
 * byte offsets).
 *
 * Generator (both this library and the test inputs implement it):
 * SplitMix64 (Steele, Lea, Flood 2014) stream with state
 * mix64(seed * 2^20 + weight_stream * 2^16 + tensor), i-th output
 * mix64(state + (i + 1) * 0x9E3779B97F4A7C15); element i of a tensor in
 * canonical row-major [out, in] order takes the basic Box-Muller transform of
 * outputs 2*(i/2) and 2*(i/2)+1 (u1 = ((z0>>11)+1)*2^-53, u2 = (z1>>11)*2^-53,
 * cosine branch for even i, sine for odd i), times init_std, rounded to float32
 * then to bf16 (nearest, ties to even).  Tensor ordinals: embedding 0,
 * lm_head 1 (untied only), layer l: 16*(l+1) + {wq 0, wk 1, wv 2, wo 3,
 * w_gate 4, w_up 5, w_down 6, bq 7, bk 8, bv 9}. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rms_eps, rope_theta, init_std;
  int32_t qkv_bias;          /* 1: Q/K/V projections carry a bias (Qwen2.5 family) */
  int32_t tied_embeddings;   /* 1: lm_head is the embedding matrix */
  int32_t dtype;             /* PARD_BF16 */
  uint32_t weight_stream;    /* generator stream id (target 0, draft 1 by convention) */
  uint64_t seed;
  /* LLaMA-3.1-style rotary frequency scaling (rope_factor 0: plain RoPE).  A
   * frequency w = rope_theta^(-2i/head_dim) whose wavelength 2 pi / w is below
   * rope_original_max_pos / rope_high_freq_factor is kept, one above
   * rope_original_max_pos / rope_low_freq_factor is divided by rope_factor,
   * and in between w becomes (1 - s) w / rope_factor + s w with
   * s = (rope_original_max_pos * w / (2 pi) - low) / (high - low).  Requires
   * rope_factor >= 1, 0 < low < high, rope_original_max_pos >= 1 (ARG otherwise). */
  float rope_factor, rope_low_freq_factor, rope_high_freq_factor;
  int32_t rope_original_max_pos;
} pard_model_spec;

typedef struct pard_ctx pard_ctx;

/* Statistics of one pard_generate call.  The phase times follow the time
 * model of Sec. 2.2 (eqs. 3-4: a step costs the draft's forward passes plus
 * one target forward): they are read on the device from its constant-rate
 * clock at the pass boundaries of every step (the first kernel of a pass, the
 * end of its step tail), so they cover the whole call, graph replays
 * included.
 *   draft_ms  -- every draft pass, from its first kernel to the end of its
 *                tail (candidates stored, verify pass staged);
 *   verify_ms -- every target pass up to and including its lm_head (the
 *                verification forward and the per-tile argmax);
 *   accept_ms -- every verify tail: the vocab argmax reduction, greedy prefix
 *                acceptance (eq. 2), KV commit/rollback and the staging of the
 *                next draft pass.
 * step_ms_p50 / step_ms_p90: median and 90th percentile of the step latency,
 * the time between the ends of consecutive verify tails (0 with fewer than two
 * steps; the last 4096 steps of the call). */
typedef struct {
  int64_t steps;             /* draft+verify steps executed */
  int64_t tokens;            /* tokens written to out_tokens */
  double elapsed_ms;         /* device time between the first and last step */
  double draft_ms, verify_ms, accept_ms;
  double step_ms_p50, step_ms_p90;
  int64_t accept_hist[33];   /* accept_hist[a] = steps that accepted a candidates */
} pard_stats;

/* Bytes of device arena needed for a target/draft pair with the given
 * capacities; 0 if the specs or capacities are invalid.  Host-only. */
size_t pard_arena_bytes(const pard_model_spec *target, const pard_model_spec *draft,
                        int32_t max_batch, int32_t max_ctx, int32_t max_k);

/* Create a context: carve the arena, generate both models' weights on the
 * device, build rotary tables.  target->vocab must equal draft->vocab;
 * mask_id in [0, vocab) is the shared mask token of the draft (Sec. 4.3).
 * max_ctx bounds every sequence's KV length (prompt + generated + 2*max_k).
 * hip_stream is a hipStream_t (NULL = the default stream).
 * Errors: ARG (bad spec/pointer), UNSUPPORTED (constraint above),
 * NOMEM (arena_bytes too small), DEVICE. */
pard_status pard_model_load(const pard_model_spec *target, const pard_model_spec *draft,
                            int32_t mask_id, int32_t max_batch, int32_t max_ctx, int32_t max_k,
                            void *dev_arena, size_t arena_bytes, void *hip_stream,
                            pard_ctx **out);

/* Prefill sequence slot `seq` (Sec. 2.1): both models ingest the n prompt
 * tokens (their KV lengths become n) and the target's greedy argmax after the
 * prompt is returned in *first_token.  That token is "pending": it is in
 * neither cache and is the first row of the next draft and verify passes.
 * Re-prefilling a slot discards its previous contents.
 * Errors: ARG, CAPACITY (n + 2*max_k + 1 > max_ctx, seq >= max_batch), DEVICE. */
pard_status pard_prefill(pard_ctx *ctx, int32_t seq, const int32_t *prompt, int32_t n,
                         int32_t *first_token);

/* Drafting stage, Sec. 3.1 eq. 7.  `prefix` is the whole committed sequence
 * (prompt and every generated token, ending with the latest pending token).
 * The draft ingests prefix[L_d : n_prefix] followed by K-1 mask tokens in one
 * forward pass (if L_d >= n_prefix it first truncates to n_prefix-1, so at
 * least the last token is re-read) and writes cand[k] = argmax of the row
 * that reads the last real token (k = 0) or mask k-1 (k >= 1), k < K.
 * Afterwards L_d = n_prefix: mask rows are never committed.  K = 1 is an
 * ordinary draft decode step.  Errors: ARG (1 <= K <= max_k, ids), STATE
 * (slot not prefilled), CAPACITY, DEVICE. */
pard_status pard_draft(pard_ctx *ctx, int32_t seq, const int32_t *prefix, int32_t n_prefix,
                       int32_t K, int32_t *cand);

/* Verification stage, Sec. 2.2 with greedy acceptance (eq. 2).  The target
 * runs [pending, cand[0..K-1]] at positions L_t .. L_t+K; with t_j its
 * argmax at row j, *n_accepted = a = the largest j with cand[i] == t_i for all
 * i < j, *bonus = t_a.  The target cache keeps a+1 rows (L_t += a+1), the
 * bonus becomes the pending token.  K = 0 is a plain greedy target step.
 * Errors: ARG, STATE, CAPACITY, DEVICE. */
pard_status pard_verify(pard_ctx *ctx, int32_t seq, const int32_t *cand, int32_t K,
                        int32_t *n_accepted, int32_t *bonus);

/* Roll the KV cache of `which` (PARD_TARGET / PARD_DRAFT) back to new_len
 * (0 <= new_len <= current length).  This is the rollback of Sec. 2.2's
 * verification stage (candidates the target does not accept are dropped, so
 * their cache rows are discarded) on a static, preallocated KV cache (the
 * setting of App. F): O(1), a length update; later passes overwrite the
 * dropped rows.  pard_verify already rolls the target back by itself; this
 * call serves rewinds and tests.  For the target, the token history the
 * library keeps is cut to the first new_len tokens and the pending token is
 * kept.  Errors: ARG (bad which, new_len outside [0, length]), STATE (slot
 * not prefilled), CAPACITY (seq outside [0, max_batch)), DEVICE. */
pard_status pard_kv_truncate(pard_ctx *ctx, int32_t seq, int32_t which, int32_t new_len);

/* Current committed KV length of `which` for slot `seq`. */
pard_status pard_kv_len(const pard_ctx *ctx, int32_t seq, int32_t which, int32_t *len);

/* Fused device-resident loop (Sec. 2.2: draft stage, verification stage) over
 * the n_seq slots seqs[0..n_seq) (distinct, prefilled): repeated draft (one
 * pass) -> verify -> accept steps with no host round trip per step.  With
 * n_seq > 1 every pass holds all unfinished slots' rows (per slot: its a+1
 * pending tokens and K-1 mask rows in the draft pass, K+1 rows in the verify
 * pass), each slot with its own positions, acceptance and KV rollback; a slot
 * that has its n_tokens leaves the batch.  Limits: n_seq <= min(max_batch,
 * 64); for n_seq > 1, n_seq*2K <= 512 and n_seq*(K+1) <= 512.
 * out_tokens is [n_seq][n_tokens] row-major: row i starts with slot seqs[i]'s
 * current pending token, then every step appends its accepted candidates and
 * bonus; exactly n_tokens tokens are written per slot (surplus tokens of the
 * last step are dropped).  max_steps > 0 caps the number of steps (then fewer
 * tokens may be written; stats->tokens is the total over the slots).  K = 0
 * runs plain greedy target steps.  stats may be NULL.
 * Errors: ARG (bad pointer, repeated slot), STATE (slot not prefilled),
 * CAPACITY (the KV would exceed max_ctx, too many slots or rows), DEVICE. */
pard_status pard_generate(pard_ctx *ctx, int32_t n_seq, const int32_t *seqs, int32_t K,
                          int32_t n_tokens, int32_t max_steps, int32_t *out_tokens,
                          pard_stats *stats);

/* pard_generate with an explicit drafting mode (PARD_MODE_PARALLEL: same as
 * pard_generate; PARD_MODE_VANILLA: each step runs K draft passes of one row
 * per slot, every pass feeding the previous candidate, then the same verify
 * pass; after verification the draft cache keeps the pending token and the
 * candidates that agree (eq. 3: T = K*T_draft + T_target per step).  Greedy
 * acceptance, outputs, limits and errors as pard_generate; ARG for an unknown
 * mode. */
pard_status pard_generate_ex(pard_ctx *ctx, int32_t n_seq, const int32_t *seqs, int32_t K,
                             int32_t mode, int32_t n_tokens, int32_t max_steps,
                             int32_t *out_tokens, pard_stats *stats);

/* Speculative sampling (Sec. 1 and Sec. 2.2: speculative decoding combined
 * with speculative sampling keeps the target's output distribution).  With
 * temperature T > 0 every later pard_prefill, pard_draft, pard_verify and
 * pard_generate samples instead of taking the argmax:
 *   - distributions are softmax(logits / T) of either model;
 *   - pard_prefill draws the first token from the target;
 *   - pard_draft draws candidate j+1 from the draft's row j (eq. 7 rows);
 *   - pard_verify keeps candidate x at position j iff u * q_j(x) < p_j(x)
 *     (p target, q draft), in order; at the first candidate not kept the
 *     step's last token is drawn from max(0, p_j - q_j) (normalised), if all
 *     K are kept from p_K; *n_accepted / *bonus report the kept count and
 *     that last token (K = 0: one token drawn from p_0).
 * Draws use the inverse CDF in token-id order.  The uniforms u come from a
 * SplitMix64 counter generator keyed by (seed, slot, the slot's verify steps
 * since its prefill, position, purpose), so results are reproducible and
 * independent of batching.  T = 0 restores greedy decoding (eq. 2).  Captured
 * step graphs are dropped (rebuilt on the next pard_generate).  With sampling,
 * pard_verify with K > 0 needs this slot's pard_draft of the same K since its
 * last verify (STATE otherwise), and PARD_MODE_VANILLA is UNSUPPORTED.
 * Errors: ARG (T negative, not finite, or in (0, 1e-3)), UNSUPPORTED (vocab above
 * 262144), DEVICE. */
pard_status pard_set_sampling(pard_ctx *ctx, float temperature, uint64_t seed);

/* Copy the fp32 logits of slot `seq`'s rows in the last lm_head pass of
 * `which` that included the slot (rows x vocab, row-major; draft rows are the
 * K candidate rows, target rows the verify rows, prefill the single
 * last-prompt row).  rows must not exceed that slot's rows.  A slot that left
 * a batched pard_generate has none until its next pass.  Parity/debug.
 * Errors: ARG, STATE, DEVICE. */
pard_status pard_read_logits(const pard_ctx *ctx, int32_t which, int32_t seq, float *out,
                             int32_t rows, int32_t vocab);

/* Read n consecutive canonical weight elements [row, col0 .. col0+n) of one
 * tensor (ordinal as in the generator comment; layer tensors use their layer's
 * ordinal) of model `which`, as float: the value the device stores (the bf16
 * weight in fp16 encoding).  Debug/parity of the generator and the on-device
 * weight layout.  Errors: ARG, DEVICE. */
pard_status pard_read_weight(const pard_ctx *ctx, int32_t which, int32_t tensor, int32_t row,
                             int32_t col0, int32_t n, float *out);

/* Per-kernel timer: HIP events around each launch of one kernel class
 * (class = which * 8 + op, op: 0 embed, 1 qkv, 2 attention (with its chunk
 * merge), 3 o-proj, 4 gate/up, 5 down, 6 lm_head, 7 argmax reduction and step
 * tail) on the context's stream, for up to max_launches launches after
 * enabling.  pard_timer_read synchronises the
 * stream and returns the number of timed launches and their summed duration.
 * kernel_class < 0 disables.  Errors: ARG, DEVICE. */
pard_status pard_timer_enable(pard_ctx *ctx, int32_t kernel_class, int32_t max_launches);
pard_status pard_timer_read(pard_ctx *ctx, int32_t *launches, double *total_ms);

/* COD training-data processing (Sec. 3.2 eqs. 9-11, Alg. 1, App. B): the
 * conditional drop-token data of PARD's mask-token training, on the device.
 * A sample of L tokens t_0..t_{L-1} has n = L-1 columns per subtask k = 1..K;
 * column j of subtask k is labelled t_{j+1} at position j, with input t_j
 * (k = 1) or mask_id (k >= 2).  Subtask 1 keeps every column.  Subtask k >= 2
 * keeps min(#valid, floor(n * gamma_k + 1/2)) columns, gamma_k =
 * max(r^(k-1), r_min) (float64), chosen among the valid ones -- j >= k-1 and
 * column j-1 of subtask k-1 kept, so every kept token's context is kept --
 * by the smallest (key, j), key = top 24 bits of output j of the SplitMix64
 * stream seeded with output k of the stream seeded with output s (the sample
 * index) of the stream seeded with `seed`.  Kept columns are packed in
 * subtask order, each in column order.  Packed token (k, j) attends to the
 * real tokens t_0..t_{j-k+1} and to the packed tokens (k', j-k+k'),
 * 2 <= k' <= k (its diagonal up to itself): the context of eq. 8.
 *
 * pard_cod_capacity: packed rows a sample of n_tokens tokens may need
 * (n + sum_{k>=2} floor(n * gamma_k + 1/2)); -1 if n_tokens is outside
 * [2, 8193] or K (1..64), r (0, 1] or r_min [0, 1] is invalid.  Host only.
 *
 * pard_cod_build: tokens (device, int32) holds the samples back to back;
 * tok_offsets (host, n_samples+1 entries) their bounds; out_offsets (host,
 * n_samples+1) the bounds of each sample's packed region in the five device
 * output arrays (ids, labels, positions, subtask k, column j; int32), each
 * region at least pard_cod_capacity of its sample; out_len (device,
 * n_samples) receives each sample's packed length; workspace (device, at
 * least pard_cod_workspace_bytes(n_samples) bytes, 256-byte aligned) holds the
 * device copy of both offset arrays during the call.  Runs on hip_stream and
 * returns after the results are complete.  The caller owns every buffer; the
 * call allocates no device memory.
 * Errors: ARG (null pointer, bad parameters, a sample outside [2, 8193]
 * tokens, misaligned workspace), CAPACITY (an output region below its
 * capacity), NOMEM (workspace too small), DEVICE. */
int64_t pard_cod_capacity(int32_t n_tokens, int32_t K, double r, double r_min);
/* pard_cod_layout: out_offsets (host, n_samples+1) = the prefix sums of the
 * samples' capacities for tok_offsets (host, n_samples+1); returns the total,
 * or -1 under the same conditions as pard_cod_capacity.  Host only. */
int64_t pard_cod_layout(const int64_t *tok_offsets, int32_t n_samples, int32_t K, double r,
                        double r_min, int64_t *out_offsets);
/* pard_cod_workspace_bytes: device workspace pard_cod_build needs for
 * n_samples samples (0 if n_samples < 1).  Host only. */
size_t pard_cod_workspace_bytes(int32_t n_samples);
/* kernel_ms (host, may be NULL) receives the kernel's device time, from HIP
 * events recorded around its launch on hip_stream. */
pard_status pard_cod_build(const int32_t *tokens, const int64_t *tok_offsets, int32_t n_samples,
                           int32_t K, double r, double r_min, int32_t mask_id, uint64_t seed,
                           const int64_t *out_offsets, int32_t *out_ids, int32_t *out_labels,
                           int32_t *out_pos, int32_t *out_section, int32_t *out_column,
                           int32_t *out_len, void *workspace, size_t workspace_bytes,
                           float *kernel_ms, void *hip_stream);

/* pard_cod_build without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc).  The device copy of the two offset arrays
 * lives in a fixed scratch array that the library holds on every GPU it runs
 * on (1 MiB each, until the process ends), so n_samples is limited to
 * PARD_COD_NOALLOC_MAX_SAMPLES (CAPACITY above it, before any device work).
 * The call allocates no device memory and reports no kernel time; the current
 * device must be the one hip_stream belongs to (the scratch of that device is
 * used; its address is looked up on the first call on each device).  Every
 * call on a GPU shares that GPU's scratch: calls that overlap on one GPU (other
 * threads, other streams) race and must be serialised by the caller.  Nothing
 * in the scratch needs clearing: each call writes both arrays before its
 * kernel reads them.  Other arguments, outputs and errors as pard_cod_build. */
#define PARD_COD_NOALLOC_MAX_SAMPLES 65535
pard_status pard_cod_build_noalloc(const int32_t *tokens, const int64_t *tok_offsets, int32_t n_samples,
                                   int32_t K, double r, double r_min, int32_t mask_id, uint64_t seed,
                                   const int64_t *out_offsets, int32_t *out_ids, int32_t *out_labels,
                                   int32_t *out_pos, int32_t *out_section, int32_t *out_column,
                                   int32_t *out_len, void *hip_stream);

/* Message of the last error on this context (never NULL; "" if none). */
const char *pard_last_error(const pard_ctx *ctx);

/* Static name of a status code. */
const char *pard_status_string(pard_status status);

/* Destroy a context (the arena stays owned by the caller).  NULL is allowed. */
void pard_free(pard_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* PARD_H */
