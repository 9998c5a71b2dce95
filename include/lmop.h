/*
 * lmop.h - C ABI of the LM-operator row-evaluation library (gfx950 / MI355X).
 *
 * The library evaluates one quantised decoder LM over every row of a table,
 * the row-wise LM function of the paper (Sec. 2.3.2 "llmmap": for each row,
 * the row's values v1..vk and the question Q form one prompt and the LM
 * returns f(Q, v1..vk)), with the return type enforced by constrained
 * decoding (Sec. 2.3 "Constrained Decoding": a declared return_type or an
 * `options` set restricts what may be generated).  The prompt's shared part
 * (instruction, type instructions, one-shot example, question: Appendix
 * "Prompts") is a *prefix* whose keys/values are computed once and reused by
 * every row (the serving setup enables prefix caching, Appendix "vLLM
 * Config"); each row contributes only its own suffix tokens.  Identical rows
 * are evaluated once (Sec. 2.4 "Early Deduplication of Database Values").
 * Joins are LLMMap over DB-built pairs (Sec. 4.1, ecomm self-join example):
 * a child prefix extends a root prefix with the left value, rows hold the
 * right value.  Weights are W4A16 (Sec. 3.2, Table "tab:models"): int4 with
 * one fp16 scale per 32 input features; embeddings and LM head are fp16.
 *
 * Conventions for every call:
 *  - Every call returns lmop_status; nothing throws across the ABI.  On
 *    error, lmop_last_error(ctx) describes the cause until the next call on
 *    that ctx, and output buffers are left unspecified.
 *  - A ctx is not thread-safe; use one ctx per host thread and stream.
 *  - The caller owns every pointer it passes and may free it when the call
 *    returns.  The library owns its device memory (weights, prefix KV,
 *    scratch) and frees it in lmop_release_prefix / lmop_destroy; scratch
 *    comes from a caller-supplied workspace instead once lmop_set_workspace
 *    has given one.
 *  - LMOP_ERR_DEVICE is sticky: after a HIP error the ctx refuses further
 *    work and must be destroyed.  For tests of that rule, the environment
 *    variable LMOP_INJECT_LAUNCH_FAILURE=<kernel name>:<n>, read by
 *    lmop_create, makes the n-th launch of that kernel on the ctx fail as a
 *    HIP launch error would, without launching it.
 *  - All calls are synchronous with respect to the host: when they return,
 *    their device work on the ctx stream has completed, also when they
 *    return an error.
 */
#ifndef LMOP_H
#define LMOP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LMOP_OK = 0,
  LMOP_ERR_INVALID_ARG = -1, /* a bad pointer, size, token id, layout or handle      */
  LMOP_ERR_STATE = -2,       /* call out of order (e.g. eval before load_weights)     */
  LMOP_ERR_OOM = -3,         /* a device or host allocation failed                    */
  LMOP_ERR_DEVICE = -4,      /* a HIP call failed; sticky, the ctx must be destroyed  */
  LMOP_ERR_UNSUPPORTED = -5  /* a model shape or option the library does not handle   */
} lmop_status;

typedef struct lmop_ctx lmop_ctx;       /* opaque */
typedef struct lmop_prefix lmop_prefix; /* opaque; owned by its ctx */

/* Decoder shape (Llama-style: RMSNorm, rotate-half RoPE, grouped-query
 * attention, SwiGLU MLP; no biases).  Supported: head_dim 64 or 128,
 * n_heads % n_kv_heads == 0, d_model % 64 == 0, group_size 32. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab, group_size;
  float rms_eps, rope_theta;
  int32_t max_seq; /* longest prefix + suffix + generated tokens; 0 = 4096, at most 2^20 */
} lmop_config;

/* Creates a ctx on HIP device `device` whose work runs on `hip_stream`
 * (a hipStream_t; NULL = the library creates its own blocking stream, which
 * is ordered after work on the null stream).  Device memory the caller
 * passes (on_device weights, a workspace) is read in the ctx stream's order:
 * work still writing it on another stream must be finished or ordered
 * before the call (on the ctx's stream or the null stream).  device = -1 creates
 * a host-only ctx: every argument check runs, but calls that would touch a
 * GPU return LMOP_ERR_UNSUPPORTED after validation.  On failure *out is NULL
 * and lmop_last_error(NULL) describes the cause (per host thread). */
lmop_status lmop_create(const lmop_config* cfg, int32_t device, void* hip_stream, lmop_ctx** out);
void lmop_destroy(lmop_ctx* ctx); /* frees everything, including live prefixes; NULL is a no-op */
const char* lmop_last_error(const lmop_ctx* ctx);
const char* lmop_status_string(lmop_status s);

/* Formats of the linear maps' weights (lmop_weights.format). */
#define LMOP_W_INT4_G32 0u /* W4A16: int4 codes, one fp16 scale per 32 input features (Sec. 3.2) */
#define LMOP_W_FP8_E4M3 1u /* FP8 checkpoints: OCP E4M3 codes, one fp32 scale per output row   */

/* One linear map y = x W^T with W [n][k].
 * LMOP_W_INT4_G32:
 *   qweight uint8 [n][kp/2], kp = k rounded up to 32: feature j is the low
 *     nibble of byte j/2 when j is even, the high nibble when j is odd; each
 *     nibble is a two's-complement int4 in [-8, 7]; pad features hold 0.
 *   scales  fp16 bit patterns [n][kp/32]: W[r][j] = q[r][j] * scales[r][j/32].
 * LMOP_W_FP8_E4M3:
 *   qweight uint8 [n][k]: OCP FP8 E4M3 codes (the "fn" variant: largest 448,
 *     no infinities; NaN codes are not allowed);
 *   scales  fp32 [n]: W[r][j] = e4m3(q[r][j]) * scales[r].
 * Activations stay fp16 in both (weight-only quantisation). */
typedef struct {
  const uint8_t* qweight;
  const void* scales;
  int32_t n, k;
} lmop_qmat;

typedef struct {
  const float* attn_norm; /* fp32 [d_model] RMSNorm gain before attention */
  const float* mlp_norm;  /* fp32 [d_model] RMSNorm gain before the MLP   */
  lmop_qmat wq;           /* [n_heads*head_dim][d_model]    */
  lmop_qmat wk, wv;       /* [n_kv_heads*head_dim][d_model] */
  lmop_qmat wo;           /* [d_model][n_heads*head_dim]    */
  lmop_qmat w_gate, w_up; /* [d_ff][d_model]                */
  lmop_qmat w_down;       /* [d_model][d_ff]                */
} lmop_layer;

typedef struct {
  const uint16_t* tok_embedding; /* fp16 [vocab][d_model] */
  const uint16_t* lm_head;       /* fp16 [vocab][d_model] */
  const float* final_norm;       /* fp32 [d_model]        */
  const lmop_layer* layers;      /* host array [n_layers] (always host memory) */
  int32_t n_layers;
  int32_t on_device; /* 0: the tensor pointers are host memory; 1: device memory on the ctx's device */
  int32_t format;    /* LMOP_W_INT4_G32 or LMOP_W_FP8_E4M3, for all seven maps of every layer */
} lmop_weights;

/* Copies the weights to the device and repacks them into the kernels'
 * tiled layout (fusing q/k/v and gate/up).  May be called again to replace
 * the weights; existing prefixes are then invalid and are released. */
lmop_status lmop_load_weights(lmop_ctx* ctx, const lmop_weights* w);

/* Computes and keeps the keys/values of a shared prompt prefix (the
 * instruction part of the LLMMap prompt, Appendix "Prompts").  parent ==
 * NULL makes a root; otherwise the prefix continues its parent's sequence
 * (positions continue, attention sees the parent's tokens) - the two-level
 * reuse of a join, root = instruction, child = instruction + left value.
 * A child's parent must be a root.  tokens: host int32 [n_tokens], n_tokens
 * >= 1, ids in [0, vocab).  The parent must stay alive while children or
 * rows use it (release order is free; a released parent lives on until its
 * last child is released). */
lmop_status lmop_set_prefix(lmop_ctx* ctx, const lmop_prefix* parent, const int32_t* tokens,
                            int32_t n_tokens, lmop_prefix** out);

/* Computes n prefixes with the same parent in one batched pass: prefix i
 * holds tokens[offsets[i] .. offsets[i+1]) (host CSR, offsets[0] = 0, every
 * prefix at least one token).  The result equals n calls of
 * lmop_set_prefix, bit for bit; it is the form a join needs, one child
 * (instruction + left value) per left value.  The n prefixes share one
 * device allocation, freed when the last of them is released; each is
 * released on its own.  n == 0 does nothing.  out: host [n]; on failure no
 * prefix is created and out is all NULL. */
lmop_status lmop_set_prefixes(lmop_ctx* ctx, const lmop_prefix* parent, const int32_t* tokens,
                              const int64_t* offsets, int32_t n, lmop_prefix** out);
lmop_status lmop_release_prefix(lmop_ctx* ctx, lmop_prefix* prefix);
/* Total sequence length of a prefix (ancestors included); -1 for NULL. */
int32_t lmop_prefix_length(const lmop_prefix* prefix);

/* Return types (Sec. 2.3 "Constrained Decoding"; `options`, Sec. 2.3.2 Example 4). */
typedef enum {
  LMOP_BOOL = 0, /* tokens = {false_token, true_token}; value 0/1                        */
  LMOP_ENUM = 1, /* tokens[i] = single-token option i; value = option index              */
  LMOP_INT = 2,  /* tokens[d] = token of digit d (n_tokens = 10), eos_token ends the
                    number; a digit string of at most max_tokens tokens (EOS included),
                    no EOS at the first step; value = decimal value of the digits       */
  LMOP_AUTOMATON = 3 /* multi-token outputs (option strings as a token trie, lists,
                    other regular types): the steps follow a token automaton            */
} lmop_kind;

/* A token automaton (Sec. 2.3 "Constrained Decoding": option strings and
 * other structured return types decoded token by token under a grammar).
 * State 0 starts.  State s has the edges edge_token[e] -> edge_next[e] for
 * e in [edge_offset[s], edge_offset[s+1]); accepting[s] != 0 lets an output
 * end in s.  A step in state s allows s's edge tokens, ordered by where
 * each token first appears in edge_token (this order breaks ties), and,
 * when s is accepting and eos_token >= 0, the EOS token last.  The output
 * ends on EOS, on reaching an accepting state without edges, or after
 * max_tokens tokens; value = the final state, or -1 if that state is not
 * accepting.  Limits: n_states in 1..65536; edges in 1..2^20; state 0 and
 * every non-accepting state have edges; a state's edge tokens are distinct
 * ids in [0, vocab); EOS is none of the edge tokens; the distinct edge
 * tokens plus EOS number at most 4096.  All arrays are host memory. */
typedef struct {
  int32_t n_states;
  const int32_t* edge_offset; /* [n_states + 1], edge_offset[0] = 0, non-decreasing */
  const int32_t* edge_token;  /* [edge_offset[n_states]] */
  const int32_t* edge_next;   /* [edge_offset[n_states]], in [0, n_states) */
  const uint8_t* accepting;   /* [n_states] */
} lmop_automaton;

typedef struct {
  int32_t kind;          /* lmop_kind */
  const int32_t* tokens; /* host [n_tokens], distinct ids in [0, vocab); AUTOMATON: unused */
  int32_t n_tokens;      /* BOOL: 2; ENUM: 1..4096; INT: 10 */
  int32_t eos_token;     /* INT: not one of the digit tokens; AUTOMATON: -1 (none) or the
                            token that ends an output in an accepting state */
  int32_t max_tokens;    /* INT, AUTOMATON: 1..8; BOOL/ENUM: ignored (1) */
  const lmop_automaton* automaton; /* AUTOMATON only */
} lmop_type;

typedef struct {
  int64_t value;      /* BOOL 0/1; ENUM option index; INT decimal value; AUTOMATON final
                         state (-1: cut off by max_tokens in a non-accepting state)        */
  float logprob;      /* sum over steps of log-softmax over that step's allowed tokens       */
  float logprob_full; /* sum over steps of log-softmax over the whole vocabulary; NaN with
                         LMOP_HEAD_RESTRICTED                                              */
  int32_t n_tokens;   /* tokens generated (EOS included)                                   */
  int32_t tokens[8];  /* generated token ids; unused entries are -1                         */
} lmop_result;

#define LMOP_NO_DEDUP 1u /* evaluate duplicate rows separately (results are identical) */
/* Restricted head: the constrained step (Sec. 2.3, "Constrained Decoding")
 * needs only the logits of the type's allowed tokens for its value and for
 * `logprob`; with this flag the library computes just those (|A| dot
 * products per row instead of the full vocabulary), `logprob_full` is NaN,
 * and debug_logits holds the allowed tokens' logits with NaN elsewhere. */
#define LMOP_HEAD_RESTRICTED 2u

typedef struct {
  uint32_t flags;           /* LMOP_NO_DEDUP | LMOP_HEAD_RESTRICTED                       */
  int32_t max_batch_tokens; /* suffix tokens per device batch; 0 = library default (16384),
                               larger values are capped at 2^21                           */
  float* debug_logits;      /* NULL or host fp32 [n_rows][max_steps][vocab]: the logits of
                               each step (max_steps = max_tokens for INT and AUTOMATON,
                               else 1); steps a row did not take are NaN                  */
  int32_t limit;            /* early exit for LIMIT queries (Sec. 2.4): 0 = evaluate every
                               row; k > 0 = rows are evaluated in table order and the call
                               stops once k rows have value == limit_value (see below)    */
  int64_t limit_value;      /* the value a row must have to count toward `limit`          */
  const uint8_t* row_mask;  /* NULL or host [n_rows]: cascade filtering (Sec. 2.4) - only
                               rows with row_mask[r] != 0 are evaluated (e.g. the rows an
                               earlier predicate kept); the others are skipped           */
} lmop_eval_opts;

/* With limit = k > 0 every row up to and including the k-th row (in table
 * order) whose value is limit_value is evaluated, as without a limit, bit
 * for bit; rows after it may be skipped.  If fewer than k rows qualify,
 * every row is evaluated.  Rows are then batched in table order, not
 * grouped by prefix.  A skipped row (by the limit or the row mask) gets
 * value -1, n_tokens 0, NaN log-probabilities, tokens -1 (and NaN debug
 * logits).  An evaluated row's result does not depend on which other rows
 * are evaluated. */

/* Evaluates the LM function on every row: row r's sequence is
 * prefix(r) ++ tokens[offsets[r] .. offsets[r+1]), where prefix(r) =
 * row_prefix[r] if row_prefix != NULL else `prefix` (either may be NULL =
 * no prefix).  tokens/offsets: host CSR, offsets[0] = 0, non-decreasing,
 * offsets[n_rows] = total.  A row with an empty suffix takes its answer from
 * the prefix's last position; a row with neither is INVALID_ARG.  Writes
 * out[r] (host) for every row.  n_rows = 0 is a no-op. */
lmop_status lmop_eval_rows(lmop_ctx* ctx, const lmop_prefix* prefix,
                           const lmop_prefix* const* row_prefix, const int32_t* tokens,
                           const int64_t* offsets, int32_t n_rows, const lmop_type* type,
                           lmop_result* out, const lmop_eval_opts* opts);

/* Scratch for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation):
 * lmop_eval_rows with every scratch buffer (activations, head partials, the
 * own-KV store of a batch or decode group) in the library's static device
 * array of LMOP_NOALLOC_SCRATCH_BYTES, one per GPU, held from the first
 * lmop_create on that GPU until the process ends.  The call makes no device,
 * pinned-host or event allocation and no memset (it clears what must start at
 * zero with a kernel); batches are sized to fit the array.  Results equal
 * lmop_eval_rows bit for bit.  Weights and prefixes must already be loaded
 * and set (those calls allocate).  Kernel timing (lmop_set_profiling) counts
 * its launches but times only those for which released events are at hand.
 * Every call on one GPU, from any ctx, shares that GPU's array: calls that
 * overlap on one GPU (two host threads, two ctxs) race and must be
 * serialised by the caller.  LMOP_ERR_OOM (with the sizes in
 * lmop_last_error) if the scratch of a batch holding the longest row, or the
 * type's tables, exceed the array; otherwise as lmop_eval_rows. */
#define LMOP_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)
lmop_status lmop_eval_rows_noalloc(lmop_ctx* ctx, const lmop_prefix* prefix,
                                   const lmop_prefix* const* row_prefix, const int32_t* tokens,
                                   const int64_t* offsets, int32_t n_rows, const lmop_type* type,
                                   lmop_result* out, const lmop_eval_opts* opts);

/* A caller-supplied workspace.  The paper's serving setup caps the GPU
 * memory the LM may take (Appendix "vLLM Config", gpu_memory_utilization)
 * and runs on a 16 GB GPU (Sec. 3.2 Setup); a caller that owns the device
 * memory (e.g. a PyTorch allocation) hands the library one region instead of
 * letting it allocate scratch.  After lmop_set_workspace(ctx, p, bytes) with
 * p != NULL, every scratch buffer of lmop_set_prefix(es) and lmop_eval_rows
 * (activations, head partials, the own-KV store of a batch or integer decode
 * group) is carved from [p, p + bytes): the library frees the scratch it had
 * allocated, sizes batches and decode groups to fit (max_batch_tokens
 * becomes an upper bound), and a call fails with LMOP_ERR_OOM, the sizes in
 * lmop_last_error, when not even one row (or one prefix) fits.  Weights and
 * prefix KV stores remain the library's own allocations.  p: device memory
 * of the ctx's device, 256-byte aligned; the caller keeps ownership, keeps
 * it alive until the workspace is replaced or the ctx destroyed, and leaves
 * it alone while a call runs (its contents are scratch).  (NULL, 0) returns
 * to library-allocated scratch.  INVALID_ARG for a misaligned or non-device
 * pointer, or one of p, bytes zero without the other. */
lmop_status lmop_set_workspace(lmop_ctx* ctx, void* dev_ptr, size_t bytes);

/* What lmop_eval_rows would do with the same arguments, without doing it:
 * validation, deduplication and the batch / decode-group plan run, no device
 * work is queued and nothing is allocated (a host-only ctx plans as well).
 * For sizing a workspace against a memory cap (Sec. 3.2, Appendix "vLLM
 * Config").  The plan is the one the call would use now: against the
 * workspace if one is set, else against library-allocated scratch.
 * opts->debug_logits only counts as NULL or not (a non-NULL pointer plans
 * the scratch of the logit dump; nothing is written to it).  Errors as
 * lmop_eval_rows (LMOP_ERR_OOM if the workspace cannot hold one row);
 * INVALID_ARG if plan is NULL. */
typedef struct {
  int32_t unique_rows;      /* rows evaluated: distinct (prefix, suffix) rows the row mask keeps */
  int32_t batches;          /* forward passes of the rows' first step                     */
  int32_t batch_tokens;     /* token budget of a pass in this plan                        */
  int32_t max_batch_tokens; /* suffix tokens of the largest pass                          */
  int32_t decode_groups;    /* groups of passes decoded together (integer and automaton
                               types: every further step is one pass per group)           */
  int32_t pad_;
  uint64_t scratch_bytes;   /* device scratch of the plan, own-KV store included          */
  uint64_t own_kv_bytes;    /* of which the own-KV store (keys and values of the rows'
                               own tokens)                                                 */
  uint64_t min_workspace_bytes; /* the smallest workspace that runs the call (with the
                                   smallest batches and decode groups); one byte less is
                                   LMOP_ERR_OOM                                           */
} lmop_eval_plan;
lmop_status lmop_plan_rows(lmop_ctx* ctx, const lmop_prefix* prefix,
                           const lmop_prefix* const* row_prefix, const int32_t* tokens,
                           const int64_t* offsets, int32_t n_rows, const lmop_type* type,
                           const lmop_eval_opts* opts, lmop_eval_plan* plan);

/* Device memory accounting of a ctx (for the 16 GB budget of Sec. 3.2). */
typedef struct {
  uint64_t device_bytes;    /* device memory the library holds now (weights, prefix KV
                               stores, scratch it allocated itself)                      */
  uint64_t device_peak;     /* the most it has held at once since lmop_create             */
  uint64_t workspace_bytes; /* size of the caller's workspace (0: none)                   */
  uint64_t workspace_peak;  /* the most of the workspace one call has used since it was set */
} lmop_memory_stats;
lmop_status lmop_get_memory(const lmop_ctx* ctx, lmop_memory_stats* out);

/* Early deduplication (Sec. 2.4): rows with equal (key, suffix) get the
 * same representative, the first such row.  keys: NULL or host [n_rows]
 * (e.g. a prefix id per row).  rep[r] = index of r's representative;
 * *n_unique = number of distinct rows.  Host only; needs no ctx. */
lmop_status lmop_dedup_rows(const int32_t* tokens, const int64_t* offsets, int32_t n_rows,
                            const int64_t* keys, int32_t* rep, int32_t* n_unique);

/* Per-kernel timing of the ctx's launches while profiling is on (off by
 * default).  Every launch is counted; a systematic sample is timed with HIP
 * events on the ctx stream (the first, (N+1)-th, (2N+1)-th ... launch of
 * each kernel for period N).  total_ms, flops and bytes cover the timed
 * launches: their mean duration is total_ms / timed_launches. */
typedef struct {
  char name[48];
  int64_t launches;       /* all launches while profiling was on */
  int64_t timed_launches; /* the sampled ones */
  double total_ms;        /* summed over the timed launches */
  double flops;           /* algorithmic FLOPs of the timed launches */
  double bytes;           /* algorithmic HBM bytes of the timed launches */
} lmop_kernel_stat;

/* period 0 turns profiling off; period N >= 1 times every N-th launch of
 * each kernel (1: all).  Each timed launch adds two events to the stream, so
 * a period above 1 keeps the timing from slowing what it measures; a period
 * with no common factor with the layer count samples every layer.  Clears
 * the counters; INVALID_ARG for a negative period. */
lmop_status lmop_set_profiling(lmop_ctx* ctx, int32_t period);
lmop_status lmop_get_kernel_stats(lmop_ctx* ctx, lmop_kernel_stat* out, int32_t max_entries,
                                  int32_t* n_entries);

#ifdef __cplusplus
}
#endif
#endif /* LMOP_H */
