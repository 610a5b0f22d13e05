/*
 * dsi.h -- C ABI of the MI355X verification step of distributed speculative
 * inference (DSI, arXiv 2405.14105).
 *
 * The paper's data-parallel step (Section 2, "Speculative Inference"): a
 * drafter proposes k tokens; the target model receives the k+1 prompts
 * x'_{<=i}, i = 0..k, as ONE batch, computes their k+1 logit rows, and from
 * them emits between 1 and k+1 tokens with a lossless accept/reject rule.
 * Each target server keeps its own KV cache and synchronises at every
 * rejection (Section 3.1, "KV cache").  DSI's orchestration of many such
 * verification tasks (Algorithm 1, speculation parallelism) is host-level
 * work above this ABI; on one GPU, concurrent verification tasks are a batch
 * of independent windows.
 *
 * Conventions
 *  - All functions return dsi_status; no C++ exception crosses the ABI.  On
 *    error, dsi_last_error() returns a thread-local message.
 *  - Host-side validation runs before anything is enqueued: a call that
 *    returns an error has no side effects.
 *  - Pointers named d_* are device pointers owned by the caller; the library
 *    never keeps them past the call.  The library owns weights, KV buffers
 *    and its own workspaces.
 *  - Work is enqueued on the stream given to dsi_model_create (a hipStream_t,
 *    NULL = the null stream) and is asynchronous unless stated otherwise.
 *  - Data-dependent errors found on the device (a token id outside [0, V),
 *    q(d) not positive and finite, an invalid token-tree parent) make the affected window output
 *    n = -1, token = -1, leave its KV length unchanged, and make the next
 *    synchronising call (dsi_sync, dsi_kv_length) return DSI_EINVAL.
 *  - A dsi_model's weights are immutable after they are set and the model
 *    may serve several dsi_kv; calls on one model (and its KV caches) must
 *    not overlap: the model's forward workspaces are shared by all of them.
 */
#ifndef DSI_H
#define DSI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DSI_OK = 0,
  DSI_EINVAL = 1,     /* invalid argument, or a device-detected input error */
  DSI_ENOMEM = 2,     /* device allocation failed */
  DSI_EHIP = 3,       /* HIP runtime error */
  DSI_ECAPACITY = 4,  /* the KV cache of a window would overflow max_len */
  DSI_ESTATE = 5      /* call out of order (e.g. a tensor was never set) */
} dsi_status;

typedef enum { DSI_F32 = 0, DSI_BF16 = 1 } dsi_dtype;

/* Verification rule.
 * DSI_SAMPLE: lossless rejection sampling -- accept d_i iff u_i < p_i(d_i)/q_i(d_i);
 *   after the first rejection draw from norm(max(0, p - q)), after k
 *   acceptances draw the bonus token from p_{k+1} (the rule the paper adopts
 *   from its cited works, Sections 2 and 3.1).
 * DSI_GREEDY: exact match against the target's argmax (Algorithm 1, the
 *   terminate / j* steps), ties to the lowest token id. */
typedef enum { DSI_SAMPLE = 0, DSI_GREEDY = 1 } dsi_mode;

/* Decoder shape.  The paper treats the target LM as a black box
 * (Appendix B); this library implements a Llama-style decoder: pre-norm
 * RMSNorm, rotate-half RoPE, causal GQA attention (query head h reads KV
 * head h / (n_heads / n_kv_heads)), SwiGLU FFN, final RMSNorm, untied head.
 * Requirements: head_dim a multiple of 32 and at most 128; d_model a
 * multiple of 32; n_heads a multiple of n_kv_heads. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab;
  float rope_base;   /* e.g. 10000 */
  float rms_eps;     /* e.g. 1e-5 */
  int32_t wdtype;    /* dsi_dtype of every weight tensor */
  int32_t kvdtype;   /* dsi_dtype of the KV cache */
} dsi_config;

typedef struct dsi_model dsi_model;  /* opaque, library-owned */
typedef struct dsi_kv dsi_kv;        /* opaque, library-owned */

/* Tensor ids for dsi_model_set_tensor.  Matrices are [out, in] row-major in
 * the model's wdtype (bf16 as raw uint16 bit patterns); norm gains are [d].
 *   global (layer = -1): EMBED [V, d], FINAL_NORM [d], LM_HEAD [V, d]
 *   per layer: ATTN_NORM [d], WQ [n_heads*hd, d], WK/WV [n_kv_heads*hd, d],
 *              WO [d, n_heads*hd], FFN_NORM [d], W_GATE/W_UP [d_ff, d],
 *              W_DOWN [d, d_ff] */
enum {
  DSI_T_EMBED = 0, DSI_T_FINAL_NORM = 1, DSI_T_LM_HEAD = 2,
  DSI_T_ATTN_NORM = 3, DSI_T_WQ = 4, DSI_T_WK = 5, DSI_T_WV = 6, DSI_T_WO = 7,
  DSI_T_FFN_NORM = 8, DSI_T_W_GATE = 9, DSI_T_W_UP = 10, DSI_T_W_DOWN = 11
};

/* Largest number of window rows B*(k+1) one dsi_verify / dsi_accept call
 * may carry. */
#define DSI_MAX_ROWS 64

/* Create a model with device storage for every weight (zero until set).
 * stream: hipStream_t used by every call on this model and its KV caches.
 * With a non-null stream, dsi_verify records its launches into a HIP graph
 * the first time it sees a combination of arguments (pointers, sizes, mode,
 * cache) and replays that graph on later calls with the same combination
 * (up to 16 are cached per model; the environment variable DSI_GRAPHS=0
 * read here disables this).  Results are identical either way. */
dsi_status dsi_model_create(const dsi_config* cfg, void* stream, dsi_model** out);

/* Upload one tensor (host memory if src_on_device == 0, else device memory).
 * nbytes must equal the tensor's element count times the wdtype size.
 * Matrices are re-laid out on the device into the library's streaming tile
 * order.  Synchronous with respect to the host. */
dsi_status dsi_model_set_tensor(dsi_model* m, int32_t layer, int32_t tensor_id,
                                const void* src, size_t nbytes, int32_t src_on_device);

/* Frees the model.  Any dsi_kv created from it must be destroyed first. */
dsi_status dsi_model_destroy(dsi_model* m);

/* KV cache for n_windows independent windows of up to max_len positions each
 * (the per-server cache of Section 3.1, one per concurrent verification
 * task).  Lengths start at 0 and live on the device. */
dsi_status dsi_kv_create(dsi_model* m, int32_t n_windows, int32_t max_len, dsi_kv** out);
dsi_status dsi_kv_destroy(dsi_kv* kv);

/* Append n prompt tokens (d_tokens [n], device) to a window: runs the target
 * over them in chunks, writes their K/V, and advances the window length by n.
 * This builds the committed prefix a target server keeps in its own KV cache
 * (Section 3.1, "KV cache"): the prompt x of the target's next-token model
 * f(x) (Appendix B, the unpadded prompt with positions from 0), and also
 * tokens a server must catch up on before verifying (committed tokens or the
 * drafts a task builds on).  d_last_logits (nullable, device [V] fp32)
 * receives the logits of the last token.  Fails with DSI_ECAPACITY if
 * length + n may exceed max_len, with no side effects.  The tokens run in
 * chunks of DSI_MAX_ROWS; a chunk holding an id outside [0, V) does not
 * advance the length and is reported by the next synchronising call
 * (DSI_EINVAL).  Stream-ordered; d_tokens is caller-owned and only read by
 * the call's stream work. */
dsi_status dsi_prefill(dsi_model* m, dsi_kv* kv, int32_t window, const int32_t* d_tokens,
                       int32_t n, float* d_last_logits);

/* One batched verification of n_windows windows window0 .. window0+B-1.
 * Window b has cached length L_b; its k+1 rows are (w0, d_1..d_k) at
 * positions L_b .. L_b+k, where w0 is the last committed token that is not
 * yet cached.  Row i attends to positions [0, L_b + i].
 *   d_tokens [B][k+1] int32: w0, d_1..d_k
 *   d_q      [B][k][V] fp32: drafter distributions q_1..q_k (sample mode;
 *            may be NULL in greedy mode).  Used as given, not renormalised.
 *   d_u      [B][k+1] fp32 in [0,1): u_1..u_k for acceptance, u_{k+1} for the
 *            single residual/bonus draw (sample mode; NULL in greedy mode)
 *   temperature > 0: p = softmax(z / temperature) (ignored in greedy mode)
 *   commit: if nonzero, window lengths become L_b + n_b + 1 (w0 and the
 *            accepted drafts stay cached; rows of rejected drafts are dead)
 *   d_logits_out (nullable) [B*(k+1)][V] fp32: the target logits
 *   d_hidden_out (nullable, diagnostics) [n_layers+1][B*(k+1)][d_model] fp32:
 *            the residual stream entering each layer and entering the head
 * Outputs (device): d_n_accepted [B] = n_b in [0, k] and d_next_token [B] =
 * the correction (n_b < k) or bonus (n_b = k) token; the window emits
 * d_1..d_{n_b}, next_token (Section 2: between 1 and k+1 tokens).
 * Numerics: fp32-accurate activations against bf16 weights, KV stored in
 * kvdtype, fp32 logits, fp64 accept/reject arithmetic. */
typedef struct {
  int32_t window0, n_windows, k;
  const int32_t* d_tokens;
  const float* d_q;
  const float* d_u;
  float temperature;
  int32_t mode;      /* dsi_mode */
  int32_t commit;
  float* d_logits_out;
  float* d_hidden_out;
} dsi_verify_args;

dsi_status dsi_verify(dsi_model* m, dsi_kv* kv, const dsi_verify_args* args,
                      int32_t* d_n_accepted, int32_t* d_next_token);

/* Token-tree verification with the exact-match rule (Algorithm 1: one
 * thread per drafter on every prefix, the terminate step, and the j* step
 * that keeps the smallest-index drafter among those that agree with the
 * target).  Each of the n_windows windows carries a tree of n_nodes nodes:
 * node 0 is w0 (the last committed token, not yet cached), node i > 0 is a
 * draft continuing node parent[i] (0 <= parent[i] < i; children of one node
 * are numbered in drafter order).  One target forward computes every node's
 * next-token logits: node i sits at cache slot L_b + i with RoPE position
 * L_b + depth(i) and attends to the prefix [0, L_b) and to its ancestors'
 * slots and its own.  The accepted path starts at the root and repeatedly
 * moves to the smallest-index child whose token equals the target's argmax
 * (ties to the lowest id) at the current node; n = its number of moves.
 *   d_tokens [B][n_nodes] int32: node tokens (node 0 = w0)
 *   d_parent [B][n_nodes] int32: parent[0] = -1, else in [0, i)
 *   commit: if nonzero, the path's K/V rows are moved to slots L_b+1..L_b+n
 *           and the window length becomes L_b + n + 1, as if w0 and the
 *           accepted drafts had been verified as one chain
 *   d_logits_out (nullable) [B*n_nodes][V] fp32: every node's target logits
 * Outputs (device): d_path [B][n_nodes] = the accepted nodes (0, a_1..a_n),
 * -1 beyond; d_n_accepted [B] = n; d_next_token [B] = the target's argmax at
 * node a_n.  A parent array that breaks the rule above or a token outside
 * [0, V) gives n = -1, token = -1, path all -1, leaves the length unchanged,
 * and makes the next synchronising call return DSI_EINVAL.  n_windows *
 * n_nodes <= DSI_MAX_ROWS; graph replay as for dsi_verify. */
typedef struct {
  int32_t window0, n_windows, n_nodes;
  const int32_t* d_tokens;
  const int32_t* d_parent;
  int32_t commit;
  float* d_logits_out;
} dsi_tree_args;

dsi_status dsi_verify_tree(dsi_model* m, dsi_kv* kv, const dsi_tree_args* args, int32_t* d_path,
                           int32_t* d_n_accepted, int32_t* d_next_token);

/* Draft k tokens for one window with a drafter model that shares the
 * target's vocabulary (Section 2: the drafter proposes the lookahead tokens
 * one at a time, each sampled from its own next-token distribution given the
 * context and the drafts before it).  The drafter's cache for `window` holds
 * the context it has seen (length L_d).
 *   d_feed [n_feed] int32: tokens the drafter has not seen yet, 1..DSI_MAX_ROWS
 *            of them (the last committed token w0, preceded after a fully
 *            accepted window by the last draft), cached at L_d ..
 *   d_u    [k] fp32 in [0,1): one uniform per draft
 *   temperature > 0
 * Outputs (device): d_tokens [k+1] = (w0, d_1..d_k), the window dsi_verify
 * takes; d_q [k][V] fp32, row i = the drafter distribution of d_{i+1}:
 * softmax(z / temperature) computed in fp64 and stored in fp32, and d_{i+1}
 * is drawn from that stored row by inverse CDF: the smallest t with
 * sum_{v<=t} q_v > u_i * sum_v q_v (sums in fp64, ascending ids), else the
 * last t with q_t > 0.  The drafter caches the feed and d_1..d_{k-1}: its
 * length becomes L_d + n_feed + k - 1.  After the target accepts n drafts,
 * roll the drafter back to keep w0, d_1..d_min(n, k-1) and feed the emitted
 * token (preceded by d_k when n = k) to the next call.  Stream-ordered;
 * feed ids outside [0, V) are reported by the next synchronising call
 * (DSI_EINVAL) as for dsi_prefill. */
dsi_status dsi_draft(dsi_model* drafter, dsi_kv* kv, int32_t window, const int32_t* d_feed,
                     int32_t n_feed, int32_t k, const float* d_u, float temperature,
                     int32_t* d_tokens, float* d_q);

/* The accept/reject step alone, on caller-provided logits
 * d_logits [B*(k+1)][V] fp32 (window-major rows); other arguments as in
 * dsi_verify.  Uses a library workspace on the current device; calls that
 * overlap on one device must be serialised by the caller. */
dsi_status dsi_accept(void* stream, int32_t n_windows, int32_t k, int32_t vocab,
                      const float* d_logits, const int32_t* d_tokens, const float* d_q,
                      const float* d_u, float temperature, int32_t mode,
                      int32_t* d_n_accepted, int32_t* d_next_token);

/* dsi_accept without any device allocation, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments, kernels and results as
 * dsi_accept (n and the token equal dsi_accept's on the same inputs).  Its
 * workspace is one fixed device array of DSI_ACCEPT_NOALLOC_BYTES per device
 * (256 bytes of it the error word), held from the first call on a device
 * until the process ends; no hipMalloc/hipFree is called.  A call whose
 * n_windows*(k+1) rows and vocabulary need more workspace than the array
 * holds fails with DSI_ECAPACITY before anything is enqueued (128256-entry
 * vocabularies fit at the 64-row maximum).  Every call on a device shares
 * that device's array: calls that overlap on one device (other streams,
 * other threads) race and must be serialised by the caller. */
#define DSI_ACCEPT_NOALLOC_BYTES (256 * 1024)
dsi_status dsi_accept_noalloc(void* stream, int32_t n_windows, int32_t k, int32_t vocab,
                              const float* d_logits, const int32_t* d_tokens, const float* d_q,
                              const float* d_u, float temperature, int32_t mode,
                              int32_t* d_n_accepted, int32_t* d_next_token);

/* Roll a window back to new_len (DSI terminates the threads that built on a
 * rejected token, Algorithm 1; their cache rows become dead).  Stream-ordered;
 * new_len must be >= 0 and not above the window's current length (checked on
 * the device: otherwise the length is unchanged and the next synchronising
 * call returns DSI_EINVAL). */
dsi_status dsi_kv_rollback(dsi_kv* kv, int32_t window, int32_t new_len);

/* Fill the dead rows of one window -- positions [length, capacity) of K and
 * V in every layer, the length being the device's when the fill runs -- with
 * NaN.  Stream-ordered.  After a rollback this turns any read of a dead row
 * (Section 3.1, "KV cache": rows of terminated threads) into NaN logits, so
 * tests can show that no kernel lets such rows reach a result.  Rows are
 * rewritten before they are read again by prefill and verification.
 * Diagnostics and tests only. */
dsi_status dsi_kv_poison(dsi_kv* kv, int32_t window);

/* Current length of a window.  Synchronises the stream. */
dsi_status dsi_kv_length(dsi_kv* kv, int32_t window, int32_t* len);

/* Synchronise the model's stream and report device-detected input errors
 * (DSI_EINVAL, clearing them) or DSI_OK. */
dsi_status dsi_sync(dsi_model* m);

/* Copy positions [0, len) of one window and layer out of (export) or into
 * (import) the cache, as K [n_kv_heads][len][head_dim] and
 * V [n_kv_heads][len][head_dim] in kvdtype.  d_k / d_v are device buffers.
 * Diagnostics and tests only; stream-ordered.  Import does not change the
 * window length. */
dsi_status dsi_kv_export(dsi_kv* kv, int32_t window, int32_t layer, int32_t len,
                         void* d_k, void* d_v);
dsi_status dsi_kv_import(dsi_kv* kv, int32_t window, int32_t layer, int32_t len,
                         const void* d_k, const void* d_v);

/* Set a window's length directly (after dsi_kv_import).  Stream-ordered. */
dsi_status dsi_kv_set_length(dsi_kv* kv, int32_t window, int32_t len);

/* Diagnostics: kernel classes of one verification step. */
enum {
  DSI_K_QKV = 1,     /* fused QKV projection + RoPE + KV append (one per layer) */
  DSI_K_ATTN = 2,    /* window attention + chunk combine (two launches per layer) */
  DSI_K_OPROJ = 3,   /* output projection + residual */
  DSI_K_GATEUP = 4,  /* gate/up projection + SwiGLU */
  DSI_K_DOWN = 5,    /* down projection + residual */
  DSI_K_HEAD = 6,    /* final RMSNorm pack + LM head */
  DSI_K_VERIFY = 7   /* accept/reject kernels */
};

/* Record a HIP event pair on the model's stream around every launch of one
 * kernel class until dsi_profile_end, which synchronises the stream and
 * returns the number of timed launches and their summed duration.  Adds a
 * little host and stream overhead; not for the timed path. */
dsi_status dsi_profile_begin(dsi_model* m, int32_t kernel_class);
dsi_status dsi_profile_end(dsi_model* m, int32_t* launches, double* total_ms);

/* Time one GEMM kernel class (DSI_K_QKV, DSI_K_OPROJ, DSI_K_GATEUP,
 * DSI_K_DOWN or DSI_K_HEAD) in isolation: `rounds` rounds, each launching
 * that GEMM once per layer (once for the head) back to back on the model's
 * stream with the row count and windows of the most recent dsi_verify,
 * between one pair of HIP events.  Every launch streams its own layer's
 * weights from HBM.  The launches read the library's current activation
 * workspace and overwrite workspace outputs and dead KV rows beyond the
 * committed lengths only.  Returns the number of launches and their average
 * duration; synchronises the stream.  Diagnostics only. */
dsi_status dsi_profile_kernel(dsi_model* m, dsi_kv* kv, int32_t kernel_class, int32_t rounds,
                              int32_t* launches, double* avg_ms);

/* Streaming read rate of the GPU (diagnostics; no model involved): the
 * ceiling the GEMM weight streams and long-prefix attention are measured
 * against.  Reads `bytes` of the caller's device buffer d_buf (16-byte
 * aligned) as `slices` equal slices, one slice per launch in turn (slices
 * whose sum exceeds the 256 MB Infinity Cache make every launch read HBM),
 * `rounds` launches after one warm-up launch, between one pair of HIP events
 * on the null stream of the current device.  A launch has `workgroups`
 * workgroups (0: 256, one per CU; at most 4096) of 8 waves; each wave reads
 * a contiguous run with 8 loads of 1 KB in flight, nontemporal when
 * `nontemporal` is nonzero.  d_sink: caller-owned device memory of at least
 * 16 bytes, written only if the data XORs to a fixed pattern.  Returns the
 * bytes one launch reads (each slice rounded down to whole 8 KB runs per
 * wave) and the average launch duration; synchronises.  DSI_EINVAL for null
 * pointers, a misaligned buffer, rounds < 1, slices < 1, workgroups outside
 * 0..4096 or slices too small for 16 MiB and an 8 KB run per wave; DSI_EHIP
 * if a launch or event fails. */
dsi_status dsi_profile_stream(const void* d_buf, uint64_t bytes, int32_t slices, int32_t nontemporal,
                              int32_t workgroups, int32_t rounds, void* d_sink, uint64_t* bytes_per_launch,
                              double* avg_ms);

/* Thread-local description of the last error. */
const char* dsi_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DSI_H */
