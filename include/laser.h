/*
 * laser.h -- C ABI of liblaser.so, the MI355X (gfx950) decode + confidence-probe
 * hot path of LASER (load-aware early exit for reasoning LLMs).
 *
 * The paper (Section 3.1, Eq. 1-2) splits a reasoning request into chain-of-thought
 * chunks separated by action transition points (ATPs).  Generating the chunks is a
 * token-by-token decode; at each ATP an answer-inducing suffix makes the model emit a
 * trial answer whose confidence, computed from the token probabilities, is compared
 * with a threshold.  LASER's contribution (Section 4) is to make that threshold and a
 * per-request budget depend on the serving load.  This library provides:
 *
 *   laser_decode_step        one greedy decode token per request over a paged KV cache
 *   laser_probe_confidence   the trial-answer probe, returning confidence and argmax ids
 *   laser_step_mixed         decode for a batch plus probe chunks for a subset, one forward
 *   laser_kv_fork, laser_forward, laser_confidence
 *                            the pieces of a probe that rides along with later decode steps
 *   laser_exit_decision      the host-side ATP decision (Eq. 5 threshold, Algorithm 1)
 *   laser_budget             the budget pre-allocation of Eq. 6-8
 *   laser_atp_match          device-side ATP detection (token-set membership)
 *   laser_simulate           the paper's serving evaluation: one FIFO server, Poisson or
 *                            phased arrivals, per-request inference time from Eq. 2
 *
 * Conventions for every function:
 *   - The return value is a laser_status; LASER_OK (0) on success, a negative code on
 *     failure.  No C++ exception, abort or exit crosses the ABI.  After a failure,
 *     laser_last_error() returns a message for the calling thread.
 *   - Arguments are validated before anything is mutated: a failing call leaves every
 *     handle, page table and device buffer as it was.
 *   - Pointers named d_* are device pointers on the model's GPU; every other pointer
 *     is host memory.  All device memory (weights, workspace, KV pools, block table,
 *     outputs) is allocated by the caller and only borrowed: the library never frees
 *     caller memory.  Handles are owned by the caller through create/destroy.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).  Device
 *     work is asynchronous on that stream; outputs are valid after the stream is
 *     synchronised.  Host bookkeeping (lengths, page tables) is updated before the call
 *     returns.
 *   - Calls on one model or KV handle must not overlap (no internal locking).
 */
#ifndef LASER_H
#define LASER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LASER_ABI_VERSION 3

typedef enum {
  LASER_OK = 0,
  LASER_ERR_INVALID_ARG = -1,   /* NULL/out-of-range argument, unknown name, wrong size */
  LASER_ERR_OUT_OF_PAGES = -2,  /* page pool cannot satisfy an allocation (nothing changed) */
  LASER_ERR_HIP = -3,           /* a HIP runtime call failed; message from hipGetErrorString */
  LASER_ERR_UNSUPPORTED = -4,   /* shape or size outside what the kernels handle */
  LASER_ERR_STATE = -5          /* call out of order (e.g. before finalize, destroyed handle) */
} laser_status;

typedef enum { LASER_DTYPE_F32 = 0, LASER_DTYPE_BF16 = 1, LASER_DTYPE_FP8_E4M3 = 2 } laser_dtype;

/* Message of the last failing call on this thread ("" if none).  Owned by the library. */
const char* laser_last_error(void);
int laser_abi_version(void);

/* ========================================================================== */
/* Host controller (Section 4).  Pure host arithmetic, no device access.       */
/* ========================================================================== */

/* Hyper-parameters.  Defaults (laser_params_default) are the paper's: Section 5.1
 * (lambda_base .95, L_target 10, beta .04, gamma 1, alpha .3, B_base 10, lambda_min .88,
 * lambda_max .97, B_min 2) and Section 4.3 (f_min .6, f_max 1.5, p_min 50, p_max 275). */
typedef struct {
  double lambda_base, beta, gamma, alpha, L_target, lambda_min, lambda_max;
  int B_base, B_min;
  double f_min, f_max;
  int p_min, p_max;
} laser_params;

/* The one scalar of controller state (Section 4.4): the EMA-smoothed load L_bar,
 * initialised to 0 (Algorithm 1). */
typedef struct {
  double L_bar;
} laser_load_state;

enum { LASER_CONTINUE = 0, LASER_EARLY_EXIT = 1, LASER_BUDGET_EXHAUSTED = 2 };

void laser_params_default(laser_params* p);

/* EMA update of Section 4.2: L_bar <- alpha * active_requests + (1 - alpha) * L_bar.
 * Errors: INVALID_ARG for NULL pointers, active_requests < 0 or alpha outside [0,1]. */
laser_status laser_ema_update(const laser_params* p, laser_load_state* state, int active_requests);

/* Eq. 5: lambda = lambda_base - beta * tanh(gamma * (L_bar - L_target) / L_target),
 * clamped to [lambda_min, lambda_max].  Errors: INVALID_ARG for NULL, L_target <= 0 or
 * lambda_min > lambda_max. */
laser_status laser_threshold(const laser_params* p, double L_bar, double* lambda_out);

/* Eq. 6-8: B = max(B_min, floor(B_base * f_diff(prompt_len) * f_load(active_requests))),
 * f_diff = clip(f_min + (prompt_len - p_min)/(p_max - p_min) * (f_max - f_min), f_min, f_max),
 * f_load = min(1, L_target / max(1, active_requests)).  The floor is of the exact value:
 * the product is formed in double precision and floored with a 1e-9 guard against
 * representation error of the decimal parameters.  Errors: INVALID_ARG for NULL,
 * prompt_len < 0, active_requests < 0, p_max <= p_min, B_min < 1. */
laser_status laser_budget(const laser_params* p, int prompt_len, int active_requests, int* B_out);

/* The decision after the probe at ATP k_done+1 of a request with budget B_i
 * (Algorithm 1 loop body): update L_bar with active_requests (the EMA above), compute
 * lambda (Eq. 5), then EARLY_EXIT if confidence > lambda (strict, Section 3.1);
 * otherwise the failed-probe count becomes k_done+1 and the decision is
 * BUDGET_EXHAUSTED if that reaches B_i (force the conclusion), else CONTINUE.
 * lambda_out may be NULL.  Errors: INVALID_ARG for NULL state/decision_out, k_done < 0,
 * k_done >= B_i, or a NaN confidence; the state is not updated on error. */
laser_status laser_exit_decision(const laser_params* p, laser_load_state* state, float confidence,
                                 int active_requests, int k_done, int B_i, int* decision_out,
                                 double* lambda_out);

/* ========================================================================== */
/* Serving simulation (Section 5.1 evaluation setup)                          */
/* ========================================================================== */
/* Discrete-event simulation of one server that takes requests first come, first served,
 * as the paper evaluates serving.  Request i's latency is its queueing delay plus its
 * inference time (Eq. 1), and the inference time follows Eq. 2 from the request's
 * reasoning trace and a cost model:
 *   prefill(p) = prefill_ms + prefill_ms_per_token * p
 *   decoding n tokens from context c = n * decode_ms + decode_ms_per_ctx * (n*c + n(n-1)/2)
 *   a probe (trial answer + confidence) at context c = probe_ms + probe_ms_per_ctx * c.
 * A trace has K_i >= 1 reasoning chunks; an ATP follows every chunk but the last, whose end
 * closes the thinking phase.  At each ATP the methods that probe pay one probe and decide
 * as Algorithm 1 does (laser_exit_decision; the fixed-threshold methods compare with
 * fixed_lambda instead of Eq. 5).  The load L(t) is the number of requests in the system,
 * waiting or in service, at time t (arrivals at exactly t included): it feeds the EMA at
 * every probe (one global L_bar, starting at 0) and Eq. 8 at the start of service.  Probe
 * tokens do not stay in the context.  After the thinking phase the conclusion's tokens are
 * decoded from the context reached.
 * Methods (Section 5.1 baselines and the Section 5.4 ablation):
 *   VANILLA         no probes: every chunk, then the conclusion
 *   FIXED           probe at every ATP, exit when confidence > fixed_lambda
 *   LASER           Eq. 5 threshold and Eq. 6-8 budget
 *   THRESHOLD_ONLY  Eq. 5 threshold, no budget
 *   BUDGET_ONLY     fixed_lambda and the Eq. 6-8 budget
 *   NOTHINKING      no reasoning chunks: prefill, then the conclusion
 * max_probes (> 0) caps the probes of the methods without a budget (a step limit);
 * max_think_tokens (> 0) ends thinking once that many reasoning tokens are generated (the
 * chunk in progress is cut there, no probe follows, the conclusion is forced). */
enum {
  LASER_SIM_VANILLA = 0, LASER_SIM_FIXED = 1, LASER_SIM_LASER = 2,
  LASER_SIM_THRESHOLD_ONLY = 3, LASER_SIM_BUDGET_ONLY = 4, LASER_SIM_NOTHINKING = 5
};
/* outcome of a request */
enum {
  LASER_SIM_FINISHED = 0,   /* the last chunk ended the thinking phase */
  LASER_SIM_EXITED = 1,     /* confidence above the threshold at an ATP */
  LASER_SIM_EXHAUSTED = 2,  /* budget or probe cap reached: conclusion forced */
  LASER_SIM_CAPPED = 3,     /* max_think_tokens reached: conclusion forced */
  LASER_SIM_SKIPPED = 4     /* NOTHINKING */
};
typedef struct {
  int method;
  double fixed_lambda;
  int max_probes, max_think_tokens;
  double prefill_ms, prefill_ms_per_token;
  double decode_ms, decode_ms_per_ctx;
  double probe_ms, probe_ms_per_ctx;
  double slo_s; /* latency deadline of the SLO rate */
} laser_sim_config;
typedef struct {
  double arrival_s; /* non-decreasing over the requests */
  int32_t prompt_len, n_chunks, conclusion_tokens;
  int32_t nothink_correct; /* correctness of the answer without reasoning (NOTHINKING) */
} laser_sim_request;
typedef struct {
  double start_s, finish_s, latency_s;
  double lambda_last; /* threshold at the last probe; NaN without probes */
  int32_t budget;     /* B_i of the budgeted methods, else 0 */
  int32_t chunks;     /* reasoning chunks generated (a cut chunk counts) */
  int32_t probes, think_tokens, outcome, correct;
} laser_sim_result;
typedef struct {
  int32_t n;
  double mean_latency_s;
  double p95_latency_s;   /* nearest rank: the ceil(0.95 n)-th smallest latency */
  double throughput_qps;  /* n / (last finish - first arrival) */
  double slo_rate;        /* fraction with latency <= slo_s */
  double accuracy;        /* fraction answered correctly */
  double mean_tokens;     /* reasoning + conclusion tokens per request */
  double early_exit_rate; /* fraction with outcome EXITED */
} laser_sim_summary;
/* Simulates n requests.  The per-chunk arrays hold sum(n_chunks) entries, request after
 * request: chunk_tokens[c] >= 1; confidence[c] of the trial answer at the ATP after chunk
 * c (not read for a request's last chunk); correct[c] nonzero if the answer given after
 * chunk c is right (for the last chunk: the answer after full reasoning).  A request that
 * stops after chunk c is scored with correct[c].  out (n entries) and summary may be NULL.
 * Host only, O(total chunks + n log n).  Errors: INVALID_ARG for NULL required arrays,
 * n < 0, an unknown method, negative costs, decreasing arrivals, n_chunks < 1 (except
 * for NOTHINKING, which reads no chunks), chunk_tokens < 1, prompt_len or
 * conclusion_tokens < 0, NaN confidence, or invalid params (as laser_budget /
 * laser_threshold). */
laser_status laser_simulate(const laser_params* p, const laser_sim_config* cfg, int n, const laser_sim_request* req,
                            const int32_t* chunk_tokens, const float* confidence, const uint8_t* correct,
                            laser_sim_result* out, laser_sim_summary* summary);

/* ========================================================================== */
/* Page pool: host bookkeeping of the paged KV cache.                          */
/* ========================================================================== */
/* The paper serves from a vLLM-style engine (Section 4.2) without stating a paging
 * policy.  This pool hands out fixed-size pages by lowest free id; a page is taken when
 * a token lands at a length that is a multiple of page_size; a sequence added with a
 * length takes its pages in ascending id order; truncation returns the pages beyond the
 * kept length.  Every allocation is all-or-nothing (OUT_OF_PAGES leaves the pool as it
 * was).  Sequence ids are 0 <= seq_id < max_seqs.  A fork shares its source's full pages
 * (reference counted: a page returns to the pool when no sequence holds it) and takes a
 * fresh lowest-id page for a copy of the source's partial last page; a truncation that
 * would end inside a shared page is refused (INVALID_ARG). */
typedef struct laser_page_pool laser_page_pool;

laser_status laser_pages_create(int num_pages, int page_size, int max_seqs, int max_pages_per_seq,
                                laser_page_pool** out);
laser_status laser_pages_add_seq(laser_page_pool* pool, int seq_id, int length);
laser_status laser_pages_append(laser_page_pool* pool, int seq_id, int n_tokens);
laser_status laser_pages_truncate(laser_page_pool* pool, int seq_id, int length);
laser_status laser_pages_free_seq(laser_page_pool* pool, int seq_id);
/* dst_seq (a free slot) gets src_seq's length and contents as described above. */
laser_status laser_pages_fork(laser_page_pool* pool, int src_seq, int dst_seq);
/* Copies the page ids of seq_id (in sequence order) to out[0..n-1]; *n_out = n.
 * INVALID_ARG if cap < n. */
laser_status laser_pages_table(const laser_page_pool* pool, int seq_id, int32_t* out, int cap, int* n_out);
laser_status laser_pages_seq_len(const laser_page_pool* pool, int seq_id, int* len_out);
laser_status laser_pages_num_free(const laser_page_pool* pool, int* n_out);
laser_status laser_pages_destroy(laser_page_pool* pool);

/* ========================================================================== */
/* Model                                                                       */
/* ========================================================================== */
/* A Qwen2/Llama-style decoder: RMSNorm, grouped-query attention with rotary position
 * embedding on half-split pairs (i, i + head_dim/2) at angle pos * rope_theta^(-2i/head_dim),
 * SwiGLU MLP, final RMSNorm, LM head (the embedding when tied_embeddings).
 * Supported: head_dim in {64, 128}; n_q_heads a multiple of n_kv_heads with
 * G = n_q_heads/n_kv_heads <= 16; d_model a multiple of 64; d_ffn a multiple of 8;
 * n_q_heads*head_dim a multiple of 64; dtype F32 or BF16 for every tensor (and the KV
 * cache unless kv_dtype says FP8_E4M3); max_positions <= 65536. */
typedef struct {
  int n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, vocab;
  int tied_embeddings, qkv_bias, dtype;
  float rope_theta, rms_eps;
  int max_positions;
  /* KV-cache element type: 0 (or dtype) = the weights' type, or LASER_DTYPE_FP8_E4M3 (bf16
   * models only): the OCP FP8 E4M3 format (bias 7, largest finite 448, NaN 0x7f/0xff), each
   * new key and value rounded to nearest even and saturated at +-448, decoded exactly. */
  int kv_dtype;
} laser_model_desc;

typedef struct laser_model laser_model;

/* Creates a host handle (no device memory).  Binds to the current HIP device. */
laser_status laser_model_create(const laser_model_desc* desc, laser_model** out);

/* Borrows a device tensor (row-major, dtype of the model) for the model's lifetime.
 * Names: "embed" [vocab, d_model]; "lm_head" [vocab, d_model] (untied only);
 * "final_norm" [d_model]; per layer i, "layers.i.attn_norm" [d], "layers.i.wq"
 * [hq*hd, d], "layers.i.wk"/"layers.i.wv" [hkv*hd, d], "layers.i.bq" [hq*hd],
 * "layers.i.bk"/"layers.i.bv" [hkv*hd] (qkv_bias only), "layers.i.wo" [d, hq*hd],
 * "layers.i.mlp_norm" [d], "layers.i.w_gate"/"layers.i.w_up" [d_ffn, d],
 * "layers.i.w_down" [d, d_ffn].  INVALID_ARG for an unknown name or a byte size that
 * does not match; STATE after finalize. */
laser_status laser_model_set_tensor(laser_model* m, const char* name, const void* d_ptr, size_t bytes);

/* Bytes of device workspace the model needs for forwards of up to max_rows rows
 * (tokens per forward: batch for decode, S*batch for a probe chunk; 1..64). */
laser_status laser_workspace_size(const laser_model* m, int max_rows, size_t* bytes);

/* Checks that every tensor is set, lays out the caller's workspace (>= the size above
 * for max_rows) and fills its constant tables (RoPE cos/sin computed on the host in
 * double precision) with asynchronous copies on `stream`.  The workspace must stay
 * allocated until laser_model_destroy. */
laser_status laser_model_finalize(laser_model* m, int max_rows, void* d_workspace, size_t bytes, void* stream);
laser_status laser_model_destroy(laser_model* m);

/* Matrix-core weight tiles (optional).  Forwards of more than 2 rows (probe chunks, batches
 * of 3 or more, prompt prefill) run the projections on the matrix cores, whose operand takes
 * each 16-row group of a weight matrix as 64 lanes x 16 bytes per 32-column step: from a
 * row-major tensor that is 64 bytes of each of 16 rows per load instruction.  With tiles set,
 * those forwards read a copy of every projection and LM-head weight kept in that order
 * (group g, step s at block g * ceil(K/32) + s; 1 KB blocks, 2 KB for fp32; columns past K
 * are zero), so every load instruction reads 1 KB contiguously and each wave's K range is
 * contiguous.  The operands and the order of operations are the same, so results are the
 * same as without tiles.  laser_model_tile_bytes gives the buffer size (about the size of
 * the projection and LM-head weights); laser_model_set_tiles fills the caller's buffer on
 * `stream` from the model's tensors (after laser_model_finalize; the tensors must not change
 * afterwards) and switches the MFMA path to it; d_buf = NULL switches back to the row-major
 * tensors.  The buffer must stay allocated while tiles are on.  Forwards with at most 2 rows
 * always read the row-major tensors. */
laser_status laser_model_tile_bytes(const laser_model* m, size_t* bytes);
laser_status laser_model_set_tiles(laser_model* m, void* d_buf, size_t bytes, void* stream);

/* ========================================================================== */
/* KV cache: device pools + page pool                                          */
/* ========================================================================== */
/* Device layout (owned by the caller, laid out by the library): K and V pools of
 * n_layers x num_pages x n_kv_heads blocks; block (layer, page, kv_head) holds 16
 * positions x head_dim values in the order the attention kernel's matrix-core
 * operands read them: K element (t, d) at ((d/32*4 + (d%32)/8)*16 + t)*8 + d%8, V element
 * (t, d) at ((d/16*4 + t/4)*16 + d%16)*4 + t%4 (t = position within the page).  The
 * block table is int32 [max_seqs][max_pages_per_seq].  Page size is 16. */
typedef struct laser_kv laser_kv;

laser_status laser_kv_pool_bytes(const laser_model* m, int num_pages, size_t* bytes_per_pool);
laser_status laser_kv_create(const laser_model* m, int num_pages, int max_seqs, int max_pages_per_seq,
                             void* d_k_pool, void* d_v_pool, int32_t* d_block_table, laser_kv** out);
/* Adds seq_id with `length` positions already present (pages allocated, contents
 * undefined until imported).  OUT_OF_PAGES / INVALID_ARG leave the cache unchanged. */
laser_status laser_kv_add_seq(laser_kv* kv, int seq_id, int length);
/* Writes positions 0..length-1 of seq_id from d_k, d_v laid out [n_layers][length]
 * [n_kv_heads][head_dim] (KV-cache element type; keys already rotated).  length must equal the
 * sequence's length. */
laser_status laser_kv_import(laser_kv* kv, int seq_id, const void* d_k, const void* d_v, int length, void* stream);
/* Inverse of import: gathers all positions of seq_id into [n_layers][len][hkv][hd]. */
laser_status laser_kv_export(const laser_kv* kv, int seq_id, void* d_k, void* d_v, void* stream);
laser_status laser_kv_free_seq(laser_kv* kv, int seq_id);
/* Forks src_seq into the free slot dst_seq (page pool rules above): dst_seq starts with
 * src_seq's length and sees the same K/V; the partial last page, if any, is copied on
 * `stream` (all layers and kv heads).  Appending to either sequence afterwards never
 * touches the other's positions.  Used to run a probe beside the request's decode. */
laser_status laser_kv_fork(laser_kv* kv, int src_seq, int dst_seq, void* stream);
laser_status laser_kv_seq_len(const laser_kv* kv, int seq_id, int* len_out);
laser_status laser_kv_page_table(const laser_kv* kv, int seq_id, int32_t* out, int cap, int* n_out);
laser_status laser_kv_destroy(laser_kv* kv);

/* ========================================================================== */
/* Hot path                                                                    */
/* ========================================================================== */

/* Runs n prompt tokens d_tokens[0..n-1] of seq_id at its current length (chunks of at
 * most max_rows rows), appending their K/V.  d_logits_last (vocab floats or NULL)
 * receives the last token's logits. */
laser_status laser_prefill(laser_model* m, laser_kv* kv, int seq_id, const int32_t* d_tokens, int n,
                           float* d_logits_last, void* stream);

/* One chain-of-thought decode step (the reasoning-chunk generation of Eq. 2): request b
 * (seq_ids[b], host array) runs token d_tokens[b] at position len(seq_ids[b]), appends its
 * K/V (taking a page when the length is a multiple of 16) and gets the greedy next token
 * d_next[b] (lowest index among equal maxima) and the maximum softmax probability
 * d_max_prob[b] = 1 / sum_j exp(l_j - l_max).  d_logits ([batch][vocab] floats) may be
 * NULL.  d_next may alias d_tokens.  1 <= batch <= max_rows; seq_ids distinct. */
laser_status laser_decode_step(laser_model* m, laser_kv* kv, int batch, const int32_t* seq_ids,
                               const int32_t* d_tokens, int32_t* d_next, float* d_max_prob, float* d_logits,
                               void* stream);

/* Allocation-free variant of laser_decode_step, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid it).
 * Same arguments, results and validation as laser_decode_step; the decode step's scratch
 * (attention split partials and statistics, the split-merge arrival counters, LM-head softmax
 * statistics, K-share partials) lives in a static device array of 32 MiB per GPU, held from
 * the library's first use on that GPU until the process ends, instead of in the model's
 * workspace.  The kernels are launched one by one (no graph is captured or instantiated), the
 * host plan is built in a buffer the model allocated at finalize, and the arrival counters
 * are cleared by a kernel at every call (the array keeps the previous call's contents).
 * Calls that overlap on one GPU (any model, any stream) race on the array: order them.
 * Errors: as laser_decode_step; LASER_ERR_UNSUPPORTED when `batch` needs more scratch than
 * the array holds (roughly n_kv_heads * 128 * batch * (n_q_heads / n_kv_heads) * (head_dim
 * + 2) * 4 bytes plus the LM-head statistics); LASER_ERR_STATE if the array's address could
 * not be resolved at finalize. */
laser_status laser_decode_step_static(laser_model* m, laser_kv* kv, int batch, const int32_t* seq_ids,
                                      const int32_t* d_tokens, int32_t* d_next, float* d_max_prob, float* d_logits,
                                      void* stream);

/* The trial-answer probe at an ATP (Section 3.1): for each request, the S suffix tokens
 * d_suffix[0..S-1] run at positions L..L+S-1 (L = the request's length), the last one's
 * distribution gives trial token t_1 and p_1, and each t_j (j < T) is fed back to give
 * t_{j+1}, p_{j+1}.  d_conf[b] = (p_1 + ... + p_T) / T, d_argmax[b*T + j-1] = t_j, and
 * d_logits ([batch][T][vocab] or NULL) the trial distributions' logits.  Afterwards every
 * request's length, page table and cached K/V below its length are as before the call
 * (the probe's pages are returned to the pool).  Requires S*batch <= max_rows. */
laser_status laser_probe_confidence(laser_model* m, laser_kv* kv, int batch, const int32_t* seq_ids,
                                    const int32_t* d_suffix, int S, int T, float* d_conf, int32_t* d_argmax,
                                    float* d_logits, void* stream);

/* Decode for every request of the batch plus, in the same forward, the probe chunk of
 * the requests probe_idx[0..n_probe-1] (indices into the batch), taken at their length
 * after this step's token; the T-1 trial tokens then run as further forwards.  Outputs
 * as laser_decode_step (d_next, d_max_prob) and laser_probe_confidence (d_conf[i],
 * d_argmax[i*T + j] for probe i).  Requires batch + S*n_probe <= max_rows. */
laser_status laser_step_mixed(laser_model* m, laser_kv* kv, int batch, const int32_t* seq_ids,
                              const int32_t* d_tokens, int32_t* d_next, float* d_max_prob, int n_probe,
                              const int32_t* probe_idx, const int32_t* d_suffix, int S, int T, float* d_conf,
                              int32_t* d_argmax, void* stream);

/* One forward over spans of rows: span i appends spans[i].n_tokens tokens to sequence
 * spans[i].seq at its current length, with input ids (tok_sel ? d_tok1 : d_tok0)
 * [tok_off .. tok_off + n_tokens - 1]; if spans[i].out is nonzero the greedy token and
 * max-softmax probability of the span's last row go to (out_sel ? d_out_tok1 : d_out_tok0)
 * [out_off] and (out_sel ? d_out_p1 : d_out_p0)[out_off], and, when the matching
 * d_out_logits0 / d_out_logits1 ([..][vocab] floats) is not NULL, its logits to row out_off
 * of it (for parity checks; NULL skips the write).  A decode step is a span of one
 * token per request; a prompt or probe chunk is a longer span; spans of different
 * sequences mix freely (this is how a probe rides along with decode steps on a fork of
 * the request: Section 3.1's probe, with the request's own tokens unaffected).  Sequences
 * are distinct across spans; the total rows are at most max_rows.  The call is one
 * forward whose first kernel reads every input token before any output is written, so
 * input and output arrays may alias, also at the same indices (a decode loop can write each
 * request's next token over its input). */
typedef struct {
  int32_t seq, n_tokens, tok_sel, tok_off, out, out_sel, out_off;
} laser_span;
laser_status laser_forward(laser_model* m, laser_kv* kv, int n_spans, const laser_span* spans,
                           const int32_t* d_tok0, const int32_t* d_tok1, int32_t* d_out_tok0, float* d_out_p0,
                           int32_t* d_out_tok1, float* d_out_p1, float* d_out_logits0, float* d_out_logits1,
                           void* stream);

/* d_conf[i] = (d_p[i*T] + ... + d_p[i*T + T-1]) / T for i < n: the confidence of
 * Section 3.1 from the trial tokens' max-softmax probabilities. */
laser_status laser_confidence(laser_model* m, const float* d_p, int T, int n, float* d_conf, void* stream);

/* ========================================================================== */
/* ATP detection and the forced conclusion                                     */
/* ========================================================================== */
/* Section 3.1 marks ATPs by linguistic cues between reasoning chunks (such as "Wait" or
 * "Alternatively").  Given the cue tokens as a set of token ids, detection is a
 * membership test of each freshly generated token, done on the device so that the decode
 * loop needs no copy to the host: d_flags[i] = 1 if d_tokens[i] is in the set, else 0
 * (ids outside [0, vocab) are never members).  The set is a bitmap of (vocab + 31) / 32
 * words, bit t % 32 of word t / 32 for token t, built on the host by laser_atp_bitmap and
 * copied to the device by the caller.  d_flags may alias d_tokens.
 * The conclusion after an exit (Algorithm 1's "generate conclusion", forced when the budget
 * is exhausted) is the closing delimiter and any answer prompt appended with laser_prefill
 * (or a laser_forward span), followed by ordinary decode steps. */
/* words_out receives (vocab + 31) / 32 words.  INVALID_ARG for NULL, n_ids < 0, vocab < 1
 * or an id outside [0, vocab). */
laser_status laser_atp_bitmap(const int32_t* ids, int n_ids, int vocab, uint32_t* words_out);
/* n >= 1 tokens; asynchronous on `stream` (the current device). */
laser_status laser_atp_match(const int32_t* d_tokens, int n, const uint32_t* d_bitmap, int vocab, int32_t* d_flags,
                             void* stream);

/* ========================================================================== */
/* Kernel timing.  While any class is enabled (a timing session), forwards launch their
 * kernels one by one (no graph replay) and every launch records a HIP event, created
 * without a system-scope fence, at its end.  A launch of a class is timed from the end of
 * the kernel launched just before it to the end of the class's last kernel (attention
 * includes its merge kernel, the LM head its reduce kernel), which with back-to-back
 * kernels equals the sum of their kernel-trace durations; each event adds about a
 * microsecond to the kernel it ends.  At most 65536 launches are timed per session. */
/* ========================================================================== */
enum {
  LASER_K_EMBED = 0, LASER_K_QKV = 1, LASER_K_ATTN = 2, LASER_K_OPROJ = 3,
  LASER_K_GATEUP = 4, LASER_K_DOWN = 5, LASER_K_LMHEAD = 6, LASER_K_OTHER = 7, LASER_K_NCLASS = 8
};
/* Enables (1) or disables (0) timing of one kernel class; clears its spans. */
laser_status laser_timing_enable(laser_model* m, int kernel_class, int enable);
/* Waits for the class's last recorded event and returns the summed duration (ms) and the
 * number of timed launches since it was enabled or last read, then clears them. */
laser_status laser_timing_read(laser_model* m, int kernel_class, double* total_ms, int* launches);

/* ========================================================================== */
/* Graph replay                                                               */
/* ========================================================================== */
/* With graphs on (the default), the kernels of a decode, probe or mixed forward are
 * captured once per launch signature (rows, outputs, attention grid width and merge
 * bound, KV cache) into a HIP graph and replayed; per-call data (positions, pages, the caller's
 * token and output buffers) travels in the plan each forward uploads.  Results are
 * bitwise identical to launching the kernels one by one, which is what happens with
 * graphs off, while any kernel class is being timed, and for laser_prefill.  Up to 16
 * graphs are kept per model; the least recently used is released first.
 * Forwards of one model must be ordered (one stream, or synchronised between streams):
 * they share the model's workspace and its one device plan slot. */
laser_status laser_model_set_graphs(laser_model* m, int enable);

/* Graph cache statistics (for callers that want to see recaptures): *captures = forwards
 * captured into graphs since the model was created, *cached = graphs held now (at most 16).
 * Host-side only.  Errors: LASER_ERR_STATE (bad model), LASER_ERR_INVALID_ARG (null). */
laser_status laser_model_graph_stats(const laser_model* m, long long* captures, int* cached);

/* Projection kernel choice on the matrix-core path (forwards of 3 to 64 rows; the linear
 * maps of the transformer block in the decode steps and the trial-answer probe of
 * Section 3.1, whose costs Eq. 2 sums).  Two kernels compute the same products: one
 * splits K over the waves of a workgroup (1-4 row groups of 16 weight rows per
 * workgroup), the other gives each of 4 waves its own row groups and stages the
 * activations once per workgroup in LDS.  mode 0 (the default) takes the second for the
 * gate/up projection of forwards of 33 to 64 rows when it has enough row groups and for
 * the O and down projections of forwards of 49 to 64 rows, and the first elsewhere; it
 * also computes the QKV projection of bf16 models in forwards of 33 to 64 rows over
 * 512-column slices of K (each slice's activations staged once in LDS for 16 row groups,
 * the slices summed by a second kernel).  1 uses only the first kernel; 2 the second
 * wherever it applies (K a multiple of 8).  The summation order differs between them, so
 * results may differ in the last bits.  Captured forwards are released when the mode
 * changes.  Errors: LASER_ERR_STATE (bad model), LASER_ERR_INVALID_ARG (mode). */
laser_status laser_model_set_gemm_kernel(laser_model* m, int mode);

/* Attention split merge.  The decode step's paged attention (Section 3.1's chain-of-thought
 * decode, whose per-token cost Eq. 2 sums) splits a long context over several workgroups per
 * KV head and combines their partial results (running max, sum of exponentials, weighted
 * values).  fused = 0 (the default): every group's partials are combined by a separate merge
 * kernel.  fused = 1: a group of one row (a plain decode row) is combined by the last of its
 * workgroups to finish, inside the attention kernel, over at most max_splits splits (56 by
 * default); other groups (probe chunks, shared-prefix families) keep the merge kernel.  The
 * summation order differs between the two, so results may differ in the last bits.  (At the
 * 7B shape, batch 1, 14k context the fused merge measured slower: the last workgroup's
 * device-scope round trips cost more than the kernel boundary.)
 * Errors: LASER_ERR_STATE (bad model), LASER_ERR_INVALID_ARG (fused not 0/1, max_splits
 * outside [2, 128]). */
laser_status laser_model_set_attn_merge(laser_model* m, int fused, int max_splits);

/* Where the attention split merge of a forward of 1-2 rows runs (the decode step of Section
 * 3.1, whose per-token cost Eq. 2 sums; with fused = 0 above).  mode 2: in the O-projection's
 * launch, whose first workgroups combine the partials and publish the output while the
 * projection's workgroups start streaming their weights, then wait for it (a bounded wait; a
 * projection whose merge never arrived writes NaN).  mode 0: a separate merge kernel.  mode 1
 * (the default): the O-projection's launch when the projection's weights take at least 16 MiB
 * (long enough a stream to hide the merge: measured faster at the 7B shape, slower at 1.5B),
 * else the merge kernel.  The two combine the partials in different orders, so results may
 * differ in the last bits.  Not used by laser_decode_step_static.
 * Errors: LASER_ERR_STATE (bad model), LASER_ERR_INVALID_ARG (mode not 0, 1 or 2). */
laser_status laser_model_set_oproj_merge(laser_model* m, int mode);

#ifdef __cplusplus
}
#endif
#endif /* LASER_H */
