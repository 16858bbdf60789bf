/*
 * pced.h - C ABI of libpced, the per-token decode step of Parallel
 * Context-of-Experts Decoding (PCED; Corallo and Papotti, arXiv 2601.08670)
 * on one AMD Instinct MI355X (gfx950).
 *
 * The method (paper, Section 3): a query q has N retrieved documents with
 * relevance scores r_1..r_N. Each document k owns a precomputed KV cache K_k; an
 * "amateur" sequence (k = 0) holds no document. The N+1 sequences ("experts")
 * decode in one batched forward pass. At each step every expert yields full
 * vocabulary logits s_k, which are fused by the retrieval-aware contrastive rule
 *     Eq. 2:  s_hat_k = (1 + beta_k) s_k - beta_k s_0 + gamma log r_k,   k = 1..N
 *     Eq. 3:  y_t = argmax_v max_{k=1..N} s_hat_k(v)
 * and y_t is appended to the shared generation history of every expert.
 *
 * What one decode step runs here, all on the device:
 *   1. the new token's K/V row (one per sequence and layer) is written into the
 *      paged KV pool (shared-history append);
 *   2. per layer, every sequence attends with its own query over its own ragged
 *      cache (grouped-query attention, scale 1/sqrt(head_dim));
 *   3. the last layer's attention output, concatenated over heads and rounded to
 *      the storage type, is each sequence's hidden state x; logits are
 *      rho * x W^T with rho = 1/sqrt(mean(x^2) + 1e-5) (norm = RMS) or 1;
 *   4. at the first step with dynamic beta: beta_k = JSD(softmax s_k || softmax s_0)
 *      in bits, frozen for the following steps;
 *   5. Eq. 2 and Eq. 3 per query; ties go to the lowest token id, and the
 *      reported expert is the lowest k reaching the maximum.
 *
 * Conventions (every function):
 *   - Device memory is owned by the caller: KV pools, workspace, weights, inputs
 *     and outputs. The library never allocates or frees device memory. It owns
 *     only the host-side context.
 *   - Work is enqueued on the caller's stream and not synchronised (the one
 *     exception: pced_load_caches waits for its copies of caches held in host
 *     memory); outputs are valid once the caller synchronises that stream. A
 *     NULL stream is the default stream.
 *   - Every argument and capacity check runs on the host before anything is
 *     enqueued. On any non-OK status nothing was enqueued and the context is
 *     unchanged; pced_last_error() returns a description (thread-local).
 *   - A context is not thread-safe; separate contexts are independent. Calls on
 *     one context must be issued on streams that order them (normally one).
 */
#ifndef PCED_H
#define PCED_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum pced_status {
  PCED_OK = 0,
  PCED_ERR_INVALID_ARG = 1,  /* NULL pointer, bad shape, value out of range      */
  PCED_ERR_CAPACITY = 2,     /* would exceed a configured maximum or a page set  */
  PCED_ERR_HIP = 3,          /* a HIP call or kernel launch failed               */
  PCED_ERR_UNSUPPORTED = 4,  /* valid but not implemented for this configuration */
  PCED_ERR_STATE = 5         /* call out of order (e.g. step before load)        */
} pced_status;

typedef enum pced_dtype {
  PCED_F32 = 0,   /* float32 storage of q, K/V, lm_head and x */
  PCED_BF16 = 1   /* bfloat16 storage (raw 16-bit patterns)   */
} pced_dtype;

typedef enum pced_aggregation {
  PCED_AGG_MAX = 0,  /* Eq. 3: y = argmax_v max_k s_hat_k(v) (the method)                        */
  PCED_AGG_MOE = 1,  /* mixture: argmax_v log sum_k pi_k softmax(c_k)(v)  (Appendix C.4 ablation) */
  PCED_AGG_POE = 2   /* product: argmax_v sum_k pi_k log softmax(c_k)(v)  (Appendix C.4 ablation) */
} pced_aggregation;

typedef enum pced_norm {
  PCED_NORM_NONE = 0,  /* logits = x W^T                               */
  PCED_NORM_RMS = 1    /* logits = x W^T / sqrt(mean(x^2) + 1e-5) per row */
} pced_norm;

/* Static shape and capacity of a context. */
typedef struct pced_config {
  int32_t n_layers;          /* L  >= 1                                          */
  int32_t n_q_heads;         /* Hq, a multiple of n_kv_heads                     */
  int32_t n_kv_heads;        /* Hkv; Hq / Hkv <= 16                              */
  int32_t head_dim;          /* D: 64 or 128                                     */
  int32_t hidden;            /* must equal Hq * D (the hidden state is the
                                concatenated per-head attention output); a
                                multiple of 256 for bf16                        */
  int32_t vocab;             /* V >= 2                                           */
  int32_t dtype;             /* pced_dtype                                       */
  int32_t page_size;         /* tokens per KV page; must be 16                   */
  int32_t max_queries;       /* B, queries per batch                             */
  int32_t max_seqs;          /* S = sum over queries of (N_b + 1)                */
  int32_t max_pages;         /* pool capacity in pages (per layer)               */
  int32_t max_pages_per_seq; /* page-table row length                            */
  int32_t norm;              /* pced_norm                                        */
  int32_t max_attn_chunks;   /* cap on the attention launch's work chunks (waves
                                per kv-head), >= 0; 0 = as many as fit on the
                                GPU at once. A smaller cap leaves compute units
                                to other work; each chunk then streams more
                                pages and may span more sequences            */
  int32_t aggregation;       /* pced_aggregation. For MoE / PoE (the paper
                                compares them with Max in Appendix C.4 without
                                formulas; reading): c_k = (1 + beta_k) s_k -
                                beta_k s_0, pi_k = r_k^gamma / sum_j r_j^gamma
                                over the query's clipped r; scores (top1, top2)
                                in log units; the reported expert maximises
                                pi_k softmax(c_k)(y)                            */
  int32_t beta_scalar;       /* dynamic beta only: 0 = one beta per expert
                                (beta_k = JSD(p_k || p_0)); 1 = one beta per
                                query, the mean of those divergences (the
                                paper's beta_0 read as a single number)       */
  int32_t ffn_dim;           /* F, MLP width of the decoder stack run by the
                                pced_model_* calls (bf16 only, a multiple of
                                64); 0 = no decoder stack (pced_step with given
                                q / k_new / v_new only)                        */
  int32_t rope_theta;        /* RoPE base of the decoder stack (500000 for
                                Llama 3); used when ffn_dim > 0               */
} pced_config;

typedef struct pced_ctx pced_ctx;

/* Bytes of one KV pool (K or V) for cfg: n_layers * max_pages * n_kv_heads *
 * page_size * head_dim * sizeof(storage). Layout (opaque to callers):
 * [layer][page][kv_head][16 x head_dim tile]; inside a bf16 tile the elements are
 * ordered so that each matrix-core operand is one contiguous 16-byte load per
 * lane. Returns 0 for an invalid cfg. */
size_t pced_pool_bytes(const pced_config* cfg);

/* Bytes of the packed LM-head weights for cfg (0 for an invalid cfg). */
size_t pced_lm_head_bytes(const pced_config* cfg);

/*
 * Re-lay the LM-head weights once (at model load) into the form every step
 * reads. w: device [V][hidden] row-major, storage type; w_packed: device,
 * pced_lm_head_bytes(cfg), caller-owned, must not overlap w. For bf16 the
 * packed form is 2 KiB tiles, one per (16 vocabulary rows, 64 hidden columns),
 * each holding two matrix-core operands in lane order, so that the LM head
 * streams W with contiguous 1 KiB wave loads (rows past V are zero); for f32 it
 * is a plain copy. Asynchronous on `stream`. Errors: INVALID_ARG, HIP.
 */
pced_status pced_pack_lm_head(const pced_config* cfg, const void* w, void* w_packed, hipStream_t stream);

/* Bytes of device workspace a context needs (0 for an invalid cfg). */
size_t pced_workspace_bytes(const pced_config* cfg);

/* Create a context over caller-owned device workspace (>= pced_workspace_bytes,
 * 256-byte aligned). Host-only: enqueues nothing. */
pced_status pced_create(const pced_config* cfg, void* d_workspace, size_t ws_bytes, pced_ctx** out);

/* Destroy a context (NULL is ignored). The caller must have synchronised any
 * stream the context used. */
void pced_destroy(pced_ctx* ctx);

/* Description of the calling thread's last non-OK status ("" if none). */
const char* pced_last_error(void);

/*
 * Load one batch: the N_b + 1 precomputed caches of each query (paper, Section 3,
 * Eq. 1 datastore: one cache per retrieved document; the amateur's cache holds
 * only the query) and the per-document relevance scores r_k.
 *
 *   n_queries       B, 1 .. max_queries
 *   n_experts       host [B]: N_b >= 1 documents of query b
 *   cache_len       host [S]: preloaded tokens of each sequence (>= 1), in order
 *                   query 0: amateur, expert 1..N_0; query 1: amateur, ...
 *   src_k, src_v    host arrays [S] of pointers, each to a contiguous
 *                   [L][cache_len[s]][Hkv][D] tensor of the storage type, in
 *                   device memory or in host memory (told apart per pointer by
 *                   hipPointerGetAttributes; pinned host memory counts as host).
 *                   Device sources are copied by a kernel on `stream` and must
 *                   stay valid until the stream has executed this call. Host
 *                   sources cross to the device during the call: the library
 *                   re-lays each host sequence into the pool's page layout in
 *                   host memory and copies it with hipMemcpyAsync on `stream`,
 *                   waiting for those copies before it returns (the one
 *                   synchronisation in the library), so host buffers may be
 *                   freed as soon as the call returns
 *   k_pool, v_pool  device, pced_pool_bytes(cfg) each, caller-owned; this call
 *                   writes the caches into them and later steps append to them
 *   page_table      host [S][max_pages_per_seq] physical page ids (>= 0,
 *                   < max_pages, distinct across the batch; -1 marks pages not
 *                   given). Page p of sequence s holds tokens 16p .. 16p+15. NULL
 *                   assigns pages in order, giving every sequence
 *                   ceil((cache_len + reserve_tokens) / 16) pages.
 *   reserve_tokens  tokens each sequence must be able to append (NULL page table
 *                   only; checked against max_pages and max_pages_per_seq)
 *   relevance       host [sum N_b] r_k; clipped to [1e-8, 1 - 1e-8] before the log
 *                   (paper, Appendix B: scores mapped into [0,1) and clipped away
 *                   from 0, eps = 1e-8)
 *   gamma           weight of the retrieval prior (paper default 2.5)
 *   beta            host [sum N_b] fixed contrastive strengths (paper, Appendix
 *                   C.1), or NULL for dynamic beta: JSD in bits between each
 *                   expert's and the amateur's next-token distributions at the first
 *                   step, kept fixed afterwards (paper, Section 3)
 * Resets the step counter. Errors: INVALID_ARG, CAPACITY (pages), HIP.
 */
pced_status pced_load_caches(pced_ctx* ctx, int32_t n_queries, const int32_t* n_experts,
                             const int32_t* cache_len, const void* const* src_k,
                             const void* const* src_v, void* k_pool, void* v_pool,
                             const int32_t* page_table, int32_t reserve_tokens,
                             const float* relevance, float gamma, const float* beta,
                             hipStream_t stream);

/* Optional device outputs of a step; any NULL member is skipped. */
typedef struct pced_step_out {
  float* attn_out;        /* [S][L][Hq][D] fp32 attention output of every layer     */
  float* logits;          /* [S][V] fp32 logits s_k (Section 3, per-expert logits)  */
  int32_t* winner;        /* [B] expert k* (1..N_b) whose score chose the token     */
  float* top1;            /* [B] fused score of the chosen token                   */
  float* top2;            /* [B] best fused score over all other tokens            */
  float* beta_used;       /* [sum N_b] beta_k used by this step                    */
  float* hidden;          /* [S][hidden] fp32 copy of the stored hidden state x;
                             pced_model_*: the final residual stream h        */
  /* Per-layer values of the decoder stack (pced_model_step / _generate only;
   * ignored by pced_step), for layer-by-layer checks against a reference: */
  float* resid_trace;     /* [L][2][S][hidden] fp32 residual stream entering
                             layer l's attention block (index 0) and its MLP
                             block (index 1)                                 */
  uint16_t* qkv_trace;    /* [L][S][Hq*D + 2*Hkv*D] bf16 q, k, v of layer l
                             after RoPE, as attended and as appended         */
  uint16_t* act_trace;    /* [L][S][ffn_dim] bf16 MLP activation
                             silu(gate) * up of layer l                      */
} pced_step_out;

/*
 * One decode step for every sequence of every loaded query (paper, Section 3:
 * batched forward pass, Eq. 2, Eq. 3, shared history).
 *   q          device [S][L][Hq][D]    this step's query vectors
 *   k_new      device [S][L][Hkv][D]   this step's K row (the shared token's)
 *   v_new      device [S][L][Hkv][D]   this step's V row
 *   lm_head    device                  LM-head weights packed by pced_pack_lm_head
 *   tokens_out device [B]              chosen token y_t per query
 *   extra      optional outputs, may be NULL
 * All in the storage type except the fp32 outputs; q, k_new and v_new must be
 * 16-byte aligned. Errors: STATE (nothing loaded), CAPACITY (a sequence has no
 * page for the new token), INVALID_ARG (NULL, misaligned), HIP.
 */
pced_status pced_step(pced_ctx* ctx, const void* q, const void* k_new, const void* v_new,
                      const void* lm_head, int32_t* tokens_out, const pced_step_out* extra,
                      hipStream_t stream);

/* Deterministic stand-in for the model's projections in multi-step generation:
 * the step-t query and K/V rows of sequence s, layer l are SplitMix64 streams
 * keyed by (seed, tag, t, s, l, y_{t-1}) where y_{t-1} is the query's previous
 * token (first_token at t = 0); values are Irwin-Hall(4) sums of 16-bit fields
 * scaled to unit variance. The exact definition is in pced_generate's source. */
typedef struct pced_synth {
  uint64_t seed;
  int32_t first_token;
} pced_synth;

/*
 * n_steps decode steps (paper, Section 3: greedy generation with the shared
 * history). Step t's q / k_new / v_new are produced on the device from the
 * previous chosen token (pced_synth), so the only host interaction is the
 * caller's final synchronisation.
 *   tokens_out  device [B][n_steps]
 *   last_extra  optional outputs of the last step
 */
pced_status pced_generate(pced_ctx* ctx, int32_t n_steps, const pced_synth* synth,
                          const void* lm_head, int32_t* tokens_out,
                          const pced_step_out* last_extra, hipStream_t stream);

/*
 * Stage entry: full-vocabulary logits for given hidden states (paper, Section 3:
 * per-expert logits s_k). x: device [n_rows][hidden] storage type; lm_head:
 * device, packed by pced_pack_lm_head; logits: device [n_rows][V] fp32;
 * n_rows <= max_seqs.
 */
pced_status pced_lmhead(pced_ctx* ctx, const void* x, int32_t n_rows, const void* lm_head,
                        float* logits, hipStream_t stream);

/*
 * Allocation-free form of pced_lmhead, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc. It needs no context and no workspace: the padded copy of x
 * that pced_lmhead stages in the context's workspace goes to a library-owned
 * device array of 4 MiB, one per GPU, held until the process ends. Same
 * arguments and results as pced_lmhead (cfg gives the shapes, dtype and norm;
 * lm_head packed by pced_pack_lm_head; x device [n_rows][hidden]; logits device
 * [n_rows][V] fp32); calls no allocating routine.
 * Limit: ceil(n_rows / 16) * 16 * hidden * sizeof(storage) <= 4 MiB (512 rows
 * at hidden 4096 in bf16), else CAPACITY. Every call on a GPU shares that GPU's
 * array: calls that overlap on one GPU (several streams or threads) race, so
 * order them, e.g. on one stream. Asynchronous on `stream`.
 * Errors: INVALID_ARG (invalid cfg, NULL, n_rows < 1), CAPACITY, HIP.
 */
pced_status pced_lmhead_noalloc(const pced_config* cfg, const void* x, int32_t n_rows, const void* lm_head,
                                float* logits, hipStream_t stream);

/*
 * Stage entry: Eq. 2 and Eq. 3 on given logits for the loaded batch.
 *   logits        device [S][V] fp32, rows in load order
 *   refresh_beta  with dynamic beta: nonzero recomputes beta from these logits
 *                 and freezes it (what the first step does); zero uses the frozen
 *                 value (STATE if none yet). Ignored with fixed beta.
 *   tokens_out    device [B]
 */
pced_status pced_fuse(pced_ctx* ctx, const float* logits, int32_t refresh_beta,
                      int32_t* tokens_out, const pced_step_out* extra, hipStream_t stream);

/*
 * Copy tokens [start, start + count) of sequence `seq` (load order), layer
 * `layer`, out of the KV pool into k_out / v_out: device, contiguous
 * [count][Hkv][D] of the storage type, caller-owned (the layout of
 * pced_load_caches' sources). Reads what the loaded caches and every append so
 * far hold, e.g. to export a cache or to inspect the rows a step appended
 * (Section 3: the chosen token joins every expert's cache). count == 0 is a
 * no-op. Asynchronous on `stream`. Errors: STATE (nothing loaded), INVALID_ARG
 * (NULL output, seq or layer out of range, a token range beyond the
 * sequence's current length), HIP.
 */
pced_status pced_read_cache(pced_ctx* ctx, int32_t seq, int32_t layer, int32_t start, int32_t count,
                            void* k_out, void* v_out, hipStream_t stream);

/* Host mirror of the current cache length of every sequence: out [S]. */
pced_status pced_get_lengths(const pced_ctx* ctx, int32_t* out, int32_t capacity);

/*
 * Diagnostic, not a step of the method: *xor_out = the XOR of every 32-bit word
 * of the `bytes` bytes at src, read once with the non-temporal 16-byte loads
 * the decode kernels stream KV pages and weights with. A streaming read of
 * known size, for calibrating memory-traffic counters (FETCH_SIZE) and for
 * checking a device's streaming bandwidth. src: device, 16-byte aligned,
 * bytes a multiple of 16 and within src's allocation (may be NULL when bytes
 * is 0); xor_out: device, one uint32 (written 0 for bytes == 0). Asynchronous
 * on `stream`.
 * Errors: INVALID_ARG (NULL, misaligned, not device memory, past the
 * allocation), HIP.
 */
pced_status pced_stream_read(const void* src, size_t bytes, uint32_t* xor_out, hipStream_t stream);

/* Retrieval score modes (paper, Appendix B: normalisation per scoring mode). */
typedef enum pced_score_mode {
  PCED_SCORE_DENSE = 0,    /* cosine similarity in [-1, 1]: r = clip((s + 1) / 2, 0, 1 - eps)     */
  PCED_SCORE_COLBERT = 1,  /* same range and rescaling as dense                                  */
  PCED_SCORE_SPARSE = 2    /* nonnegative, unbounded: r = clip((2/pi) atan(max(s, 0)), 0, 1 - eps) */
} pced_score_mode;

/*
 * Host helper: relevance scores r_k for pced_load_caches from raw retrieval
 * scores and reranker logits (paper: Section 3, "Retrieval and relevance
 * scoring"; Appendix B, the per-mode normalisation, the reranker's sigmoid and
 * the harmonic-mean fusion), eps = 1e-8:
 *     r_ret = per mode (see pced_score_mode)
 *     r_rer = clip(1 / (1 + exp(-z)), 0, 1 - eps)
 *     r     = 2 r_ret r_rer / (r_ret + r_rer + eps)
 * With reranker_logits NULL, r = r_ret. Evaluated in double precision, stored
 * as float. All pointers are host memory of n elements; relevance may alias
 * neither input. No device work and no context involved.
 * Errors: INVALID_ARG (NULL retrieval or relevance, n < 0, unknown mode, a NaN
 * input).
 */
pced_status pced_relevance(int32_t mode, int32_t n, const float* retrieval, const float* reranker_logits,
                           float* relevance);

/*
 * Decoder stack around the step (bf16, cfg.ffn_dim > 0). The paper runs the
 * N+1 experts through the language model in one batched forward pass and
 * processes the query into every expert's cache (Section 3); it does not
 * restate the model. The stack here is a Llama-3-style decoder:
 *   h = E[y];  per layer:
 *     a = RMSNorm(h) g_attn;  q, k, v = a Wq^T, a Wk^T, a Wv^T;
 *     q, k rotated (RoPE, pairs (2i, 2i+1), angle pos * rope_theta^(-2i/D));
 *     k, v appended to the layer's cache at position pos;
 *     h += Attn(q, cache) Wo^T;
 *     b = RMSNorm(h) g_mlp;  h += (silu(b Wg^T) * (b Wu^T)) Wd^T;
 *   logits = RMSNorm(h) g_final W_lm^T, then Eq. 2 / Eq. 3 as in pced_step.
 * RMSNorm(h) = h / sqrt(mean(h^2) + 1e-5). pos is the sequence's own cache
 * length before the append (each expert's document was encoded from
 * position 0). Precision: h is fp32; a normalised product is computed as
 * rho * (bf16(h * g) W^T) with rho from the fp32 h; q, k, v are rounded to bf16
 * after RoPE, the attention output and silu(gate) * up to bf16 before their
 * projections; products accumulate in fp32.
 *
 * Weights live in one caller-owned device buffer of pced_model_bytes(cfg),
 * filled once by pced_pack_model_layer (every layer) and pced_pack_model_globals.
 * The buffer holds each layer's four matrices twice: in the matrix-core tile
 * order that the decode kernels stream, and row-major for the library GEMMs
 * (rocBLAS) that compute the projections of passes with more than 48 rows
 * (the prefill's chunks).
 */

/* Bytes of the packed decoder-stack weights (0 if cfg is invalid or ffn_dim == 0). */
size_t pced_model_bytes(const pced_config* cfg);

/*
 * Pack layer `layer`'s weights into `model`. tensors: host array of 9 DEVICE
 * pointers to bf16 row-major tensors, in this order:
 *   attn_norm [hidden], wq [Hq*D][hidden], wk [Hkv*D][hidden], wv [Hkv*D][hidden],
 *   wo [hidden][Hq*D], mlp_norm [hidden], w_gate [F][hidden], w_up [F][hidden],
 *   w_down [hidden][F]
 * (matrices are [out][in]). The sources may be freed once the stream has
 * executed the call. Errors: INVALID_ARG (NULL, layer out of range, no stack
 * configured), HIP.
 */
pced_status pced_pack_model_layer(const pced_config* cfg, int32_t layer, const void* const* tensors, void* model,
                                  hipStream_t stream);

/* Pack the token embedding (device bf16 [V][hidden]) and the final norm weight
 * (device bf16 [hidden]) into `model`. Errors: INVALID_ARG, HIP. */
pced_status pced_pack_model_globals(const pced_config* cfg, const void* embed, const void* final_norm, void* model,
                                    hipStream_t stream);

/*
 * Query-suffix prefill (paper, Section 3: the query is processed into every
 * expert's cache): appends tokens[b][0 .. n_tokens-1] to every sequence of
 * query b. The tokens go through the stack in chunks of up to
 * max(2304, max_seqs) / S tokens, all (sequence, token) rows of a chunk in one
 * pass; each token attends to the cache and to the suffix tokens before it
 * (causal). No logits.
 *   model   device, packed weights
 *   tokens  device int32 [B][n_tokens]; ids outside [0, V) are clamped
 * Errors: STATE (nothing loaded), CAPACITY (pages, or an attention plan whose
 * chunks or partial states exceed the workspace), INVALID_ARG, HIP.
 */
pced_status pced_model_prefill(pced_ctx* ctx, const void* model, int32_t n_tokens, const int32_t* tokens,
                               hipStream_t stream);

/*
 * One decode step through the decoder stack: in_tokens[b] (the query's last
 * token: the final suffix token, then each chosen token) is appended to every
 * sequence of query b, the stack and the LM head run for all S sequences, and
 * Eq. 2 / Eq. 3 pick tokens_out[b]. Dynamic beta is computed at the first step
 * that produces logits after a load.
 *   in_tokens   device int32 [B] (clamped to [0, V))
 *   tokens_out  device int32 [B]
 *   lm_head     device, packed by pced_pack_lm_head
 * Errors: as pced_model_prefill.
 */
pced_status pced_model_step(pced_ctx* ctx, const void* model, const void* lm_head, const int32_t* in_tokens,
                            int32_t* tokens_out, const pced_step_out* extra, hipStream_t stream);

/*
 * n_steps of pced_model_step, each feeding the previous chosen token; the
 * first step feeds first_tokens (device int32 [B]). tokens_out: device int32
 * [B][n_steps]; last_extra: optional outputs of the last step.
 */
pced_status pced_model_generate(pced_ctx* ctx, const void* model, const void* lm_head, int32_t n_steps,
                                const int32_t* first_tokens, int32_t* tokens_out,
                                const pced_step_out* last_extra, hipStream_t stream);

/* Kernel timing with HIP events attached to each kernel dispatch (start when
 * the kernel begins, stop when it completes). Classes: */
enum {
  PCED_PROF_APPEND = 0,  /* shared-history append and work planning */
  PCED_PROF_ATTN = 1,    /* decode attention, one launch per layer (bf16
                            pced_step: each launch after the first also
                            merges the previous layer's split partials) */
  PCED_PROF_LMHEAD = 2,  /* LM head                                */
  PCED_PROF_BETA = 3,    /* dynamic beta (first step only)         */
  PCED_PROF_FUSE = 4,    /* Eq. 2 + Eq. 3 over materialised logits:
                            the slice pass (k_fuse)               */
  PCED_PROF_SYNTH = 5,   /* pced_generate's input synthesis        */
  PCED_PROF_COMBINE = 6, /* merge of split attention partials as a launch
                            of its own (bf16 pced_step: last layer only) */
  PCED_PROF_EMBED = 7,   /* decoder stack: token embedding          */
  PCED_PROF_QKV = 8,     /* decoder stack: norm + QKV + RoPE + append */
  PCED_PROF_OPROJ = 9,   /* decoder stack: O projection + residual  */
  PCED_PROF_GATEUP = 10, /* decoder stack: norm + gate/up + SwiGLU  */
  PCED_PROF_DOWN = 11,   /* decoder stack: down projection + residual */
  PCED_PROF_FUSE_MERGE = 12, /* per-query merge of the slice candidates
                                (k_fuse_final): after the LM head's fused
                                Eq. 2 epilogue (steps after the first) or
                                after the slice pass of PCED_PROF_FUSE     */
  PCED_PROF_NCLASS = 13
};
typedef struct pced_profile {
  int64_t launches[PCED_PROF_NCLASS];
  double total_ms[PCED_PROF_NCLASS];
  double bytes[PCED_PROF_NCLASS];   /* algorithmic bytes of the timed launches */
  double flops[PCED_PROF_NCLASS];   /* algorithmic flops of the timed launches */
} pced_profile;

/* Start (nonzero) or stop (zero) recording; starting clears the totals. */
pced_status pced_profile_enable(pced_ctx* ctx, int32_t on);
/* Totals of the launches recorded so far; the caller must have synchronised the
 * stream. */
pced_status pced_profile_read(pced_ctx* ctx, pced_profile* out);

#ifdef __cplusplus
}
#endif
#endif /* PCED_H */
