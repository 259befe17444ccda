/*
 * moa.h -- C ABI of the MI355X (gfx950) ragged mixture-of-agents generation engine.
 *
 * What it computes. The paper's workload (Section "Problem Setting") is a
 * fixed batch of pre-routed model calls: every (query, expert) pair chosen by
 * the upstream router is an independent generation by that expert, and the
 * aggregator call (Section "MOSAIC: Adaptive Aggregation", Eq. 11) is one more
 * generation on the query followed by the expert outputs. Generation length
 * drives the cost (Section "Workload Characterisation"), and decode is bound
 * by memory bandwidth once a few prompts are in flight (appendix "Pitfalls of
 * Data Concurrency and Over-Sharding"). This engine keeps every model
 * co-resident on one GPU, shares one paged KV pool between them, and runs all
 * models' requests in one ragged continuous batch per step: each call
 * greedily decodes exactly max_new_tokens tokens (no end-of-sequence token).
 *
 * Conventions for every call:
 *   - returns moa_status; MOA_OK == 0, errors are negative; no exception or
 *     signal crosses the ABI;
 *   - pointers named host_* / tokens / res / tok_buf are host memory, copied
 *     before the call returns (the caller keeps ownership);
 *   - dev_arena is device memory owned by the caller; the engine
 *     sub-allocates weights, the KV pool and its workspace inside it and never
 *     calls hipMalloc after moa_create; the arena and the stream must outlive
 *     the engine;
 *   - device work is enqueued on the caller's stream; a bf16 engine with
 *     max_models > 1 also runs part of a step's layers on one internal stream
 *     that waits for the caller's stream when the step starts and that the
 *     caller's stream waits for before the step's final norm and LM head, so
 *     the caller's stream still orders every step (MOA_FLAG_ONE_STREAM keeps
 *     everything on the caller's stream);
 *   - single host thread: an engine is not thread-safe;
 *   - after MOA_EHIP only moa_destroy is valid on that engine.
 */
#ifndef MOA_H
#define MOA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOA_OK = 0,
  MOA_EINVAL = -1, /* bad argument (shape, id, length, capacity) */
  MOA_ENOMEM = -2, /* arena, token store or block-list store too small */
  MOA_ENOSPC = -3, /* request can never fit the KV pool */
  MOA_ESTATE = -4, /* call not valid in the engine's current state */
  MOA_EHIP = -5    /* HIP runtime error; the engine is unusable */
} moa_status;

enum { MOA_F32 = 0, MOA_BF16 = 1 };

/* flags */
enum {
  /* Scheduler dry run: every call does its host bookkeeping but no device
   * work is enqueued and no tokens are computed (collected tokens read -1).
   * dev_arena and hip_stream may be NULL. */
  MOA_FLAG_PLAN_ONLY = 1,
  /* Run every kernel on the caller's stream. By default a bf16 engine with
   * several models splits each step's model groups in two halves and runs
   * the second half's layers on an internal stream (its own split-K
   * workspace in the arena), so the halves' kernels overlap. Every launch
   * is planned over the whole step either way, so the results are
   * bit-identical; the flag gives launch durations that are not shared with
   * concurrent kernels. */
  MOA_FLAG_ONE_STREAM = 2
};

/* Decoder geometry (Llama-style pre-norm decoder: RMSNorm, GQA attention with
 * rotate-half RoPE, SwiGLU MLP, untied LM head). */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rope_theta, rms_eps;
} moa_model_cfg;

typedef struct {
  moa_model_cfg model;        /* geometry shared by every model of the engine */
  int32_t dtype;              /* MOA_F32 or MOA_BF16: weights, activations, KV */
  int32_t kv_block_size;      /* token slots per KV block; must be 16 */
  int32_t num_kv_blocks;      /* blocks in the shared KV pool (all layers) */
  int32_t max_num_seqs;       /* running requests at once */
  int32_t max_prefill_tokens; /* prompt tokens processed per step */
  int32_t max_model_len;      /* max prompt + generated tokens of a request */
  int32_t max_models;         /* models the arena reserves room for */
  int32_t flags;              /* MOA_FLAG_* */
  int64_t token_store;        /* device slots for prompt+output tokens of live requests (0: default) */
  int64_t block_store;        /* device slots for block lists of live requests (0: default) */
} moa_engine_cfg;

typedef struct moa_engine moa_engine;

typedef struct {
  int64_t step;            /* index of the step just enqueued; -1: nothing to run */
  int32_t admitted;        /* requests admitted this step */
  int32_t prefill_tokens;  /* prompt positions processed */
  int32_t decode_rows;     /* decode positions processed */
  int32_t finished;        /* requests retired this step */
  int32_t running;         /* running after the step */
  int32_t pending;         /* waiting for admission after the step */
  int32_t free_blocks;     /* free KV blocks after the step */
  int32_t emitted;         /* tokens the step produces: its decode rows plus the
                              requests whose prompt completes in it */
} moa_step_info;

typedef struct {
  int64_t request_id;
  int32_t model_id;
  int32_t n_tokens;        /* == max_new_tokens of the request */
  int64_t tok_offset;      /* where its tokens start in the caller's tok_buf */
  int64_t finish_step;     /* step at which it retired */
} moa_result;

/* Device bytes moa_create + max_models moa_load_expert calls need in the arena.
 * EINVAL: inconsistent cfg. */
moa_status moa_arena_bytes(const moa_engine_cfg* cfg, size_t* bytes);

/* Create an engine. cfg is copied. Lays out the KV pool and workspace inside
 * dev_arena (arena_bytes >= moa_arena_bytes()). hip_stream is a hipStream_t.
 * EINVAL: bad cfg (kv_block_size != 16, head_dim not 64/128 in bf16 mode,
 * n_heads not a multiple of n_kv_heads, non-positive sizes). ENOMEM: arena too
 * small. EHIP: runtime failure (no engine is returned). */
moa_status moa_create(const moa_engine_cfg* cfg, void* dev_arena, size_t arena_bytes,
                      void* hip_stream, moa_engine** out);

/* Load one model (Section "MOSAIC: Multi-Model Scheduling", subsection
 * "Problem Setting": the deployment draws its experts from a pool of
 * heterogeneous models; here every expert and the aggregator are resident
 * at once, so the per-model load cost l_m of that subsection is paid once,
 * here, instead of per session). host_weights is the packed blob: tensors in the order
 *   embed[V,d], { attn_norm[d], wq[nh*hd,d], wk[nkv*hd,d], wv[nkv*hd,d],
 *   wo[d,nh*hd], mlp_norm[d], w_gate[ffn,d], w_up[ffn,d], w_down[d,ffn] } x L,
 *   final_norm[d], lm_head[V,d]
 * each row-major [out, in], elements in the engine dtype (fp32, or bf16 bits),
 * no padding. The engine re-lays the matrices out for its kernels. Model ids
 * are dense, in load order; the aggregator is just another model. Blocks
 * until the weights are resident. EINVAL: cfg differs from the engine's
 * geometry or nbytes is wrong. ENOMEM: more than max_models. ESTATE: called
 * after the first moa_step. */
moa_status moa_load_expert(moa_engine* e, const moa_model_cfg* cfg, const void* host_weights,
                           size_t nbytes, int32_t* model_id);

/* Queue one generation call (subsection "Problem Setting": the fixed prompt
 * set, routed before scheduling, is a batch of (prompt, expert) calls;
 * subsection "MOSAIC: Adaptive Aggregation": the aggregator call is one more
 * such call on the query followed by the expert outputs): prompt
 * tokens[0..n_tokens) for model model_id, emitting exactly max_new_tokens tokens. Request ids are dense and increase
 * in submit order. The request waits in a FIFO until its KV blocks
 * ceil((n_tokens + max_new_tokens - 1) / 16) and a seat are free.
 * EINVAL: n_tokens < 1, max_new_tokens < 1, unknown model, token id outside
 * [0, vocab) (not checked in a MOA_FLAG_PLAN_ONLY dry run), n_tokens +
 * max_new_tokens - 1 > max_model_len, or max_prefill_tokens == 0.
 * ENOSPC: the request needs more blocks than the pool has.
 * ENOMEM: token or block-list store full (collect finished requests first). */
moa_status moa_submit(moa_engine* e, const int32_t* tokens, int32_t n_tokens, int32_t model_id,
                      int32_t max_new_tokens, int64_t* request_id);

/* Queue a call that arrives with a KV history instead of a prompt to prefill
 * (a long generation already in progress): positions 0..ctx_len-1 of every
 * layer hold the given K/V, the call feeds seed_token at position ctx_len and
 * emits exactly max_new_tokens tokens. It needs
 * ceil((ctx_len + max_new_tokens) / 16) blocks and skips the prefill phase.
 * host_kv: [n_layers][2 (K, V)][ctx_len][n_kv_heads][head_dim] elements of the
 * engine dtype (K after RoPE), copied before the call returns and written into
 * the request's blocks when it is admitted (that step drains the stream).
 * host_kv == NULL: the history is filled on the device with values in
 * [-1, 1) from a hash of (request id, layer, K|V, position, head, dim).
 * EINVAL: bad id, ctx_len < 0, max_new_tokens < 1, seed token outside the
 * vocabulary, or ctx_len + max_new_tokens > max_model_len. ENOSPC / ENOMEM as
 * for moa_submit. */
moa_status moa_submit_with_history(moa_engine* e, int32_t model_id, int32_t seed_token, int32_t ctx_len,
                                   const void* host_kv, int32_t max_new_tokens, int64_t* request_id);

/* Plan one step on the host and enqueue its kernels on the stream (the
 * generation phase that subsection "Workload Characterisation" makes the
 * dominant cost, run as continuous batching of every resident model's calls,
 * which appendix "The Pitfalls of Data Concurrency and Over-Sharding" needs
 * to keep decode bound by memory bandwidth):
 *   1 admit FIFO heads while a seat and their blocks are free (head-of-line
 *     blocking); a request gets the smallest free block ids, ascending;
 *   2 prefill: running requests in admission order take prompt positions up
 *     to the per-step budget; completing a prompt emits token 0;
 *   3 decode: every other running request with tokens left feeds its last
 *     token and emits the next one;
 *   4 retire requests that have emitted all tokens; their blocks are freed.
 * Does not wait for the device (the sampled tokens stay on the device and feed
 * the next step). info may be NULL; info->step == -1 when nothing is queued
 * or running. EHIP on a runtime failure. */
moa_status moa_step(moa_engine* e, moa_step_info* info);

/* moa_step for callers that cannot allocate (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): the same step --
 * the same plan and kernels, bit-identical results -- that calls no HIP
 * allocation routine (no hipMalloc / hipHostMalloc / hipFree /
 * hipEventCreate). Its kernels' split-K and split-KV partial sums live in the
 * library's static per-GPU scratch array (64 MiB, one copy on each GPU the
 * library runs on, held until the process ends) instead of the arena; the
 * metadata goes through the pinned staging sized at moa_create; prompts and
 * block lists are uploaded from the engine's own host copies; kernel timing
 * (moa_debug_time_kernels) is skipped for these steps.
 * ENOMEM, with nothing changed: the engine's planned partials (split-K
 * partials of every model stream plus split-KV slots) exceed 64 MiB (then
 * use moa_step). Every moa_step_noalloc on one GPU shares that GPU's array:
 * calls whose steps overlap on the device (engines stepping on different
 * streams at once) race; steps of one engine are ordered by its stream.
 * Other errors as moa_step. */
moa_status moa_step_noalloc(moa_engine* e, moa_step_info* info);

/* Hand back finished calls (subsection "MOSAIC: Adaptive Aggregation": the
 * expert outputs a query's aggregator call, or the confidence gate of Eq. 11,
 * is waiting for). Return requests retired at steps <= upto_step (upto_step < 0: every step
 * enqueued so far) that were not collected yet, in retirement order (step,
 * then admission order), waiting for that step to finish on the device.
 * Tokens are written back to back into tok_buf. If cap or tok_cap is too
 * small nothing is drained, *n_out is set to the number of results that are
 * ready and EINVAL is returned. */
moa_status moa_collect(moa_engine* e, int64_t upto_step, moa_result* res, int32_t cap,
                       int32_t* n_out, int32_t* tok_buf, int64_t tok_cap);

/* Wait for every enqueued step. */
moa_status moa_sync(moa_engine* e);

/* Wait for the engine's streams, then free what the engine allocated
 * (host state, pinned staging, streams and events). The device arena stays
 * the caller's: free it after this returns. NULL is a no-op. */
void moa_destroy(moa_engine* e);
/* Static description of a status code ("MOA_OK", "MOA_EINVAL: invalid
 * argument", ...); never NULL. */
const char* moa_status_str(moa_status s);

/* ---- inspection hooks (tests) ---- */

typedef struct {
  int32_t model_id, prompt_len, max_new_tokens, n_blocks;
  int64_t admit_step, finish_step; /* -1 until it happens */
  int32_t n_chunks;                /* prefill chunks so far */
  int32_t state;                   /* 0 pending, 1 running, 2 retired, 3 collected */
} moa_request_info;

moa_status moa_debug_request(moa_engine* e, int64_t request_id, moa_request_info* info);

/* The request's KV block ids (ascending, as admitted). n_out = count. */
moa_status moa_debug_block_table(moa_engine* e, int64_t request_id, int32_t* out, int32_t cap,
                                 int32_t* n_out);

/* The request's prefill chunks as (step, start, length) triples. */
moa_status moa_debug_chunks(moa_engine* e, int64_t request_id, int64_t* out, int32_t cap_triples,
                            int32_t* n_out);

/* Per-step bookkeeping rows (step, admitted, prefill_tokens, decode_rows,
 * finished, free_blocks_after), 6 int64 per step, oldest first, into out
 * (caller-owned, cap_steps rows). *n_out is always set to the number of
 * steps recorded; MOA_EINVAL without writing when cap_steps is smaller (a
 * call with out = NULL and cap_steps = 0 asks for the count) or when e or
 * n_out is NULL. */
moa_status moa_debug_steps(moa_engine* e, int64_t* out, int64_t cap_steps, int64_t* n_out);

/* How the last moa_step split its models over the model streams (a
 * MOA_FLAG_PLAN_ONLY bf16 engine plans the split a GPU engine with two
 * streams would make, so this can be inspected without a GPU).
 *   *n_shares: shares used, 1 .. 4;
 *   *n_models: models with rows in the step;
 *   models[i], i < n_models: those models in the step's row order;
 *   cost[i]: the split's cost of models[i]: its weight bytes times
 *     max(1, rows / 96) plus the K/V bytes its rows' attention reads;
 *   share_models0[u], share_row0[u], share_lm0[u], u <= n_shares: index in
 *     models, row and LM row where share u starts (the last entries are
 *     n_models and the step's row and LM-row counts).
 * share_* hold at least 5 entries, models and cost max_models. */
moa_status moa_debug_step_shares(moa_engine* e, int32_t* n_shares, int32_t* n_models, int32_t* models,
                                 double* cost, int32_t* share_models0, int32_t* share_row0,
                                 int32_t* share_lm0);

/* Capture the fp32 logits row of every token request_id emits: row j (the
 * logits that produced output token j) is copied to host_logits + j * vocab
 * once the step that computes it completes. cap: floats host_logits holds;
 * EINVAL (nothing registered) when it is below max_new_tokens * vocab. The
 * buffer must stay valid until the request is collected. ESTATE when the
 * request's prefill has already completed (register before it). */
moa_status moa_debug_capture_logits(moa_engine* e, int64_t request_id, float* host_logits, int64_t cap);

/* Kernel classes of one step (for moa_debug_time_kernels). */
enum {
  MOA_K_EMBED = 0, MOA_K_NORM, MOA_K_GEMM_QKV, MOA_K_ROPE_KV, MOA_K_ATTN, MOA_K_ATTN_REDUCE,
  MOA_K_GEMM_O, MOA_K_GEMM_GATEUP, MOA_K_GEMM_DOWN, MOA_K_GEMM_LMHEAD, MOA_K_ARGMAX, MOA_K_PREFILL_ATTN,
  /* Two views of the GEMM launches above, by the kernel that runs them: every
   * qkv / o / gate-up / down / LM-head launch is counted once more in exactly
   * one of these (the workgroup-tile kernel of small and medium row counts,
   * or the 128-row-tile matrix-core kernel of large row counts). A sum over
   * classes must leave them out. */
  MOA_K_GEMM_SMALL_M, MOA_K_GEMM_LARGE_M,
  MOA_K_COUNT
};

/* Per-class launch statistics of the sampled steps. bytes/flops are the
 * algorithmic figures of those launches: for a GEMM the bf16 weights it
 * streams (N*K*2 per model group) plus its split-bf16 input (M*K*4) and fp32
 * output (M*N*4), flops 2*M*N*K; for attention the bf16 K/V it reads
 * (keys*2*head_dim*2 per KV head) plus q (fp32) and its output; for causal
 * prefill attention each block's keys once per KV head, and 4*head_dim flops
 * per (query head, query, visible key). */
typedef struct {
  int64_t launches;   /* timed launches (sampled steps) */
  double ms;          /* their summed durations (HIP events around each launch; sampled
                         steps run on one stream, so no other stream's kernels overlap them) */
  double bytes;       /* their algorithmic bytes */
  double flops;       /* their algorithmic flops */
  int64_t launches_all; /* every launch since the reset */
  double bytes_all, flops_all;
  double roof_ms_all; /* sum over every launch of max(bytes / peak_bw, flops / peak_flops) */
} moa_kernel_stats;

/* Reset the statistics; from now on account every launch (bytes, flops,
 * roofline time at the given peaks, bytes/s and flop/s) and time every launch
 * of one step out of `every` (every <= 0: no timing) with an event pair
 * around it on the engine's stream. A timed step runs all of its kernels on
 * the caller's stream (a two-stream engine included; the results are the
 * same bits), so a timed launch carries the whole step and runs beside no
 * other stream's kernels. */
moa_status moa_debug_time_kernels(moa_engine* e, int32_t every, double peak_bw, double peak_flops);

/* Statistics per class, out[MOA_K_COUNT]. Waits for the stream. */
moa_status moa_debug_kernel_stats(moa_engine* e, moa_kernel_stats* out);

/* What this GPU sustains, measured on the engine's stream (the device work
 * runs now; the call returns when it is done): *read_bytes_per_s = streaming
 * HBM read bandwidth over up to 8 GiB of the KV pool (read only; the pool must
 * be at least 1 GiB), *mfma_flops_per_s = bf16 matrix-core throughput of the
 * 32x32x16 MFMA (dense, 2*32*32*16 flops per instruction). Each is the best of
 * five timed runs after a warm-up. Uses the logits workspace as scratch
 * (overwritten; call between steps). EINVAL: null outputs or a pool under
 * 1 GiB; ESTATE: plan-only engine or unusable engine; EHIP: runtime error. */
moa_status moa_debug_measure_peaks(moa_engine* e, double* read_bytes_per_s, double* mfma_flops_per_s);

#ifdef __cplusplus
}
#endif
#endif /* MOA_H */
