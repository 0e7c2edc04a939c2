/*
 * rl_decode.h -- C ABI of the MI355X (gfx950) RL-rollout decode library.
 *
 * The library runs the generation step of an RL iteration: a policy decoder
 * extends a batch of sampled responses by one token per call and returns,
 * with every token, its log-probability (RLinf, arXiv 2509.15965, Sec. 2.1:
 * GRPO generates several responses per query and the RL loss consumes their
 * per-token log-probabilities; Sec. 5.1.2: one forward pass yields both the
 * action token and its log-probability).  Generation is the bandwidth-bound
 * phase of the iteration (Sec. 2.1, characteristics of RL workflows) and its
 * speed is set by how much KV cache the engine can keep (Sec. 5.1.1).
 *
 * The decoder is a pre-norm transformer: RMSNorm, fused q|k|v projection,
 * rotate-half RoPE, grouped-query attention over a per-sequence KV cache,
 * output projection, RMSNorm, SwiGLU MLP, final RMSNorm, untied LM head,
 * then temperature-scaled log-softmax with Gumbel-max sampling keyed by a
 * counter-based generator (Philox4x32-10, Salmon et al., SC'11).
 *
 * Conventions for every entry point:
 *  - All device memory (weights, KV pool, workspace, token and output
 *    buffers) is owned by the caller and borrowed by the library; it must
 *    outlive the context.  The library never frees it.
 *  - "host" arguments are read before the call returns; "device" arguments
 *    are read or written asynchronously on the context's stream.
 *  - Every call returns an rl_status.  Arguments are validated on the host
 *    before anything is enqueued: a call that returns an error has enqueued
 *    no work and changed no state.  RL_ERR_HIP reports a failed HIP runtime
 *    call (including a device fault surfaced by the runtime).
 *  - Work is asynchronous: outputs are valid once the caller synchronises
 *    the stream.  No entry point synchronises the stream, except
 *    rl_decode_create, rl_decode_kernel_stats and rl_decode_destroy.
 *  - A context is used by one host thread at a time.
 */
#ifndef RL_DECODE_H
#define RL_DECODE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rl_status {
    RL_OK = 0,
    RL_ERR_INVALID_ARG = 1,   /* null pointer, bad value, duplicate slot ...      */
    RL_ERR_UNSUPPORTED = 2,   /* shape the kernels do not handle                  */
    RL_ERR_CAPACITY = 3,      /* too many rows / positions, buffer too small      */
    RL_ERR_HIP = 4,           /* HIP runtime error                                */
    RL_ERR_STATE = 5          /* destroyed or corrupted context                   */
} rl_status;

typedef enum rl_dtype {
    RL_DTYPE_FP32 = 0,        /* weights, activations and KV in fp32              */
    RL_DTYPE_BF16 = 1         /* weights, GEMM inputs and KV in bf16              */
} rl_dtype;

/* Decoder shape and capacity.
 * Supported: head_dim in {64, 128}; n_q_heads a multiple of n_kv_heads with
 * n_q_heads / n_kv_heads <= 16; hidden, ffn and vocab multiples of 8; in
 * bf16 every weight matrix (the LM head, gate|up, q|k|v, o, down) under
 * 4 GiB.  rms_eps > 0, rope_theta > 1.  Capacity: max_seqs KV slots (also the most
 * rows one rl_decode_step takes), max_ctx positions per slot, and
 * max_prefill_tokens packed prompt tokens per rl_prefill call. */
typedef struct rl_model_config {
    int32_t n_layers;
    int32_t hidden;
    int32_t n_q_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t ffn;
    int32_t vocab;
    int32_t dtype;                /* rl_dtype */
    double  rms_eps;
    double  rope_theta;
    int32_t max_seqs;
    int32_t max_ctx;
    int32_t max_prefill_tokens;
    int32_t kv_page_size;         /* 0: contiguous slots; else positions per K/V page (a multiple of 32 in [32, 65536]) */
    int32_t kv_pages;             /* pages in the pool (0: max_seqs * ceil(max_ctx / kv_page_size)); 0 without pages */
    /* Mixture of experts (Sec. 5.1.1's Qwen3-30B-A3B policy): n_experts > 0
     * replaces each layer's MLP by n_experts SwiGLU experts of width
     * expert_ffn of which each token uses its top_k (bf16 only; n_experts
     * <= 1024, top_k <= min(n_experts, 16), expert_ffn a multiple of 16,
     * hidden a multiple of 16 and <= 4096; ffn is then not used).  A token's
     * router row r = h . W_r^T (fp32); its experts are the top_k largest
     * entries (equal values: the lower expert first) and their weights the
     * softmax of those entries; the MLP output is the weighted sum of the
     * chosen experts' outputs. */
    int32_t n_experts;
    int32_t top_k;
    int32_t expert_ffn;
    int32_t reserved;             /* must be 0 */
} rl_model_config;

/* Device pointers to the weights, all in the model dtype, row-major
 * [out][in]; layer tensors are stacked over layers (layer-major).
 * With Hq = n_q_heads, Hkv = n_kv_heads, d = head_dim, H = hidden, F = ffn:
 *   embed      [vocab][H]
 *   attn_norm  [L][H]
 *   w_qkv      [L][(Hq + 2*Hkv)*d][H]   q rows (head-major), then k, then v
 *   w_o        [L][H][Hq*d]
 *   mlp_norm   [L][H]
 *   w_gate_up  [L][2*F][H]              gate rows first, then up rows
 *   w_down     [L][H][F]
 *   final_norm [H]
 *   lm_head    [vocab][H]
 * and for a mixture of experts (E = n_experts, Fe = expert_ffn), in place of
 * w_gate_up and w_down (which may then be NULL):
 *   w_router       [L][E][H]
 *   w_exp_gate_up  [L][E][2*Fe][H]     per expert: gate rows, then up rows
 *   w_exp_down     [L][E][H][Fe]
 * q-head j attends with kv-head j / (Hq / Hkv).  Every row must be 16-byte
 * aligned (guaranteed by the multiple-of-8 shape rules for bf16 and fp32). */
typedef struct rl_weights {
    const void* embed;
    const void* attn_norm;
    const void* w_qkv;
    const void* w_o;
    const void* mlp_norm;
    const void* w_gate_up;
    const void* w_down;
    const void* final_norm;
    const void* lm_head;
    const void* w_router;
    const void* w_exp_gate_up;
    const void* w_exp_down;
} rl_weights;

/* Sampling: seed keys the generator; temperature T >= 0 divides the logits
 * both for sampling and for the reported log-probability.  T == 0 selects
 * the arg-max token (lowest index on ties) and reports its T = 1
 * log-probability.  A NaN logit never wins: a row with NaN entries samples
 * among its other entries and reports a NaN log-probability; a row of NaN
 * logits gets token -1 (an input row of zeros if fed back) and NaN. */
typedef struct rl_sample_params {
    uint64_t seed;
    float    temperature;
    int32_t  reserved;            /* must be 0 */
} rl_sample_params;

typedef struct rl_decode_ctx rl_decode_ctx;

/* ---------------------------------------------------------------------
 * Sizes.
 *
 * KV pool layout (model dtype), with S = max_seqs, cap = max_ctx rounded
 * up to a multiple of 32, and E = element size:
 *   K slab at byte offset 0:
 *     K[l][s][h][t][i]  at element  (((l*S + s)*Hkv + h)*cap + t)*d + i
 *   V slab at byte offset rl_decode_kv_bytes(cfg) / 2, in 8-position blocks:
 *     V[l][s][h][t][i]  at element  ((((l*S + s)*Hkv + h)*(cap/8) + t/8)*d + i)*8 + t%8
 * Position t of a slot holds the token at position t of that sequence.
 *
 * Paged pool (kv_page_size = P > 0, NP = kv_pages or max_seqs * ceil(max_ctx / P)):
 *     K[l][s][h][t][i]  at element  ((l*NP + pg)*Hkv + h)*B + (t%P)*d + i
 *     V[l][s][h][t][i]  at element  ((l*NP + pg)*Hkv + h)*B + (((t%P)/8)*d + i)*8 + t%8
 * with pg the page that holds positions [P*(t/P), P*(t/P + 1)) of slot s and
 * B * E = P*d*E bytes rounded up to an odd multiple of 256 (so that blocks
 * are never a power of two apart; K and V slabs are 2*L*NP*Hkv*B*E bytes
 * together).  A
 * slot is given pages as its length grows (prefill, decode steps, scoring,
 * set lengths, onload) and gives them back when released or shortened, so a
 * pool of fewer pages than max_seqs * max_ctx positions serves sequences of
 * uneven lengths; a call that would need more pages than are free fails with
 * RL_ERR_CAPACITY and changes nothing.  The slots of a GRPO group (prefill
 * or scoring with group > 1) share the pages their prompt fills completely:
 * those K/V rows are written once and held by every slot of the group until
 * the last one lets them go; the rest of the prompt and each response are
 * in pages of the slot's own.  A slot whose length is set to end inside a
 * shared page first gets its own copy of that page (rl_set_slot_lengths).
 * The page table travels with each call's metadata
 * (4 * max_seqs * ceil(max_ctx / P) bytes).
 * Returns 0 when cfg is invalid or unsupported.
 * ------------------------------------------------------------------- */
size_t rl_decode_kv_bytes(const rl_model_config* cfg);

/* Workspace bytes: activations for max(max_seqs, max_prefill_tokens) rows,
 * split-K and split-KV partial sums, fp32 logits for max_seqs rows, the
 * RoPE table and per-call index metadata.  0 when cfg is invalid. */
size_t rl_decode_workspace_bytes(const rl_model_config* cfg);

/* ---------------------------------------------------------------------
 * Life cycle.
 * ------------------------------------------------------------------- */

/* Create a context on the current HIP device.  The context is the rollout
 * engine's state for one policy model: its KV capacity (max_seqs slots of
 * max_ctx positions) bounds how many responses generate at once, which is
 * what sets rollout speed (Sec. 5.1.1, larger KV-cache allocations).
 *  cfg        host; copied.
 *  w          host struct of device pointers; copied (the memory is borrowed).
 *  kv_pool    device, kv_bytes >= rl_decode_kv_bytes(cfg), 256-byte aligned.
 *  workspace  device, ws_bytes >= rl_decode_workspace_bytes(cfg), 256-byte aligned.
 *  stream     hipStream_t to run on (NULL = the null stream); borrowed.
 *  out        receives the context; set to NULL on error.
 * Every slot starts empty (length 0).  Uploads the RoPE table and
 * synchronises the stream once.  The context owns host memory only
 * (metadata and a small pinned staging ring). */
rl_status rl_decode_create(const rl_model_config* cfg, const rl_weights* w,
                           void* kv_pool, size_t kv_bytes,
                           void* workspace, size_t ws_bytes,
                           void* stream, rl_decode_ctx** out);

/* Free the context's host state.  NULL is accepted (no-op).  Waits for the
 * context's outstanding work first.  The context must not be used again. */
rl_status rl_decode_destroy(rl_decode_ctx* ctx);

/* ---------------------------------------------------------------------
 * Prefill (generation start, Sec. 2.1: G responses per query).
 *
 * Runs the causal forward over n_prompts packed prompts, each computed once,
 * writes each prompt's K/V into all `group` slots of its group, and samples
 * the first response token of every slot.
 *  n_prompts, group   >= 1, n_prompts*group <= max_seqs.
 *  slots          host [n_prompts*group]; slots of prompt p are
 *                 slots[p*group .. p*group+group-1]; distinct, < max_seqs.
 *  seq_uids       host [n_prompts*group]; per-sequence sampling identity.
 *  prompt_offsets host [n_prompts+1], CSR offsets into tokens; offsets[0] = 0,
 *                 every prompt length in [1, max_ctx - 1], total
 *                 <= max_prefill_tokens.
 *  tokens         device int32 [offsets[n_prompts]]; an id v >= 0 selects
 *                 embedding row v (< vocab); an id v < 0 selects row -v-1 of
 *                 `embeds` (< n_embed_rows).  Out-of-range ids embed as zeros.
 *  embeds         device [n_embed_rows][hidden] model dtype, or NULL.
 *  forced_first   device int32 [n_prompts*group] or NULL: when given, the
 *                 log-probability reported is that of this token.
 *  sp             host.
 *  out_tok        device int32 [n_prompts*group]: the sampled first tokens.
 *  out_logp       device float [n_prompts*group].
 *  out_logits     device float [n_prompts][vocab] (logits of each prompt's
 *                 last position) or NULL.
 * Afterwards each slot's length is its prompt length; the sampled token
 * takes position `length` and is fed back through rl_decode_step.
 * With group > 1 the slots of a group share the prompt for decode attention
 * (RL_OPT_SHARED_PREFIX) until one of them is released, prefilled or scored
 * again, or has its length set: then that slot and every slot reading
 * through it go back to their own copies.  K/V the caller writes into the
 * pool must be declared with rl_set_slot_lengths. */
rl_status rl_prefill(rl_decode_ctx* ctx, int32_t n_prompts, int32_t group,
                     const int32_t* slots, const uint64_t* seq_uids,
                     const int32_t* prompt_offsets, const int32_t* tokens,
                     const void* embeds, int32_t n_embed_rows,
                     const int32_t* forced_first, const rl_sample_params* sp,
                     int32_t* out_tok, float* out_logp, float* out_logits);

/* ---------------------------------------------------------------------
 * Inference stage: log-probabilities of given responses (Sec. 2.1, GRPO:
 * after generation the per-token log-probabilities of the responses are
 * computed by a forward pass over prompt + response, with no sampling).
 *
 * Sequence s (< n_prompts*group) is prompt p = s / group followed by
 * response s.  One causal forward over all tokens: each prompt is computed
 * once and its K/V written to all `group` slots of its group; the response
 * tokens of sequence s continue its slot at positions P, P+1, ...
 *  n_prompts, group, slots, prompt_offsets, prompt_tokens, embeds,
 *                 n_embed_rows: as rl_prefill.
 *  resp_offsets   host [n_prompts*group + 1], CSR offsets into resp_tokens;
 *                 resp_offsets[0] = 0; every response length m >= 1 with
 *                 P + m <= max_ctx.  All prompt plus all response tokens
 *                 <= max_prefill_tokens.
 *  resp_tokens    device int32 [resp_offsets[n]].
 *  temperature    >= 0; 0 reports the T = 1 value (as the arg-max sampler).
 *  out_logp       device float [resp_offsets[n]]:
 *                 out_logp[resp_offsets[s] + j] = fl32(z_y / T) - LSE(fl32(z / T))
 *                 with y = response token j and z the logits after the
 *                 prompt and response tokens 0..j-1; NaN when y is outside
 *                 [0, vocab).
 * The slots serve as scratch: their K/V is overwritten and they are empty
 * (length 0) afterwards.  The LM head runs in chunks of rows whose fp32
 * logits fit the workspace (max_seqs rows, or more when the MLP activation
 * buffer, free by then, holds more). */
rl_status rl_score(rl_decode_ctx* ctx, int32_t n_prompts, int32_t group, const int32_t* slots,
                   const int32_t* prompt_offsets, const int32_t* prompt_tokens,
                   const void* embeds, int32_t n_embed_rows,
                   const int32_t* resp_offsets, const int32_t* resp_tokens,
                   float temperature, float* out_logp);

/* ---------------------------------------------------------------------
 * One decode step (the rollout's hot loop: Sec. 2.1, generation extends every
 * unfinished response by one token and the RL loss later consumes each
 * token's log-probability; Sec. 5.1.2, the token and its log-probability come
 * from the same forward pass; Sec. 5.2, temperature).
 *
 * For each row i < n: appends in_tok[i] to slot slots[i] at position
 * p = length(slot), attends over positions 0..p, and samples the token of
 * position p + 1 with noise keyed by (sp->seed, seq_uids[i], p + 1, vocab
 * index) -- independent of the slot and of the other rows.
 *  n          0 <= n <= max_seqs (0 is a no-op).
 *  slots      host int32 [n], distinct, each with length < max_ctx.
 *  seq_uids   host uint64 [n].
 *  in_tok     device int32 [n]; out-of-range ids embed as zeros.
 *  forced_tok device int32 [n] or NULL (teacher forcing: report the
 *             log-probability of this token instead of the sampled one).
 *  out_tok    device int32 [n]  sampled token.
 *  out_logp   device float [n]  log-probability (forced or sampled token).
 *  out_logits device float [n][vocab] or NULL.
 * Every slot's length grows by one.  Nothing synchronises the stream. */
rl_status rl_decode_step(rl_decode_ctx* ctx, int32_t n, const int32_t* slots,
                         const uint64_t* seq_uids, const int32_t* in_tok,
                         const int32_t* forced_tok, const rl_sample_params* sp,
                         int32_t* out_tok, float* out_logp, float* out_logits);

/* Sample from caller-provided fp32 logits with the same rule as the step.
 *  logits   device float [n][vocab];  n <= max_seqs.
 *  seq_uids host uint64 [n]; pos_new host int32 [n] (position the sampled
 *           token takes, >= 0).
 *  forced   device int32 [n] or NULL.  out_tok/out_logp device [n]. */
rl_status rl_sample_logits(rl_decode_ctx* ctx, int32_t n, const float* logits,
                           const uint64_t* seq_uids, const int32_t* pos_new,
                           const int32_t* forced, const rl_sample_params* sp,
                           int32_t* out_tok, float* out_logp);

/* Allocation-free variant of rl_sample_logits, for callers that cannot
 * allocate device memory or own a workspace: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  Needs no context,
 * calls no allocating routine, and gives the same tokens and
 * log-probabilities as rl_sample_logits for the same inputs.
 *  n          rows, 0 <= n <= 2^20 (0 is a no-op).
 *  vocab      entries per row, a multiple of 4, <= 2^24.
 *  logits     device float [n][ld], 16-byte aligned; ld >= vocab, ld % 4 == 0.
 *  seq_uids   device uint64 [n]; pos_new device int32 [n] (>= 0): the noise
 *             key of each row, as in rl_decode_step.
 *  forced     device int32 [n] or NULL.  sp host (as rl_decode_step).
 *  out_tok, out_logp  device [n].
 *  stream     hipStream_t of the current device.
 * The per-chunk partial results go to a fixed device array of the library
 * (4096 entries of 16 bytes, 64 KiB; every n fits), one per device, held
 * until the process ends.  Every call on a device shares that array: calls
 * that overlap on one device (two streams, or two threads) race and give
 * wrong results; calls on one stream are ordered and safe.
 * RL_ERR_INVALID_ARG for bad sizes or pointers, RL_ERR_CAPACITY if a launch
 * would need more partials than the array holds, RL_ERR_HIP if the launch
 * or the array's lookup fails. */
rl_status rl_sample_logits_noalloc(int32_t n, int32_t vocab, const float* logits, int32_t ld,
                                   const uint64_t* seq_uids, const int32_t* pos_new, const int32_t* forced,
                                   const rl_sample_params* sp, int32_t* out_tok, float* out_logp, void* stream);

/* ---------------------------------------------------------------------
 * Slot bookkeeping (host only; nothing is enqueued).
 * ------------------------------------------------------------------- */

/* Mark slots empty (length 0) so they can take new sequences. */
rl_status rl_release_slots(rl_decode_ctx* ctx, int32_t n, const int32_t* slots);

/* Declare lengths of slots whose K/V the caller wrote into the pool itself
 * (layout above), or cut sequences short.  lengths[i] in [0, max_ctx].  On a
 * paged pool a length that ends inside a page shared with other slots
 * enqueues a copy of that page on the context's stream. */
rl_status rl_set_slot_lengths(rl_decode_ctx* ctx, int32_t n, const int32_t* slots,
                              const int32_t* lengths);

/* Length of a slot, or -1 for an invalid context or slot. */
int32_t rl_slot_length(const rl_decode_ctx* ctx, int32_t slot);

/* Free pages of a paged K/V pool (admission control: a prompt group of
 * length p and group g needs floor(p/P) shared pages plus, per slot, the
 * pages of the rest of its length); -1 for a contiguous pool or an invalid
 * context. */
int64_t rl_kv_free_pages(const rl_decode_ctx* ctx);

/* ---------------------------------------------------------------------
 * Context switching (Sec. 3: in temporal mode a worker's GPU state is
 * offloaded so that the next stage can use the devices, and reloaded when
 * it runs again; Sec. 5.1.1 counts that cost in "Others").
 *
 * Packed K/V of slot s (length n = its current length, E = element size):
 * for every layer l and kv-head h (index l*Hkv + h): n K rows of head_dim
 * elements, then ceil(n/8) V blocks of 8 positions (the pool's own layouts),
 * i.e. n_layers * Hkv * (n + ceil8(n)) * head_dim * E bytes; slots follow
 * one another in the order given.  The copies go through the workspace (a
 * chunk of whole slots at a time); the host buffer should be pinned
 * (hipHostMalloc) for full PCIe speed.  Weights are the caller's tensors and
 * are moved by the caller.
 * ------------------------------------------------------------------- */

/* Bytes rl_kv_offload writes for these slots; 0 for an invalid context or
 * slot. */
size_t rl_kv_offload_bytes(const rl_decode_ctx* ctx, int32_t n, const int32_t* slots);

/* Copy the live K/V of n distinct slots to host_dst (host_bytes >= the size
 * above).  Asynchronous: host_dst is complete once the stream is
 * synchronised.  Slot state is unchanged (release the slots to reuse them).
 * RL_ERR_CAPACITY when one slot's K/V exceeds the workspace's staging region
 * (the activation buffers). */
rl_status rl_kv_offload(rl_decode_ctx* ctx, int32_t n, const int32_t* slots, void* host_dst,
                        size_t host_bytes);

/* Copy packed K/V from host_src into n distinct slots and set their
 * lengths (lengths[i] in [0, max_ctx]; the layout above for these
 * lengths).  The slots need not be those it was offloaded from.  They read
 * their own copies afterwards (no prompt sharing). */
rl_status rl_kv_onload(rl_decode_ctx* ctx, int32_t n, const int32_t* slots, const int32_t* lengths,
                       const void* host_src, size_t host_bytes);

/* Point the context at new device buffers (same sizes and alignment rules
 * as rl_decode_create), e.g. after the caller freed the old ones during a
 * context switch.  Waits for the context's outstanding work, then writes the
 * RoPE table into the new workspace (synchronises the stream).  Slot lengths are kept: reload their K/V with rl_kv_onload, or
 * release them. */
rl_status rl_decode_rebind(rl_decode_ctx* ctx, const rl_weights* w, void* kv_pool, size_t kv_bytes,
                           void* workspace, size_t ws_bytes);

/* ---------------------------------------------------------------------
 * Options and measurement.
 * ------------------------------------------------------------------- */

typedef enum rl_option {
    RL_OPT_ATTN_CHUNK = 1,   /* positions per split-KV chunk: 0 = automatic
                                (decode steps that read shared prompts: 256;
                                other decode steps: the largest power of two
                                that still gives about 1024 work items;
                                prefill and scoring: 1024), else a multiple of
                                32 in [32, 65536]; doubled as needed so no
                                sequence has more than 64 chunks and the work
                                items fit the workspace                        */
    RL_OPT_PROFILE = 2,      /* bit mask over rl_kernel_class: launches of the
                                selected classes are timed with HIP events on
                                the context's stream (the bf16 decode
                                attention by events stamped at the kernel's
                                own start and end; the other classes by an
                                event pair around the launch, which also spans
                                the dispatch gap); 0 = off (default),
                                -1 = every class                              */
    RL_OPT_GEMM_PLAN = 3,    /* bf16 GEMM kernel override (testing every tile
                                kernel on small models): 0 = the cost-model
                                planner (default); else
                                  bits 0-7:   rl_gemm_kernel of all columns
                                              (or of the first half, below),
                                  bits 8-15:  split-K count s (0 or 1 = none,
                                              else <= 32; the K slices are
                                              whole 64-wide blocks, so the
                                              count used is K over
                                              ceil(K/s) rounded up to 64),
                                  bits 16-23: rl_gemm_kernel of the second
                                              half of the output columns
                                              (0 = one segment; no split-K).
                                A GEMM the override cannot serve (GEMV with
                                M > 32, direct-load or wide GEMV with M > 64,
                                a tile kernel or either GEMV with K not a
                                multiple of 64, a wide GEMV whose split-K
                                partials would exceed 32 Mi floats) keeps
                                the planner's choice.  Results stay within the
                                parity tolerances for every choice; the bits
                                differ (fp32 summation order).               */
    RL_OPT_SHARED_PREFIX = 4, /* 1 (default): decode attention of the slots of
                                one rl_prefill group reads the prompt's K/V
                                from the group's first slot (every slot of
                                the group holds the same copy), in 32-position
                                steps, and keeps the readers of one prompt
                                chunk on one XCD, so each prompt chunk is read
                                from HBM about once per group; 0: every slot
                                reads its own copy.  The same function; the
                                bits differ (fp32 summation order).        */
    RL_OPT_PREFILL_ATTENTION = 5 /* attention of rl_prefill and rl_score: 0
                                (default) workgroups of consecutive query
                                tokens sharing each K/V step through LDS; 1:
                                the decode kernel's split-KV work items
                                (RL_OPT_ATTN_CHUNK applies).  Results agree
                                within the parity tolerances.             */
} rl_option;

typedef enum rl_gemm_kernel {
    RL_GEMM_DIRECT = 1,      /* direct-load MFMA kernel (M <= 64)            */
    RL_GEMM_GEMV = 2,        /* 16 weight rows x all K per workgroup (M <= 32) */
    RL_GEMM_T256 = 3,        /* 256 x 256 tiles, 8 waves                      */
    RL_GEMM_T128X256 = 4,    /* 128 x 256 tiles, 8 waves                      */
    RL_GEMM_T128 = 5,        /* 128 x 128 tiles, 4 waves, two per CU          */
    RL_GEMM_T128_DEEP = 6,   /* 128 x 128 tiles, 4 waves, 4-stage ring        */
    RL_GEMM_GEMV_WIDE = 7    /* 64 weight rows x a K slice per workgroup
                                (M <= 64; split-K allowed)                    */
} rl_gemm_kernel;

rl_status rl_decode_set_option(rl_decode_ctx* ctx, int32_t option, int64_t value);

typedef enum rl_kernel_class {
    RL_K_EMBED = 0, RL_K_RMSNORM, RL_K_GEMM_QKV, RL_K_ROPE_APPEND, RL_K_ATTENTION,
    RL_K_ATTN_COMBINE, RL_K_GEMM_O, RL_K_GEMM_GATE_UP, RL_K_GEMM_DOWN, RL_K_GEMM_LM_HEAD,
    RL_K_SPLITK_REDUCE, RL_K_SAMPLE,
    RL_K_MOE_ROUTE,          /* router projection, top-k and grouping by expert */
    RL_K_MOE_EXPERTS,        /* the grouped expert projections */
    RL_K_COUNT
} rl_kernel_class;

/* Measured GEMM plans.  The decode batch of a rollout shrinks from the whole
 * batch to a few long responses (Sec. 2.2, the long tail), so the bf16
 * projections run at every row count from max_seqs down to 1.  For each
 * batch size in `sizes` (host array of n_sizes strictly increasing values in
 * [1, max_seqs]) and each of the q|k|v, o, gate-up, down and LM-head
 * projections, every plan of the cost model's search space (tile kernel or
 * GEMV form, split-K count, two-segment launch) is timed on the context's stream with
 * HIP events, each together with the kernel that consumes its output as a
 * decode step issues it; the fastest few and the cost model's plan are then
 * timed inside whole decode steps of that many rows, one projection at a
 * time, and the fastest step's plan is kept.  A GEMM of M rows then uses the
 * plan measured for the smallest listed size >= M; larger M keep the cost
 * model, and RL_OPT_GEMM_PLAN still overrides.  n_sizes = 0 clears the
 * table.  The context must hold no live sequence (every slot length 0:
 * before the first prefill, or after releasing every slot; RL_ERR_INVALID_ARG
 * otherwise): the measuring steps decode slots 0 .. largest size - 1 at a
 * short context, overwrite their K/V and the workspace, and leave every
 * length at 0 (on a paged pool they take pages and return every one; a pool
 * too small for them fails with RL_ERR_CAPACITY, the table cleared).
 * Synchronises the stream.  Every plan gives results within
 * the parity tolerances; the bits depend on the plan (fp32 summation
 * order), so the table is part of a run's configuration.  Dense bf16 models
 * only (RL_ERR_UNSUPPORTED for fp32 or a mixture of experts when
 * n_sizes > 0).  Takes about 0.3 s per
 * size at the 7B shape. */
rl_status rl_decode_tune_gemms(rl_decode_ctx* ctx, int32_t n_sizes, const int32_t* sizes);

/* The plan a projection of class kclass (one of the five GEMM classes) at
 * `rows` rows (1 .. max(max_seqs, max_prefill_tokens)) uses now, as an
 * RL_OPT_GEMM_PLAN code in *plan_code, and its measured microseconds per
 * layer (unit time with its consumer) in *tuned_us (may be NULL), or -1 when
 * the plan comes from the cost model or the override.  bf16 models only. */
rl_status rl_decode_gemm_plan(rl_decode_ctx* ctx, int32_t kclass, int32_t rows, int64_t* plan_code,
                              float* tuned_us);

/* Accumulated per-class figures since the last reset, collected for the
 * launches made while RL_OPT_PROFILE selects the class (launches made with
 * the class deselected are neither counted nor timed).  alg_bytes / alg_flops are the algorithmic HBM bytes
 * and FLOPs of the launches (what the operation must move or compute, not
 * what the kernel happens to move).  Synchronises the stream. */
typedef struct rl_kernel_stats {
    int64_t launches;
    double  total_ms;
    double  alg_bytes;
    double  alg_flops;
    char    name[48];
} rl_kernel_stats;

rl_status rl_decode_kernel_stats(rl_decode_ctx* ctx, int32_t kclass, rl_kernel_stats* out);

/* Shape of the decode attention's work-item plans, summed over the
 * rl_decode_step calls since the last reset (one plan serves every layer of
 * a call).  Host-side counters, always collected; nothing is synchronised.
 * A work item is one wave's key range for up to 16 query columns; a pair
 * item serves two sequences that read the same shared prompt chunk
 * (RL_OPT_SHARED_PREFIX); an LDS workgroup is a workgroup of four items over
 * one shared chunk that stages each K/V step through LDS once. */
typedef struct rl_attn_plan_stats {
    int64_t steps;            /* rl_decode_step calls counted               */
    int64_t items;            /* work items (padding excluded)              */
    int64_t shared_items;     /* items over a shared prompt chunk           */
    int64_t pair_items;       /* items serving two sequences                */
    int64_t lds_workgroups;   /* workgroups staging a shared chunk in LDS   */
} rl_attn_plan_stats;

rl_status rl_decode_attn_plan_stats(const rl_decode_ctx* ctx, rl_attn_plan_stats* out);

/* Zero the kernel-class figures and the attention plan counters. */
rl_status rl_decode_reset_stats(rl_decode_ctx* ctx);

/* Plain device-to-device copy kernel (16-byte vector loads and stores) of
 * `bytes` bytes (a multiple of 16; both pointers 16-byte aligned) on
 * `stream`.  Used to calibrate hardware byte counters against a known size. */
rl_status rl_probe_copy(void* dst, const void* src, size_t bytes, void* stream);

/* Measured peaks beside the published ones.  rl_probe_read: a read-only
 * stream of `bytes` bytes at src (a multiple of 16; 16-byte aligned) by
 * n_blocks (1..65536) workgroups, four 16-byte loads in flight per thread;
 * out (device, n_blocks uint32) receives each workgroup's XOR of the words
 * it read (so the reads cannot be elided; the XOR of all entries is the XOR
 * of every 32-bit word of the buffer).  rl_probe_mfma: n_blocks (1..65536)
 * workgroups of four waves, each wave iters (1..2^20) rounds of eight
 * independent 32x32x16 bf16 MFMAs (32768 FLOPs each) on operands of 1.0 and
 * no memory traffic; out (device, 4 * n_blocks floats) receives 128 * iters
 * per wave.  Both asynchronous on `stream`; RL_ERR_INVALID_ARG for bad
 * sizes or pointers.  Test probes, not part of the decode path. */
rl_status rl_probe_read(const void* src, size_t bytes, int32_t n_blocks, uint32_t* out, void* stream);
rl_status rl_probe_mfma(int32_t n_blocks, int32_t iters, float* out, void* stream);

/* Check of the two upper bounds of the Gumbel noise g(x) = fl32(-log(-log u)),
 * u = (x + 1/2) 2^-32, that the sampler uses to skip the exact fp64 noise of
 * entries that cannot win (the sample stays the exhaustive arg-max only if
 * both hold), evaluated with the sampler's own device code over the noise
 * words [lo, lo + count), count <= 2^32 and lo + count <= 2^32:
 *   x <  0xFF000000: the fp32 hardware-logarithm bound >= g(x), 5.56 >= g(x);
 *   x >= 0xFF000000: 22.9 >= g(x).
 * viol and min_margin are device arrays of n_blocks (1..65536) entries; each
 * workgroup writes its count of violations and the smallest margin of the
 * fp32 bound over its words (+inf if it saw none below 0xFF000000).
 * Asynchronous on `stream`.  A test probe, not part of the decode path. */
rl_status rl_probe_gumbel_bound(uint32_t lo, uint64_t count, int32_t n_blocks, uint32_t* viol, float* min_margin,
                                void* stream);

/* Static description of a status code. */
const char* rl_status_string(rl_status s);

/* Message describing the last error seen by this context ("" if none). */
const char* rl_decode_last_error(const rl_decode_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* RL_DECODE_H */
