/*
 * dlm.h -- C ABI of the MI355X (gfx950) refinement-step library.
 *
 * The library runs the refinement stage of draft-then-refine decoding for
 * diffusion language models (paper: Sec. 4.2 "Bidirectional Refinement"):
 * the refiner receives a fixed prompt and a complete draft, runs a
 * bidirectional (non-causal) transformer forward over the whole sequence,
 * reduces each draft position's vocabulary logits to a top-1 token and its
 * confidence, and applies a threshold rule that re-edits draft tokens and
 * unmasks [MASK] positions.  The pass budget is an upper bound: the loop stops
 * once a pass changes nothing (App. C.4; one refine threshold, Table 10).
 *
 * Conventions for every entry point
 *   - Pointers named d_* are device pointers (HIP device memory on the current
 *     device); h_* are host pointers.  The caller owns every buffer: weights,
 *     workspace, tokens and outputs.  The library owns only the small host
 *     handle returned by dlm_load_synthetic_weights, freed by dlm_free.
 *   - hip_stream is a hipStream_t passed as void* (NULL = the default stream).
 *     All device work is enqueued on it; entry points return without waiting
 *     unless stated.
 *   - Return value: DLM_OK (0) or a negative dlm_status.  On error nothing is
 *     launched, and dlm_last_error() returns a message (thread-local).  No C++
 *     exception crosses this boundary.
 *   - Integers are int32 unless stated; token arrays are row-major int32
 *     [batch][len].  Floats are IEEE binary32.
 */
#ifndef DLM_H
#define DLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DLM_OK = 0,
    DLM_ERR_INVALID_ARG = -1,   /* bad shape, null pointer, non-finite threshold ... */
    DLM_ERR_HIP = -3,           /* a HIP runtime call failed                          */
    DLM_ERR_UNSUPPORTED = -4,   /* a shape the kernels do not implement              */
    DLM_ERR_WORKSPACE = -5,     /* weights or workspace buffer too small             */
    DLM_ERR_NO_MEMORY = -6,     /* a host memory allocation inside the library failed */
    DLM_ERR_INTERNAL = -7       /* any other unexpected host-side failure            */
} dlm_status;

/*
 * Refiner shape.  Architecture (the paper does not describe the refiner's
 * internals, Sec. 5.1): pre-norm RMSNorm blocks, rotate-half RoPE on q and k
 * with positions 0..S-1 of each sequence, non-causal grouped-query attention,
 * then either a dense SwiGLU FFN (n_experts == 0) or a softmax-routed top-k
 * SwiGLU mixture of experts renormalised over the k selected, plus
 * n_shared_experts (0 or 1) always-on experts of width expert_ffn_dim; a final
 * RMSNorm and an untied LM head.  mask_id is the [MASK] token id.
 * Supported: head_dim 64 or 128; d_model, n_heads*head_dim multiples of 128;
 * ffn widths multiples of 64; n_experts <= 256; top_k <= 8; vocab >= 2.
 * Shapes: batch * (prompt_len + draft_len) tokens times max(d_model,
 * n_heads*head_dim) bf16 values must stay below 2 GiB (the kernels address
 * activations with 32-bit offsets); larger shapes are DLM_ERR_INVALID_ARG.
 */
typedef struct dlm_config {
    int32_t n_layers;
    int32_t d_model;
    int32_t n_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t ffn_dim;           /* dense SwiGLU width (n_experts == 0)           */
    int32_t n_experts;         /* routed experts, 0 = dense FFN                  */
    int32_t top_k;
    int32_t expert_ffn_dim;    /* width of routed and shared experts            */
    int32_t n_shared_experts;  /* 0 or 1                                        */
    int32_t vocab;
    int32_t mask_id;           /* 0 <= mask_id < vocab                          */
    float rope_theta;          /* e.g. 10000                                    */
    float norm_eps;            /* e.g. 1e-6                                     */
    float init_std;            /* synthetic weight standard deviation (0.02)    */
    float lm_head_scale;       /* extra factor on the LM head's init std (1.0)  */
} dlm_config;

typedef struct dlm_model dlm_model;   /* opaque host handle */

/* Counters of one pass or of a whole refine call. */
typedef struct dlm_stats {
    int32_t n_unmasked;     /* [MASK] slots that took a token                    */
    int32_t n_edited;       /* real-token slots that changed                     */
    int32_t n_masked_left;  /* [MASK] slots left at the end (dlm_refine only)    */
    int32_t steps_run;      /* passes executed (dlm_refine only)                 */
    int32_t n_invalid;      /* token ids outside [0, vocab), or mask_id in the   */
                            /* prompt, seen by the pass (it then wrote nothing)  */
} dlm_stats;

/*
 * Token validation (Sec. 4.2: the prompt is fixed context, only the draft is
 * editable, so the prompt holds real tokens).  Every pass checks on the device
 * that each token id lies in [0, vocab) and that no prompt slot holds mask_id.
 * A pass that finds such an id updates no slot and counts the ids in
 * dlm_stats.n_invalid.  The entry points that synchronise once per pass
 * (dlm_refine, dlm_refine_ex, dlm_refine_local, dlm_draft, dlm_cascade) read
 * the count at that synchronisation and return DLM_ERR_INVALID_ARG; the
 * asynchronous single-pass entry points (dlm_refine_step*, dlm_draft_step)
 * report it through d_stats only.
 */

/* Bytes of device memory the weights of cfg occupy (0 if cfg is invalid). */
size_t dlm_weights_bytes(const dlm_config* cfg);

/* Bytes of device workspace one pass over a [batch][prompt_len + draft_len]
 * token array needs (0 if the arguments are invalid). */
size_t dlm_workspace_bytes(const dlm_config* cfg, int32_t batch, int32_t prompt_len,
                           int32_t draft_len);

/*
 * Fill d_weights (>= dlm_weights_bytes(cfg) bytes, 256-byte aligned) with the
 * synthetic weights of cfg for `seed`, on hip_stream, and return a handle in
 * *out.  Weight element i (row-major in the logical [out_features x
 * in_features] matrix) of tensor `tid` is
 *     n = sum of the four 16-bit halves of words 0,1 of
 *         Philox4x32-10(counter = (i_lo, i_hi, tid, 0), key = (seed_lo, seed_hi))
 *         minus 131070,
 *     w = bf16_round_nearest_even(float(n) * float(init_std * s * sqrt(3) / 65536))
 * with s = lm_head_scale for the LM head and 1 otherwise; tid =
 * (layer_field << 20) | (kind << 12) | expert with layer_field 0 for the
 * embedding (kind 0) and the LM head (kind 1), and l+1 for layer l with kinds
 * Wq 0, Wk 1, Wv 2, Wo 3, dense gate 4 / up 5 / down 6, router 7, expert gate 8
 * / up 9 / down 10, shared gate 11 / up 12 / down 13.  RMSNorm gains are 1.
 * The handle keeps d_weights (not owned); the buffer must outlive it.
 */
dlm_status dlm_load_synthetic_weights(const dlm_config* cfg, uint64_t seed, void* d_weights,
                                      size_t weights_bytes, void* hip_stream, dlm_model** out);

/*
 * One refinement pass (Sec. 4.2) over d_tokens [batch][prompt_len + draft_len]
 * (in/out): forward over all positions with no attention mask, then for every
 * draft position p the top-1 token t* (lowest id among equal maxima) and its
 * confidence conf = 1 / sum_v exp(z_v - max z), then all draft positions are
 * updated at once: a slot takes t* when t* != mask_id and conf >= threshold.
 * Prompt slots are never written.  Draft slots may hold mask_id; the prompt
 * may not (see token validation above: such a pass writes nothing and
 * d_stats->n_invalid counts the offending ids).
 * Optional outputs (NULL to skip), device pointers:
 *   d_top1 int32 [batch][draft_len], d_conf float [batch][draft_len],
 *   d_stats dlm_stats (n_unmasked, n_edited, n_invalid of this pass; other
 *   fields 0).
 * threshold must not be NaN (any other float is accepted; > 1 edits nothing,
 * <= 0 takes every top-1 that is not mask_id).
 * The call only enqueues kernels and device-to-device copies on hip_stream;
 * it allocates nothing, records no memset and never waits on the host, so it
 * may be captured in a HIP graph (stream capture) and replayed (as may
 * dlm_refine_step_static and dlm_refine_step_ex).
 */
dlm_status dlm_refine_step(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                           int32_t* d_tokens, float threshold, void* d_workspace,
                           size_t workspace_bytes, void* hip_stream, int32_t* d_top1,
                           float* d_conf, dlm_stats* d_stats);

/*
 * dlm_refine_step for callers that cannot allocate device memory or pass a
 * workspace (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same pass and the same results, with the workspace in
 * a static device array of DLM_STATIC_SCRATCH_BYTES that the library holds on
 * every GPU it runs on until the process ends.  The call allocates nothing.
 * Shapes whose workspace (dlm_workspace_bytes) exceeds the array return
 * DLM_ERR_WORKSPACE with nothing launched.  The model's device (current when
 * its weights were loaded) must be current.  Every call on one GPU uses the
 * same array: calls that overlap on one GPU (other streams, other threads,
 * other models) race and must be serialised by the caller.  Arguments and
 * results as dlm_refine_step.
 */
#define DLM_STATIC_SCRATCH_BYTES (64u << 20)
dlm_status dlm_refine_step_static(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                                  int32_t* d_tokens, float threshold, void* hip_stream, int32_t* d_top1,
                                  float* d_conf, dlm_stats* d_stats);

/*
 * Refine a draft: slots with d_mask[b][i] != 0 start as mask_id (d_mask may be
 * NULL = empty mask set), then up to n_steps passes of dlm_refine_step,
 * stopping after a pass that changed no slot.  d_prompt int32 [batch][prompt_len]
 * is read only; d_draft int32 [batch][draft_len] is updated in place.  Blocks
 * the calling thread once per pass (a 16-byte device-to-host copy) to decide the
 * early stop.  h_stats (host, may be NULL) receives totals over all passes.
 * n_steps = 0 only applies the mask set.  A pass that finds an invalid token id
 * ends the call with DLM_ERR_INVALID_ARG and d_draft unchanged.
 */
dlm_status dlm_refine(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                      const int32_t* d_prompt, int32_t* d_draft, const uint8_t* d_mask,
                      int32_t n_steps, float threshold, void* d_workspace, size_t workspace_bytes,
                      void* hip_stream, dlm_stats* h_stats);

/*
 * Editing rule with separate thresholds and an EOS stop (App. C.4: the native
 * token-editing rule ends a refinement early once no confident edit remains or
 * an EOS token is produced; the reading used here):
 *   a [MASK] draft slot takes t* when t* != mask_id and conf >= unmask_threshold;
 *   a real-token draft slot takes t* when t* != mask_id and conf >= edit_threshold;
 *   with eos_id >= 0, a pass that writes eos_id into at least one draft slot
 *   (a slot that did not already hold it) ends dlm_refine_ex after that pass.
 * unmask_threshold == edit_threshold with eos_id < 0 is the rule of
 * dlm_refine_step.  Thresholds must not be NaN; eos_id < vocab.
 */
typedef struct dlm_edit_rule {
    float unmask_threshold;
    float edit_threshold;
    int32_t eos_id;            /* < 0: no EOS stop */
} dlm_edit_rule;

/*
 * dlm_refine_step under *rule (host pointer).  d_eos_written (device int32,
 * may be NULL) receives the number of draft slots this pass set to eos_id
 * (0 when rule->eos_id < 0).  Other arguments as dlm_refine_step.
 */
dlm_status dlm_refine_step_ex(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                              int32_t* d_tokens, const dlm_edit_rule* rule, void* d_workspace,
                              size_t workspace_bytes, void* hip_stream, int32_t* d_top1, float* d_conf,
                              dlm_stats* d_stats, int32_t* d_eos_written);

/*
 * dlm_refine under *rule: stops after a pass that changed no slot, or (eos_id
 * >= 0) after a pass that wrote eos_id into a draft slot.  h_stop_reason (host,
 * may be NULL): 0 = pass budget used up (or n_steps = 0), 1 = a pass changed
 * nothing, 2 = EOS written.  Other arguments as dlm_refine.
 */
dlm_status dlm_refine_ex(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                         const int32_t* d_prompt, int32_t* d_draft, const uint8_t* d_mask, int32_t n_steps,
                         const dlm_edit_rule* rule, void* d_workspace, size_t workspace_bytes,
                         void* hip_stream, dlm_stats* h_stats, int32_t* h_stop_reason);

/*
 * Local refinement (Sec. 6.3 / Table 10: refinement applied to 64-token
 * chunks of the generated span instead of the whole span; App. D.4: staged
 * schedules such as two passes at span 256 then two at 512).  Reading used
 * here: a chunk is refined on its own, attending to the prompt and the chunk
 * only, its tokens keeping their positions in the full sequence.
 *
 * dlm_refine_step_span: one pass over d_tokens [batch][prompt_len + span_len]
 *   = prompt ‖ span, whose span token i sits at position prompt_len +
 *   span_start + i (RoPE); otherwise as dlm_refine_step_ex.
 * dlm_refine_local: for each stage g < n_stages (host arrays h_span, h_passes),
 *   the draft is cut into chunks of h_span[g] tokens (the last may be shorter)
 *   and each chunk gets up to h_passes[g] passes of dlm_refine_step_span,
 *   stopping after a pass that changed nothing in it; the whole run ends after
 *   a pass that wrote rule->eos_id (eos_id >= 0).  Slots with d_mask != 0
 *   (may be NULL) start as mask_id; d_draft [batch][draft_len] is updated in
 *   place.  The workspace is the one of (batch, prompt_len, draft_len).
 *   h_stats: totals over all passes; h_stop_reason: 0 = some chunk used its
 *   whole pass budget, 1 = every chunk stopped on a pass without change, 2 =
 *   EOS written.  A schedule of one stage with span >= draft_len is
 *   dlm_refine_ex.
 */
dlm_status dlm_refine_step_span(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t span_len,
                                int32_t span_start, int32_t* d_tokens, const dlm_edit_rule* rule, void* d_workspace,
                                size_t workspace_bytes, void* hip_stream, int32_t* d_top1, float* d_conf,
                                dlm_stats* d_stats, int32_t* d_eos_written);
dlm_status dlm_refine_local(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                            const int32_t* d_prompt, int32_t* d_draft, const uint8_t* d_mask, int32_t n_stages,
                            const int32_t* h_span, const int32_t* h_passes, const dlm_edit_rule* rule,
                            void* d_workspace, size_t workspace_bytes, void* hip_stream, dlm_stats* h_stats,
                            int32_t* h_stop_reason);

/*
 * Block-AR drafting (Sec. 3.3 Block Autoregressive Diffusion, Sec. 4.1
 * Drafting; the b/s/t settings of Table 9 and Table 10: block size, steps per
 * block, confidence threshold).
 *
 * The draft_len response positions after the prompt are cut into blocks of
 * block_len (1..1024; the last block may be shorter), generated in order.
 * Visibility is block-causal: a position of block k attends to the prompt,
 * to blocks 0..k-1 and to its own block; the prompt attends to itself.  K and
 * V of the prompt and of finished blocks are computed once, from their final
 * tokens, and kept per layer in the workspace.  Each block starts all
 * [MASK]; one step is a forward of the block's rows followed by the
 * unmasking: with n masked slots in the block (per sequence) and r steps left
 * for it, quota = ceil(n / r); every masked slot whose confidence (softmax
 * probability of its top-1) is >= threshold takes its top-1, or, when those
 * are fewer than the quota, the quota most confident masked slots do (equal
 * confidences: lower position first).  Drafting never changes a real token.
 * A block ends once no sequence of the batch has a [MASK] in it, at the
 * latest after steps_per_block steps.
 *
 * dlm_draft_workspace_bytes: device workspace size for the drafting entry
 *   points at (batch, prompt_len, draft_len, block_len); 0 for an invalid
 *   shape.  It holds the per-layer K/V caches of all prompt_len + draft_len
 *   positions.
 * dlm_draft: d_prompt int32 [batch][prompt_len] (may be NULL when prompt_len
 *   is 0), d_draft int32 [batch][draft_len] (output; every slot is
 *   written).  h_stats (host, may be NULL): n_unmasked = slots given a real
 *   token, n_edited = 0, n_masked_left = [MASK] slots left in the draft (a
 *   step may select a slot whose top-1 is mask_id itself), steps_run = steps
 *   over all blocks.  h_block_steps (host, may be NULL): steps of each block,
 *   ceil(draft_len / block_len) entries.  Synchronises the stream once per
 *   step (the block's stop test) and returns when the draft is written.
 * dlm_draft_step: one step on block block_index of d_tokens int32
 *   [batch][prompt_len + draft_len] (prompt, finished blocks, the block in
 *   progress; later positions are not read), with steps_left (>= 1) steps
 *   left for the block; the K/V of the prompt and of the earlier blocks are
 *   computed from d_tokens first.  The block's slots are updated in place;
 *   d_top1 / d_conf / d_max_logit (device, may be NULL) receive the top-1,
 *   its confidence and the max logit of the block's rows [batch][block rows]
 *   (before the update); d_stats (device, may be NULL):
 *   n_unmasked, n_edited = 0, n_masked_left in the block, steps_run = 1.
 *   Asynchronous on hip_stream.
 * Errors: NULL handle / buffers, block_len outside 1..1024, steps < 1,
 * block_index out of range, NaN threshold -> DLM_ERR_INVALID_ARG; workspace
 * too small -> DLM_ERR_WORKSPACE.  Token ids must lie in [0, vocab).
 */
size_t dlm_draft_workspace_bytes(const dlm_config* cfg, int32_t batch, int32_t prompt_len, int32_t draft_len,
                                 int32_t block_len);
dlm_status dlm_draft(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len, const int32_t* d_prompt,
                     int32_t* d_draft, int32_t block_len, int32_t steps_per_block, float threshold,
                     void* d_workspace, size_t workspace_bytes, void* hip_stream, dlm_stats* h_stats,
                     int32_t* h_block_steps);
dlm_status dlm_draft_step(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len, int32_t block_len,
                          int32_t block_index, int32_t steps_left, float threshold, int32_t* d_tokens,
                          void* d_workspace, size_t workspace_bytes, void* hip_stream, int32_t* d_top1,
                          float* d_conf, float* d_max_logit, dlm_stats* d_stats);

/*
 * Speculative correction with two models (Sec. 4.3: a smaller drafter, the
 * larger refiner; Sec. 4.2: the cost counted as K x T_d drafting passes plus
 * T_r refinement passes; Sec. 5.3 / App. A: model time = drafting + refinement
 * time only).
 *
 * dlm_cascade: dlm_draft with `drafter` (blocks of block_len, up to
 *   steps_per_block steps, draft_threshold), then dlm_refine_ex with `refiner`
 *   on the finished draft (no mask set; up to n_refine_steps passes under
 *   *rule).  The two models must share vocab and mask_id.  d_prompt int32
 *   [batch][prompt_len] (may be NULL when prompt_len is 0), d_draft int32
 *   [batch][draft_len] receives the refined draft.  One workspace serves both
 *   stages (they run one after the other): dlm_cascade_workspace_bytes, the
 *   larger of the two stages' sizes.  h_stats (host, may be NULL): the draft
 *   and refine stats, the pass counts of each stage, the refine stop reason
 *   (as dlm_refine_ex) and the host wall-clock milliseconds of each stage
 *   (each stage returns with its output written).  Synchronises the stream.
 *   Errors as dlm_draft and dlm_refine_ex; models of different vocabularies
 *   -> DLM_ERR_INVALID_ARG.
 */
typedef struct dlm_cascade_stats {
    dlm_stats draft;           /* as dlm_draft's h_stats */
    dlm_stats refine;          /* as dlm_refine_ex's h_stats */
    int32_t draft_passes;      /* K x (steps used per block), summed over blocks */
    int32_t refine_passes;     /* T_r actually run */
    int32_t refine_stop_reason;
    int32_t reserved;
    double draft_ms;
    double refine_ms;
} dlm_cascade_stats;

size_t dlm_cascade_workspace_bytes(const dlm_config* drafter_cfg, const dlm_config* refiner_cfg, int32_t batch,
                                   int32_t prompt_len, int32_t draft_len, int32_t block_len);
dlm_status dlm_cascade(dlm_model* drafter, dlm_model* refiner, int32_t batch, int32_t prompt_len, int32_t draft_len,
                       const int32_t* d_prompt, int32_t* d_draft, int32_t block_len, int32_t steps_per_block,
                       float draft_threshold, int32_t n_refine_steps, const dlm_edit_rule* rule, void* d_workspace,
                       size_t workspace_bytes, void* hip_stream, dlm_cascade_stats* h_stats);

/*
 * Test hooks (same kernels as dlm_refine_step, intermediate results exposed).
 *
 * dlm_debug_forward: forward over d_tokens without the reduction; writes the
 *   residual stream after the last layer (before the final norm) to d_hidden
 *   float [batch*(prompt_len+draft_len)][d_model], and, when d_max_logit is
 *   not NULL, the per-draft-position max logit, top-1 and confidence of the
 *   fused reduction to d_max_logit / d_top1 / d_conf [batch*draft_len].
 *   When d_logits is not NULL it also writes full float logits of the draft
 *   rows [batch*draft_len][vocab] through the same LM-head GEMM (test-only:
 *   the refine path never materialises logits).  For a mixture-of-experts
 *   model, d_route_ids (may be NULL) receives every block's selected experts
 *   int32 [n_layers][batch*(prompt_len+draft_len)][top_k] in selection order
 *   and d_router_logits (may be NULL) the router logits they were selected
 *   from, float [n_layers][batch*(prompt_len+draft_len)][n_experts].
 * dlm_debug_layer: one block `layer` applied to the float residual stream
 *   d_x_in [batch*seq][d_model], result to d_x_out (may equal d_x_in); for a
 *   mixture-of-experts layer d_route_ids (may be NULL) receives the selected
 *   experts int32 [batch*seq][top_k] in selection order and d_router_logits
 *   (may be NULL) the router logits float [batch*seq][n_experts] they were
 *   selected from.
 * dlm_debug_head: final norm + LM head + fused reduction on a float residual
 *   stream d_x [batch*(prompt_len+draft_len)][d_model] (draft rows used).
 */
dlm_status dlm_debug_forward(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                             const int32_t* d_tokens, void* d_workspace, size_t workspace_bytes,
                             void* hip_stream, float* d_hidden, float* d_max_logit,
                             int32_t* d_top1, float* d_conf, float* d_logits, int32_t* d_route_ids,
                             float* d_router_logits);
dlm_status dlm_debug_layer(dlm_model* m, int32_t layer, int32_t batch, int32_t seq_len,
                           const float* d_x_in, float* d_x_out, void* d_workspace,
                           size_t workspace_bytes, void* hip_stream, int32_t* d_route_ids,
                           float* d_router_logits);
dlm_status dlm_debug_head(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                          const float* d_x, void* d_workspace, size_t workspace_bytes,
                          void* hip_stream, float* d_max_logit, int32_t* d_top1, float* d_conf);

/* dlm_debug_gemm: the library's bf16 MFMA GEMM on its own (for tests and
 *   measurements): d_c float [m][n] = d_a bf16 [m][k] * d_b bf16 [n][k]^T, with a
 *   tile of tile_m x tile_n (256x256, 256x128, 128x256, 128x128 or 128x64);
 *   tile_m >> 16 selects an alternative K pipeline (1: 256x256 with 32-wide K
 *   steps and 4 stages, 128x128 with 3 stages, 256x128 with 2 stages);
 *   k must be a multiple of 64. */
dlm_status dlm_debug_gemm(const void* d_a, const void* d_b, float* d_c, int32_t m, int32_t n,
                          int32_t k, int32_t tile_m, int32_t tile_n, void* hip_stream);

/* Device pointer and byte size of one logical weight tensor (for tests):
 * kind/layer/expert as in dlm_load_synthetic_weights; *d_ptr receives the
 * base of the tensor's storage and *layout a code: 0 = plain row-major
 * [out][in]; 1 = gate/up interleaved in 32-row blocks with its partner. */
dlm_status dlm_weight_info(dlm_model* m, int32_t layer_field, int32_t kind, int32_t expert,
                           void** d_ptr, int32_t* layout);

/*
 * Kernel timing with HIP events recorded on the launch stream around every
 * launch whose kernel name equals name_filter ("*" = every launch, NULL = off).
 * Each dlm_set_profiling call clears what was recorded.
 * dlm_profile_read waits for the recorded events and writes up to max_entries
 * (kernel name, milliseconds) pairs, one per launch in launch order; it
 * returns the number written, or -1 on error.  Names are static strings.
 */
dlm_status dlm_set_profiling(dlm_model* m, const char* name_filter);
int32_t dlm_profile_read(dlm_model* m, const char** names, float* ms, int32_t max_entries);

/*
 * Test hook for the library's own host allocations (plans, the model object,
 * profiling records): the n-th allocation point passed from now fails as if
 * the host were out of memory (n = 0: none).  The entry point that meets it
 * returns DLM_ERR_NO_MEMORY with nothing half-built left behind (no model
 * handle is returned; no kernel has been launched when a plan fails).  No
 * C++ exception ever leaves an entry point.  n < 0 -> DLM_ERR_INVALID_ARG.
 * Process-wide; for single-threaded tests.
 */
dlm_status dlm_debug_fail_host_alloc(int32_t n);

void dlm_free(dlm_model* m);
const char* dlm_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DLM_H */
