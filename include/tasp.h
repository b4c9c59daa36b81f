/*
 * tasp.h - C ABI of the compiled structured-sparse decoder runtime for MI355X (gfx950).
 *
 * A structured mask removes, per decoder layer, whole GQA KV groups together with their query
 * heads, single query heads inside a kept group, and SwiGLU channels (gate row, up row and down
 * column together). The mask is closed under those dependencies (paper, Sec. "Dependency-Closed
 * Masks and Cache-Consistent Routing") and then compiled once into a plan: the retained rows and
 * columns of every projection are copied into dense INT8 panels (same section, and the appendix
 * paragraph "Backing-store semantics"), so that every later decode step and prefill launches only
 * the smaller contractions. One plan serves a whole request, its prefill and all of its decode
 * steps; a cache filled under one mask is refused by a plan of another mask (same section).
 *
 * Model: Llama-3 style decoder layer. Per layer and token, with residual r (float32):
 *   n = RMSNorm(r; gamma_attn); [q; k; v] = Wqkv n; RoPE(q, k) at the token position;
 *   append BF16 k, v to the cache; o = softmax(q K^T / sqrt(d_h)) V per retained head;
 *   r += Wo o; n2 = RMSNorm(r; gamma_ffn); h = silu(Wg n2) * (Wu n2); r += Wd h.
 * A stack applies L layers, then logits = W_lm RMSNorm(r; gamma_final) with a dense BF16 LM head.
 *
 * Conventions used by every entry point
 *   - Weights: INT8, row-major [out][in], one float32 scale per output row (W = q * s).
 *   - Query head h belongs to KV group h / (n_q_heads / n_kv_heads); heads are never regrouped.
 *   - RoPE: rotate-half pairs (i, i + d_h/2), angle = pos * theta^(-2i/d_h).
 *   - KV cache: BF16, K and V separate, [n_layers][batch][n_kv_heads][max_seq][head_dim]. Only
 *     retained groups' rows are read or written. Decode at `pos` writes row `pos` and attends
 *     over rows 0..pos inclusive, reading the stored BF16 values.
 *   - Activations x / out: float32; rows of `d_model` (decode: [batch][d_model]).
 *   - Pointers marked (device) are HIP device pointers; (host) are host pointers.
 *   - Streams are `hipStream_t` passed as void*; NULL is the default stream.
 *   - Every device buffer is owned by the caller. The library allocates no device memory and owns
 *     only a plan's host metadata until tasp_plan_destroy.
 *   - Errors: all arguments are validated on the host before any work is enqueued; on error
 *     nothing is enqueued and the status says why. tasp_last_error() gives thread-local detail.
 *     HIP failures map to TASP_ERR_HIP with the runtime's message. No C++ exception crosses the ABI.
 */
#ifndef TASP_H
#define TASP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t tasp_status;
enum {
  TASP_OK = 0,
  TASP_ERR_INVALID_ARG = -1,      /* null pointer, negative size, wrong enum value        */
  TASP_ERR_SHAPE = -2,            /* model or call shape not supported / inconsistent      */
  TASP_ERR_MASK = -3,             /* mask byte other than 0 or 1                           */
  TASP_ERR_WORKSPACE = -4,        /* workspace too small or misaligned                     */
  TASP_ERR_POS_RANGE = -5,        /* pos / pos0 + T outside the cache or the plan's limits */
  TASP_ERR_CACHE_PLAN_MISMATCH = -6, /* cache bound to a plan of another mask              */
  TASP_ERR_HIP = -7,              /* HIP runtime error                                     */
  TASP_ERR_UNSUPPORTED = -8,      /* valid request this build does not implement           */
  TASP_ERR_INTERNAL = -9          /* device result disagrees with the host's check         */
};

typedef struct tasp_plan_s* tasp_plan;   /* opaque; immutable after tasp_compile_plan */

/* Model geometry and the plan's capacity limits.
 *   n_layers >= 1; d_model % 16 == 0; head_dim in {64, 128}; n_q_heads % n_kv_heads == 0 with
 *   n_q_heads / n_kv_heads <= 8; d_ffn % 16 == 0; vocab = 0 for a bare layer stack (decode
 *   returns the residual) or > 0 for a stack ending in the BF16 LM head (decode returns logits).
 *   max_batch in 1..8 (decode batch), max_seq = cache rows per sequence, max_prefill = largest
 *   prefill chunk T (0: prefill unused, no prefill scratch is reserved). */
typedef struct {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, vocab;
  int32_t max_batch, max_seq, max_prefill;
  float rms_eps;
  float reserved0;
  double rope_theta;
} tasp_model_desc;

typedef struct {
  const int8_t* w;        /* (device) int8 [out][in], row-major, 16-byte aligned */
  const float* scale;     /* (device) float32 [out] */
} tasp_qmat;

/* One layer of the INT8 store: wq [Hq*dh][d], wk/wv [Hkv*dh][d], wo [d][Hq*dh],
 * wg/wu [d_ffn][d], wd [d][d_ffn]; attn_norm / ffn_norm are BF16 gains [d] (device). */
typedef struct {
  tasp_qmat wq, wk, wv, wo, wg, wu, wd;
  const uint16_t* attn_norm;
  const uint16_t* ffn_norm;
} tasp_layer;

/* The store: layers (host array of n_layers), and for vocab > 0 the final BF16 norm gain [d]
 * and the dense BF16 LM head [vocab][d] (device). The plan copies what it needs, so the store
 * may be freed once tasp_compile_plan's stream work has completed. */
typedef struct {
  const tasp_layer* layers;
  const uint16_t* final_norm;
  const uint16_t* lm_head;
} tasp_store;

/* Host bytes in {0, 1}: q_keep [n_layers][n_q_heads], kv_keep [n_layers][n_kv_heads] (NULL: all
 * kept), ffn_keep [n_layers][d_ffn]. A NULL tasp_mask* means the dense (all-kept) plan. A mask
 * that is not dependency-closed is closed, not rejected: a head in a dropped group is dropped,
 * and a group with no retained head is dropped. */
typedef struct {
  const uint8_t* q_keep;
  const uint8_t* kv_keep;
  const uint8_t* ffn_keep;
} tasp_mask;

/* A caller-owned KV cache (device BF16 arrays, layout above). plan_sig records the plan the
 * cache contents belong to; it is set by tasp_kv_bind and checked by decode and prefill. */
typedef struct {
  void* k;
  void* v;
  int32_t batch;          /* sequences in the cache, 1..max_batch */
  int32_t max_seq;        /* rows per sequence, <= the plan's max_seq */
  uint64_t plan_sig;
} tasp_kv_cache;

/* Index lists of tasp_plan_indices. */
enum { TASP_IDX_Q = 0, TASP_IDX_KV = 1, TASP_IDX_QKVSLOT = 2, TASP_IDX_FFN = 3 };
/* Panels of tasp_plan_panel. */
enum { TASP_PANEL_QKV = 0, TASP_PANEL_O = 1, TASP_PANEL_GATE = 2, TASP_PANEL_UP = 3,
       TASP_PANEL_DOWN = 4 };

/* Workspace bytes that tasp_compile_plan needs for this mask (paper, Sec. "Dependency-Closed
 * Masks and Cache-Consistent Routing": each mask's retained units are packed into contiguous
 * tensors; Eqs. flop-attn and flop-mlp give the retained panel shapes): panels, copies of the
 * gains and LM head, RoPE table, decode and prefill scratch. The mask is closed on the host to
 * size it. desc, mask: host; *bytes (host) receives the size. Errors: TASP_ERR_SHAPE for an
 * unsupported desc, TASP_ERR_MASK for a byte other than 0 / 1. */
tasp_status tasp_plan_workspace_bytes(const tasp_model_desc* desc, const tasp_mask* mask,
                                      size_t* bytes);

/* Compile a plan (paper, Sec. "Dependency-Closed Masks and Cache-Consistent Routing": one
 * compiled launch plan per mask over the INT8 store). Uploads the mask, runs the closure/index kernel (one workgroup per layer; integer-only), gathers
 * the retained rows / columns and their scales into the panels inside `workspace` (device, 256-byte
 * aligned, >= tasp_plan_workspace_bytes), and zeroes the decode scratch. Synchronises `stream`
 * once to read the index lists back; returns TASP_ERR_INTERNAL if they differ from the host's
 * closure. The workspace must outlive the plan and must not be shared between plans. */
tasp_status tasp_compile_plan(const tasp_model_desc* desc, const tasp_store* store,
                              const tasp_mask* mask, void* workspace, size_t workspace_bytes,
                              void* stream, tasp_plan* out);

/* ---- shared-store plans (paper, appendix "Backing-store semantics": every mask indexes one
 * immutable packed store and owns no weight bytes, so memory grows only by plan metadata; Table
 * "configuration": symmetric groupwise INT8, group size 128, BF16 scales).
 *
 * Groupwise matrix: w int8 [out][in] row-major (16-byte aligned), scale BF16 bits
 * [out][in / 128] (2-byte aligned); W[o][i] = w[o][i] * scale[o][i / 128]. */
typedef struct {
  const int8_t* w;
  const uint16_t* scale;
} tasp_gqmat;

/* One layer of the packed groupwise store: wqkv [(n_q_heads + 2 n_kv_heads) head_dim][d] holds
 * every query head's rows, then every K row, then every V row; wo [d][n_q_heads head_dim];
 * wg / wu [d_ffn][d]; wd [d][d_ffn]; gains BF16 [d] (device). */
typedef struct {
  tasp_gqmat wqkv, wo, wg, wu, wd;
  const uint16_t* attn_norm;
  const uint16_t* ffn_norm;
} tasp_glayer;

/* The packed store (host array of n_layers layers; final BF16 gain and dense BF16 LM head
 * [vocab][d] on the device for vocab > 0). Plans keep pointers into it: it must outlive them. */
typedef struct {
  const tasp_glayer* layers;
  const uint16_t* final_norm;
  const uint16_t* lm_head;
} tasp_gstore;

/* Bytes of a shared-store plan (paper, appendix "Backing-store semantics": a plan over the one
 * store is block-selection and launch metadata). *plan_bytes: masks, index lists, the maps into
 * the store and the RoPE table, the same for every mask. *scratch_bytes: the decode (max_batch
 * sequences) and prefill (max_prefill tokens) scratch, which any number of shared plans of equal
 * scratch size may share (see tasp_compile_shared_plan). d_model, n_q_heads * head_dim and d_ffn
 * must be divisible by 128. */
tasp_status tasp_shared_plan_workspace_bytes(const tasp_model_desc* desc, size_t* plan_bytes,
                                             size_t* scratch_bytes);

/* Compile a plan over the shared store: closes the mask (as tasp_compile_plan), builds on the
 * device the maps from plan rows / column pieces to store rows / columns (QKV rows of the
 * retained heads and groups, W_o columns of the retained heads, gate / up rows and W_down column
 * blocks of the retained channels) and checks them on the host; copies no weights. The retained
 * channels of every layer must come in aligned blocks of 16 (else TASP_ERR_UNSUPPORTED; the
 * paper's channel groups are 1,024 wide). Such a plan serves every call a per-row plan serves
 * (decode at batch 1..max_batch, prefill, tasp_generate, tasp_serve_turn, the profiling calls),
 * reading the store in place: batch 1 with per-lane group scales, batches and prefill on the
 * matrix cores with each weight times its group scale split exactly into BF16 hi and lo parts;
 * only tasp_plan_panel returns TASP_ERR_UNSUPPORTED (there are no panels). Its signature differs
 * from a per-row plan of the same mask, so caches are not shared between the two formats.
 * `workspace` (256-byte aligned, plan_bytes) holds the plan's metadata. `scratch` (256-byte
 * aligned, scratch_bytes) is its scratch arena and may be passed to several shared plans: their
 * calls, and this compile (it clears the arena's counters), must then be ordered one after
 * another (one stream, or synchronised streams); overlapping calls race. With scratch NULL the
 * arena is the workspace's tail (workspace_bytes >= plan_bytes + scratch_bytes). Both buffers stay
 * owned by the caller and must outlive the plan. Synchronises `stream`. */
tasp_status tasp_compile_shared_plan(const tasp_model_desc* desc, const tasp_gstore* store,
                                     const tasp_mask* mask, void* workspace,
                                     size_t workspace_bytes, void* scratch, size_t scratch_bytes,
                                     void* stream, tasp_plan* out);

/* Retained counts of one layer after closure (paper, Eqs. flop-attn and flop-mlp: m^q, m^kv and
 * c of that layer): query heads, KV groups, SwiGLU channels, written to host int32s.
 * TASP_ERR_INVALID_ARG for a NULL pointer or a layer outside 0..n_layers-1. */
tasp_status tasp_plan_counts(tasp_plan plan, int32_t layer, int32_t* m_q, int32_t* m_kv,
                             int32_t* n_ffn);

/* Copy one ascending index list of a layer as computed on the device by the closure (paper,
 * Sec. "Dependency-Closed Masks and Cache-Consistent Routing": a KV group stays active while any
 * of its query heads is retained, heads keep their group, and a SwiGLU channel is kept or removed
 * in gate, up and down together) into host dst of cap entries: TASP_IDX_Q retained query heads,
 * TASP_IDX_KV retained KV groups, TASP_IDX_QKVSLOT the rank of each retained head's group among
 * the retained groups, TASP_IDX_FFN retained channels. *n (if not NULL) receives the list length; dst NULL
 * only queries it. TASP_ERR_INVALID_ARG if the length exceeds cap, or for a bad layer / `which`. */
tasp_status tasp_plan_indices(tasp_plan plan, int32_t layer, int32_t which, int32_t* dst,
                              int32_t cap, int32_t* n);

/* Where a panel of a layer lives (paper, appendix "Backing-store semantics": the contiguous
 * retained tensors a plan launches on): device int8 rows [rows][ld] (columns >= cols are zero)
 * and its float32 scales [rows], both inside the plan's workspace (not owned by the caller's
 * pointers; valid until tasp_plan_destroy). QKV rows: retained q heads, then K, then V rows of
 * retained groups. TASP_ERR_UNSUPPORTED for a shared-store plan (it has no panels). */
tasp_status tasp_plan_panel(tasp_plan plan, int32_t layer, int32_t which, const int8_t** w,
                            const float** scale, int64_t* rows, int64_t* cols, int64_t* ld);

/* Analytical active-FLOP ratio of the decoder projections (paper, Eqs. flop-attn and flop-mlp;
 * LM head excluded), retained INT8 weight bytes, float32 scale bytes, and the plan signature
 * (a hash of the model shape and the closed mask; equal masks give equal signatures). */
tasp_status tasp_plan_ledger(tasp_plan plan, double* active_flop_ratio, uint64_t* weight_bytes,
                             uint64_t* scale_bytes, uint64_t* signature);

/* Release a plan's host metadata (paper, appendix "Backing-store semantics": a mask owns plan
 * metadata only). The workspace given to the compile call stays the caller's to free once the
 * plan's queued work has completed. NULL is accepted. */
tasp_status tasp_plan_destroy(tasp_plan plan);

/* Adopt a cache whose rows 0..pos-1 were filled outside the library (already rotated keys) for
 * this plan (paper, Sec. "Dependency-Closed Masks and Cache-Consistent Routing": cache contents
 * belong to one mask and are not carried to an incompatible one): checks its shape against the
 * plan (TASP_ERR_SHAPE: batch outside 1..max_batch, max_seq above the plan's) and sets
 * cache->plan_sig (host struct; the device arrays are not touched). */
tasp_status tasp_kv_bind(tasp_plan plan, tasp_kv_cache* cache);

/* One decode step (paper, Sec. "Dependency-Closed Masks and Cache-Consistent Routing": the
 * plan chosen for a turn runs every decode step; Table "systems": the timed decode latency) for
 * cache->batch sequences that share `pos` (prior positions, 0 <= pos < cache->max_seq, else
 * TASP_ERR_POS_RANGE; a cache bound to another plan gives TASP_ERR_CACHE_PLAN_MISMATCH). x (device) float32 [batch][d_model]; out (device) float32 [batch][d_model], or
 * logits [batch][vocab] when the plan has an LM head. x and out may not overlap. Stream-ordered
 * and asynchronous; launches only the plan's kernels and allocates nothing, so it may be captured
 * into a HIP graph. Calls on one plan must be ordered (they share the plan's scratch). */
tasp_status tasp_decode_step(tasp_plan plan, const float* x, tasp_kv_cache* cache, int32_t pos,
                             float* out, void* stream);

/* Prefill of T tokens of one sequence (cache->batch must be 1) at positions pos0..pos0+T-1
 * (paper, Sec. "Dependency-Closed Masks and Cache-Consistent Routing": the plan fixed at the start
 * of a turn serves the prompt and every later decode step; Table "configuration": the timed
 * request begins with a prefill). 1 <= T <= max_prefill (TASP_ERR_UNSUPPORTED for a plan compiled with
 * max_prefill 0), pos0 + T <= cache->max_seq (else TASP_ERR_POS_RANGE). x (device) float32
 * [T][d_model]; out (device, not overlapping x) float32 [T][d_model], or logits [T][vocab] with
 * an LM head. Token t attends causally over rows 0..pos0+t; rows pos0..pos0+T-1 of every
 * retained group receive the BF16 k and v of the tokens. pos0 == 0 binds the cache to the plan;
 * pos0 > 0 requires it bound (else TASP_ERR_CACHE_PLAN_MISMATCH). Projections and attention run
 * on the matrix cores with activations split into hi/lo BF16 pairs. Stream-ordered, capturable;
 * calls on one plan must be ordered (they share the plan's scratch). */
tasp_status tasp_prefill(tasp_plan plan, const float* x, int32_t T, tasp_kv_cache* cache,
                         int32_t pos0, float* out, void* stream);

/* The same prefill returning only the last token's logits (paper, Sec. "Dependency-Closed Masks
 * and Cache-Consistent Routing" and Table "configuration": greedy decoding continues from the
 * prompt's last position, so no other position's logits are needed). Arguments and errors as
 * tasp_prefill, with out (device, not overlapping x) float32 [vocab]: the final RMSNorm and LM
 * head of token T - 1 only, by the decode LM head kernel (TASP_ERR_UNSUPPORTED without an LM
 * head). The cache rows and every other effect are those of tasp_prefill. tasp_generate and
 * tasp_serve_turn prefill this way. */
tasp_status tasp_prefill_last(tasp_plan plan, const float* x, int32_t T, tasp_kv_cache* cache,
                              int32_t pos0, float* out, void* stream);

/* One request under the plan (paper, Sec. "Dependency-Closed Masks and Cache-Consistent Routing":
 * the plan stays fixed through prefill and every decode step; Table "configuration": the timed
 * request is a prefill followed by greedy decoding). The prompt's ids (device int32 [T]) are
 * embedded from the dense INT8 table (device int8 [vocab][d_model] with float32 row scales
 * [vocab]), prefilled at positions 0..T-1 (binding the cache), and the greedy id of the last
 * position goes to out_ids[0]; then n_new decode steps feed out_ids[i] at position T + i and
 * write the greedy id of its logits to out_ids[i + 1]. Greedy = highest logit, lowest id on ties;
 * ids stay on the device, so nothing waits for the host between tokens.
 *   Requires an LM head (else TASP_ERR_UNSUPPORTED), cache batch 1, 1 <= T <= max_prefill and
 *   T + n_new <= cache->max_seq (else TASP_ERR_POS_RANGE).
 *   out_ids: device int32 [n_new + 1]; x_scratch: device float32 [T][d_model]; logits: device
 *   float32 [T][vocab] (holds the last step's logits afterwards). Stream-ordered. */
tasp_status tasp_generate(tasp_plan plan, const int8_t* embed, const float* embed_scale,
                          const int32_t* prompt, int32_t T, int32_t n_new, tasp_kv_cache* cache,
                          int32_t* out_ids, float* x_scratch, float* logits, void* stream);

/* Profiling variant of tasp_prefill (per-kernel split of the prefill time of Table "systems"):
 * an event pair around every kernel; kinds as for tasp_decode_step_timed, plus 7 for the RoPE /
 * cache-append kernel. kernel_ms, kinds: host arrays of cap entries; *n the kernels launched.
 * Synchronises `stream`. */
tasp_status tasp_prefill_timed(tasp_plan plan, const float* x, int32_t T, tasp_kv_cache* cache,
                               int32_t pos0, float* out, void* stream, float* kernel_ms,
                               int32_t* kinds, int32_t cap, int32_t* n);

/* Profiling variant of tasp_decode_step (per-kernel split of the decode latency of Table
 * "systems"): records a HIP event pair around every kernel it launches,
 * synchronises `stream`, and writes each kernel's duration in milliseconds to kernel_ms[i] and a
 * kernel-kind code to kinds[i] (0 QKV, 1 attention, 2 O, 3 gate/up, 4 down, 5 LM head, 6 batched
 * operand preparation) for up to
 * cap kernels; *n receives the number launched. Not capturable (it synchronises). */
tasp_status tasp_decode_step_timed(tasp_plan plan, const float* x, tasp_kv_cache* cache,
                                   int32_t pos, float* out, void* stream, float* kernel_ms,
                                   int32_t* kinds, int32_t cap, int32_t* n);

/* Profiling (the timing protocol of Sec. "Experimental Design": back-to-back runs between
 * events, here for one stage): average duration of one stage of layer `layer`, measured as n_plans * reps
 * back-to-back launches between two HIP events on `stream` (layer -1: every layer that has the stage,
 * in order, so that each launch of a stack reads another layer's panel). Stage `kind`: 1 attention at `pos`
 * (split-KV partials, merged by the last split of each group slot; rewrites cache row pos with
 * the same values, or for layer -1 every layer's row pos with the last decoded layer's k, v), 3 the gate/up projection (RMSNorm + SwiGLU), 4 the down projection (writes the plan's
 * scratch, not a caller buffer). Launch i uses plans[i % n_plans] with caches[i % n_plans] (bound
 * to that plan; its batch selects the batch-1 or the batched kernels), so distinct plan copies
 * keep every launch streaming from HBM rather than from cache. Each plan must have run a
 * tasp_decode_step with that cache at `pos` (its scratch holds the stage's input). Synchronises
 * `stream`; writes the mean milliseconds per launch. Not capturable. */
tasp_status tasp_profile_stage(const tasp_plan* plans, const tasp_kv_cache* caches,
                               int32_t n_plans, int32_t layer, int32_t kind, int32_t pos,
                               int32_t reps, void* stream, float* ms_per_launch);

/* Greedy dependency-closed mask construction (paper, Sec. "Dependency-Closed Masks and
 * Cache-Consistent Routing"; costs from Eqs. flop-attn and flop-mlp). Candidates are every query
 * head and every SwiGLU group of `granule` consecutive channels (gate row, up row and down column
 * jointly). They are ranked by score / active FLOPs in float64 (a head: 4 d d_h plus 1/r of its
 * KV group's 4 d d_h; a channel group: 6 d granule), equal keys by ascending candidate index
 * (layer-major, a layer's heads before its channel groups), and accepted in that order when the
 * marginal cost (a head whose KV group is not open yet also pays the group) fits the budget
 * floor(target x full-width decoder FLOPs); a candidate that does not fit is skipped. Outputs are
 * dependency-closed by construction.
 *   head_scores (device) float32 [n_layers][n_q_heads]; chan_scores (device) float32
 *   [n_layers][d_ffn / granule]; all finite (else TASP_ERR_INVALID_ARG).
 *   q_keep [L][Hq], kv_keep [L][Hkv], ffn_keep [L][d_ffn] (device, caller-owned) receive 0/1.
 *   granule must divide d_ffn (else TASP_ERR_SHAPE); 0 <= target <= 1.
 *   workspace: device, 256-byte aligned, at least tasp_mask_workspace_bytes.
 * Synchronises `stream` (it reads back the status and the FLOPs spent, *flops_spent if given). */
tasp_status tasp_mask_workspace_bytes(const tasp_model_desc* desc, int32_t granule, size_t* bytes);
tasp_status tasp_build_mask(const tasp_model_desc* desc, const float* head_scores,
                            const float* chan_scores, int32_t granule, double target,
                            void* workspace, size_t workspace_bytes, uint8_t* q_keep,
                            uint8_t* kv_keep, uint8_t* ffn_keep, uint64_t* flops_spent,
                            void* stream);

/* ---- routing (paper, Sec. "Dependency-Closed Masks and Cache-Consistent Routing": a three-layer
 * MLP router picks one task plan per user turn, or the dense plan when its temperature-scaled
 * confidence is below tau; appendix "Router feature specification": the feature vector).
 *
 * Feature vector of a prompt (float32, proj_dim + 11 entries, in this order):
 *   [0, proj_dim)  proj x tf, tf[bin] = (number of the prompt's byte trigrams, ASCII letters
 *                  case-folded, whose 32-bit FNV-1a hash is bin modulo n_bins) / max(1, bytes - 2);
 *   then ln(1 + bytes), the proxy-LM mean token log-probability (an input), ln(1 + count) of
 *   digits, of operators (+ - * / = < > % ^), of code punctuation ({ } [ ] ( ) ; _ # ` \ | &) and
 *   of question marks, and five 0/1 descriptors: numbered list (a line opening with 1-3 digits,
 *   '.' or ')', a space), code fence (three backticks), translate cue ("translat", case-folded),
 *   multiple-choice pattern (lines opening with option labels A and B, as "X.", "X)" or "(X)"
 *   then a space), retrieval cue (case-folded who / when / where / which at a word start and
 *   not followed by a letter).
 * MLP: h1 = ReLU(w1 f + b1), h2 = ReLU(w2 h1 + b2), z = w3 h2 + b3; p = softmax(z / temperature);
 * choice = the lowest task index of max p, or -1 (dense plan) when max p < tau. float32
 * arithmetic; the text scan is integer. */
#define TASP_ROUTER_SCALARS 11
#define TASP_ROUTER_MAX_TASKS 16
#define TASP_ROUTER_MAX_BINS 16384

typedef struct {
  int32_t n_bins;       /* hashed trigram bins (paper: 2,048), 1..16384 */
  int32_t proj_dim;     /* width of the frozen random projection (paper: 256), >= 1 */
  int32_t hidden1;      /* MLP hidden widths (paper: 512 and 256), >= 1 */
  int32_t hidden2;
  int32_t n_tasks;      /* task plans (paper: 5), 1..16 */
  float temperature;    /* > 0; divides the logits */
  float tau;            /* confidence threshold of the dense fallback (paper: 0.85) */
  const float* proj;    /* device float32 [proj_dim][n_bins] */
  const float* w1;      /* device float32 [hidden1][proj_dim + 11] */
  const float* b1;      /* [hidden1] */
  const float* w2;      /* [hidden2][hidden1] */
  const float* b2;      /* [hidden2] */
  const float* w3;      /* [n_tasks][hidden2] */
  const float* b3;      /* [n_tasks] */
} tasp_router;

/* Device workspace bytes for routing n_prompts prompts (also covers tasp_serve_turn with
 * n_prompts = 1). */
tasp_status tasp_router_workspace_bytes(const tasp_router* router, int32_t n_prompts,
                                        size_t* bytes);

/* Route n_prompts prompts. text (device bytes, n_text of them) holds the prompts back to back;
 * offsets (device int32 [n_prompts + 1]) bounds prompt i as [offsets[i], offsets[i + 1]), each
 * bound clamped to [0, n_text] on the device (a decreasing pair is an empty prompt); offsets NULL
 * means one prompt, the whole text (n_prompts must be 1). proxy_logprob: device float32
 * [n_prompts]. Outputs (device): features float32 [n_prompts][proj_dim + 11] (may be NULL),
 * probs float32 [n_prompts][n_tasks], choice int32 [n_prompts]. workspace: device, 256-byte
 * aligned, at least tasp_router_workspace_bytes. Stream-ordered and asynchronous (five kernels,
 * no allocation), so it may be captured into a HIP graph. Errors: TASP_ERR_INVALID_ARG for NULL
 * pointers, sizes out of range (n_prompts 1..65535, n_text >= 0) or a temperature <= 0;
 * TASP_ERR_WORKSPACE for a short workspace. */
tasp_status tasp_route(const tasp_router* router, const uint8_t* text, int32_t n_text,
                       const int32_t* offsets, int32_t n_prompts, const float* proxy_logprob,
                       void* workspace, size_t workspace_bytes, float* features, float* probs,
                       int32_t* choice, void* stream);

/* Routing for callers that cannot allocate (code under HIP graph capture, serving loops and
 * harnesses that forbid allocation): tasp_route without a workspace argument. Its scratch is a
 * fixed TASP_ROUTE_NOALLOC_SCRATCH_BYTES array that the library holds in each GPU's memory
 * until the process ends; the call allocates nothing. A call whose scratch need
 * (tasp_router_workspace_bytes for the same router and n_prompts) exceeds that size returns
 * TASP_ERR_WORKSPACE and enqueues nothing (about 12 KB per prompt at the paper's router shape,
 * so ~340 prompts per call). Every call on one GPU uses that GPU's one array: calls that overlap
 * on one GPU (concurrent streams, or host threads without ordering) race and must be serialised
 * by the caller; calls on one stream are ordered. The array's contents are left over from the
 * last call and need no clearing (every byte a call reads, that call writes first). The first
 * call on a device looks up the array's device address (not enqueued). Arguments, outputs and
 * errors otherwise as tasp_route; the results equal tasp_route's bit for bit. */
#define TASP_ROUTE_NOALLOC_SCRATCH_BYTES ((size_t)4 << 20)
tasp_status tasp_route_noalloc(const tasp_router* router, const uint8_t* text, int32_t n_text,
                               const int32_t* offsets, int32_t n_prompts,
                               const float* proxy_logprob, float* features, float* probs,
                               int32_t* choice, void* stream);

/* One user turn with routing and dispatch (paper, Sec. "Dependency-Closed Masks and
 * Cache-Consistent Routing"): one routing decision per turn; the plan it picks runs all of that
 * turn's prefill and decode work; cache rows written under one closed mask are kept only when the
 * same plan serves the next turn, and are otherwise discarded and rebuilt.
 *   1. routes the turn's text (device bytes [n_text], one prompt) with proxy_logprob (device
 *      float32 [1]) and waits for the decision (this synchronises `stream`);
 *   2. takes task_plans[choice], or dense_plan for choice -1 (all n_tasks + 1 plans must share
 *      one model shape with an LM head);
 *   3. if 0 < n_cached < T and the cache is bound to the chosen plan, its rows 0..n_cached-1 (the
 *      conversation so far, written under that plan) are kept and prompt ids n_cached..T-1 are
 *      prefilled at those positions (*reused = 1); otherwise the cache is invalidated: all T ids
 *      are prefilled from position 0 and the cache is bound to the chosen plan (*reused = 0);
 *   4. decodes greedily as tasp_generate: out_ids[0] from the last prompt position, then n_new
 *      steps. After the turn the cache holds T + n_new valid rows (the last id is not fed).
 *   prompt: device int32 [T] (the whole conversation's ids); x_scratch: device float32
 *   [T][d_model]; logits: device float32 [T][vocab]; out_ids: device int32 [n_new + 1];
 *   workspace: tasp_router_workspace_bytes(router, 1). *chosen receives the choice (-1 dense).
 *   Errors as tasp_route and tasp_generate; T - prefilled start must fit the plan's max_prefill. */
tasp_status tasp_serve_turn(const tasp_router* router, const tasp_plan* task_plans,
                            tasp_plan dense_plan, const uint8_t* text, int32_t n_text,
                            const float* proxy_logprob, const int8_t* embed,
                            const float* embed_scale, const int32_t* prompt, int32_t T,
                            int32_t n_cached, int32_t n_new, tasp_kv_cache* cache,
                            int32_t* out_ids, float* x_scratch, float* logits, void* workspace,
                            size_t workspace_bytes, int32_t* chosen, int32_t* reused,
                            void* stream);

/* Plain streaming copy of `bytes` (multiple of 16) from src to dst (device, not overlapping):
 * the reference kernel whose counter readings calibrate memory-traffic measurements (the byte
 * ledger of appendix "FLOP and storage validation" checked against hardware counters).
 * TASP_ERR_INVALID_ARG for NULL pointers or a size not a multiple of 16. */
tasp_status tasp_copy_probe(void* dst, const void* src, size_t bytes, void* stream);

/* Text of a status code, and the thread-local detail of the last failing call on this thread
 * (static / thread-owned strings; the caller does not free them). They report the host-side
 * validation that precedes every enqueue (all entry points above). */
const char* tasp_status_string(tasp_status s);
const char* tasp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* TASP_H */
