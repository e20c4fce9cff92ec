/*
 * infs -- shared-prefix continuous-sampling decode attention for one MI355X
 * (gfx950).  C ABI: plain pointers and sizes only.
 *
 * The operations follow the problem statement of "Infinite Sampling"
 * (arXiv 2506.22950):
 *   - the G completions of a prompt share one prefill KV cache, kept for the
 *     whole group (Section 3.1, "KV Cache Pooling"; Section 3.2, "Shared
 *     Prompt KV and Sample-Level Cache Lifecycle")          -> infs_prefill_shared
 *   - a fixed pool holds the response KV of the m live slots; every running
 *     step decodes one token for each live slot, through every layer
 *     (Section 2.1; Section 5.1, definition of a running step)
 *                                                          -> infs_decode_step, infs_decode_step_layers,
 *                                                             infs_end_step
 *   - a finished sample releases its slot and buffer, and the slot is refilled
 *     at once with a pending sample that starts at the next step
 *     (Section 3.2; Algorithm 1, phase 2)                  -> infs_retire_slot, infs_refill_slot
 *   - the refill order: naive micro groups (Section 3.1), fixed-slot rows
 *     (Section 3.2), FIFO, shortest-job-first on predicted lengths
 *     (Algorithm 3), FPTAS grouping (Algorithm 2) alone or followed by SJF
 *     (Algorithm 1), longest-first                          -> infs_sched_*, infs_fptas_assign
 *   - prefix reuse: every sample first decodes k probe tokens, whose KV is
 *     kept; a dispatched sample resumes at token k+1 (Section 4)
 *                                                          -> infs_probe_step, infs_probe_step_layers,
 *                                                             infs_end_probe_step, infs_release_sample
 *   - optionally an FP8 (E4M3) KV cache, in the direction of the KV-cache
 *     compression the paper leaves as future work           -> INFS_FLAG_KV_FP8
 *
 * Attention computed by infs_decode_step, per live slot s holding sample i of
 * prompt p with t generated tokens (the token of this step included), per
 * query head h:
 *     g   = h / (Hq / Hkv)                       (grouped-query KV head)
 *     K   = [ prefix_p K[0:P_p, g] ; response_(p,i) K[0:t, g] ]   (V alike)
 *     o_h = softmax(scale * K q_h) V,  scale = 1/sqrt(head_dim) unless set.
 *
 * Conventions for every call:
 *   - Every function returns an infs_status; nothing throws or aborts across
 *     the ABI.  infs_last_error() gives the message of the last failure.
 *   - Arguments and state are validated on the host before anything is
 *     enqueued, so argument and state errors are synchronous and leave the
 *     context unchanged.  A failed HIP call or kernel launch makes the
 *     context return INFS_E_DEVICE from then on.
 *   - Device work is enqueued on the HIP stream given to infs_create; no call
 *     synchronises except infs_sync, infs_sample_tokens, infs_timing_end,
 *     infs_read_prefix, infs_read_response and infs_destroy.
 *   - "_dev" pointers are device (HBM) pointers owned by the caller; they
 *     must stay valid until the stream work that reads or writes them is
 *     done.  Host pointers are read or written before the call returns.
 *   - Element type of Q/K/V buffers is the context dtype (fp32, or bf16 as
 *     raw 16-bit patterns); O is always fp32.  Buffers handed to kernels are
 *     16-byte aligned.
 *   - A context must be used from one host thread at a time.
 */
#ifndef INFS_H
#define INFS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define INFS_ABI_VERSION 3

typedef enum infs_status {
    INFS_OK = 0,
    INFS_E_ARG = -1,       /* invalid argument (shape, index, null pointer, unsupported shape) */
    INFS_E_STATE = -2,     /* call not allowed in the current slot / step state */
    INFS_E_CAPACITY = -3,  /* a response would exceed max_suffix_len, or the page pool is full */
    INFS_E_DUP = -4,       /* the sample id was already dispatched (or released) in this group */
    INFS_E_NOMEM = -5,     /* device allocation failed */
    INFS_E_DEVICE = -6     /* a HIP call failed; sticky for the context */
} infs_status;

typedef enum infs_dtype { INFS_F32 = 0, INFS_BF16 = 1 } infs_dtype;

/* Refill policies of the host scheduler. */
typedef enum infs_policy {
    INFS_NAIVE = 0,      /* micro groups one after another: refill only when all m slots are empty,
                            with the next m sample ids (Section 3.1) */
    INFS_FIXED_ROW = 1,  /* fixed-slot continuous sampling: slot s runs s, s+m, s+2m, ... (Section 3.2) */
    INFS_FIFO = 2,       /* continuous refill with the lowest pending sample id */
    INFS_SJF = 3,        /* continuous refill with the smallest predicted length, ties to the
                            lowest id (Algorithm 3) */
    INFS_FPTAS = 4,      /* static pre-planning only: Algorithm 2 groups the samples into m bins by
                            predicted length (epsilon INFS_FPTAS_EPSILON) and slot s runs bin s in
                            position order (Table 2, "FPTAS only") */
    INFS_FPTAS_SJF = 5,  /* Algorithm 1: each slot starts with position 0 of its bin, every later
                            refill is SJF (Table 2, "Infinite") */
    INFS_LPT = 6         /* continuous refill with the largest predicted length, ties to the lowest
                            id; given the true lengths, a post-hoc list schedule whose step count is
                            an upper bound on the post-hoc optimum of Tables 1 and 2 ("Infinite*",
                            infs_sched_optimum), at most 4/3 - 1/(3m) times it (Graham 1969) */
} infs_policy;

#define INFS_FPTAS_EPSILON 0.1

/* Bookkeeping only: no device memory, no kernels, pointers are not read.
   Lets the slot / page / step state machine run on a host without a GPU. */
#define INFS_FLAG_DRY_RUN 1u

/* Store the KV cache (prefix store and response pages) as OCP E4M3 bytes: half the bytes of bf16 per
   token, in the direction of the KV-cache compression the paper names as future work.  K/V still
   come in as bf16 and are rounded to nearest even (magnitudes beyond 448 saturate) when stored;
   attention reads the stored values (the newest token included) and computes as for bf16.  Needs
   dtype INFS_BF16, head_dim 128 and at least 16 prefix rows (slots_per_prompt * heads per KV head). */
#define INFS_FLAG_KV_FP8 2u

typedef struct infs_config {
    int32_t num_layers;          /* >= 1 */
    int32_t num_q_heads;         /* Hq, a multiple of num_kv_heads */
    int32_t num_kv_heads;        /* Hkv */
    int32_t head_dim;            /* d: 64 or 128 */
    int32_t num_prompts;         /* prompts decoded in one batch, 1..16 */
    int32_t slots_per_prompt;    /* m live slots per prompt; slot s serves prompt s / m */
    int32_t samples_per_prompt;  /* G: sample ids of a prompt are 0..G-1 */
    int32_t max_prompt_len;      /* capacity of the shared prefix per prompt, >= 0 */
    int32_t max_suffix_len;      /* capacity of one response, >= 1 */
    int32_t page_tokens;         /* tokens per response page; 0 or 16 */
    int32_t num_pages;           /* response page pool size; 0: enough for every slot at capacity, plus
                                    every sample's probe tokens */
    int32_t split_tokens;        /* split-K chunk length of responses in tokens; 0: 256; a multiple of 128
                                    up to 4096.  Prefixes are split in 128-token chunks when they run on
                                    MFMA tiles, else in split_tokens chunks; prefix plus response chunks
                                    of one slot must not exceed 128 */
    int32_t dtype;               /* infs_dtype of Q, K, V */
    float scale;                 /* softmax scale; 0: 1/sqrt(head_dim) */
    uint32_t flags;              /* INFS_FLAG_* */
    int32_t probe_tokens;        /* prefix reuse (Section 4): k probe tokens every sample decodes before it
                                    is dispatched (infs_probe_step); 0 = no probe phase.  In [0, max_suffix_len] */
} infs_config;

typedef struct infs_ctx infs_ctx;

/* Totals since creation or the last infs_reset (host-side counts). */
typedef struct infs_stats {
    int64_t steps;               /* infs_end_step calls */
    int64_t launches;            /* attention kernel launches (one per decode_step or probe_step) */
    int64_t tokens;              /* tokens generated (live slots summed over steps, probe tokens included) */
    double alg_bytes;            /* algorithmic HBM bytes of all decode_step and probe_step launches: prefix K/V
                                    once per prompt with a live slot, each live slot's stored response K/V,
                                    new K/V read and append write, Q read, O write (K/V at their stored
                                    size) */
    double alg_flops;            /* 4 * Hq * d * (P + t) per live slot and layer */
} infs_stats;

int32_t infs_abi_version(void);

/* Create a context: validates cfg, allocates the prefix store, the response page pool, the slot
   table and the split-K workspace on the current HIP device (all zero-initialised), and records
   `hip_stream` (a hipStream_t; NULL = default stream) for all later work.  E_ARG also when a derived
   size leaves its index range: the page table or the split-K output workspace at 2 GiB or more (the
   workspace is addressed with 32-bit offsets), or a page pool beyond INT32_MAX pages.  On failure *out
   is NULL and infs_last_error(NULL) describes why. */
infs_status infs_create(const infs_config* cfg, void* hip_stream, infs_ctx** out);

/* Free everything infs_create allocated.  Waits for the context's stream first.  NULL is a no-op. */
void infs_destroy(infs_ctx* ctx);

/* Return to the just-created state (no prefix prefilled, every slot empty, no sample dispatched,
   token counters zero, stats zero), keeping allocations.  Enqueues a clear of the device counters. */
infs_status infs_reset(infs_ctx* ctx);

/* Copy one prompt's prefill K and V for one layer into the shared-prefix store (Section 3.1:
   the prompt's KV cache is kept and shared by every micro group).
   k_dev, v_dev: [prompt_len, Hkv, head_dim] row-major, context dtype, 16-byte aligned.  prompt_len in
   [0, max_prompt_len]; every layer of a prompt must use the same prompt_len.  Not allowed while
   a step is open (between the first decode_step of a step and end_step). */
infs_status infs_prefill_shared(infs_ctx* ctx, int32_t prompt, int32_t layer, int32_t prompt_len,
                                const void* k_dev, const void* v_dev);

/* Give empty slot `slot` the sample `sample_id` of `prompt` (which must be slot / m).  The sample
   starts with the probe tokens it decoded in the probe phase (none without probe_tokens): its
   KV pages are reused, and it decodes its next token at the next decode step (Section 4,
   prefix reuse: decoding resumes at token k+1).
   E_STATE: slot is live, or a step is open.  E_DUP: sample_id already dispatched for this prompt. */
infs_status infs_refill_slot(infs_ctx* ctx, int32_t slot, int32_t prompt, int64_t sample_id);

/* Release a live slot: its response pages return to the pool (the sample's buffer is recycled on
   completion, Section 3.2).  E_STATE: slot is empty, or a step is open. */
infs_status infs_retire_slot(infs_ctx* ctx, int32_t slot);

/* ---------------------------------------------------------------------------------------------
 * Probe phase of prefix reuse (Section 4, "Prefix Reuse Optimization"; contexts with
 * probe_tokens = k > 0).  Before the decode, every sample decodes its first k tokens against the
 * shared prompt so that its length can be predicted from them; the KV of those tokens is kept, and
 * a sample dispatched later resumes at token k+1 (infs_refill_slot).  A probe step decodes one
 * token for a batch of samples of one prompt through every layer, like a decode step whose slots
 * are the batch's samples: all n*hpk query rows of a KV head share each prefix K/V byte.
 * ------------------------------------------------------------------------------------------- */

/* One layer of a probe step for samples first_sample .. first_sample+n-1 of `prompt`.
   live_host: n bytes, nonzero = the sample appends its next probe token (at position = its probe
   length) and attends over [prefix ; its probe tokens]; zero = idle (O rows written 0).  NULL = all
   live.  q_dev [n, Hq, d], k_new_dev / v_new_dev [n, Hkv, d] (context dtype), o_dev [n, Hq, d] fp32,
   all 16-byte aligned.  1 <= n <= the probe batch (min(64, G, R / hpk) with R = 128 on MFMA tiles,
   16 otherwise).  Every layer once per probe step, each with the same batch; close with
   infs_end_probe_step.  E_STATE: a decode step is open, the batch differs from the open probe
   step's, the layer was already probed, a live sample was already dispatched or released, or its
   prompt is not prefilled for the layer.  E_CAPACITY: a live sample already has k probe tokens, or
   the page pool is empty. */
infs_status infs_probe_step(infs_ctx* ctx, int32_t layer, int32_t prompt, int32_t first_sample, int32_t n,
                            const uint8_t* live_host, const void* q_dev, const void* k_new_dev,
                            const void* v_new_dev, float* o_dev);

/* Every layer of one probe step in a single launch: the same results as infs_probe_step for layers
   0 .. num_layers-1 with the same batch, with the layer order, strides (in bytes; 0 = one layer's n
   rows), bounded waits and residency of infs_decode_step_layers (Section 2.1; Section 4 for the probe
   phase).  Layer l reads q_dev + l * q_layer_stride ([n, Hq, d]), k_new_dev / v_new_dev + l *
   kv_layer_stride ([n, Hkv, d]) and writes o_dev + l * o_layer_stride ([n, Hq, d] fp32).  E_STATE: a
   layer of this probe step was already probed, a decode step is open, the prompt lacks a prefilled
   layer, or the device cannot hold the launch; E_ARG and E_CAPACITY as infs_probe_step, and for
   strides below one layer's rows or not multiples of 16.  Close with infs_end_probe_step;
   infs_get_stats counts the call as one launch. */
infs_status infs_probe_step_layers(infs_ctx* ctx, int32_t prompt, int32_t first_sample, int32_t n,
                                   const uint8_t* live_host, const void* q_dev, const void* k_new_dev,
                                   const void* v_new_dev, float* o_dev, int64_t q_layer_stride,
                                   int64_t kv_layer_stride, int64_t o_layer_stride);

/* Close the probe step: every live sample's probe length grows by one.  E_STATE unless every layer
   was probed exactly once. */
infs_status infs_end_probe_step(infs_ctx* ctx);

/* Largest n of infs_probe_step (0 without a probe phase; -1 for a NULL context). */
int32_t infs_probe_batch(const infs_ctx* ctx);

/* Probe tokens decoded so far by a sample (0 without a probe phase). */
infs_status infs_probe_state(const infs_ctx* ctx, int32_t prompt, int64_t sample_id, int32_t* probe_len);

/* A sample that will not be dispatched (for instance, it finished within its probe tokens) returns
   its probe pages to the pool and can no longer be dispatched.  E_STATE without a probe phase or
   while a step is open; E_DUP if it was already dispatched or released. */
infs_status infs_release_sample(infs_ctx* ctx, int32_t prompt, int64_t sample_id);

/* One layer of one running step for every slot:
   live slots append this step's K/V (position = current length) to their response, then attend
   over [prefix ; response]; idle slots' rows are ignored and their O rows are written as 0.
   q_dev: [S, Hq, d]; k_new_dev, v_new_dev: [S, Hkv, d] (context dtype); o_dev: [S, Hq, d] fp32,
   with S = num_prompts * slots_per_prompt, slot-major; all four 16-byte aligned (E_ARG otherwise).
   Each layer must be decoded exactly once
   per step.  E_STATE: layer already decoded in this step, or a live slot's prompt has no prefix
   for this layer.  E_CAPACITY: a response would pass max_suffix_len or the page pool is empty. */
infs_status infs_decode_step(infs_ctx* ctx, int32_t layer, const void* q_dev, const void* k_new_dev,
                             const void* v_new_dev, float* o_dev);

/* For callers that cannot allocate device memory during the decode loop (code under HIP graph capture,
   tight serving loops, harnesses that forbid hipMalloc): infs_decode_step with the same arguments,
   validation, state rules and results, except that the launch's split-K workspace (partial outputs and
   (max, sum) records) and its arrival counters live in a static device array of the library
   (INFS_STATIC_SCRATCH_BYTES per GPU, 256-byte aligned, held until the process ends; its device address
   is looked up once per device in infs_create) instead of the context's own workspace.  The call itself
   allocates nothing: it enqueues a small kernel that zeroes the counters it uses, then the decode launch.
   E_CAPACITY (before anything is enqueued) if the context's workspace and counters, laid out as
   counters [S][Hkv] x 128 bytes, then (max, sum) records, then partial outputs (each part 256-byte
   aligned), exceed INFS_STATIC_SCRATCH_BYTES.  Every call on one GPU shares that GPU's array and it keeps
   the last call's contents: calls whose stream work overlaps on one GPU (two streams, two threads, two
   contexts) race and give invalid outputs; order them on one stream.  Mixing it with infs_decode_step
   layer by layer within a step is allowed. */
#define INFS_STATIC_SCRATCH_BYTES (16u << 20)
infs_status infs_decode_step_static(infs_ctx* ctx, int32_t layer, const void* q_dev, const void* k_new_dev,
                                    const void* v_new_dev, float* o_dev);

/* Every layer of one running step in a single launch (Section 2.1: a decode step passes through all
   layers; Section 5.1: one running step decodes one token for every live slot): the same results as
   infs_decode_step for layers 0 .. num_layers-1 in order.  Layer l reads q_dev + l * q_layer_stride
   ([S, Hq, d]), k_new_dev / v_new_dev + l * kv_layer_stride ([S, Hkv, d]) and writes o_dev + l *
   o_layer_stride ([S, Hq, d] fp32); strides are in bytes, multiples of 16, and 0 means one layer's rows
   (dense [L, S, H, d] buffers).  All four buffers stay with the caller until the stream work is done.
   The launch keeps as many work-groups as the GPU holds resident at once (infs_step_launch_workgroups)
   and walks the layers in order: the queries and new K/V rows of layer l are read only after every
   merge of layer l-1 of the same prompt has written its O rows (as a model's layer l would need), while
   the cached prefix and response K/V of layer l may be loaded earlier.  Split-K partials follow the
   exchange mode of infs_set_exchange, as in infs_decode_step (in mode 1 the merges load them past the
   CU's L1: the launch rewrites them in every layer).  Every device wait is bounded
   (infs_set_merge_wait); a wait that gives up makes the
   next synchronising call return E_DEVICE.  The launch needs all its work-groups on the GPU at once: other
   work running on the same GPU at the same time can delay it until its waits give up.
   E_STATE: a layer of this step was already decoded, a probe step is open, a live slot's prompt lacks
   a prefilled layer, or the device cannot hold the launch (infs_step_launch_workgroups() == 0).
   E_CAPACITY as infs_decode_step.  E_ARG: null or misaligned buffers, strides below one layer's rows.
   Close the step with infs_end_step; infs_get_stats counts the call as one launch. */
infs_status infs_decode_step_layers(infs_ctx* ctx, const void* q_dev, const void* k_new_dev, const void* v_new_dev,
                                    float* o_dev, int64_t q_layer_stride, int64_t kv_layer_stride,
                                    int64_t o_layer_stride);

/* Work-groups of an infs_decode_step_layers launch (the occupancy of its kernel times the compute
   units; 0 on a dry-run context or when the device cannot hold one producer and one merge work-group per
   KV head); -1 for a NULL context. */
int32_t infs_step_launch_workgroups(const infs_ctx* ctx);

/* Close the step: every live slot's length grows by one.  E_STATE unless every layer was decoded
   exactly once since the previous end_step (a step with no live slot needs no decode). */
infs_status infs_end_step(infs_ctx* ctx);

/* Read-back of the stores (synchronises; for checks and debugging).  Elements come back as stored:
   fp32, bf16 bit patterns, or E4M3 codes for an FP8 KV cache.
   infs_read_prefix: one prompt's prefilled K and V of one layer, [prompt_len, Hkv, d] each.
   infs_read_response: the response K and V of a live slot's sample for one layer, [len, Hkv, d]
   each, len = the slot's current length (infs_slot_state).  E_STATE in a dry-run context, for an
   unprefilled prompt or empty slot, or while a step is open. */
infs_status infs_read_prefix(infs_ctx* ctx, int32_t prompt, int32_t layer, void* k_host, void* v_host);
infs_status infs_read_response(infs_ctx* ctx, int32_t slot, int32_t layer, void* k_host, void* v_host);

/* Host mirror of a slot: *sample_id = -1 and *len = 0 when empty. */
infs_status infs_slot_state(const infs_ctx* ctx, int32_t slot, int64_t* sample_id, int32_t* len);

/* Synchronise and copy the device per-sample token counters of `prompt` (tokens appended at layer
   0, counted on the GPU) into counts_host[0..n).  n must equal samples_per_prompt. */
infs_status infs_sample_tokens(infs_ctx* ctx, int32_t prompt, int32_t* counts_host, int32_t n);

/* Wait for all work enqueued by the context.  Also reports (E_DEVICE) a decode launch whose merge
   stage stopped waiting for its producers, which leaves that launch's outputs invalid (NaN). */
infs_status infs_sync(infs_ctx* ctx);

/* Bound on how many times a merge work-group polls for its producers before it gives up (default
   2^20, far beyond any wait of a healthy launch; the work-group then writes NaN and the next
   synchronising call returns E_DEVICE).  max_polls < 0: merges give up at once -- a way to exercise
   that error path from the host.  E_STATE while a step is open. */
infs_status infs_set_merge_wait(infs_ctx* ctx, int32_t max_polls);

/* How work-groups of one decode or step launch hand their split-K partials to the merging
   work-group.
   mode 0: stores written through to the device coherence point, loads from it: correct wherever
           work-groups run.
   mode 1: through the L2 of the XCD that runs a KV head's work-groups (fewer trips to the
           coherence point).  Available when infs_create saw, in a probe launch, work-group b run on
           XCD b % n for the device's n XCDs and num_kv_heads is a multiple of n; then it is the
           default.  Every work-group checks its XCD again; a mismatch makes the next synchronising
           call return E_DEVICE (outputs of that launch are invalid).
   mode 2: mode 1 with every work-group's check made to fail, so the error path can be tested.
   E_STATE while a step is open or when mode 1/2 is unavailable (always on dry-run contexts). */
infs_status infs_set_exchange(infs_ctx* ctx, int32_t mode);

/* How an infs_decode_step_layers launch divides a step's work among its producer work-groups.
   mode 1 (default): the chunks of mode 0 while every response work-group takes at most one;
           otherwise each live response is cut into near-equal page ranges (at most one per response
           work-group when the live slots allow) and the number of prefix work-groups is chosen with
           the cuts, so that the most tokens one work-group reads after its layer's queries arrive is
           as small as it can be (a work-group holds one round of 256 tokens in registers before
           then).
   Where the per-layer prefix chunks would give some work-group two items, mode 1 also takes the
   prefix in chunks of 256 tokens on MFMA tiles, bf16 or E4M3 cache (two per-layer chunks, walked by
   the same work-group), which leaves more work-groups for the responses.
   mode 0: responses in chunks of split_tokens, the prefix in the per-layer launch's chunks, and
           work-groups divided in proportion to the chunk counts, the partition of infs_decode_step:
           outputs then differ from a per-layer decode only in the order the merges add partials.
   Both give the same results up to rounding (mode 1 moves the split-K boundaries).  E_ARG for another
   mode; E_STATE while a step is open. */
infs_status infs_set_step_split(infs_ctx* ctx, int32_t mode);

/* The work split a step launch in `mode` (as infs_set_step_split) uses for one step, with nj
   work-groups per KV head (infs_step_launch_workgroups / num_kv_heads), S slots of which slot s holds
   len[s] tokens (0 = idle), n_prefix_items prefix chunks of prefix_split tokens (a step launch in mode 1
   takes the prefix in chunks of 128 tokens on MFMA tiles, or of 256 where the
   128-token ones would give some work-group two items, and of split_tokens on the wavefront path),
   response chunks of
   `split` tokens (split_tokens of the context, 256 for 0) and at most scmax of them per slot
   (ceil(max_suffix_len / split)).  Writes pieces[0..S) (response items per slot) and roles[0..5) =
   {prefix work-groups, response work-groups, merge work-groups, response items, 1 if the responses
   are cut into near-equal page ranges else 0 for chunks of `split` tokens}.  A pure function for
   diagnostics and tests.  E_ARG: nj < 2, S outside [1, 64], split not a multiple of 16 in [16, 4096],
   scmax < 1, a len outside [0, scmax * split], mode not 0 or 1, null arrays. */
infs_status infs_step_split_plan(int32_t nj, int32_t S, int32_t n_prefix_items, int32_t prefix_split,
                                 const int32_t* len, int32_t split, int32_t scmax, int32_t mode, int32_t* pieces,
                                 int32_t* roles);

/* The current exchange mode (0, 1 or 2); -1 for a NULL context. */
int32_t infs_exchange_mode(const infs_ctx* ctx);

infs_status infs_get_stats(const infs_ctx* ctx, infs_stats* out);

/* The decode kernel instantiation a context runs, fixed by infs_create from the element type, head
   size, heads per KV head and m * hpk prefix rows: bf16 (0: fp32 Q/K/V, 1: bf16), head_dim, hpk,
   mfma (1: the prefix contractions run on 16x16x32 MFMA tiles, 0: on wavefront dot products),
   prefix_rows (the row tile, padded: 8/16 on the wavefront path, 16/32/64/128 on MFMA tiles),
   kv_fp8 (1: K/V stored as E4M3).  probe_* describe the kernel of infs_probe_step launches
   (probe_prefix_rows = 0 without a probe phase).  For diagnostics and tests; dry-run contexts
   answer too. */
typedef struct infs_kernel_info {
    int32_t bf16, head_dim, hpk, mfma, prefix_rows, kv_fp8;
    int32_t probe_mfma, probe_prefix_rows;
} infs_kernel_info;
infs_status infs_get_kernel_info(const infs_ctx* ctx, infs_kernel_info* out);

/* Kernel timing.  Between begin and end every decode_step and probe_step launch records, on the
   device wall clock, the start of its first work-group and the end of its last one.  infs_timing_end
   synchronises and returns the summed kernel time (ms) of the timed launches, their number, and
   the time between the two calls measured by HIP events on the context's stream (region_ms,
   which also covers gaps between launches and any other work on the stream). */
infs_status infs_timing_begin(infs_ctx* ctx);
infs_status infs_timing_end(infs_ctx* ctx, double* kernel_ms, double* region_ms, int64_t* launches);

/* Message of the last failed call on ctx (NULL ctx: last failed infs_create / infs_sched_create
   of this thread).  Never NULL. */
const char* infs_last_error(const infs_ctx* ctx);

/* ---------------------------------------------------------------------------------------------
 * Host scheduler (CPU only, no device): chooses which sample a freed slot receives.
 * One scheduler serves one prompt's m slots (local slot ids 0..m-1) and G samples.
 * Use: after the retirements of a step, call infs_sched_next for every empty slot in ascending
 * slot order; a returned id is dispatched (pass it to infs_refill_slot).  Call infs_sched_done
 * when a slot's sample finishes.
 * ------------------------------------------------------------------------------------------- */
typedef struct infs_sched infs_sched;

/* pred_len: G predicted lengths (float64), required for INFS_SJF, INFS_FPTAS, INFS_FPTAS_SJF and
   INFS_LPT, ignored otherwise (may be NULL).  The array is copied. */
infs_status infs_sched_create(int32_t G, int32_t m, int32_t policy, const double* pred_len,
                              infs_sched** out);

/* Next sample for empty slot `slot`: *sample_out = id, or -1 when the policy dispatches nothing
   now (naive: some slot of the current micro group still runs; every policy: no candidate left).
   E_STATE if the slot already holds a sample. */
infs_status infs_sched_next(infs_sched* s, int32_t slot, int64_t* sample_out);

/* The sample in `slot` finished; the slot becomes empty.  E_STATE if the slot is empty. */
infs_status infs_sched_done(infs_sched* s, int32_t slot);

/* Samples not yet dispatched. */
int32_t infs_sched_pending(const infs_sched* s);

void infs_sched_destroy(infs_sched* s);

/* FPTAS-based micro-group assignment (Algorithm 2), on the host.  With S the sum of pred_len (summed
   in id order) and K = (epsilon * S) / N, sample i has integer size ceil(pred_len[i] / K) and the
   bin capacity is ceil(sum of sizes / N).  Samples are placed largest size first (equal sizes:
   lower id first) into the first bin whose load stays within the capacity; a sample that fits no
   bin goes to the bin with the least load (lowest index among equals) -- a case the paper leaves
   open.  Writes group_out[i] (bin of sample i, 0..N-1) and pos_out[i] (its position in the bin).
   pred_len: G finite values >= 0 with a positive sum; epsilon > 0.  E_ARG otherwise. */
infs_status infs_fptas_assign(int32_t G, int32_t N, const double* pred_len, double epsilon, int32_t* group_out,
                              int32_t* pos_out);

/* The post-hoc optimum that Tables 1 and 2 compare against ("Infinite*": every response placed after
   generation, with the fewest running steps possible; Table 1 caption, Section 5.4).  A slot runs the
   samples it is given back to back, so a schedule's running steps are its largest per-slot sum of true
   lengths, and the optimum is the minimum of that over all assignments of the G samples to the m slots
   (the makespan problem P||Cmax).  Exact branch and bound, host only.
   lengths: G true lengths >= 1.  max_nodes: search budget (>= 0; about 10^7 nodes take a second).
   Writes *best_out (running steps of the best schedule found) and *lower_out (a proven lower bound);
   they are equal when the optimum is proven, else the budget ran out and lower <= optimum <= best.
   slot_out (G entries, or NULL): the slot of every sample in that best schedule.  E_ARG otherwise. */
infs_status infs_sched_optimum(int32_t G, int32_t m, const int32_t* lengths, int64_t max_nodes, int64_t* best_out,
                               int64_t* lower_out, int32_t* slot_out);

#ifdef __cplusplus
}
#endif

#endif /* INFS_H */
