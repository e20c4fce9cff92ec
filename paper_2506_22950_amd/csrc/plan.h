// Per-launch plan of one decode step, passed to the attention kernel by value.
//
// The host knows every slot's length, so it plans the split-K work of a step
// on the CPU and hands it over in the kernel argument block: no per-step
// host-to-device copy is needed.  The same plan serves every layer of a step.
#pragma once
#include <stddef.h>
#include <stdint.h>

namespace infs {

constexpr int kMaxSlots = 64;      // S = num_prompts * slots_per_prompt; also the largest probe batch
constexpr int kMaxPrompts = 16;
constexpr int kPageTokens = 16;    // tokens per response page
constexpr int kBlockThreads = 256; // 4 wavefronts of 64
constexpr int kWaves = kBlockThreads / 64;
constexpr int kMfmaBlock = 32;     // prefix tokens per MFMA block
constexpr int kMfmaPrefixSplit = 4 * kMfmaBlock;  // MFMA prefix chunk: one block per wavefront
constexpr int kStepPrefixSplit = 2 * kMfmaPrefixSplit;  // MFMA prefix chunk of a step launch (step_plan.h)
constexpr int kMaxPartials = 128;  // prefix + response chunks merged for one slot
constexpr int kMaxSplit = 4096;    // split-K chunk length limit (a wavefront covers <= 64 pages)

constexpr int kMergeSpins = 1 << 20;   // bound on a merge block's wait for its producers
constexpr int kCounterStride = 32;     // int32 per arrival counter: each counter has a 128-byte line of its own
constexpr int kRecordsPerLine = 16;   // (max, sum) records of 8 bytes per 128-byte line
constexpr int kClockSlots = 16;        // timing slots per launch (see StepArgs::clock_start)
constexpr int kClockStride = 16;       // uint64 per timing slot: one 128-byte line each
constexpr int kMateWaitTicks = 2000;   // bound on a step-launch work-group's wait for its CU mate (100 MHz ticks)
// Size of the file-scope device array that holds the split-K workspace and the
// arrival counters of infs_decode_step_static (one copy per GPU, kept until the
// process ends).
constexpr size_t kStaticScratchBytes = size_t(16) << 20;

// Work item kinds, in grid order: prefix chunks, response chunks, idle slots,
// then one merge item per live slot.  Grid x = item * Hkv + kv_head, so with 8
// KV heads each head's items stay on one XCD (work-groups are dealt
// round-robin over the 8 XCDs).  Merge items come last so that every XCD has
// dispatched all of its producer work-groups before any merge work-group,
// whose only wait is for producers to finish.

struct SlotPlan {
  int32_t len;         // response length after this step's append; 0 = idle
  int32_t item_begin;  // first response item of this slot
  int32_t cur_page;    // page holding position len-1 (where this step's K/V go)
  int32_t sample;      // sample id (token counters)
  int32_t target;      // slot counter value once this launch's producers for the slot (its response
                       // chunks and its prompt's prefix chunks) have all arrived; in a step launch
                       // through every layer, the value before the launch (each layer adds the
                       // slot's producer count)
  int32_t seq;         // page-table row of the sample's response (a sequence handle)
  int32_t pieces;      // response items of the slot: ceil(len / split) chunks in a per-layer launch; in a
                       // step launch, near-equal page ranges (see step_plan.h), item_begin counting them
  int32_t pad_;
};

struct PromptPlan {
  int32_t plen;        // prefix length
  int32_t nchunks;     // prefix chunks this step (0 when the prompt has no live slot)
  int32_t item_begin;  // first prefix item
  int32_t pad_;
};

struct StepArgs {
  // caller buffers
  const void* q;       // [S, Hq, d]
  const void* knew;    // [S, Hkv, d]
  const void* vnew;    // [S, Hkv, d]
  float* o;            // [S, Hq, d]
  // library buffers (already offset to this layer)
  const void* prefix;  // shared-prefix store of this layer
  void* pool;          // response page pool of this layer
  int32_t* page_table; // [sequence handles][pages_per_slot]
  float* ws_o;         // partial outputs   [..., d]
  float* ws_ml;        // partial (max, sum) [..., 2]
  int32_t* counters;   // arrival counters [S][Hkv], kCounterStride apart: a prefix chunk counts on every
                       // live slot of its prompt, a response chunk on its own slot.  They only grow
                       // (wrapping); each launch carries the values they reach once its producers
                       // have all arrived.
  int32_t* tokens;     // [num_prompts, G] per-sample token counters
  int32_t* status;     // device status word: 1 after a merge wait hit its bound, 2 after a work-group
                       // of an XCD-local exchange ran on another XCD than planned
  // Timing mode (else null): kClockSlots start/end slots of this launch,
  // kClockStride apart; block b folds its start into the minimum of slot
  // b % kClockSlots and its end into the maximum of that slot (spread over
  // cache lines so the atomics do not queue on one line).
  unsigned long long* clock_start;
  unsigned long long* clock_end;
  // geometry
  int32_t S, m, G, Hq, Hkv, prefix_rows;  // prefix_rows = m * hpk (real rows)
  int32_t max_prompt_len;     // prefix store row capacity (multiple of 32)
  int32_t pages_per_slot;
  int32_t split;              // response chunk length in tokens
  int32_t prefix_split;       // prefix chunk length in tokens
  int32_t prefix_chunks_max;  // ceil(max_prompt_len / prefix_split)
  int32_t suffix_chunks_max;  // ceil(max_suffix_len / split)
  int32_t count_tokens;       // 1 on layer 0
  float scale_log2;           // softmax scale * log2(e)
  uint32_t ws_o_bytes;        // size of ws_o (below 2^31)
  uint32_t ws_ml_bytes;       // size of ws_ml
  int32_t l2_xcds;            // > 0: partials exchanged through the XCD's L2; work-group b runs on XCD
                              // b % l2_xcds (0: written through to the device coherence point)
  int32_t l2_check_shift;     // 0; 1 makes every work-group's XCD check fail (error-path tests)
  int32_t merge_polls;        // bound on a merge block's polls of its counters (kMergeSpins; < 0: none)
  // Step launch through every layer (infs_decode_step_layers); unused by per-layer launches.
  // Layer l reads q + l * q_layer_stride (knew, vnew alike) and writes o + l * o_layer_stride; the
  // prefix store and page pool of layer l are prefix + l * prefix_layer_bytes and pool + l *
  // pool_layer_bytes.  Per KV head (work-groups j = 0 .. n_pre_wg + n_suf_wg + n_merge_wg - 1), the
  // first n_pre_wg take the prefix items round robin, j = merge_j0 .. merge_j0 + n_merge_wg - 1 do
  // one slot's merge (or zeroing) per wavefront, and the others, in order, the response items.
  int32_t num_layers;
  int32_t n_pre_wg, n_suf_wg, n_merge_wg;
  int32_t resp_cut;                    // 1: slot s's response items are its slot[s].pieces near-equal page
                                       // ranges (step_plan.h); 0: chunks of `split` tokens
  int32_t merge_j0;                    // first merge work-group of a KV head (>= n_pre_wg)
  int64_t q_layer_stride, kv_layer_stride, o_layer_stride;
  int64_t prefix_layer_bytes, pool_layer_bytes;
  int32_t* merged;                     // per prompt, kCounterStride apart: merges completed (they only grow);
                                       // then per (prompt, KV head) the layer-done flags
  int32_t merged_base[kMaxPrompts];    // value of each prompt's merged counter before this launch
  int32_t merged_per_layer[kMaxPrompts];  // merges of each prompt per layer: its live slots * Hkv
  uint64_t live_mask;                  // bit s set: slot s is live this step
  int32_t* peer;                       // per work-group of the launch, kCounterStride apart: words 0..3 =
                                       // peer_base + l + 1 once its wavefront w (a producer: the whole
                                       // work-group, word 0) is done with layer l; word 4 = its CU id + 1
  int32_t peer_base;                   // progress value before this launch (grows by num_layers a launch)
  // this step
  int32_t n_prefix_items, n_suffix_items, n_zero_items, n_merge_items;
  int32_t num_prompts;
  PromptPlan prompt[kMaxPrompts];
  SlotPlan slot[kMaxSlots];
  int8_t zero_slot[kMaxSlots];
  int8_t live_slot[kMaxSlots];
};

}  // namespace infs
