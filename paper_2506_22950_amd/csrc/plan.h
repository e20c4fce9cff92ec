// Per-launch plan of one decode step, passed to the attention kernel by value.
//
// The host knows every slot's length, so it plans the split-K work of a step
// on the CPU and hands it over in the kernel argument block: no per-step
// host-to-device copy is needed.  The same plan serves every layer of a step.
#pragma once
#include <stdint.h>

namespace infs {

constexpr int kMaxSlots = 64;      // S = num_prompts * slots_per_prompt
constexpr int kMaxPrompts = 16;
constexpr int kPageTokens = 16;    // tokens per response page
constexpr int kBlockThreads = 256; // 4 wavefronts of 64
constexpr int kMfmaBlock = 32;     // prefix tokens per MFMA block

// Work item kinds, in grid order: prefix chunks, response chunks, idle slots.
// Grid x = item * Hkv + kv_head, so with 8 KV heads each head's items stay on
// one XCD (work-groups are dealt round-robin over the 8 XCDs).

struct SlotPlan {
  int32_t len;         // response length after this step's append; 0 = idle
  int32_t item_begin;  // first response-chunk item of this slot
  int32_t cur_page;    // page holding position len-1 (where this step's K/V go)
  int32_t sample;      // sample id (token counters)
  int32_t n_expect;    // partials merged for this slot: prefix chunks + response chunks
  int32_t pad_[3];
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
  int32_t* page_table; // [S, pages_per_slot]
  float* ws_o;         // partial outputs   [..., d]
  float* ws_ml;        // partial (max, sum) [..., 2]
  int32_t* counters;   // [S, Hkv] arrivals per (slot, kv head); the merging block resets it
  int32_t* tokens;     // [num_prompts, G] per-sample token counters
  // geometry
  int32_t S, m, G, Hq, Hkv, prefix_rows;  // prefix_rows = m * hpk (real rows)
  int32_t max_prompt_len;     // prefix store row capacity (multiple of 32)
  int32_t pages_per_slot;
  int32_t split;              // chunk length in tokens (prefix and response)
  int32_t prefix_chunks_max;  // ceil(max_prompt_len / split)
  int32_t suffix_chunks_max;  // ceil(max_suffix_len / split)
  int32_t count_tokens;       // 1 on layer 0
  float scale_log2;           // softmax scale * log2(e)
  // this step
  int32_t n_prefix_items, n_suffix_items, n_zero_items;
  int32_t num_prompts;
  PromptPlan prompt[kMaxPrompts];
  SlotPlan slot[kMaxSlots];
  int8_t zero_slot[kMaxSlots];
};

}  // namespace infs
