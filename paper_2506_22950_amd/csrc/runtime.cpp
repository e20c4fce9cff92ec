// Host runtime of the C ABI: context, validation, slot table, response page
// allocator, per-step split-K plan, kernel launches, statistics and timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <functional>
#include <new>
#include <queue>
#include <string>
#include <vector>

#include "infs.h"
#include "kernels.h"
#include "step_plan.h"
#include "plan.h"

using infs::KernelKey;
using infs::StepArgs;

static_assert(sizeof(StepArgs) <= 4096, "kernel argument block must fit 4 KiB");
static_assert(INFS_STATIC_SCRATCH_BYTES == infs::kStaticScratchBytes, "static scratch size: header and library agree");

namespace {
thread_local std::string g_thread_error = "no error";

// Timing mode: each decode launch folds its blocks' device wall-clock start
// and end times into one {min start, max end} pair of a device array; a HIP
// event pair brackets the whole timed region on the context's stream.
struct Timing {
  bool on = false;
  unsigned long long* clocks = nullptr;  // [capacity][kClockSlots * kClockStride] starts, then ends
  int64_t capacity = 0;
  int64_t used = 0;                      // pairs written since the last harvest
  double kernel_ms = 0.0;
  int64_t launches = 0;
  hipEvent_t region[2] = {nullptr, nullptr};
  double ticks_per_ms = 0.0;
};
}  // namespace

constexpr size_t kClockWords = (size_t)infs::kClockSlots * infs::kClockStride;  // per launch

struct infs_ctx {
  infs_config cfg{};
  bool dry = false;
  hipStream_t stream = nullptr;
  KernelKey key{};
  int S = 0, m = 0, G = 0, hpk = 0, D = 0, Hkv = 0, Hq = 0, L = 0, NP = 0;
  int pmax_pad = 0, split = 0, prefix_split = 0, pages_per_slot = 0, num_pages = 0, pcmax = 0, scmax = 0;
  int l2_xcds = 0;    // > 0: work-group b was seen on XCD b % l2_xcds and Hkv is a multiple of it
  size_t es = 0;      // bytes per Q / K / V element handed over the ABI
  size_t kv_es = 0;   // bytes per stored K / V element (prefix store and pages)
  size_t prefix_layer_bytes = 0, pool_layer_bytes = 0;
  int64_t ws_records = 0;
  // device memory
  char* prefix = nullptr;
  char* pool = nullptr;
  int32_t* page_table = nullptr;
  float* ws_o = nullptr;
  float* ws_ml = nullptr;
  int32_t* counters = nullptr;
  int32_t* tokens = nullptr;
  int32_t* status = nullptr;
  void* scratch = nullptr;  // this device's static scratch array (infs_decode_step_static)
  int layers_resident = 0;  // work-groups of the step-launch kernel resident at once (0: no step launch)
  int players_resident = 0; // the same for the probe kernel's step launch (0: none)
  // host state
  std::vector<int32_t> plen;                       // per prompt, -1 before its first prefill
  std::vector<std::vector<uint8_t>> prefilled;     // [prompt][layer]
  std::vector<int64_t> slot_sample;                // -1: empty
  std::vector<int32_t> slot_len;
  // Sequence handles: each live response has a page-table row.  Without probes
  // the handle of a slot's response is the slot; with probes (prefix reuse)
  // it is prompt * G + sample, so a sample keeps its probe pages when it is
  // dispatched.
  int H = 0;
  std::vector<int32_t> slot_handle;                // -1: empty slot
  std::vector<std::vector<int32_t>> seq_pages;     // host copy of each handle's page list
  std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>> free_pages;
  std::vector<std::vector<uint8_t>> dispatched;    // [prompt][G]
  // Arrivals each slot's device counter has been sent so far (the same for
  // every KV head): its response chunks and its prompt's prefix chunks.
  std::vector<uint32_t> slot_arrivals;
  // Merges each prompt's "merged" counter has counted so far (step launches only).
  std::vector<uint32_t> merged_arrivals;
  uint32_t peer_progress = 0;  // peer-line progress value reached by the step launches so far
  uint32_t probe_merged_arrivals = 0;  // merges counted by probe step launches so far
  bool step_open = false;
  // Probe phase of prefix reuse.
  int step_split = 1;                              // infs_set_step_split: 1 planned pieces, 0 per-layer chunks
  int probe_k = 0;                                 // probe tokens per sample (0: no prefix reuse)
  int probe_batch = 0;                             // most samples per probe launch
  KernelKey pkey{};                                // kernel of probe launches
  std::vector<std::vector<int32_t>> probe_len;     // [prompt][G] probe tokens decoded
  bool probe_open = false;
  std::vector<uint8_t> probe_layer_done;
  int probe_layers_done = 0;
  int pb_prompt = -1, pb_first = 0, pb_n = 0;      // the open probe step's batch
  uint8_t pb_live[infs::kMaxSlots] = {};
  StepArgs pplan{};
  int pgrid = 0;
  double pstep_bytes = 0, pstep_flops = 0;
  std::vector<uint32_t> probe_slot_arrivals;
  std::vector<uint8_t> layer_done;
  int layers_done = 0;
  StepArgs plan{};
  int grid = 0;
  double step_bytes = 0, step_flops = 0;
  infs_stats stats{};
  bool dead = false;
  std::string dead_msg;  // the device error that made the context unusable
  std::string err = "no error";
  Timing timing;
};

namespace {

infs_status fail(infs_ctx* c, infs_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c)
    c->err = buf;
  else
    g_thread_error = buf;
  return st;
}

infs_status device_fail(infs_ctx* c, hipError_t e, const char* what) {
  const infs_status st = fail(c, e == hipErrorOutOfMemory ? INFS_E_NOMEM : INFS_E_DEVICE, "%s failed: %s", what,
                              hipGetErrorString(e));
  if (c) {
    c->dead = true;
    c->dead_msg = c->err;
  }
  return st;
}

#define HIP_TRY(ctx, expr)                                  \
  do {                                                      \
    hipError_t e_ = (expr);                                 \
    if (e_ != hipSuccess) return device_fail(ctx, e_, #expr); \
  } while (0)

#define CHECK_CTX(c)                                                                  \
  do {                                                                                \
    if (!(c)) return fail(nullptr, INFS_E_ARG, "null context");                      \
    if ((c)->dead) return fail(c, INFS_E_DEVICE, "context unusable after a device error: %s", (c)->dead_msg.c_str()); \
  } while (0)

int ceil_div(int a, int b) { return (a + b - 1) / b; }

void free_device(infs_ctx* c) {
  if (c->dry) return;
  (void)hipFree(c->prefix);
  (void)hipFree(c->pool);
  (void)hipFree(c->page_table);
  (void)hipFree(c->ws_o);
  (void)hipFree(c->ws_ml);
  (void)hipFree(c->counters);
  (void)hipFree(c->tokens);
  (void)hipFree(c->status);
}

// Counters: one per (slot, KV head) for decode launches [S][Hkv], then the
// probe launches' own [kMaxSlots][Hkv], then for step launches one "merged"
// counter per prompt, one layer-done flag per (prompt, KV head) and one peer
// line per work-group; each on a 128-byte line of its own.
size_t probe_merged_lines(const infs_ctx* c) { return c->probe_k > 0 ? 1 + (size_t)c->Hkv : 0; }
size_t counter_lines(const infs_ctx* c) {
  return (size_t)(c->S + infs::kMaxSlots) * c->Hkv + c->NP + (size_t)c->NP * c->Hkv + probe_merged_lines(c) +
         (size_t)std::max(c->layers_resident, c->players_resident);
}
size_t counter_bytes(const infs_ctx* c) { return sizeof(int32_t) * infs::kCounterStride * counter_lines(c); }
int32_t* merged_counters(const infs_ctx* c) {
  return c->counters + (size_t)(c->S + infs::kMaxSlots) * c->Hkv * infs::kCounterStride;
}
// The merged counter and layer flags of probe step launches (one prompt's layout).
int32_t* probe_merged_counters(const infs_ctx* c) {
  return merged_counters(c) + ((size_t)c->NP + (size_t)c->NP * c->Hkv) * infs::kCounterStride;
}
int32_t* peer_lines(const infs_ctx* c) { return probe_merged_counters(c) + probe_merged_lines(c) * infs::kCounterStride; }

// Split-K record capacities.  Records are numbered (prompt, KV head)-major for
// prefix chunks and (slot, KV head)-major for response chunks, so padding the
// chunks per (prompt | slot, KV head) to fill whole 128-byte lines of (max,
// sum) records gives every line to one KV head: in the XCD-local exchange no
// two XCDs then write the same line.
int lines_of_records(int chunks, int rows) {
  const int per_line = std::max(1, infs::kRecordsPerLine / rows);
  return (chunks + per_line - 1) / per_line * per_line;
}
int prefix_chunk_capacity(const infs::KernelKey& key, const infs::KernelKey* probe_key, int chunks) {
  const int rows = probe_key ? std::min(key.prefix_rows, probe_key->prefix_rows) : key.prefix_rows;
  return lines_of_records(chunks, rows);
}
int response_chunk_capacity(const infs::KernelKey& key, int chunks) { return lines_of_records(chunks, key.hpk); }

void reset_host(infs_ctx* c) {
  c->plen.assign(c->NP, -1);
  c->prefilled.assign(c->NP, std::vector<uint8_t>(c->L, 0));
  c->slot_sample.assign(c->S, -1);
  c->slot_len.assign(c->S, 0);
  c->slot_handle.assign(c->S, -1);
  c->seq_pages.assign(c->H, {});
  c->free_pages = {};
  for (int i = 0; i < c->num_pages; ++i) c->free_pages.push(i);
  c->dispatched.assign(c->NP, std::vector<uint8_t>(c->G, 0));
  c->slot_arrivals.assign(c->S, 0);
  c->merged_arrivals.assign(c->NP, 0);
  c->peer_progress = 0;
  c->probe_merged_arrivals = 0;
  c->step_open = false;
  c->probe_len.assign(c->probe_k > 0 ? c->NP : 0, std::vector<int32_t>(c->G, 0));
  c->probe_open = false;
  c->probe_layer_done.assign(c->L, 0);
  c->probe_layers_done = 0;
  c->probe_slot_arrivals.assign(infs::kMaxSlots, 0);
  c->layer_done.assign(c->L, 0);
  c->layers_done = 0;
  c->stats = infs_stats{};
}

// Build the plan of the step that is about to open: lengths after the append,
// pages, chunk items.  Validates before changing anything.
infs_status open_step(infs_ctx* c) {
  int need_pages = 0;
  for (int s = 0; s < c->S; ++s) {
    if (c->slot_sample[s] < 0) continue;
    if (c->slot_len[s] + 1 > c->cfg.max_suffix_len)
      return fail(c, INFS_E_CAPACITY, "slot %d: response would exceed max_suffix_len=%d", s, c->cfg.max_suffix_len);
    if (c->slot_len[s] % infs::kPageTokens == 0) ++need_pages;
  }
  if ((size_t)need_pages > c->free_pages.size())
    return fail(c, INFS_E_CAPACITY, "page pool exhausted: need %d pages, %zu free", need_pages, c->free_pages.size());

  StepArgs& a = c->plan;
  a.prefix_split = c->prefix_split;  // a step launch may have lengthened the chunks of the last step
  int items = 0;
  std::vector<int> live(c->NP, 0);
  for (int s = 0; s < c->S; ++s)
    if (c->slot_sample[s] >= 0) ++live[s / c->m];
  for (int p = 0; p < c->NP; ++p) {
    if (live[p] > 0 && c->plen[p] < 0)
      return fail(c, INFS_E_STATE, "prompt %d has live slots but no prefilled prefix", p);
  }
  double bytes = 0, flops = 0;
  const double kvrow = (double)c->Hkv * c->D * c->kv_es;    // one stored K or V row, all heads
  const double kvrow_in = (double)c->Hkv * c->D * c->es;    // one caller K or V row
  for (int p = 0; p < c->NP; ++p) {
    infs::PromptPlan& pp = a.prompt[p];
    pp.plen = std::max(c->plen[p], 0);
    pp.nchunks = live[p] > 0 ? ceil_div(pp.plen, c->prefix_split) : 0;
    pp.item_begin = items;
    items += pp.nchunks;
    if (live[p] > 0) bytes += 2.0 * pp.plen * kvrow;
  }
  a.n_prefix_items = items;
  items = 0;
  int zeros = 0, lives = 0;
  for (int s = 0; s < c->S; ++s) {
    infs::SlotPlan& sp = a.slot[s];
    sp = infs::SlotPlan{};
    if (c->slot_sample[s] < 0) {
      sp.item_begin = items;
      a.zero_slot[zeros++] = (int8_t)s;
      continue;
    }
    const int len = c->slot_len[s] + 1;
    const int pos = len - 1;
    const int h = c->slot_handle[s];
    if (pos % infs::kPageTokens == 0) {
      c->seq_pages[h].push_back(c->free_pages.top());
      c->free_pages.pop();
    }
    a.live_slot[lives++] = (int8_t)s;
    sp.len = len;
    sp.item_begin = items;
    sp.seq = h;
    sp.cur_page = c->seq_pages[h][pos / infs::kPageTokens];
    sp.sample = (int32_t)c->slot_sample[s];
    const int nch = ceil_div(len, c->split);
    sp.pieces = nch;
    items += nch;
    const int P = a.prompt[s / c->m].plen;
    bytes += 2.0 * (len - 1) * kvrow + 2.0 * kvrow_in + 2.0 * kvrow + (double)c->Hq * c->D * (c->es + 4);
    flops += 4.0 * c->Hq * c->D * (double)(P + len);
  }
  a.n_suffix_items = items;
  a.n_zero_items = zeros;
  a.n_merge_items = lives;
  a.live_mask = 0;
  for (int s = 0; s < c->S; ++s)
    if (a.slot[s].len > 0) a.live_mask |= uint64_t(1) << s;
  c->grid = (a.n_prefix_items + a.n_suffix_items + a.n_zero_items + a.n_merge_items) * c->Hkv;
  c->step_bytes = bytes;
  c->step_flops = flops;
  c->step_open = true;
  std::fill(c->layer_done.begin(), c->layer_done.end(), 0);
  c->layers_done = 0;
  return INFS_OK;
}

// Build the plan of a probe step for samples first .. first+n-1 of prompt p
// (live[j] != 0: sample first+j decodes its next probe token).  The probe plan
// is a one-prompt decode plan whose slots are the batch's samples; the launch
// offsets the prefix, token-counter and counter pointers to prompt p and to
// the probe counters.  Validates before changing anything.
infs_status open_probe(infs_ctx* c, int p, int first, int n, const uint8_t* live) {
  int need_pages = 0, nlive = 0;
  for (int j = 0; j < n; ++j) {
    if (!live[j]) continue;
    const int i = first + j;
    ++nlive;
    if (c->dispatched[p][i])
      return fail(c, INFS_E_STATE, "sample %d of prompt %d was already dispatched or released", i, p);
    if (c->probe_len[p][i] >= c->probe_k)
      return fail(c, INFS_E_CAPACITY, "sample %d of prompt %d already has probe_tokens=%d probe tokens", i, p,
                  c->probe_k);
    if (c->probe_len[p][i] % infs::kPageTokens == 0) ++need_pages;
  }
  if ((size_t)need_pages > c->free_pages.size())
    return fail(c, INFS_E_CAPACITY, "page pool exhausted: need %d pages, %zu free", need_pages, c->free_pages.size());
  if (nlive > 0 && c->plen[p] < 0) return fail(c, INFS_E_STATE, "prompt %d has no prefilled prefix", p);
  StepArgs& a = c->pplan;
  a = c->plan;
  a.prefix_split = c->prefix_split;
  a.S = n;
  a.m = n;
  a.num_prompts = 1;
  a.prefix_rows = n * c->hpk;
  a.clock_start = a.clock_end = nullptr;
  for (int q = 0; q < infs::kMaxPrompts; ++q) a.prompt[q] = infs::PromptPlan{};
  const double kvrow = (double)c->Hkv * c->D * c->kv_es;    // one stored K or V row, all heads
  const double kvrow_in = (double)c->Hkv * c->D * c->es;    // one caller K or V row
  double bytes = 0, flops = 0;
  infs::PromptPlan& pp = a.prompt[0];
  pp.plen = std::max(c->plen[p], 0);
  pp.nchunks = nlive > 0 ? ceil_div(pp.plen, c->prefix_split) : 0;
  pp.item_begin = 0;
  if (nlive > 0) bytes += 2.0 * pp.plen * kvrow;
  int items = 0, zeros = 0, lives = 0;
  a.n_prefix_items = pp.nchunks;
  for (int j = 0; j < n; ++j) {
    infs::SlotPlan& sp = a.slot[j];
    sp = infs::SlotPlan{};
    if (!live[j]) {
      sp.item_begin = items;
      a.zero_slot[zeros++] = (int8_t)j;
      continue;
    }
    const int i = first + j, h = p * c->G + i;
    const int len = c->probe_len[p][i] + 1, pos = len - 1;
    if (pos % infs::kPageTokens == 0) {
      c->seq_pages[h].push_back(c->free_pages.top());
      c->free_pages.pop();
    }
    a.live_slot[lives++] = (int8_t)j;
    sp.len = len;
    sp.item_begin = items;
    sp.seq = h;
    sp.sample = i;
    sp.cur_page = c->seq_pages[h][pos / infs::kPageTokens];
    items += ceil_div(len, c->split);
    bytes += 2.0 * (len - 1) * kvrow + 2.0 * kvrow_in + 2.0 * kvrow + (double)c->Hq * c->D * (c->es + 4);
    flops += 4.0 * c->Hq * c->D * (double)(pp.plen + len);
  }
  a.n_suffix_items = items;
  a.n_zero_items = zeros;
  a.n_merge_items = lives;
  a.live_mask = 0;
  for (int j = 0; j < n; ++j)
    if (a.slot[j].len > 0) a.live_mask |= uint64_t(1) << j;
  c->pgrid = (a.n_prefix_items + a.n_suffix_items + a.n_zero_items + a.n_merge_items) * c->Hkv;
  c->pstep_bytes = bytes;
  c->pstep_flops = flops;
  c->pb_prompt = p;
  c->pb_first = first;
  c->pb_n = n;
  std::memcpy(c->pb_live, live, n);
  c->probe_open = true;
  std::fill(c->probe_layer_done.begin(), c->probe_layer_done.end(), 0);
  c->probe_layers_done = 0;
  return INFS_OK;
}

// Start times to all ones (so the first block's minimum wins), end times to 0.
infs_status arm_clocks(infs_ctx* c) {
  Timing& t = c->timing;
  const size_t n = (size_t)t.capacity * kClockWords;
  HIP_TRY(c, hipMemsetAsync(t.clocks, 0xFF, sizeof(unsigned long long) * n, c->stream));
  HIP_TRY(c, hipMemsetAsync(t.clocks + n, 0, sizeof(unsigned long long) * n, c->stream));
  return INFS_OK;
}

// Add up the durations of the launches timed so far and re-arm the arrays.
infs_status harvest_clocks(infs_ctx* c) {
  Timing& t = c->timing;
  if (t.used > 0) {
    const size_t n = (size_t)t.capacity * kClockWords;
    std::vector<unsigned long long> h(2 * n);
    HIP_TRY(c, hipStreamSynchronize(c->stream));
    HIP_TRY(c, hipMemcpy(h.data(), t.clocks, h.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost));
    for (int64_t i = 0; i < t.used; ++i) {
      unsigned long long a = ~0ull, b = 0;
      for (int k = 0; k < infs::kClockSlots; ++k) {
        const size_t x = (size_t)i * kClockWords + (size_t)k * infs::kClockStride;
        if (h[n + x] == 0) continue;  // slot not reached by any block
        a = std::min(a, h[x]);
        b = std::max(b, h[n + x]);
      }
      if (b > a) t.kernel_ms += (double)(b - a) / t.ticks_per_ms;
    }
    t.launches += t.used;
    t.used = 0;
  }
  return arm_clocks(c);
}

// After a synchronisation: report a merge block that stopped waiting.
infs_status check_status(infs_ctx* c) {
  int32_t st = 0;
  HIP_TRY(c, hipMemcpy(&st, c->status, sizeof st, hipMemcpyDeviceToHost));
  if (st != 0) {
    fail(c, INFS_E_DEVICE, st == 2 ? "a work-group ran on another XCD than the XCD-local exchange of partials "
                                     "assumes; outputs are invalid (infs_set_exchange(ctx, 0) avoids it)"
                                   : "a decode launch gave up waiting (a merge for its producers, or a layer of a "
                                     "step launch for the previous layer); outputs are invalid");
    c->dead = true;
    c->dead_msg = c->err;
    return INFS_E_DEVICE;
  }
  return INFS_OK;
}

// Advance the arrival targets by this launch's producers.
void set_targets(infs_ctx* c) {
  StepArgs& a = c->plan;
  for (int s = 0; s < c->S; ++s) {
    if (a.slot[s].len > 0)
      c->slot_arrivals[s] += (uint32_t)(ceil_div(a.slot[s].len, c->split) + a.prompt[s / c->m].nchunks);
    a.slot[s].target = (int32_t)c->slot_arrivals[s];
  }
}

// Launch one decode or probe kernel (or, with `layers`, the step launch through
// every layer); in timing mode it records its start and end.
infs_status timed_launch(infs_ctx* c, const KernelKey& key, StepArgs& a, int grid, bool layers = false) {
  Timing& t = c->timing;
  a.clock_start = a.clock_end = nullptr;
  if (t.on) {
    if (t.used == t.capacity) {
      infs_status st = harvest_clocks(c);
      if (st != INFS_OK) return st;
    }
    a.clock_start = t.clocks + (size_t)t.used * kClockWords;
    a.clock_end = t.clocks + ((size_t)t.capacity + t.used) * kClockWords;
    ++t.used;
  }
  HIP_TRY(c, layers ? infs::launch_layers(key, a, grid, c->stream) : infs::launch_decode(key, a, grid, c->stream));
  return INFS_OK;
}

// Layout of a decode launch's split-K exchange in the static scratch array:
// the arrival counters [S][Hkv] (one 128-byte line each), then the (max, sum)
// records, then the partial outputs, each part 256-byte aligned.  Returns the
// bytes needed.
struct StaticLayout {
  size_t counters = 0, ml = 0, o = 0, ml_bytes = 0, o_bytes = 0, total = 0;
};
StaticLayout static_layout(const infs_ctx* c) {
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  StaticLayout s;
  const int64_t recs = infs::workspace_records(c->key, c->NP, c->Hkv, c->pcmax, c->S, c->scmax);
  s.counters = 0;
  s.ml = up(sizeof(int32_t) * infs::kCounterStride * (size_t)c->S * c->Hkv);
  s.ml_bytes = sizeof(float) * 2 * (size_t)recs;
  s.o = s.ml + up(s.ml_bytes);
  s.o_bytes = sizeof(float) * (size_t)c->D * recs;
  s.total = s.o + up(s.o_bytes);
  return s;
}

// Where work-groups run: a probe launch of kProbeBlocks work-groups records
// each one's XCD.  If work-group b ran on XCD b % n for n distinct XCDs and Hkv
// is a multiple of n, every KV head's work-groups share one XCD (item * Hkv + g
// is g modulo n), and partials can be exchanged through that XCD's L2.
infs_status probe_xcds(infs_ctx* c) {
  constexpr int kProbeBlocks = 4096;
  c->l2_xcds = 0;
  int32_t* d = nullptr;
  hipError_t e = hipMalloc((void**)&d, sizeof(int32_t) * kProbeBlocks);
  if (e != hipSuccess) return device_fail(nullptr, e, "hipMalloc(XCD probe)");
  std::vector<int32_t> h(kProbeBlocks);
  e = infs::launch_xcd_probe(d, kProbeBlocks, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e == hipSuccess) e = hipMemcpy(h.data(), d, sizeof(int32_t) * kProbeBlocks, hipMemcpyDeviceToHost);
  (void)hipFree(d);
  if (e != hipSuccess) return device_fail(nullptr, e, "XCD probe");
  const int n = *std::max_element(h.begin(), h.end()) + 1;
  bool ok = n >= 1 && c->Hkv % n == 0;
  for (int b = 0; ok && b < kProbeBlocks; ++b) ok = h[b] == b % n;
  if (ok) c->l2_xcds = n;
  return INFS_OK;
}

}  // namespace

extern "C" {

int32_t infs_abi_version(void) { return INFS_ABI_VERSION; }

const char* infs_last_error(const infs_ctx* ctx) { return ctx ? ctx->err.c_str() : g_thread_error.c_str(); }

infs_status infs_create(const infs_config* cfg, void* hip_stream, infs_ctx** out) {
  if (!out) return fail(nullptr, INFS_E_ARG, "out is null");
  *out = nullptr;
  if (!cfg) return fail(nullptr, INFS_E_ARG, "cfg is null");
  const infs_config& k = *cfg;
  if (k.num_layers < 1 || k.num_layers > 4096) return fail(nullptr, INFS_E_ARG, "num_layers must be in [1, 4096]");
  if (k.num_kv_heads < 1 || k.num_q_heads < 1 || k.num_q_heads % k.num_kv_heads)
    return fail(nullptr, INFS_E_ARG, "num_q_heads must be a positive multiple of num_kv_heads");
  if (k.head_dim != 64 && k.head_dim != 128) return fail(nullptr, INFS_E_ARG, "head_dim must be 64 or 128");
  if (k.num_prompts < 1 || k.num_prompts > infs::kMaxPrompts)
    return fail(nullptr, INFS_E_ARG, "num_prompts must be in [1, %d]", infs::kMaxPrompts);
  if (k.slots_per_prompt < 1 || (int64_t)k.num_prompts * k.slots_per_prompt > infs::kMaxSlots)
    return fail(nullptr, INFS_E_ARG, "num_prompts * slots_per_prompt must be in [1, %d]", infs::kMaxSlots);
  if (k.samples_per_prompt < 1 || k.samples_per_prompt > (1 << 24))
    return fail(nullptr, INFS_E_ARG, "samples_per_prompt must be in [1, 2^24]");
  if (k.max_prompt_len < 0 || k.max_prompt_len > (1 << 20))
    return fail(nullptr, INFS_E_ARG, "max_prompt_len must be in [0, 2^20]");
  if (k.max_suffix_len < 1 || k.max_suffix_len > (1 << 20))
    return fail(nullptr, INFS_E_ARG, "max_suffix_len must be in [1, 2^20]");
  if (k.page_tokens != 0 && k.page_tokens != infs::kPageTokens)
    return fail(nullptr, INFS_E_ARG, "page_tokens must be 0 or %d", infs::kPageTokens);
  if (k.split_tokens < 0 || k.split_tokens % 128 || k.split_tokens > infs::kMaxSplit)
    return fail(nullptr, INFS_E_ARG, "split_tokens must be 0 or a multiple of 128 up to %d", infs::kMaxSplit);
  if (k.num_pages < 0) return fail(nullptr, INFS_E_ARG, "num_pages must be >= 0");
  if (k.dtype != INFS_F32 && k.dtype != INFS_BF16) return fail(nullptr, INFS_E_ARG, "dtype must be INFS_F32 or INFS_BF16");
  if (!(k.scale >= 0.f) || !std::isfinite(k.scale)) return fail(nullptr, INFS_E_ARG, "scale must be finite and >= 0");
  if (k.flags & ~(INFS_FLAG_DRY_RUN | INFS_FLAG_KV_FP8)) return fail(nullptr, INFS_E_ARG, "unknown flags");
  const int kv8 = (k.flags & INFS_FLAG_KV_FP8) ? 1 : 0;
  if (k.probe_tokens < 0 || k.probe_tokens > k.max_suffix_len)
    return fail(nullptr, INFS_E_ARG, "probe_tokens must be in [0, max_suffix_len]");

  const int hpk = k.num_q_heads / k.num_kv_heads;
  KernelKey key{};
  if (kv8 && (k.dtype != INFS_BF16 || k.head_dim != 128 || k.slots_per_prompt * hpk < 16))
    return fail(nullptr, INFS_E_ARG,
                "INFS_FLAG_KV_FP8 needs bf16, head_dim 128 and at least 16 prefix rows (slots_per_prompt * heads_per_kv)");
  if (!infs::select_kernel(k.dtype == INFS_BF16, k.head_dim, hpk, k.slots_per_prompt * hpk, kv8, &key))
    return fail(nullptr, INFS_E_ARG,
                "no kernel for dtype=%s head_dim=%d heads_per_kv=%d prefix rows=%d (bf16 supports up to 128 rows, "
                "fp32 up to 16)",
                k.dtype == INFS_BF16 ? "bf16" : "f32", k.head_dim, hpk, k.slots_per_prompt * hpk);
  // Probe launches put up to probe_batch samples' rows on one prefix work item,
  // on the prefix path of the decode kernel (the prefix store layout is shared).
  KernelKey pkey{};
  int probe_batch = 0;
  if (k.probe_tokens > 0) {
    const int max_rows = key.mfma ? 128 : 16;
    probe_batch = std::min({infs::kMaxSlots, max_rows / hpk, k.samples_per_prompt});
    if (probe_batch < 1 ||
        !infs::select_kernel_path(k.dtype == INFS_BF16, k.head_dim, hpk, probe_batch * hpk, key.mfma, kv8, &pkey))
      return fail(nullptr, INFS_E_ARG, "no probe kernel for heads_per_kv=%d", hpk);
  }
  {
    const int split = k.split_tokens ? k.split_tokens : 256;
    const int psplit = key.mfma ? infs::kMfmaPrefixSplit : split;
    const int parts = (k.max_prompt_len + psplit - 1) / psplit + (k.max_suffix_len + split - 1) / split;
    if (parts > infs::kMaxPartials)
      return fail(nullptr, INFS_E_ARG,
                  "max_prompt_len and max_suffix_len need %d split-K chunks per slot (limit %d): raise split_tokens",
                  parts, infs::kMaxPartials);
    const int pcm = prefix_chunk_capacity(key, k.probe_tokens > 0 ? &pkey : nullptr,
                                          std::max(1, (k.max_prompt_len + psplit - 1) / psplit));
    const int scm = response_chunk_capacity(key, (k.max_suffix_len + split - 1) / split);
    int64_t recs = infs::workspace_records(key, k.num_prompts, k.num_kv_heads, pcm, k.num_prompts * k.slots_per_prompt, scm);
    if (k.probe_tokens > 0)
      recs = std::max(recs, infs::workspace_records(pkey, 1, k.num_kv_heads, pcm, probe_batch, scm));
    const int64_t ws_bytes = recs * k.head_dim * (int64_t)sizeof(float);
    if (ws_bytes >= (int64_t(1) << 31))
      return fail(nullptr, INFS_E_ARG, "split-K workspace of %lld bytes exceeds 2 GiB: lower num_kv_heads or raise split_tokens",
                  (long long)ws_bytes);
  }
  infs_ctx* c = new (std::nothrow) infs_ctx;
  if (!c) return fail(nullptr, INFS_E_NOMEM, "host allocation failed");
  c->cfg = k;
  c->dry = (k.flags & INFS_FLAG_DRY_RUN) != 0;
  c->stream = (hipStream_t)hip_stream;
  c->key = key;
  c->pkey = pkey;
  c->probe_k = k.probe_tokens;
  c->probe_batch = probe_batch;
  c->NP = k.num_prompts;
  c->m = k.slots_per_prompt;
  c->S = c->NP * c->m;
  c->G = k.samples_per_prompt;
  c->hpk = hpk;
  c->D = k.head_dim;
  c->Hkv = k.num_kv_heads;
  c->Hq = k.num_q_heads;
  c->L = k.num_layers;
  c->es = k.dtype == INFS_BF16 ? 2 : 4;
  c->kv_es = key.kv8 ? 1 : c->es;
  c->split = k.split_tokens ? k.split_tokens : 256;
  c->pmax_pad = std::max(32, (k.max_prompt_len + 31) / 32 * 32);
  c->pages_per_slot = ceil_div(k.max_suffix_len, infs::kPageTokens);
  c->H = c->probe_k > 0 ? c->NP * c->G : c->S;
  if ((int64_t)c->H * c->pages_per_slot * (int64_t)sizeof(int32_t) >= (int64_t(1) << 31)) {
    const int seqs = c->H, pps = c->pages_per_slot;
    delete c;
    return fail(nullptr, INFS_E_ARG, "page table of %d sequences x %d pages exceeds 2 GiB", seqs, pps);
  }
  {
    const int64_t pages = k.num_pages ? (int64_t)k.num_pages
                                      : (int64_t)c->S * c->pages_per_slot +
                                            (c->probe_k > 0 ? (int64_t)c->NP * c->G * ceil_div(c->probe_k, infs::kPageTokens)
                                                            : 0);
    if (pages > INT32_MAX) {
      delete c;
      return fail(nullptr, INFS_E_ARG, "a page pool of %lld pages is beyond the page index range", (long long)pages);
    }
    c->num_pages = (int)pages;
  }
  c->prefix_split = key.mfma ? infs::kMfmaPrefixSplit : c->split;
  c->pcmax = prefix_chunk_capacity(key, c->probe_k > 0 ? &pkey : nullptr,
                                   std::max(1, ceil_div(k.max_prompt_len, c->prefix_split)));
  c->scmax = response_chunk_capacity(key, ceil_div(k.max_suffix_len, c->split));
  c->prefix_layer_bytes = (size_t)c->NP * c->Hkv * infs::prefix_elems_per_head(key, c->pmax_pad) * c->kv_es;
  c->pool_layer_bytes = (size_t)c->num_pages * c->Hkv * 2 * infs::kPageTokens * c->D * c->kv_es;
  c->ws_records = infs::workspace_records(key, c->NP, c->Hkv, c->pcmax, c->S, c->scmax);
  if (c->probe_k > 0)
    c->ws_records =
        std::max(c->ws_records, infs::workspace_records(pkey, 1, c->Hkv, c->pcmax, c->probe_batch, c->scmax));
  reset_host(c);

  StepArgs& a = c->plan;
  a.S = c->S;
  a.m = c->m;
  a.G = c->G;
  a.Hq = c->Hq;
  a.Hkv = c->Hkv;
  a.prefix_rows = c->m * hpk;
  a.max_prompt_len = c->pmax_pad;
  a.pages_per_slot = c->pages_per_slot;
  a.split = c->split;
  a.prefix_split = c->prefix_split;
  a.prefix_chunks_max = c->pcmax;
  a.suffix_chunks_max = c->scmax;
  a.num_prompts = c->NP;
  const float scale = k.scale > 0.f ? k.scale : 1.0f / std::sqrt((float)k.head_dim);
  a.scale_log2 = scale * 1.4426950408889634f;
  a.ws_o_bytes = (uint32_t)(c->ws_records * c->D * sizeof(float));
  a.ws_ml_bytes = (uint32_t)(c->ws_records * 2 * sizeof(float));
  a.merge_polls = infs::kMergeSpins;

  if (!c->dry) {
    auto alloc = [&](void** p, size_t bytes, const char* what) -> infs_status {
      hipError_t e = hipMalloc(p, std::max<size_t>(bytes, 256));
      if (e != hipSuccess) {
        return fail(nullptr, e == hipErrorOutOfMemory ? INFS_E_NOMEM : INFS_E_DEVICE, "hipMalloc(%s, %zu bytes): %s",
                    what, bytes, hipGetErrorString(e));
      }
      e = hipMemset(*p, 0, std::max<size_t>(bytes, 256));
      if (e != hipSuccess) return fail(nullptr, INFS_E_DEVICE, "hipMemset(%s): %s", what, hipGetErrorString(e));
      return INFS_OK;
    };
    const hipError_t oe = infs::layers_resident(key, &c->layers_resident);
    if (oe != hipSuccess) {
      delete c;
      return device_fail(nullptr, oe, "occupancy query of the step launch");
    }
    // a step launch needs at least one producer and one merge work-group per KV head
    if (c->layers_resident / c->Hkv < 2) c->layers_resident = 0;
    if (c->probe_k > 0) {
      const hipError_t pe = infs::layers_resident(c->pkey, &c->players_resident);
      if (pe != hipSuccess) {
        delete c;
        return device_fail(nullptr, pe, "occupancy query of the probe step launch");
      }
      if (c->players_resident / c->Hkv < 2) c->players_resident = 0;
    }
    infs_status st = INFS_OK;
    if (st == INFS_OK) st = alloc((void**)&c->prefix, c->prefix_layer_bytes * c->L, "prefix store");
    if (st == INFS_OK) st = alloc((void**)&c->pool, c->pool_layer_bytes * c->L, "page pool");
    if (st == INFS_OK) st = alloc((void**)&c->page_table, sizeof(int32_t) * c->H * c->pages_per_slot, "page table");
    if (st == INFS_OK) st = alloc((void**)&c->ws_o, sizeof(float) * c->ws_records * c->D, "workspace");
    if (st == INFS_OK) st = alloc((void**)&c->ws_ml, sizeof(float) * c->ws_records * 2, "workspace");
    if (st == INFS_OK) st = alloc((void**)&c->counters, counter_bytes(c), "counters");
    if (st == INFS_OK) st = alloc((void**)&c->tokens, sizeof(int32_t) * c->NP * c->G, "token counters");
    if (st == INFS_OK) st = alloc((void**)&c->status, sizeof(int32_t), "status word");
    if (st != INFS_OK) {
      free_device(c);
      delete c;
      return st;
    }
    st = probe_xcds(c);
    if (st != INFS_OK) {
      free_device(c);
      delete c;
      return st;
    }
    const hipError_t se = infs::static_scratch_ptr(&c->scratch);
    if (se != hipSuccess) {
      free_device(c);
      delete c;
      return device_fail(nullptr, se, "hipGetSymbolAddress(static scratch)");
    }
    a.l2_xcds = c->l2_xcds;
    a.page_table = c->page_table;
    a.ws_o = c->ws_o;
    a.ws_ml = c->ws_ml;
    a.counters = c->counters;
    a.tokens = c->tokens;
    a.status = c->status;
  }
  *out = c;
  return INFS_OK;
}

void infs_destroy(infs_ctx* c) {
  if (!c) return;
  if (!c->dry) {
    (void)hipStreamSynchronize(c->stream);
    if (c->timing.clocks) (void)hipFree(c->timing.clocks);
    for (auto e : c->timing.region)
      if (e) (void)hipEventDestroy(e);
    free_device(c);
  }
  delete c;
}

infs_status infs_reset(infs_ctx* c) {
  CHECK_CTX(c);
  reset_host(c);
  if (!c->dry) {
    HIP_TRY(c, hipMemsetAsync(c->tokens, 0, sizeof(int32_t) * c->NP * c->G, c->stream));
    HIP_TRY(c, hipMemsetAsync(c->counters, 0, counter_bytes(c), c->stream));
  }
  return INFS_OK;
}

infs_status infs_prefill_shared(infs_ctx* c, int32_t prompt, int32_t layer, int32_t prompt_len, const void* k_dev,
                                const void* v_dev) {
  CHECK_CTX(c);
  if (prompt < 0 || prompt >= c->NP) return fail(c, INFS_E_ARG, "prompt %d out of range [0, %d)", prompt, c->NP);
  if (layer < 0 || layer >= c->L) return fail(c, INFS_E_ARG, "layer %d out of range [0, %d)", layer, c->L);
  if (prompt_len < 0 || prompt_len > c->cfg.max_prompt_len)
    return fail(c, INFS_E_ARG, "prompt_len %d out of range [0, %d]", prompt_len, c->cfg.max_prompt_len);
  if (c->plen[prompt] >= 0 && c->plen[prompt] != prompt_len)
    return fail(c, INFS_E_ARG, "prompt %d was prefilled with %d tokens in another layer", prompt, c->plen[prompt]);
  if (c->step_open || c->probe_open) return fail(c, INFS_E_STATE, "prefill while a step is open");
  if (!c->dry && prompt_len > 0 && (!k_dev || !v_dev)) return fail(c, INFS_E_ARG, "null K/V pointer");
  if (!c->dry && prompt_len > 0 && (((uintptr_t)k_dev | (uintptr_t)v_dev) & 15))
    return fail(c, INFS_E_ARG, "K/V must be 16-byte aligned");
  if (!c->dry) {
    HIP_TRY(c, infs::launch_prefill(c->key, c->prefix + c->prefix_layer_bytes * layer, k_dev, v_dev, prompt,
                                    prompt_len, c->Hkv, c->pmax_pad, c->stream));
  }
  c->plen[prompt] = prompt_len;
  c->prefilled[prompt][layer] = 1;
  return INFS_OK;
}

infs_status infs_refill_slot(infs_ctx* c, int32_t slot, int32_t prompt, int64_t sample_id) {
  CHECK_CTX(c);
  if (slot < 0 || slot >= c->S) return fail(c, INFS_E_ARG, "slot %d out of range [0, %d)", slot, c->S);
  if (prompt != slot / c->m) return fail(c, INFS_E_ARG, "slot %d serves prompt %d, not %d", slot, slot / c->m, prompt);
  if (sample_id < 0 || sample_id >= c->G)
    return fail(c, INFS_E_ARG, "sample_id %lld out of range [0, %d)", (long long)sample_id, c->G);
  if (c->step_open) return fail(c, INFS_E_STATE, "refill while a step is open");
  if (c->slot_sample[slot] >= 0) return fail(c, INFS_E_STATE, "slot %d is live", slot);
  if (c->dispatched[prompt][sample_id])
    return fail(c, INFS_E_DUP, "sample %lld of prompt %d was already dispatched", (long long)sample_id, prompt);
  if (c->probe_open) return fail(c, INFS_E_STATE, "refill while a probe step is open");
  c->dispatched[prompt][sample_id] = 1;
  c->slot_sample[slot] = sample_id;
  if (c->probe_k > 0) {
    c->slot_handle[slot] = prompt * c->G + (int32_t)sample_id;
    c->slot_len[slot] = c->probe_len[prompt][sample_id];  // decoding resumes after the probe tokens
  } else {
    c->slot_handle[slot] = slot;
    c->slot_len[slot] = 0;
  }
  return INFS_OK;
}

infs_status infs_retire_slot(infs_ctx* c, int32_t slot) {
  CHECK_CTX(c);
  if (slot < 0 || slot >= c->S) return fail(c, INFS_E_ARG, "slot %d out of range [0, %d)", slot, c->S);
  if (c->step_open) return fail(c, INFS_E_STATE, "retire while a step is open");
  if (c->slot_sample[slot] < 0) return fail(c, INFS_E_STATE, "slot %d is empty", slot);
  std::vector<int32_t>& pages = c->seq_pages[c->slot_handle[slot]];
  for (int32_t pg : pages) c->free_pages.push(pg);
  pages.clear();
  c->slot_sample[slot] = -1;
  c->slot_len[slot] = 0;
  c->slot_handle[slot] = -1;
  return INFS_OK;
}

infs_status infs_release_sample(infs_ctx* c, int32_t prompt, int64_t sample_id) {
  CHECK_CTX(c);
  if (c->probe_k == 0) return fail(c, INFS_E_STATE, "release_sample needs a context with probe_tokens > 0");
  if (prompt < 0 || prompt >= c->NP) return fail(c, INFS_E_ARG, "prompt %d out of range [0, %d)", prompt, c->NP);
  if (sample_id < 0 || sample_id >= c->G)
    return fail(c, INFS_E_ARG, "sample_id %lld out of range [0, %d)", (long long)sample_id, c->G);
  if (c->step_open || c->probe_open) return fail(c, INFS_E_STATE, "release while a step is open");
  if (c->dispatched[prompt][sample_id])
    return fail(c, INFS_E_DUP, "sample %lld of prompt %d was already dispatched or released", (long long)sample_id,
                prompt);
  c->dispatched[prompt][sample_id] = 1;
  std::vector<int32_t>& pages = c->seq_pages[prompt * c->G + (int32_t)sample_id];
  for (int32_t pg : pages) c->free_pages.push(pg);
  pages.clear();
  return INFS_OK;
}

}  // extern "C"

namespace {

// Roles, counter targets and launch of a step launch through every layer of
// plan `a` (a decode step or a probe step) with nj work-groups per KV head.
// slot_arrivals[s] and merged_arrivals[p] are the host's running values of the
// plan's slot counters and per-prompt merged counters (a.merged); both advance
// by the launch's layers.
infs_status launch_step_layers(infs_ctx* c, const KernelKey& key, StepArgs& a, int nj, uint32_t* slot_arrivals,
                               uint32_t* merged_arrivals) {
  a.peer = peer_lines(c);
  a.peer_base = (int32_t)c->peer_progress;
  // Work-groups per KV head: one merge wavefront per slot, the rest split between prefix chunks
  // and response pieces so that no producer reads many more tokens than the others.
  int32_t lens[infs::kMaxSlots], pieces[infs::kMaxSlots];
  for (int s = 0; s < a.S; ++s) lens[s] = a.slot[s].len;
  const infs::StepRoles roles =
      c->step_split ? infs::plan_step_roles(nj, a.S, a.n_prefix_items, a.prefix_split, lens, c->split, c->scmax,
                                            pieces)
                    : infs::plan_step_roles_chunks(nj, a.S, a.n_prefix_items, lens, c->split, pieces);
  if ((a.n_prefix_items > 0 && roles.n_pre < 1) || (roles.n_suffix_items > 0 && roles.n_suf < 1))
    return fail(c, INFS_E_STATE, "no step launch on this device: %d work-groups per KV head cannot take prefix "
                "chunks, response chunks and merges", nj);
  a.n_merge_wg = roles.n_merge;
  a.n_pre_wg = roles.n_pre;
  a.n_suf_wg = roles.n_suf;
  for (int s = 0, items = 0; s < a.S; ++s) {
    a.slot[s].pieces = pieces[s];
    a.slot[s].item_begin = items;
    items += pieces[s];
  }
  a.n_suffix_items = roles.n_suffix_items;
  a.resp_cut = roles.cut ? 1 : 0;
  // Merges go opposite the prefix work-groups (index j shares its CU with j + nj/2, see
  // mate_gate), else after the response work-groups.
  a.merge_j0 = (nj % 2 == 0 && a.n_pre_wg <= nj / 2 && a.n_merge_wg <= nj / 2) ? nj / 2 : a.n_pre_wg + a.n_suf_wg;
  // counter targets: each slot counts its producers once per layer, each prompt its merges
  for (int s = 0; s < a.S; ++s) {
    a.slot[s].target = (int32_t)slot_arrivals[s];
    if (a.slot[s].len > 0)
      slot_arrivals[s] += (uint32_t)c->L * (uint32_t)(a.slot[s].pieces + a.prompt[s / a.m].nchunks);
  }
  for (int p = 0; p < a.num_prompts; ++p) {
    int live = 0;
    for (int s = p * a.m; s < (p + 1) * a.m; ++s) live += a.slot[s].len > 0;
    a.merged_base[p] = (int32_t)merged_arrivals[p];
    a.merged_per_layer[p] = live * c->Hkv;
    merged_arrivals[p] += (uint32_t)c->L * (uint32_t)(live * c->Hkv);
  }
  infs_status st = timed_launch(c, key, a, c->Hkv * (a.n_pre_wg + a.n_suf_wg + a.n_merge_wg), true);
  if (st != INFS_OK) return st;
  c->peer_progress += (uint32_t)c->L;
  return INFS_OK;
}

// One layer of the open (or opening) step; with `static_ws` the split-K
// workspace and arrival counters are taken from the static scratch array.
infs_status decode_layer(infs_ctx* c, int32_t layer, const void* q_dev, const void* k_new_dev, const void* v_new_dev,
                         float* o_dev, bool static_ws) {
  CHECK_CTX(c);
  if (layer < 0 || layer >= c->L) return fail(c, INFS_E_ARG, "layer %d out of range [0, %d)", layer, c->L);
  if (!c->dry && (!q_dev || !k_new_dev || !v_new_dev || !o_dev)) return fail(c, INFS_E_ARG, "null buffer");
  if (!c->dry && (((uintptr_t)q_dev | (uintptr_t)k_new_dev | (uintptr_t)v_new_dev | (uintptr_t)o_dev) & 15))
    return fail(c, INFS_E_ARG, "q, k_new, v_new and o must be 16-byte aligned");
  if (static_ws) {
    const StaticLayout sl = static_layout(c);
    if (sl.total > infs::kStaticScratchBytes)
      return fail(c, INFS_E_CAPACITY,
                  "decode_step_static needs %zu bytes of static scratch for this context's split-K workspace "
                  "(limit %zu): use infs_decode_step, or fewer slots, KV heads or split-K chunks",
                  sl.total, infs::kStaticScratchBytes);
  }
  if (c->probe_open) return fail(c, INFS_E_STATE, "decode_step while a probe step is open");
  if (c->step_open && c->layer_done[layer])
    return fail(c, INFS_E_STATE, "layer %d already decoded in this step", layer);
  for (int p = 0; p < c->NP; ++p) {
    bool live = false;
    for (int s = p * c->m; s < (p + 1) * c->m; ++s) live |= c->slot_sample[s] >= 0;
    if (live && !c->prefilled[p][layer])
      return fail(c, INFS_E_STATE, "prompt %d has live slots but layer %d is not prefilled", p, layer);
  }
  if (!c->step_open) {
    infs_status st = open_step(c);
    if (st != INFS_OK) return st;
  }
  if (!c->dry) {
    StepArgs& a = c->plan;
    a.q = q_dev;
    a.knew = k_new_dev;
    a.vnew = v_new_dev;
    a.o = o_dev;
    a.prefix = c->prefix + c->prefix_layer_bytes * layer;
    a.pool = c->pool + c->pool_layer_bytes * layer;
    a.count_tokens = layer == 0;
    if (!static_ws) {
      set_targets(c);
      infs_status st = timed_launch(c, c->key, a, c->grid);
      if (st != INFS_OK) return st;
    } else {
      // The counters start from zero in every call (the array keeps whatever
      // the last call on this GPU left), so each merge waits for exactly this
      // launch's arrivals; the context's own counters and targets are untouched.
      const StaticLayout sl = static_layout(c);
      char* base = (char*)c->scratch;
      StepArgs sa = a;
      sa.counters = (int32_t*)(base + sl.counters);
      sa.ws_ml = (float*)(base + sl.ml);
      sa.ws_o = (float*)(base + sl.o);
      sa.ws_ml_bytes = (uint32_t)sl.ml_bytes;
      sa.ws_o_bytes = (uint32_t)sl.o_bytes;
      for (int s = 0; s < c->S; ++s)
        sa.slot[s].target = sa.slot[s].len > 0 ? ceil_div(sa.slot[s].len, c->split) + sa.prompt[s / c->m].nchunks : 0;
      HIP_TRY(c, infs::launch_zero_words((uint32_t*)sa.counters, (int64_t)infs::kCounterStride * c->S * c->Hkv,
                                         c->stream));
      infs_status st = timed_launch(c, c->key, sa, c->grid);
      if (st != INFS_OK) return st;
    }
  }
  c->layer_done[layer] = 1;
  ++c->layers_done;
  ++c->stats.launches;
  c->stats.alg_bytes += c->step_bytes;
  c->stats.alg_flops += c->step_flops;
  return INFS_OK;
}

}  // namespace

extern "C" {

infs_status infs_decode_step(infs_ctx* c, int32_t layer, const void* q_dev, const void* k_new_dev,
                             const void* v_new_dev, float* o_dev) {
  return decode_layer(c, layer, q_dev, k_new_dev, v_new_dev, o_dev, false);
}

infs_status infs_decode_step_static(infs_ctx* c, int32_t layer, const void* q_dev, const void* k_new_dev,
                                    const void* v_new_dev, float* o_dev) {
  return decode_layer(c, layer, q_dev, k_new_dev, v_new_dev, o_dev, true);
}

infs_status infs_decode_step_layers(infs_ctx* c, const void* q_dev, const void* k_new_dev, const void* v_new_dev,
                                    float* o_dev, int64_t q_layer_stride, int64_t kv_layer_stride,
                                    int64_t o_layer_stride) {
  CHECK_CTX(c);
  const int64_t q_bytes = (int64_t)c->S * c->Hq * c->D * (int64_t)c->es;
  const int64_t kv_bytes = (int64_t)c->S * c->Hkv * c->D * (int64_t)c->es;
  const int64_t o_bytes = (int64_t)c->S * c->Hq * c->D * (int64_t)sizeof(float);
  if (q_layer_stride == 0) q_layer_stride = q_bytes;
  if (kv_layer_stride == 0) kv_layer_stride = kv_bytes;
  if (o_layer_stride == 0) o_layer_stride = o_bytes;
  if (q_layer_stride < q_bytes || kv_layer_stride < kv_bytes || o_layer_stride < o_bytes)
    return fail(c, INFS_E_ARG, "layer strides must be 0 or at least one layer's rows (%lld, %lld, %lld bytes)",
                (long long)q_bytes, (long long)kv_bytes, (long long)o_bytes);
  if ((q_layer_stride | kv_layer_stride | o_layer_stride) & 15)
    return fail(c, INFS_E_ARG, "layer strides must be multiples of 16 bytes");
  if (!c->dry && (!q_dev || !k_new_dev || !v_new_dev || !o_dev)) return fail(c, INFS_E_ARG, "null buffer");
  if (!c->dry && (((uintptr_t)q_dev | (uintptr_t)k_new_dev | (uintptr_t)v_new_dev | (uintptr_t)o_dev) & 15))
    return fail(c, INFS_E_ARG, "q, k_new, v_new and o must be 16-byte aligned");
  if (c->probe_open) return fail(c, INFS_E_STATE, "decode_step_layers while a probe step is open");
  if (c->step_open && c->layers_done > 0)
    return fail(c, INFS_E_STATE, "decode_step_layers needs a step with no layer decoded yet (%d decoded)",
                c->layers_done);
  if (!c->dry && c->layers_resident == 0)
    return fail(c, INFS_E_STATE, "no step launch on this device: too few work-groups resident per KV head");
  for (int p = 0; p < c->NP; ++p) {
    bool live = false;
    for (int s = p * c->m; s < (p + 1) * c->m; ++s) live |= c->slot_sample[s] >= 0;
    for (int layer = 0; live && layer < c->L; ++layer)
      if (!c->prefilled[p][layer])
        return fail(c, INFS_E_STATE, "prompt %d has live slots but layer %d is not prefilled", p, layer);
  }
  if (!c->step_open) {
    infs_status st = open_step(c);
    if (st != INFS_OK) return st;
  }
  if (!c->dry) {
    StepArgs& a = c->plan;
    a.q = q_dev;
    a.knew = k_new_dev;
    a.vnew = v_new_dev;
    a.o = o_dev;
    a.prefix = c->prefix;
    a.pool = c->pool;
    a.count_tokens = 1;
    a.num_layers = c->L;
    a.q_layer_stride = q_layer_stride;
    a.kv_layer_stride = kv_layer_stride;
    a.o_layer_stride = o_layer_stride;
    a.prefix_layer_bytes = (int64_t)c->prefix_layer_bytes;
    a.pool_layer_bytes = (int64_t)c->pool_layer_bytes;
    a.merged = merged_counters(c);
    int32_t lens[infs::kMaxSlots];
    for (int s = 0; s < c->S; ++s) lens[s] = a.slot[s].len;
    if (c->step_split && c->key.mfma &&
        infs::longer_prefix_chunks(c->layers_resident / c->Hkv, c->S, a.n_prefix_items, lens, c->split)) {
      // MFMA prefix chunks of kStepPrefixSplit tokens (bf16 or E4M3 cache) when the per-layer
      // chunks would give some producer two items: half as many prefix work-groups, each walking
      // twice the blocks with the next block in flight, leave more work-groups to the responses
      // (the records of 128-token chunks have room for them).
      a.prefix_split = infs::kStepPrefixSplit;
      int items = 0;
      for (int p = 0; p < c->NP; ++p) {
        infs::PromptPlan& pp = a.prompt[p];
        pp.nchunks = pp.nchunks > 0 ? ceil_div(pp.plen, a.prefix_split) : 0;
        pp.item_begin = items;
        items += pp.nchunks;
      }
      a.n_prefix_items = items;
    }
    infs_status st = launch_step_layers(c, c->key, a, c->layers_resident / c->Hkv, c->slot_arrivals.data(),
                                        c->merged_arrivals.data());
    if (st != INFS_OK) return st;
  }
  std::fill(c->layer_done.begin(), c->layer_done.end(), 1);
  c->layers_done = c->L;
  ++c->stats.launches;
  c->stats.alg_bytes += c->step_bytes * c->L;
  c->stats.alg_flops += c->step_flops * c->L;
  return INFS_OK;
}

int32_t infs_step_launch_workgroups(const infs_ctx* c) { return c ? c->layers_resident : -1; }

infs_status infs_end_step(infs_ctx* c) {
  CHECK_CTX(c);
  if (!c->step_open || c->layers_done != c->L)
    return fail(c, INFS_E_STATE, "end_step needs every layer decoded once (%d of %d)", c->step_open ? c->layers_done : 0,
                c->L);
  for (int s = 0; s < c->S; ++s)
    if (c->slot_sample[s] >= 0) {
      ++c->slot_len[s];
      ++c->stats.tokens;
    }
  c->step_open = false;
  ++c->stats.steps;
  return INFS_OK;
}

infs_status infs_probe_step(infs_ctx* c, int32_t layer, int32_t prompt, int32_t first_sample, int32_t n,
                            const uint8_t* live_host, const void* q_dev, const void* k_new_dev, const void* v_new_dev,
                            float* o_dev) {
  CHECK_CTX(c);
  if (c->probe_k == 0) return fail(c, INFS_E_STATE, "probe_step needs a context with probe_tokens > 0");
  if (layer < 0 || layer >= c->L) return fail(c, INFS_E_ARG, "layer %d out of range [0, %d)", layer, c->L);
  if (prompt < 0 || prompt >= c->NP) return fail(c, INFS_E_ARG, "prompt %d out of range [0, %d)", prompt, c->NP);
  if (n < 1 || n > c->probe_batch) return fail(c, INFS_E_ARG, "n=%d out of range [1, %d]", n, c->probe_batch);
  if (first_sample < 0 || first_sample > c->G - n)
    return fail(c, INFS_E_ARG, "samples %d..%d out of range [0, %d)", first_sample, first_sample + n - 1, c->G);
  if (!c->dry && (!q_dev || !k_new_dev || !v_new_dev || !o_dev)) return fail(c, INFS_E_ARG, "null buffer");
  if (!c->dry && (((uintptr_t)q_dev | (uintptr_t)k_new_dev | (uintptr_t)v_new_dev | (uintptr_t)o_dev) & 15))
    return fail(c, INFS_E_ARG, "q, k_new, v_new and o must be 16-byte aligned");
  if (c->step_open) return fail(c, INFS_E_STATE, "probe_step while a decode step is open");
  uint8_t live[infs::kMaxSlots];
  for (int j = 0; j < n; ++j) live[j] = live_host ? (live_host[j] != 0) : 1;
  if (c->probe_open) {
    if (prompt != c->pb_prompt || first_sample != c->pb_first || n != c->pb_n || std::memcmp(live, c->pb_live, n))
      return fail(c, INFS_E_STATE, "every layer of a probe step must decode the same batch");
    if (c->probe_layer_done[layer]) return fail(c, INFS_E_STATE, "layer %d already probed in this step", layer);
  }
  bool any = false;
  for (int j = 0; j < n; ++j) any |= live[j] != 0;
  if (any && !c->prefilled[prompt][layer])
    return fail(c, INFS_E_STATE, "prompt %d has no prefix for layer %d", prompt, layer);
  if (!c->probe_open) {
    infs_status st = open_probe(c, prompt, first_sample, n, live);
    if (st != INFS_OK) return st;
  }
  if (!c->dry) {
    StepArgs& a = c->pplan;
    a.q = q_dev;
    a.knew = k_new_dev;
    a.vnew = v_new_dev;
    a.o = o_dev;
    a.prefix = c->prefix + c->prefix_layer_bytes * layer +
               (size_t)prompt * c->Hkv * infs::prefix_elems_per_head(c->key, c->pmax_pad) * c->kv_es;
    a.pool = c->pool + c->pool_layer_bytes * layer;
    a.tokens = c->tokens + (size_t)prompt * c->G;
    a.counters = c->counters + (size_t)c->S * c->Hkv * infs::kCounterStride;
    a.count_tokens = layer == 0;
    for (int j = 0; j < n; ++j) {
      if (a.slot[j].len > 0)
        c->probe_slot_arrivals[j] += (uint32_t)(ceil_div(a.slot[j].len, c->split) + a.prompt[0].nchunks);
      a.slot[j].target = (int32_t)c->probe_slot_arrivals[j];
    }
    infs_status st = timed_launch(c, c->pkey, a, c->pgrid);
    if (st != INFS_OK) return st;
  }
  c->probe_layer_done[layer] = 1;
  ++c->probe_layers_done;
  ++c->stats.launches;
  c->stats.alg_bytes += c->pstep_bytes;
  c->stats.alg_flops += c->pstep_flops;
  return INFS_OK;
}

infs_status infs_probe_step_layers(infs_ctx* c, int32_t prompt, int32_t first_sample, int32_t n,
                                   const uint8_t* live_host, const void* q_dev, const void* k_new_dev,
                                   const void* v_new_dev, float* o_dev, int64_t q_layer_stride,
                                   int64_t kv_layer_stride, int64_t o_layer_stride) {
  CHECK_CTX(c);
  if (c->probe_k == 0) return fail(c, INFS_E_STATE, "probe_step_layers needs a context with probe_tokens > 0");
  if (prompt < 0 || prompt >= c->NP) return fail(c, INFS_E_ARG, "prompt %d out of range [0, %d)", prompt, c->NP);
  if (n < 1 || n > c->probe_batch) return fail(c, INFS_E_ARG, "n=%d out of range [1, %d]", n, c->probe_batch);
  if (first_sample < 0 || first_sample > c->G - n)
    return fail(c, INFS_E_ARG, "samples %d..%d out of range [0, %d)", first_sample, first_sample + n - 1, c->G);
  const int64_t q_bytes = (int64_t)n * c->Hq * c->D * (int64_t)c->es;
  const int64_t kv_bytes = (int64_t)n * c->Hkv * c->D * (int64_t)c->es;
  const int64_t o_bytes = (int64_t)n * c->Hq * c->D * (int64_t)sizeof(float);
  if (q_layer_stride == 0) q_layer_stride = q_bytes;
  if (kv_layer_stride == 0) kv_layer_stride = kv_bytes;
  if (o_layer_stride == 0) o_layer_stride = o_bytes;
  if (q_layer_stride < q_bytes || kv_layer_stride < kv_bytes || o_layer_stride < o_bytes)
    return fail(c, INFS_E_ARG, "layer strides must be 0 or at least one layer's rows (%lld, %lld, %lld bytes)",
                (long long)q_bytes, (long long)kv_bytes, (long long)o_bytes);
  if ((q_layer_stride | kv_layer_stride | o_layer_stride) & 15)
    return fail(c, INFS_E_ARG, "layer strides must be multiples of 16 bytes");
  if (!c->dry && (!q_dev || !k_new_dev || !v_new_dev || !o_dev)) return fail(c, INFS_E_ARG, "null buffer");
  if (!c->dry && (((uintptr_t)q_dev | (uintptr_t)k_new_dev | (uintptr_t)v_new_dev | (uintptr_t)o_dev) & 15))
    return fail(c, INFS_E_ARG, "q, k_new, v_new and o must be 16-byte aligned");
  if (c->step_open) return fail(c, INFS_E_STATE, "probe_step_layers while a decode step is open");
  if (c->probe_open)
    return fail(c, INFS_E_STATE, "probe_step_layers needs a probe step with no layer probed yet (%d probed)",
                c->probe_layers_done);
  if (!c->dry && c->players_resident == 0)
    return fail(c, INFS_E_STATE, "no probe step launch on this device: too few work-groups resident per KV head");
  uint8_t live[infs::kMaxSlots];
  bool any = false;
  for (int j = 0; j < n; ++j) {
    live[j] = live_host ? (live_host[j] != 0) : 1;
    any |= live[j] != 0;
  }
  for (int layer = 0; any && layer < c->L; ++layer)
    if (!c->prefilled[prompt][layer])
      return fail(c, INFS_E_STATE, "prompt %d has no prefix for layer %d", prompt, layer);
  infs_status st = open_probe(c, prompt, first_sample, n, live);
  if (st != INFS_OK) return st;
  if (!c->dry) {
    StepArgs& a = c->pplan;
    a.q = q_dev;
    a.knew = k_new_dev;
    a.vnew = v_new_dev;
    a.o = o_dev;
    a.prefix = c->prefix + (size_t)prompt * c->Hkv * infs::prefix_elems_per_head(c->key, c->pmax_pad) * c->kv_es;
    a.pool = c->pool;
    a.tokens = c->tokens + (size_t)prompt * c->G;
    a.counters = c->counters + (size_t)c->S * c->Hkv * infs::kCounterStride;
    a.count_tokens = 1;
    a.num_layers = c->L;
    a.q_layer_stride = q_layer_stride;
    a.kv_layer_stride = kv_layer_stride;
    a.o_layer_stride = o_layer_stride;
    a.prefix_layer_bytes = (int64_t)c->prefix_layer_bytes;
    a.pool_layer_bytes = (int64_t)c->pool_layer_bytes;
    a.merged = probe_merged_counters(c);
    st = launch_step_layers(c, c->pkey, a, c->players_resident / c->Hkv, c->probe_slot_arrivals.data(),
                            &c->probe_merged_arrivals);
    if (st != INFS_OK) return st;
  }
  std::fill(c->probe_layer_done.begin(), c->probe_layer_done.end(), 1);
  c->probe_layers_done = c->L;
  ++c->stats.launches;
  c->stats.alg_bytes += c->pstep_bytes * c->L;
  c->stats.alg_flops += c->pstep_flops * c->L;
  return INFS_OK;
}

infs_status infs_end_probe_step(infs_ctx* c) {
  CHECK_CTX(c);
  if (!c->probe_open || c->probe_layers_done != c->L)
    return fail(c, INFS_E_STATE, "end_probe_step needs every layer probed once (%d of %d)",
                c->probe_open ? c->probe_layers_done : 0, c->L);
  for (int j = 0; j < c->pb_n; ++j)
    if (c->pb_live[j]) {
      ++c->probe_len[c->pb_prompt][c->pb_first + j];
      ++c->stats.tokens;
    }
  c->probe_open = false;
  return INFS_OK;
}

int32_t infs_probe_batch(const infs_ctx* c) { return c ? c->probe_batch : -1; }

infs_status infs_set_merge_wait(infs_ctx* c, int32_t max_polls) {
  CHECK_CTX(c);
  if (c->step_open || c->probe_open) return fail(c, INFS_E_STATE, "set_merge_wait while a step is open");
  c->plan.merge_polls = max_polls < 0 ? -1 : max_polls;
  return INFS_OK;
}

infs_status infs_set_exchange(infs_ctx* c, int32_t mode) {
  CHECK_CTX(c);
  if (mode < 0 || mode > 2) return fail(c, INFS_E_ARG, "exchange mode must be 0, 1 or 2");
  if (c->step_open || c->probe_open) return fail(c, INFS_E_STATE, "set_exchange while a step is open");
  if (mode > 0 && c->l2_xcds == 0)
    return fail(c, INFS_E_STATE, "no XCD-local exchange: %s",
                c->dry ? "dry-run context" : "work-groups of one KV head do not share an XCD on this device");
  c->plan.l2_xcds = mode > 0 ? c->l2_xcds : 0;
  c->plan.l2_check_shift = mode == 2 ? 1 : 0;
  return INFS_OK;
}

infs_status infs_step_split_plan(int32_t nj, int32_t S, int32_t n_prefix_items, int32_t prefix_split,
                                 const int32_t* len, int32_t split, int32_t scmax, int32_t mode, int32_t* pieces,
                                 int32_t* roles) {
  if (nj < 2 || S < 1 || S > infs::kMaxSlots || n_prefix_items < 0 || prefix_split < 1 || split < infs::kPageTokens ||
      split > infs::kMaxSplit || split % infs::kPageTokens || scmax < 1 || mode < 0 || mode > 1)
    return fail(nullptr, INFS_E_ARG, "step_split_plan: nj >= 2, S in [1, %d], split a page multiple up to %d, "
                "scmax >= 1 and mode 0 or 1", infs::kMaxSlots, infs::kMaxSplit);
  if (!len || !pieces || !roles) return fail(nullptr, INFS_E_ARG, "step_split_plan: null array");
  for (int s = 0; s < S; ++s)
    if (len[s] < 0 || len[s] > scmax * split)
      return fail(nullptr, INFS_E_ARG, "step_split_plan: len[%d] = %d outside [0, scmax * split]", s, len[s]);
  const infs::StepRoles r = mode ? infs::plan_step_roles(nj, S, n_prefix_items, prefix_split, len, split, scmax, pieces)
                                 : infs::plan_step_roles_chunks(nj, S, n_prefix_items, len, split, pieces);
  roles[0] = r.n_pre;
  roles[1] = r.n_suf;
  roles[2] = r.n_merge;
  roles[3] = r.n_suffix_items;
  roles[4] = r.cut ? 1 : 0;
  return INFS_OK;
}

infs_status infs_set_step_split(infs_ctx* c, int32_t mode) {
  CHECK_CTX(c);
  if (mode < 0 || mode > 1) return fail(c, INFS_E_ARG, "step split mode must be 0 or 1");
  if (c->step_open || c->probe_open) return fail(c, INFS_E_STATE, "set_step_split while a step is open");
  c->step_split = mode;
  return INFS_OK;
}

int32_t infs_exchange_mode(const infs_ctx* c) {
  if (!c) return -1;
  return c->plan.l2_xcds == 0 ? 0 : c->plan.l2_check_shift ? 2 : 1;
}

infs_status infs_probe_state(const infs_ctx* c, int32_t prompt, int64_t sample_id, int32_t* probe_len) {
  if (!c) return fail(nullptr, INFS_E_ARG, "null context");
  infs_ctx* cc = const_cast<infs_ctx*>(c);
  if (prompt < 0 || prompt >= c->NP) return fail(cc, INFS_E_ARG, "prompt %d out of range", prompt);
  if (sample_id < 0 || sample_id >= c->G) return fail(cc, INFS_E_ARG, "sample_id out of range");
  if (!probe_len) return fail(cc, INFS_E_ARG, "null output pointer");
  *probe_len = c->probe_k > 0 ? c->probe_len[prompt][sample_id] : 0;
  return INFS_OK;
}

infs_status infs_read_prefix(infs_ctx* c, int32_t prompt, int32_t layer, void* k_host, void* v_host) {
  CHECK_CTX(c);
  if (c->dry) return fail(c, INFS_E_STATE, "no device memory in a dry-run context");
  if (prompt < 0 || prompt >= c->NP) return fail(c, INFS_E_ARG, "prompt %d out of range [0, %d)", prompt, c->NP);
  if (layer < 0 || layer >= c->L) return fail(c, INFS_E_ARG, "layer %d out of range [0, %d)", layer, c->L);
  if (!c->prefilled[prompt][layer]) return fail(c, INFS_E_STATE, "prompt %d layer %d is not prefilled", prompt, layer);
  const int P = c->plen[prompt], D = c->D, Hkv = c->Hkv;
  if (P > 0 && (!k_host || !v_host)) return fail(c, INFS_E_ARG, "null output pointer");
  const size_t es = c->kv_es;
  const size_t head_elems = (size_t)infs::prefix_elems_per_head(c->key, c->pmax_pad);
  std::vector<uint8_t> buf(head_elems * Hkv * es);
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  HIP_TRY(c, hipMemcpy(buf.data(), c->prefix + c->prefix_layer_bytes * layer + (size_t)prompt * Hkv * head_elems * es,
                       buf.size(), hipMemcpyDeviceToHost));
  uint8_t* out[2] = {(uint8_t*)k_host, (uint8_t*)v_host};
  auto put = [&](int kind, int tok, int g, int d, const uint8_t* src) {
    std::memcpy(out[kind] + (((size_t)tok * Hkv + g) * D + d) * es, src, es);
  };
  for (int g = 0; g < Hkv; ++g) {
    const uint8_t* head = buf.data() + (size_t)g * head_elems * es;
    if (!c->key.mfma) {  // [K|V][max_prompt_len][D] rows
      for (int kind = 0; kind < 2; ++kind)
        for (int tok = 0; tok < P; ++tok)
          for (int d = 0; d < D; ++d) put(kind, tok, g, d, head + (((size_t)kind * c->pmax_pad + tok) * D + d) * es);
      continue;
    }
    // MFMA blocks of 32 tokens: K as [2 halves][D/32][64 lanes][8], V as [D/16][64 lanes][8] (see the kernels)
    const int KB = D / 32, DB = D / 16;
    for (int tok = 0; tok < P; ++tok) {
      const int b = tok / infs::kMfmaBlock, r = tok % infs::kMfmaBlock;
      const uint8_t* blk = head + (size_t)b * 2 * infs::kMfmaBlock * D * es;
      const int mb = r / 16, i = r % 16;
      for (int d = 0; d < D; ++d) {
        const int kb = d / 32, q = (d % 32) / 8, e = d % 8;
        put(0, tok, g, d, blk + ((size_t)((mb * KB + kb) * 64 + q * 16 + i) * 8 + e) * es);
      }
      // token r sits at lane quarter q, element e with r = 4q+e (e < 4) or 16+4q+(e-4)
      const int q = (r % 16) / 4, e = (r < 16 ? 0 : 4) + r % 4;
      for (int d = 0; d < D; ++d) {
        const int db = d / 16, j = d % 16;
        put(1, tok, g, d, blk + ((size_t)infs::kMfmaBlock * D + (size_t)((db * 64 + q * 16 + j) * 8 + e)) * es);
      }
      (void)DB;
    }
  }
  return INFS_OK;
}

infs_status infs_read_response(infs_ctx* c, int32_t slot, int32_t layer, void* k_host, void* v_host) {
  CHECK_CTX(c);
  if (c->dry) return fail(c, INFS_E_STATE, "no device memory in a dry-run context");
  if (slot < 0 || slot >= c->S) return fail(c, INFS_E_ARG, "slot %d out of range [0, %d)", slot, c->S);
  if (layer < 0 || layer >= c->L) return fail(c, INFS_E_ARG, "layer %d out of range [0, %d)", layer, c->L);
  if (c->slot_sample[slot] < 0) return fail(c, INFS_E_STATE, "slot %d is empty", slot);
  if (c->step_open || c->probe_open) return fail(c, INFS_E_STATE, "read while a step is open");
  const int len = c->slot_len[slot], D = c->D, Hkv = c->Hkv;
  if (len > 0 && (!k_host || !v_host)) return fail(c, INFS_E_ARG, "null output pointer");
  const size_t es = c->kv_es, rowb = (size_t)D * es, pageb = (size_t)infs::kPageTokens * rowb;
  const std::vector<int32_t>& pages = c->seq_pages[c->slot_handle[slot]];
  std::vector<uint8_t> buf((size_t)Hkv * 2 * pageb);
  uint8_t* out[2] = {(uint8_t*)k_host, (uint8_t*)v_host};
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  for (int lp = 0; lp * infs::kPageTokens < len; ++lp) {
    HIP_TRY(c, hipMemcpy(buf.data(), c->pool + c->pool_layer_bytes * layer + (size_t)pages[lp] * buf.size(), buf.size(),
                         hipMemcpyDeviceToHost));
    for (int r = 0; r < infs::kPageTokens && lp * infs::kPageTokens + r < len; ++r) {
      const int tok = lp * infs::kPageTokens + r;
      for (int g = 0; g < Hkv; ++g) {
        const uint8_t* kp = buf.data() + (size_t)g * 2 * pageb;
        const uint8_t* vp = kp + pageb;
        uint8_t* kd = out[0] + ((size_t)tok * Hkv + g) * rowb;
        uint8_t* vd = out[1] + ((size_t)tok * Hkv + g) * rowb;
        if (!c->key.bf16) {  // fp32 pages: token rows
          std::memcpy(kd, kp + (size_t)r * rowb, rowb);
          std::memcpy(vd, vp + (size_t)r * rowb, rowb);
          continue;
        }
        // bf16 / E4M3 pages in MFMA operand order: K unit (kb, lane) holds token
        // lane % 16, dims 32 kb + 8 (lane / 16) + e; V unit (db, lane) holds dim
        // 16 db + lane % 16, tokens 4 (lane / 16) + e.
        for (int d = 0; d < D; ++d) {
          const size_t ku = (size_t)((d / 32) * 64 + ((d % 32) / 8) * 16 + r) * 8 + d % 8;
          const size_t vu = (size_t)((d / 16) * 64 + (r / 4) * 16 + d % 16) * 4 + r % 4;
          std::memcpy(kd + d * es, kp + ku * es, es);
          std::memcpy(vd + d * es, vp + vu * es, es);
        }
      }
    }
  }
  return INFS_OK;
}

infs_status infs_slot_state(const infs_ctx* c, int32_t slot, int64_t* sample_id, int32_t* len) {
  if (!c) return fail(nullptr, INFS_E_ARG, "null context");
  if (slot < 0 || slot >= c->S) return fail(const_cast<infs_ctx*>(c), INFS_E_ARG, "slot %d out of range", slot);
  if (!sample_id || !len) return fail(const_cast<infs_ctx*>(c), INFS_E_ARG, "null output pointer");
  *sample_id = c->slot_sample[slot];
  *len = c->slot_len[slot];
  return INFS_OK;
}

infs_status infs_sample_tokens(infs_ctx* c, int32_t prompt, int32_t* counts_host, int32_t n) {
  CHECK_CTX(c);
  if (prompt < 0 || prompt >= c->NP) return fail(c, INFS_E_ARG, "prompt %d out of range", prompt);
  if (!counts_host || n != c->G) return fail(c, INFS_E_ARG, "counts must hold samples_per_prompt=%d entries", c->G);
  if (c->dry) return fail(c, INFS_E_STATE, "no device counters in a dry-run context");
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  HIP_TRY(c, hipMemcpy(counts_host, c->tokens + (size_t)prompt * c->G, sizeof(int32_t) * c->G, hipMemcpyDeviceToHost));
  return check_status(c);
}

infs_status infs_sync(infs_ctx* c) {
  CHECK_CTX(c);
  if (c->dry) return INFS_OK;
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  return check_status(c);
}

infs_status infs_get_stats(const infs_ctx* c, infs_stats* out) {
  if (!c || !out) return fail(nullptr, INFS_E_ARG, "null argument");
  *out = c->stats;
  return INFS_OK;
}

infs_status infs_get_kernel_info(const infs_ctx* c, infs_kernel_info* out) {
  if (!c || !out) return fail(nullptr, INFS_E_ARG, "null argument");
  *out = infs_kernel_info{c->key.bf16, c->key.head_dim, c->key.hpk, c->key.mfma, c->key.prefix_rows, c->key.kv8,
                          c->probe_batch > 0 ? c->pkey.mfma : 0, c->probe_batch > 0 ? c->pkey.prefix_rows : 0};
  return INFS_OK;
}

infs_status infs_timing_begin(infs_ctx* c) {
  CHECK_CTX(c);
  if (c->dry) return fail(c, INFS_E_STATE, "no timing in a dry-run context");
  Timing& t = c->timing;
  if (!t.clocks) {
    t.capacity = 1 << 12;
    HIP_TRY(c, hipMalloc((void**)&t.clocks, sizeof(unsigned long long) * 2 * t.capacity * kClockWords));
    HIP_TRY(c, hipEventCreate(&t.region[0]));
    HIP_TRY(c, hipEventCreate(&t.region[1]));
    int dev = 0, khz = 0;
    HIP_TRY(c, hipGetDevice(&dev));
    HIP_TRY(c, hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev));
    if (khz <= 0) return fail(c, INFS_E_DEVICE, "device wall clock rate unavailable");
    t.ticks_per_ms = (double)khz;
  }
  t.used = 0;
  t.kernel_ms = 0.0;
  t.launches = 0;
  infs_status st = arm_clocks(c);
  if (st != INFS_OK) return st;
  HIP_TRY(c, hipEventRecord(t.region[0], c->stream));
  t.on = true;
  return INFS_OK;
}

infs_status infs_timing_end(infs_ctx* c, double* kernel_ms, double* region_ms, int64_t* launches) {
  CHECK_CTX(c);
  Timing& t = c->timing;
  if (!t.on) return fail(c, INFS_E_STATE, "timing not started");
  if (!kernel_ms || !region_ms || !launches) return fail(c, INFS_E_ARG, "null output pointer");
  HIP_TRY(c, hipEventRecord(t.region[1], c->stream));
  HIP_TRY(c, hipEventSynchronize(t.region[1]));
  float ms = 0.f;
  HIP_TRY(c, hipEventElapsedTime(&ms, t.region[0], t.region[1]));
  infs_status st = harvest_clocks(c);
  if (st != INFS_OK) return st;
  t.on = false;
  c->plan.clock_start = c->plan.clock_end = nullptr;
  *kernel_ms = t.kernel_ms;
  *region_ms = ms;
  *launches = t.launches;
  return INFS_OK;
}

}  // extern "C"
