// Host refill scheduler: which pending sample a freed slot receives.
//
// Policies (one prompt, m slots, G samples):
//   NAIVE      micro groups decoded one after another (Section 3.1): a new
//              group of the next m ids opens only once every slot is empty.
//   FIXED_ROW  fixed-slot continuous sampling (Section 3.2): slot s runs
//              samples s, s+m, s+2m, ... back to back.
//   FIFO       continuous refill with the lowest pending id.
//   SJF        shortest-job-first refill (Algorithm 3): the pending sample with
//              the smallest predicted length, ties to the lowest id.  The
//              candidates are the samples not yet dispatched.
// FIFO and SJF rank candidates by a key fixed before decoding starts, so the
// dispatch order is a precomputed list and each refill is O(1).
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <new>
#include <numeric>
#include <string>
#include <vector>

#include "infs.h"

struct infs_sched {
  int32_t G = 0, m = 0, policy = 0;
  std::vector<int64_t> slot;      // sample held by each slot, -1 if empty
  std::vector<int32_t> order;     // FIFO / SJF dispatch order
  size_t cursor = 0;              // next position in `order`
  std::vector<int32_t> row_next;  // FIXED_ROW: next id of each slot
  int32_t naive_next = 0;         // NAIVE: next id to hand out
  int32_t naive_left = 0;         // NAIVE: ids left in the open group
  int32_t pending = 0;
};

extern "C" {

infs_status infs_sched_create(int32_t G, int32_t m, int32_t policy, const double* pred_len, infs_sched** out) {
  if (!out) return INFS_E_ARG;
  *out = nullptr;
  if (G < 1 || m < 1) return INFS_E_ARG;
  if (policy < INFS_NAIVE || policy > INFS_SJF) return INFS_E_ARG;
  if (policy == INFS_SJF) {
    if (!pred_len) return INFS_E_ARG;
    for (int32_t i = 0; i < G; ++i)
      if (!std::isfinite(pred_len[i])) return INFS_E_ARG;
  }
  infs_sched* s = new (std::nothrow) infs_sched;
  if (!s) return INFS_E_NOMEM;
  s->G = G;
  s->m = m;
  s->policy = policy;
  s->slot.assign(m, -1);
  s->pending = G;
  if (policy == INFS_FIFO || policy == INFS_SJF) {
    s->order.resize(G);
    std::iota(s->order.begin(), s->order.end(), 0);
    if (policy == INFS_SJF) {
      std::vector<double> key(pred_len, pred_len + G);
      std::stable_sort(s->order.begin(), s->order.end(),
                       [&](int32_t a, int32_t b) { return key[a] < key[b] || (key[a] == key[b] && a < b); });
    }
  }
  if (policy == INFS_FIXED_ROW) {
    s->row_next.resize(m);
    std::iota(s->row_next.begin(), s->row_next.end(), 0);
  }
  *out = s;
  return INFS_OK;
}

infs_status infs_sched_next(infs_sched* s, int32_t slot, int64_t* sample_out) {
  if (!s || !sample_out) return INFS_E_ARG;
  if (slot < 0 || slot >= s->m) return INFS_E_ARG;
  if (s->slot[slot] >= 0) return INFS_E_STATE;
  int64_t id = -1;
  switch (s->policy) {
    case INFS_NAIVE:
      if (s->naive_left == 0) {
        const bool all_empty = std::all_of(s->slot.begin(), s->slot.end(), [](int64_t x) { return x < 0; });
        if (all_empty && s->naive_next < s->G) s->naive_left = std::min(s->m, s->G - s->naive_next);
      }
      if (s->naive_left > 0) {
        id = s->naive_next++;
        --s->naive_left;
      }
      break;
    case INFS_FIXED_ROW:
      if (s->row_next[slot] < s->G) {
        id = s->row_next[slot];
        s->row_next[slot] += s->m;
      }
      break;
    default:  // FIFO, SJF
      if (s->cursor < s->order.size()) id = s->order[s->cursor++];
      break;
  }
  if (id >= 0) {
    s->slot[slot] = id;
    --s->pending;
  }
  *sample_out = id;
  return INFS_OK;
}

infs_status infs_sched_done(infs_sched* s, int32_t slot) {
  if (!s) return INFS_E_ARG;
  if (slot < 0 || slot >= s->m) return INFS_E_ARG;
  if (s->slot[slot] < 0) return INFS_E_STATE;
  s->slot[slot] = -1;
  return INFS_OK;
}

int32_t infs_sched_pending(const infs_sched* s) { return s ? s->pending : -1; }

void infs_sched_destroy(infs_sched* s) { delete s; }

}  // extern "C"
