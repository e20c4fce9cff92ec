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
//   FPTAS      static pre-planning only: Algorithm 2 groups the samples into m
//              bins on their predicted lengths and slot s runs bin s in
//              position order.
//   FPTAS_SJF  the two-stage plan of Algorithm 1: each slot's first sample is
//              position 0 of its bin (Algorithm 2), every later refill is SJF.
//   LPT        continuous refill with the largest predicted length, ties to
//              the lowest id (on true lengths: the post-hoc list schedule).
// FIFO, SJF and LPT rank candidates by a key fixed before decoding starts, so
// the dispatch order is a precomputed list walked by a cursor that skips
// samples already dispatched.
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
  std::vector<int32_t> order;     // FIFO / SJF / LPT dispatch order
  size_t cursor = 0;              // next position in `order`
  std::vector<uint8_t> taken;     // dispatched samples
  std::vector<int32_t> row_next;  // FIXED_ROW: next id of each slot
  std::vector<std::vector<int32_t>> bins;  // FPTAS, FPTAS_SJF: bin s in position order
  std::vector<int32_t> bin_next;  // FPTAS: next position of each slot's bin
  std::vector<uint8_t> started;   // FPTAS_SJF: slot has had its first sample
  int32_t naive_next = 0;         // NAIVE: next id to hand out
  int32_t naive_left = 0;         // NAIVE: ids left in the open group
  int32_t pending = 0;
};

namespace {

// Algorithm 2.  Sizes are the predicted lengths in units of K = eps * S / N,
// rounded up; the capacity is the rounded-up mean size per bin.  Samples go,
// largest size first (equal sizes: lower id first), into the first bin whose
// load stays within the capacity; one that fits nowhere goes to the bin with
// the least load (lowest index among equals).  S is summed in id order.
infs_status fptas(int32_t G, int32_t N, const double* pred, double eps, int32_t* group, int32_t* pos) {
  if (G < 1 || N < 1 || !pred || !group || !pos || !(eps > 0.0) || !std::isfinite(eps)) return INFS_E_ARG;
  double S = 0.0;
  for (int32_t i = 0; i < G; ++i) {
    if (!std::isfinite(pred[i]) || pred[i] < 0.0) return INFS_E_ARG;
    S += pred[i];
  }
  const double K = (eps * S) / N;
  if (!(K > 0.0)) return INFS_E_ARG;
  std::vector<int64_t> size(G);
  int64_t total = 0;
  for (int32_t i = 0; i < G; ++i) {
    const double q = std::ceil(pred[i] / K);
    if (q > 4.0e15) return INFS_E_ARG;
    size[i] = (int64_t)q;
    total += size[i];
  }
  const int64_t cap = (total + N - 1) / N;
  std::vector<int32_t> idx(G);
  std::iota(idx.begin(), idx.end(), 0);
  std::stable_sort(idx.begin(), idx.end(), [&](int32_t a, int32_t b) { return size[a] > size[b]; });
  std::vector<int64_t> load(N, 0);
  std::vector<int32_t> count(N, 0);
  for (int32_t i : idx) {
    int32_t n = 0;
    while (n < N && load[n] + size[i] > cap) ++n;
    if (n == N) n = (int32_t)(std::min_element(load.begin(), load.end()) - load.begin());
    group[i] = n;
    pos[i] = count[n]++;
    load[n] += size[i];
  }
  return INFS_OK;
}

bool needs_pred(int32_t policy) {
  return policy == INFS_SJF || policy == INFS_FPTAS || policy == INFS_FPTAS_SJF || policy == INFS_LPT;
}

int64_t take_next_in_order(infs_sched* s) {
  while (s->cursor < s->order.size() && s->taken[s->order[s->cursor]]) ++s->cursor;
  return s->cursor < s->order.size() ? s->order[s->cursor++] : -1;
}

}  // namespace

extern "C" {

infs_status infs_fptas_assign(int32_t G, int32_t N, const double* pred_len, double epsilon, int32_t* group_out,
                              int32_t* pos_out) {
  return fptas(G, N, pred_len, epsilon, group_out, pos_out);
}

infs_status infs_sched_create(int32_t G, int32_t m, int32_t policy, const double* pred_len, infs_sched** out) {
  if (!out) return INFS_E_ARG;
  *out = nullptr;
  if (G < 1 || m < 1) return INFS_E_ARG;
  if (policy < INFS_NAIVE || policy > INFS_LPT) return INFS_E_ARG;
  if (needs_pred(policy)) {
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
  s->taken.assign(G, 0);
  s->pending = G;
  if (policy == INFS_FIFO || policy == INFS_SJF || policy == INFS_FPTAS_SJF || policy == INFS_LPT) {
    s->order.resize(G);
    std::iota(s->order.begin(), s->order.end(), 0);
    if (policy != INFS_FIFO) {
      const double sign = policy == INFS_LPT ? -1.0 : 1.0;
      std::stable_sort(s->order.begin(), s->order.end(),
                       [&](int32_t a, int32_t b) { return sign * pred_len[a] < sign * pred_len[b]; });
    }
  }
  if (policy == INFS_FPTAS || policy == INFS_FPTAS_SJF) {
    std::vector<int32_t> group(G), pos(G);
    const infs_status st = fptas(G, m, pred_len, INFS_FPTAS_EPSILON, group.data(), pos.data());
    if (st != INFS_OK) {
      delete s;
      return st;
    }
    s->bins.assign(m, {});
    for (int32_t n = 0; n < m; ++n) s->bins[n].reserve(G / m + 1);
    std::vector<int32_t> by(G);
    std::iota(by.begin(), by.end(), 0);
    std::sort(by.begin(), by.end(), [&](int32_t a, int32_t b) {
      return group[a] < group[b] || (group[a] == group[b] && pos[a] < pos[b]);
    });
    for (int32_t i : by) s->bins[group[i]].push_back(i);
    s->bin_next.assign(m, 0);
    s->started.assign(m, 0);
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
    case INFS_FPTAS:
      if (s->bin_next[slot] < (int32_t)s->bins[slot].size()) id = s->bins[slot][s->bin_next[slot]++];
      break;
    case INFS_FPTAS_SJF:
      if (!s->started[slot]) {
        s->started[slot] = 1;
        if (!s->bins[slot].empty() && !s->taken[s->bins[slot][0]]) id = s->bins[slot][0];
      }
      if (id < 0) id = take_next_in_order(s);
      break;
    default:  // FIFO, SJF, LPT
      id = take_next_in_order(s);
      break;
  }
  if (id >= 0) {
    s->slot[slot] = id;
    s->taken[id] = 1;
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
