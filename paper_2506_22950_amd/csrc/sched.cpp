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
//              the lowest id (on true lengths: a post-hoc list schedule, an
//              upper bound on the post-hoc optimum computed by
//              infs_sched_optimum).
// FIFO, SJF and LPT rank candidates by a key fixed before decoding starts, so
// the dispatch order is a precomputed list walked by a cursor that skips
// samples already dispatched.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <numeric>
#include <string>
#include <unordered_set>
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

// Micro-group assignment of Algorithm 2, as first-fit decreasing bin packing:
// the predicted lengths, in units of K = eps * S / N (S summed in id order),
// rounded up, are the item sizes; every one of the N bins holds the rounded-up
// mean size; items go largest first (equal sizes: lower id first) into the
// lowest-numbered bin with room for them.  An item no bin has room for (the
// algorithm leaves that case open) goes to the least-loaded bin, lowest index
// among equals.  The free room of the bins sits in a max-tree, so both the
// first bin with room and the least-loaded bin are found in O(log N).
class RoomTree {
 public:
  RoomTree(int n, int64_t room) : leaves_(1) {
    while (leaves_ < n) leaves_ *= 2;
    node_.assign(2 * leaves_, INT64_MIN);
    for (int i = 0; i < n; ++i) node_[leaves_ + i] = room;
    for (int i = leaves_ - 1; i >= 1; --i) node_[i] = std::max(node_[2 * i], node_[2 * i + 1]);
  }
  // Lowest bin whose room is at least `need`, or -1.
  int first_with(int64_t need) const {
    if (node_[1] < need) return -1;
    int i = 1;
    while (i < leaves_) i = node_[2 * i] >= need ? 2 * i : 2 * i + 1;
    return i - leaves_;
  }
  int most_room() const { return first_with(node_[1]); }
  void take(int bin, int64_t amount) {
    int i = leaves_ + bin;
    node_[i] -= amount;
    for (i /= 2; i >= 1; i /= 2) node_[i] = std::max(node_[2 * i], node_[2 * i + 1]);
  }

 private:
  int leaves_;
  std::vector<int64_t> node_;
};

infs_status fptas(int32_t G, int32_t N, const double* pred, double eps, int32_t* group, int32_t* pos) {
  if (G < 1 || N < 1 || !pred || !group || !pos || !(eps > 0.0) || !std::isfinite(eps)) return INFS_E_ARG;
  double S = 0.0;
  for (int32_t i = 0; i < G; ++i) {
    if (!std::isfinite(pred[i]) || pred[i] < 0.0) return INFS_E_ARG;
    S += pred[i];
  }
  const double K = (eps * S) / N;
  if (!(K > 0.0)) return INFS_E_ARG;
  std::vector<std::pair<int64_t, int32_t>> items(G);  // (-size, id): ascending = largest first, lower id first
  int64_t total = 0;
  for (int32_t i = 0; i < G; ++i) {
    const double q = std::ceil(pred[i] / K);
    if (q > 4.0e15) return INFS_E_ARG;
    items[i] = {-(int64_t)q, i};
    total += (int64_t)q;
  }
  std::sort(items.begin(), items.end());
  RoomTree room(N, (total + N - 1) / N);
  std::vector<int32_t> filled(N, 0);
  for (const auto& it : items) {
    const int64_t size = -it.first;
    int bin = room.first_with(size);
    if (bin < 0) bin = room.most_room();
    room.take(bin, size);
    group[it.second] = bin;
    pos[it.second] = filled[bin]++;
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

// ---------------------------------------------------------------------------
// Infinite*: the fewest running steps of a post-hoc schedule (Table 1 caption,
// Section 5.4).  A slot runs its samples back to back, so the steps of an
// assignment of samples to slots are its largest slot sum, and the optimum is
// the makespan problem P||Cmax.  Branch and bound on that makespan:
//   * lower bound: max(ceil(sum / m), the longest sample, and -- with more
//     samples than slots -- the m-th plus the (m+1)-th longest, two of the m+1
//     longest sharing a slot);
//   * first incumbent: longest-processing-time list scheduling;
//   * then repeated depth-first searches for a schedule shorter than the
//     incumbent, samples longest first, each placed on a slot in order of
//     increasing load (equal loads tried once), with three cuts: the
//     remaining samples must fit in the free room below the target; room that
//     no remaining sample fits into is lost; a sample that fills a slot to the
//     target exactly goes there only.  A (next sample, multiset of loads)
//     state that cannot reach a target cannot reach a lower one either, so
//     failed states are kept across searches.
// The search ends when the incumbent meets the lower bound or a search fails
// (the incumbent is optimal), or after max_nodes search nodes (unsolved).
// ---------------------------------------------------------------------------
struct OptSearch {
  int m = 0, n = 0;
  std::vector<int64_t> size;   // samples, longest first
  std::vector<int64_t> rest;   // rest[i] = sum of size[i..n)
  std::vector<int64_t> load;
  std::vector<int32_t> where;  // slot of size[i] in the current branch
  std::vector<int32_t> found;  // slot of size[i] in the last schedule found
  int64_t target = 0, nodes = 0, max_nodes = 0;
  bool out_of_nodes = false;
  std::unordered_set<std::string> failed;
  static constexpr size_t kMaxFailed = size_t(1) << 22;

  std::string state_key(int i) const {
    std::vector<int64_t> l(load);
    std::sort(l.begin(), l.end());
    std::string k(sizeof(int32_t) + l.size() * sizeof(int64_t), '\0');
    std::memcpy(&k[0], &i, sizeof(int32_t));
    std::memcpy(&k[sizeof(int32_t)], l.data(), l.size() * sizeof(int64_t));
    return k;
  }

  bool search(int i) {
    if (i == n) {
      found = where;
      return true;
    }
    if (++nodes > max_nodes) {
      out_of_nodes = true;
      return false;
    }
    int64_t room = 0, usable = 0;
    const int64_t smallest = size[n - 1];
    for (int s = 0; s < m; ++s) {
      const int64_t gap = target - load[s];
      room += gap;
      if (gap >= smallest) usable += gap;
    }
    if (room < rest[i] || usable < rest[i]) return false;
    const std::string key = state_key(i);
    if (failed.count(key)) return false;
    const int64_t x = size[i];
    std::vector<int> order;
    order.reserve(m);
    for (int s = 0; s < m; ++s)
      if (load[s] + x == target) {
        order.push_back(s);
        break;
      }
    if (order.empty()) {
      std::vector<int> idx(m);
      std::iota(idx.begin(), idx.end(), 0);
      std::stable_sort(idx.begin(), idx.end(), [&](int a, int b) { return load[a] < load[b]; });
      for (int k = 0; k < m; ++k) {
        const int s = idx[k];
        if (load[s] + x > target) break;
        if (k > 0 && load[idx[k - 1]] == load[s]) continue;
        order.push_back(s);
      }
    }
    for (int s : order) {
      load[s] += x;
      where[i] = s;
      const bool ok = search(i + 1);
      load[s] -= x;
      if (ok) return true;
      if (out_of_nodes) return false;
    }
    if (failed.size() < kMaxFailed) failed.insert(key);
    return false;
  }
};

}  // namespace

extern "C" {

infs_status infs_sched_optimum(int32_t G, int32_t m, const int32_t* lengths, int64_t max_nodes, int64_t* best_out,
                               int64_t* lower_out, int32_t* slot_out) {
  if (G < 1 || m < 1 || !lengths || !best_out || !lower_out || max_nodes < 0) return INFS_E_ARG;
  for (int32_t i = 0; i < G; ++i)
    if (lengths[i] < 1) return INFS_E_ARG;
  OptSearch o;
  o.m = m;
  o.n = G;
  std::vector<int32_t> id(G);
  std::iota(id.begin(), id.end(), 0);
  std::stable_sort(id.begin(), id.end(), [&](int32_t a, int32_t b) { return lengths[a] > lengths[b]; });
  o.size.resize(G);
  for (int32_t k = 0; k < G; ++k) o.size[k] = lengths[id[k]];
  o.rest.assign(G + 1, 0);
  for (int32_t k = G - 1; k >= 0; --k) o.rest[k] = o.rest[k + 1] + o.size[k];
  int64_t lower = std::max((o.rest[0] + m - 1) / m, o.size[0]);
  if (G > m) lower = std::max(lower, o.size[m - 1] + o.size[m]);
  // Incumbent: longest-processing-time list scheduling (least loaded slot, lowest index).
  std::vector<int64_t> lpt(m, 0);
  std::vector<int32_t> best(G);
  for (int32_t k = 0; k < G; ++k) {
    const int s = (int)(std::min_element(lpt.begin(), lpt.end()) - lpt.begin());
    lpt[s] += o.size[k];
    best[k] = s;
  }
  int64_t ub = *std::max_element(lpt.begin(), lpt.end());
  o.load.assign(m, 0);
  o.where.assign(G, 0);
  o.max_nodes = max_nodes;
  bool solved = ub == lower;
  while (!solved) {
    o.target = ub - 1;
    std::fill(o.load.begin(), o.load.end(), 0);
    if (o.search(0)) {
      std::vector<int64_t> l(m, 0);
      for (int32_t k = 0; k < G; ++k) l[o.found[k]] += o.size[k];
      ub = *std::max_element(l.begin(), l.end());
      best = o.found;
      solved = ub == lower;
    } else if (o.out_of_nodes) {
      break;
    } else {
      lower = ub;  // no schedule below the incumbent
      solved = true;
    }
  }
  *best_out = ub;
  *lower_out = lower;
  if (slot_out)
    for (int32_t k = 0; k < G; ++k) slot_out[id[k]] = best[k];
  return INFS_OK;
}

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
