// Work split of a step launch through every layer (infs_decode_step_layers):
// how many work-groups of a KV head take prefix chunks, and where each live
// slot's response is cut into pieces for the response work-groups.
//
// A producer work-group loads one round of K/V into registers while the
// previous layer finishes, so that round is ready when the layer's queries
// arrive; whatever else it reads for the layer is loaded only after the
// queries (its registers hold the previous round until then) and lengthens
// the layer.  The per-layer launch's response chunks (a round each) fit this
// while every response work-group takes at most one.  When there are more
// chunks than response work-groups, the plan cuts each live response into
// `pieces` page ranges of near-equal length instead (piece c of a response
// of P pages holds pages [c*P/n, (c+1)*P/n)), at most one per response
// work-group, and picks the number of prefix work-groups with the cuts, so
// that the most tokens one producer reads is as small as it can be.  The
// split only decides which partial softmax holds which tokens; the merge
// combines whatever partials there are.
//
// Plain C++ with constexpr helpers (usable from host and device code) so that
// host tests can check the planner on its own.
#pragma once
#include <stdint.h>

#include "plan.h"

namespace infs {

// A wavefront holds the page numbers of its range one per lane, so a piece
// spans at most kWaves * 64 pages.
constexpr int kPiecePagesMax = kWaves * 64;
// Smallest piece the plan cuts on purpose: one page per wavefront.
constexpr int kPiecePagesMin = kWaves;

// First page of piece c of a response of `pages` pages cut into n pieces.
constexpr int piece_first_page(int c, int pages, int n) { return c * pages / n; }
// Pages per wavefront in a piece of `piece_pages` pages (wavefront w takes the
// w-th run of that many, the last runs may be short or empty).
constexpr int piece_wave_pages(int piece_pages) { return (piece_pages + kWaves - 1) / kWaves; }

struct StepRoles {
  int n_pre, n_suf, n_merge;  // work-groups per KV head taking prefix chunks, response pieces, merges
  int n_suffix_items;         // response items of the step (sum of pieces[])
  bool cut;                   // near-equal pieces chosen by the plan (else the per-layer launch's chunks)
};

namespace step_plan_detail {
inline int cdiv(int a, int b) { return (a + b - 1) / b; }
inline int pieces_at(int pages, int scmax, int t) {
  const int lo = cdiv(pages, kPiecePagesMax), hi = pages < scmax ? pages : scmax;
  int n = cdiv(pages, t);
  if (n < lo) n = lo;
  if (n > hi) n = hi;
  return n;
}
}  // namespace step_plan_detail

// Cut the live responses (len[s] > 0 tokens, s < S) into at most w pieces in
// total, each slot into at most scmax and at least ceil(pages / kPiecePagesMax),
// with the largest piece as small as it can be (pieces of at least
// kPiecePagesMin pages where a response has them).  Writes pieces[s] (0 for an
// idle slot) and returns the largest piece in pages, or -1 when the slots
// cannot fit in w pieces.
inline int cut_responses(const int32_t* len, int S, int w, int scmax, int32_t* pieces) {
  using namespace step_plan_detail;
  auto total = [&](int t) {
    int n = 0;
    for (int s = 0; s < S; ++s)
      if (len[s] > 0) n += pieces_at(cdiv(len[s], kPageTokens), scmax, t);
    return n;
  };
  if (total(kPiecePagesMax) > w) return -1;
  int lo = kPiecePagesMin, hi = kPiecePagesMax;  // smallest t with total(t) <= w
  while (lo < hi) {
    const int mid = (lo + hi) / 2;
    if (total(mid) <= w)
      hi = mid;
    else
      lo = mid + 1;
  }
  int largest = 0;
  for (int s = 0; s < S; ++s) {
    pieces[s] = 0;
    if (len[s] <= 0) continue;
    const int pages = cdiv(len[s], kPageTokens);
    pieces[s] = pieces_at(pages, scmax, lo);
    const int big = cdiv(pages, pieces[s]);
    if (big > largest) largest = big;
  }
  return largest;
}

// The split with the per-layer launch's chunks: one merge wavefront per slot,
// the producers divided between prefix and response chunks in proportion to
// their counts (at least one each when there are any), pieces[s] = the slot's
// chunks of `split` tokens.
inline StepRoles plan_step_roles_chunks(int nj, int S, int n_prefix_items, const int32_t* len, int split,
                                        int32_t* pieces) {
  using namespace step_plan_detail;
  StepRoles r{};
  r.n_merge = cdiv(S, kWaves) < nj - 1 ? cdiv(S, kWaves) : nj - 1;
  const int prod = nj - r.n_merge;
  for (int s = 0; s < S; ++s) {
    pieces[s] = len[s] > 0 ? cdiv(len[s], split) : 0;
    r.n_suffix_items += pieces[s];
  }
  const int npi = n_prefix_items, nsi = r.n_suffix_items;
  int pre = 0;
  if (npi > 0) {
    pre = (int)((int64_t)prod * npi / (npi + nsi > 1 ? npi + nsi : 1));
    pre = pre < 1 ? 1 : pre > npi ? npi : pre;
    if (nsi > 0 && pre > prod - 1) pre = prod - 1;
  }
  r.n_pre = pre > 0 ? pre : 0;
  r.n_suf = prod - r.n_pre;
  return r;
}

// Whether a step launch takes the prefix in chunks of kStepPrefixSplit tokens
// rather than the per-layer launch's (n_prefix_items of them): when the
// per-layer chunks would leave some producer two items.  Longer chunks free
// work-groups for the responses, but each prefix work-group then walks twice
// the blocks after its layer's queries arrive, which lengthens a layer that
// had room to spare.
inline bool longer_prefix_chunks(int nj, int S, int n_prefix_items, const int32_t* len, int split) {
  int32_t pieces[kMaxSlots];
  const StepRoles r = plan_step_roles_chunks(nj, S, n_prefix_items, len, split, pieces);
  return r.n_suffix_items > r.n_suf || r.n_pre < n_prefix_items;
}

// Roles of the nj work-groups per KV head and the response pieces of a step.
// n_prefix_items prefix chunks of prefix_split tokens; live slot s has len[s]
// tokens; the per-layer launch cuts responses into chunks of `split` tokens,
// at most scmax per slot.  Writes pieces[s].
//
// While the per-layer chunks leave every response work-group at most one
// chunk, they are kept: all of a producer's tokens are then in registers when
// its layer starts, and cutting finer only spreads the same bytes over more
// work-groups and partials (which measured slower).  Otherwise the number of
// prefix work-groups is chosen among the fewest that take k chunks each
// (k = 1, 2, ...) to minimise the largest per-producer token count, prefix
// tokens counted twice (every slot's merge waits for all prefix chunks, so a
// prefix work-group's second chunk delays the whole layer), and the responses
// are cut into pieces, at most one per remaining work-group; when the live
// slots outnumber those work-groups the chunks stay, dealt round robin.
inline StepRoles plan_step_roles(int nj, int S, int n_prefix_items, int prefix_split, const int32_t* len, int split,
                                 int scmax, int32_t* pieces) {
  using namespace step_plan_detail;
  StepRoles r = plan_step_roles_chunks(nj, S, n_prefix_items, len, split, pieces);
  if (r.n_suffix_items <= r.n_suf) return r;
  const int prod = nj - r.n_merge, chunks = r.n_suffix_items;
  int best = -1, best_pre = r.n_pre;
  const int kmax = n_prefix_items > 0 ? n_prefix_items : 1;
  for (int k = 1; k <= kmax; ++k) {
    const int n_pre = n_prefix_items > 0 ? cdiv(n_prefix_items, k) : 0;
    if (k > 1 && n_pre == cdiv(n_prefix_items, k - 1)) continue;
    const int w = prod - n_pre;
    if (w < 1) continue;
    const int pre_tokens = n_pre > 0 ? 2 * cdiv(n_prefix_items, n_pre) * prefix_split : 0;
    const int big = cut_responses(len, S, w, scmax, pieces);
    const int resp_tokens = big > 0 ? big * kPageTokens : cdiv(chunks, w) * split;
    const int cost = pre_tokens > resp_tokens ? pre_tokens : resp_tokens;
    if (best < 0 || cost < best) {
      best = cost;
      best_pre = n_pre;
    }
  }
  if (best < 0) {  // no split beats the chunks (a single producer)
    plan_step_roles_chunks(nj, S, n_prefix_items, len, split, pieces);
    return r;
  }
  r.n_pre = best_pre;
  r.n_suf = prod - best_pre;
  const int big = cut_responses(len, S, r.n_suf, scmax, pieces);
  r.cut = big > 0;
  if (!r.cut)
    for (int s = 0; s < S; ++s) pieces[s] = len[s] > 0 ? cdiv(len[s], split) : 0;
  r.n_suffix_items = 0;
  for (int s = 0; s < S; ++s) r.n_suffix_items += pieces[s];
  return r;
}

}  // namespace infs
