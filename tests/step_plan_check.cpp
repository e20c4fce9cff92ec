// Host check of the step launch's work split (csrc/step_plan.h), built with g++
// by tests/test_step_plan.py.  For random slot lengths and launch shapes it
// checks the roles add up, that every live response's pieces are whole page
// ranges covering it exactly (also per wavefront, as the kernel cuts them),
// the bounds on pieces per slot and pages per piece, and that the cut is the
// smallest largest piece a brute force over all piece counts finds; and that
// the step launch takes longer prefix chunks exactly when the per-layer chunks
// would give some producer two items.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "step_plan.h"

using namespace infs;

static int fails = 0;
#define CHECK(cond, ...)                              \
  do {                                                \
    if (!(cond)) {                                    \
      if (++fails < 20) {                             \
        std::printf("FAIL %s: ", #cond);              \
        std::printf(__VA_ARGS__);                     \
        std::printf("\n");                            \
      }                                               \
    }                                                 \
  } while (0)

static int cdiv(int a, int b) { return (a + b - 1) / b; }

// Pieces of one response as the kernel cuts them: token ranges of every
// wavefront must be page aligned, at most 64 pages, and tile [0, len).
static void check_cover(int len, int n, int case_id) {
  const int pages = cdiv(len, kPageTokens);
  int next = 0;
  for (int c = 0; c < n; ++c) {
    const int pg0 = piece_first_page(c, pages, n), pg1 = piece_first_page(c + 1, pages, n);
    CHECK(pg1 > pg0, "case %d: empty piece %d of %d (pages %d)", case_id, c, n, pages);
    CHECK(pg1 - pg0 <= kPiecePagesMax, "case %d: piece of %d pages", case_id, pg1 - pg0);
    const int ppw = piece_wave_pages(pg1 - pg0);
    CHECK(ppw <= 64, "case %d: %d pages per wavefront", case_id, ppw);
    const int t1 = pg1 * kPageTokens < len ? pg1 * kPageTokens : len;
    for (int w = 0; w < kWaves; ++w) {
      int wt0 = (pg0 + w * ppw) * kPageTokens;
      if (wt0 > t1) wt0 = t1;
      int wt1 = wt0 + ppw * kPageTokens;
      if (wt1 > t1) wt1 = t1;
      if (wt1 == wt0) continue;
      CHECK(wt0 % kPageTokens == 0, "case %d: unaligned wavefront start %d", case_id, wt0);
      CHECK(wt0 == next, "case %d: gap or overlap at token %d (expected %d)", case_id, wt0, next);
      next = wt1;
    }
  }
  CHECK(next == len, "case %d: pieces cover %d of %d tokens", case_id, next, len);
}

// Smallest largest piece (pages) over all piece counts n_s in [lo_s, hi_s]
// with sum <= w, by exhaustive search (few slots only).
static int brute_cut(const std::vector<int>& pages, int w, int scmax) {
  const int k = (int)pages.size();
  std::vector<int> lo(k), hi(k), n(k);
  for (int i = 0; i < k; ++i) {
    lo[i] = cdiv(pages[i], kPiecePagesMax);
    hi[i] = pages[i] < scmax ? pages[i] : scmax;
    n[i] = lo[i];
  }
  int best = -1;
  while (true) {
    int sum = 0, big = 0;
    for (int i = 0; i < k; ++i) {
      sum += n[i];
      big = std::max(big, cdiv(pages[i], n[i]));
    }
    if (sum <= w && (best < 0 || big < best)) best = big;
    int i = 0;
    while (i < k && n[i] == hi[i]) n[i] = lo[i], ++i;
    if (i == k) break;
    ++n[i];
  }
  return best;
}

int main(int argc, char** argv) {
  const int cases = argc > 1 ? std::atoi(argv[1]) : 20000;
  std::mt19937 rng(12345);
  auto uni = [&](int a, int b) { return std::uniform_int_distribution<int>(a, b)(rng); };
  int cut_cases = 0, fixed_cases = 0;
  for (int cs = 0; cs < cases; ++cs) {
    const int nj = (int[]){8, 16, 32, 64, 128}[uni(0, 4)];
    const int S = uni(1, kMaxSlots);
    const int split = (int[]){128, 256, 512, 4096}[uni(0, 3)];
    const int max_len = uni(1, 3) == 1 ? uni(1, 300) : uni(1, 8192);
    const int scmax = cdiv(max_len, split);
    const int prefix_split = 128;
    std::vector<int32_t> len(S, 0), pieces(S, -1);
    int live = 0;
    const int idle_pct = uni(0, 60);
    for (int s = 0; s < S; ++s)
      if (uni(0, 99) >= idle_pct) {
        len[s] = uni(1, max_len);
        ++live;
      }
    const int npi = live > 0 ? uni(0, 64) : 0;
    // Longer prefix chunks exactly when dealing the per-layer chunks round robin over the
    // chunk plan's work-groups would give some producer a second item (with two producers
    // or more: with one, the runtime refuses the step launch).
    if (nj - std::min(cdiv(S, kWaves), nj - 1) >= 2) {
      std::vector<int32_t> chunk_pieces(S, -1);
      const StepRoles c = plan_step_roles_chunks(nj, S, npi, len.data(), split, chunk_pieces.data());
      int most = 0;
      for (int i = 0; i < npi; ++i) most = std::max(most, i / std::max(c.n_pre, 1) + 1);
      for (int i = 0; i < c.n_suffix_items; ++i) most = std::max(most, i / std::max(c.n_suf, 1) + 1);
      CHECK(longer_prefix_chunks(nj, S, npi, len.data(), split) == (most > 1),
            "case %d: longer prefix chunks %d with at most %d items per producer", cs,
            (int)longer_prefix_chunks(nj, S, npi, len.data(), split), most);
      if (npi > 0) CHECK(c.n_pre >= 1, "case %d: prefix chunks but no prefix work-group", cs);
      if (c.n_suffix_items > 0) CHECK(c.n_suf >= 1, "case %d: response chunks but no response work-group", cs);
    }
    const StepRoles r = plan_step_roles(nj, S, npi, prefix_split, len.data(), split, scmax, pieces.data());
    const int merge = std::min(cdiv(S, kWaves), nj - 1);
    CHECK(r.n_merge == merge, "case %d: %d merge work-groups, expected %d", cs, r.n_merge, merge);
    CHECK(r.n_pre >= 0 && r.n_suf >= 0 && r.n_pre + r.n_suf + r.n_merge == nj, "case %d: roles %d+%d+%d != %d", cs,
          r.n_pre, r.n_suf, r.n_merge, nj);
    const int prod = nj - merge;
    if (live > 0 && npi > 0 && prod >= 2) CHECK(r.n_pre >= 1 && r.n_suf >= 1, "case %d: a kind of work has no producer", cs);
    if (live > 0 && npi == 0) CHECK(r.n_pre == 0 && r.n_suf == prod, "case %d: no prefix but %d prefix work-groups", cs, r.n_pre);
    if (r.n_pre > 0) CHECK(r.n_pre <= npi, "case %d: %d prefix work-groups for %d chunks", cs, r.n_pre, npi);
    int total = 0;
    for (int s = 0; s < S; ++s) {
      if (len[s] == 0) {
        CHECK(pieces[s] == 0, "case %d: idle slot with %d pieces", cs, pieces[s]);
        continue;
      }
      const int pages = cdiv(len[s], kPageTokens);
      CHECK(pieces[s] >= 1 && pieces[s] <= pages && pieces[s] <= scmax, "case %d: %d pieces (pages %d, limit %d)", cs,
            pieces[s], pages, scmax);
      if (!r.cut) CHECK(pieces[s] == cdiv(len[s], split), "case %d: uncut slot with %d pieces", cs, pieces[s]);
      total += pieces[s];
      if (pieces[s] >= 1 && pieces[s] <= pages) check_cover(len[s], pieces[s], cs);
    }
    CHECK(total == r.n_suffix_items, "case %d: %d pieces, plan says %d", cs, total, r.n_suffix_items);
    if (r.cut) {
      ++cut_cases;
      CHECK(total <= r.n_suf, "case %d: %d pieces for %d response work-groups", cs, total, r.n_suf);
    } else if (live > 0 && r.n_suf > 0) {
      ++fixed_cases;
    }
    // The cut is optimal: no piece counts within the bounds and the work-group count have a
    // smaller largest piece, except that pieces are not cut below kPiecePagesMin pages.
    if (r.cut && live <= 4) {
      std::vector<int> pg;
      int big = 0;
      for (int s = 0; s < S; ++s)
        if (len[s] > 0) {
          pg.push_back(cdiv(len[s], kPageTokens));
          big = std::max(big, cdiv(pg.back(), pieces[s]));
        }
      bool small = true;
      long combos = 1;
      for (int p : pg) combos *= std::min(p, scmax);
      small = combos <= 200000;
      if (small) {
        const int opt = brute_cut(pg, r.n_suf, scmax);
        CHECK(big >= opt, "case %d: largest piece %d below the optimum %d", cs, big, opt);
        CHECK(big <= std::max(opt, kPiecePagesMin), "case %d: largest piece %d, optimum %d", cs, big, opt);
      }
    }
  }
  std::printf("cases %d: cut %d, per-layer chunks %d, failures %d\n", cases, cut_cases, fixed_cases, fails);
  return fails ? 1 : 0;
}
