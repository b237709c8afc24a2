// Host-only checks of the attention work lists: the executor plans every iteration
// into the same DecodePlan / PrefillPlan objects, so a plan must carry nothing over
// from the previous iteration; a prefill plan covers every (entry, kv-head, query
// block) with one item over all its key tiles or with contiguous key ranges whose
// partial slots one merge job names.  Built with the host compiler against
// decode_plan.cpp (no device code); prints "ok" or the first violation.
#include <algorithm>
#include <cstdio>
#include <map>
#include <set>
#include <tuple>
#include <vector>

#include "decode_plan.hpp"

using namespace hxf;

static int fail(const char* what, int it) {
  std::printf("iteration %d: %s\n", it, what);
  return 1;
}

// the counts the executor reads must describe the items of this plan alone
static int check(const DecodePlan& P, int G, int64_t expect_rows, int it) {
  const int R1 = decode_rows_narrow(G);
  int64_t wide = 0, rows = 0;
  for (const DecodeItem& d : P.items) wide += d.n_rows > R1;
  if (P.n_wide != wide) return fail("n_wide differs from the wide items present", it);
  if (P.n_wide < 0 || P.n_wide > (int64_t)P.items.size()) return fail("n_wide out of range", it);
  for (size_t k = 0; k < P.items.size(); ++k)
    if ((k < P.items.size() - (size_t)P.n_wide) != (P.items[k].n_rows <= R1))
      return fail("one-tile items do not precede the wide ones", it);
  for (const MergeItem& m : P.merges) rows += m.kvh == 0;
  if (rows != expect_rows) return fail("merge jobs from another iteration", it);
  return 0;
}

// every query block's key tiles [0, ceil((pos0 + q0 + nq) / 32)) exactly once
static int check_prefill(const std::vector<PrefillEntry>& E, int hkv, int qpi, int it) {
  PrefillPlan P;
  plan_prefill(E, hkv, qpi, P);
  using Key = std::tuple<int, int, int>;
  std::map<Key, std::vector<std::pair<int, int>>> cover;   // (entry, kvh, q0) -> key-tile ranges
  std::map<Key, int> whole_items;
  std::set<int> parts;
  int64_t n_whole = 0;
  for (const PrefillEntry& e : E) n_whole += (int64_t)hkv * ((e.n + qpi - 1) / qpi);
  for (const PrefillItem& x : P.items) {
    if (x.t0 < 0 || x.t1 <= x.t0 || x.nq < 1 || x.nq > qpi) return fail("bad prefill item", it);
    cover[Key{x.entry, x.kvh, x.q0}].push_back({x.t0, x.t1});
    if (x.part < 0) {
      ++whole_items[Key{x.entry, x.kvh, x.q0}];
    } else if (!parts.insert(x.part).second || x.part >= P.n_parts) {
      return fail("a partial slot used twice or out of range", it);
    }
  }
  if (!P.merges.empty() && n_whole >= kPrefillResident / 2) return fail("items split with one per CU", it);
  for (const PrefillMerge& m : P.merges) {
    for (int k = 0; k < m.n_part; ++k)
      if (!parts.count(m.part0 + k)) return fail("a merge names a slot no item writes", it);
    if (whole_items.count(Key{m.entry, m.kvh, m.q0})) return fail("a merged block also has a whole item", it);
  }
  for (const PrefillEntry& e : E)
    for (int h = 0; h < hkv; ++h)
      for (int q0 = 0; q0 < e.n; q0 += qpi) {
        auto r = cover[Key{e.entry, h, q0}];
        std::sort(r.begin(), r.end());
        const int nq = std::min(qpi, e.n - q0), t1 = (e.pos0 + q0 + nq + 31) / 32;
        int at = 0;
        for (auto& [a, b] : r) {
          if (a != at) return fail("key tiles missed or attended twice", it);
          at = b;
        }
        if (at != t1) return fail("key tiles missed at the end", it);
      }
  return 0;
}

int main() {
  const int hkv = 8, G = 4;   // 32 query heads over 8 kv-heads: one tile holds 4 rows, two hold 8
  // a parent of 600 tokens and 8 forks sharing its 37 full pages, as candidates decoding together
  std::vector<int32_t> parent(64), pages[8];
  for (int j = 0; j < 64; ++j) parent[j] = j;
  std::vector<DecodeSeq> forks;
  for (int i = 0; i < 8; ++i) {
    pages[i] = parent;
    for (int j = 37; j < 64; ++j) pages[i][j] = 100 + 64 * i + j;
    forks.push_back(DecodeSeq{i, 601 + i, pages[i].data()});
  }
  std::vector<int32_t> solo(64);
  for (int j = 0; j < 64; ++j) solo[j] = 1000 + j;
  const std::vector<DecodeSeq> none, one{DecodeSeq{0, 300, solo.data()}};

  DecodePlan P;
  plan_decode(forks, hkv, G, P);
  if (check(P, G, 8, 0)) return 1;
  if (P.n_wide == 0) return fail("eight forks sharing full pages gave no two-tile item", 0);
  plan_decode(none, hkv, G, P);            // a prefill-only iteration
  if (check(P, G, 0, 1)) return 1;
  if (!P.items.empty() || P.n_parts != 0 || P.kv_tokens != 0) return fail("an empty plan kept work", 1);
  plan_decode(forks, hkv, G, P);
  if (check(P, G, 8, 2)) return 1;
  plan_decode(one, hkv, G, P);             // one sequence: no groups
  if (check(P, G, 1, 3)) return 1;
  if (P.n_wide != 0) return fail("a lone sequence kept two-tile items", 3);

  PrefillPlan Q;
  plan_prefill({PrefillEntry{0, 4080, 16}}, hkv, 32, Q);      // 8 items of 128 key tiles
  if (Q.merges.size() != 8) return fail("a 16-query chunk at 4080 was not split", 4);
  plan_prefill({}, hkv, 32, Q);
  if (!Q.items.empty() || !Q.merges.empty() || Q.n_parts || Q.tiles) return fail("an empty prefill plan kept work", 5);
  const std::vector<std::vector<PrefillEntry>> cases = {
      {{0, 0, 2048}}, {{0, 6144, 2048}}, {{0, 4352, 512}}, {{0, 4080, 16}},
      {{0, 0, 300}, {1, 2000, 40}, {2, 17, 1}}, {{0, 0, 1}}, {{3, 100, 77}, {5, 513, 130}}};
  int k = 6;
  for (const auto& c : cases)
    for (int qpi : {16, 25, 32, 64})
      if (check_prefill(c, hkv, qpi, k++)) return 1;
  std::printf("ok\n");
  return 0;
}
