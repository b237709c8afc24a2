// Host-only check of the attention work lists' reuse contract: the executor plans
// every iteration into the same DecodePlan / PrefillPlan objects, so a plan must
// carry nothing over from the previous iteration.  Built with the host compiler
// against decode_plan.cpp (no device code); prints "ok" or the first violation.
#include <cstdio>
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
  plan_prefill({PrefillEntry{0, 4096, 2048}}, hkv, 32, Q);
  if (Q.merges.empty()) return fail("a 6144-token chunk was not split", 4);
  plan_prefill({}, hkv, 32, Q);
  if (!Q.items.empty() || !Q.merges.empty() || Q.n_parts || Q.tiles) return fail("an empty prefill plan kept work", 5);
  std::printf("ok\n");
  return 0;
}
