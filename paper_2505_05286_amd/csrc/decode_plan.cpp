// Attention work lists: decode (prefix groups, partitions, partial slots) and
// chunked prefill (query blocks, key-range splits).
#include "decode_plan.hpp"

#include <algorithm>

namespace hxf {

namespace {

struct Stream {
  int64_t len;      // tokens
  int first;        // first token
  int rows[kDecodeRows];
  int n_rows;       // sequences served (indices into seqs)
  int slot_off;     // offset of this stream's pieces inside each row's slot block
};

}  // namespace

void plan_decode(const std::vector<DecodeSeq>& seqs, int hkv, int G, DecodePlan& out) {
  // every field is overwritten: the caller reuses one plan across iterations, and a stale
  // count of wide items with no items behind it would send the two-tile kernel past them
  out.items.clear();
  out.merges.clear();
  out.n_parts = 0;
  out.kv_tokens = 0;
  out.n_wide = 0;
  const int n = (int)seqs.size();
  if (n == 0) return;
  const int R1 = decode_rows_narrow(G), R = decode_rows_wide(G);

  // prefix groups: equal first page, shared length = the shortest common run of full pages
  std::vector<int> order, shared(n, 0);
  for (int i = 0; i < n; ++i)
    if (seqs[i].pages) order.push_back(i);
  std::stable_sort(order.begin(), order.end(),
                   [&](int a, int b) { return seqs[a].pages[0] < seqs[b].pages[0]; });
  std::vector<std::vector<int>> groups;
  const int n_known = (int)order.size();
  for (int i = 0; i < n_known;) {
    int j = i + 1;
    while (j < n_known && seqs[order[j]].pages[0] == seqs[order[i]].pages[0]) ++j;
    if (j - i >= 2) {
      const DecodeSeq& lead = seqs[order[i]];
      int s = lead.ctx / kPage;
      for (int k = i + 1; k < j; ++k) {
        const DecodeSeq& m = seqs[order[k]];
        int c = 0;
        const int lim = std::min(s, m.ctx / kPage);
        while (c < lim && m.pages[c] == lead.pages[c]) ++c;
        s = c;
      }
      if (s > 0) {
        std::vector<int> g(order.begin() + i, order.begin() + j);
        std::sort(g.begin(), g.end());
        for (int k : g) shared[k] = s * kPage;
        groups.push_back(std::move(g));
      }
    }
    i = j;
  }

  // streams: shared prefixes (R sequences at a time), then every sequence's own tokens
  std::vector<Stream> streams;
  for (const auto& g : groups) {
    for (size_t c = 0; c < g.size(); c += R) {
      Stream st{shared[g[0]], 0, {0}, 0, 0};
      for (size_t k = c; k < g.size() && k < c + R; ++k) st.rows[st.n_rows++] = g[k];
      streams.push_back(st);
    }
  }
  for (int i = 0; i < n; ++i)
    if (seqs[i].ctx > shared[i]) {
      Stream st{seqs[i].ctx - shared[i], shared[i], {i}, 1, 0};
      streams.push_back(st);
    }
  int64_t total = 0;
  for (const auto& st : streams) total += st.len;
  const int64_t target = decode_target_tokens(total, (int64_t)streams.size(), hkv);

  // pieces per stream; slot blocks per sequence (shared pieces first, then own pieces)
  std::vector<int> plen(streams.size()), npieces(streams.size()), nslots(n, 0);
  for (size_t k = 0; k < streams.size(); ++k) {
    plen[k] = decode_part_len((int)streams[k].len, target);
    npieces[k] = (int)((streams[k].len + plen[k] - 1) / plen[k]);
    streams[k].slot_off = nslots[streams[k].rows[0]];
    for (int r = 0; r < streams[k].n_rows; ++r) nslots[streams[k].rows[r]] += npieces[k];
  }
  std::vector<int64_t> base(n);   // slot of (sequence i, kv-head 0); kv-head h adds h * nslots[i]
  int64_t slot = 0;
  for (int i = 0; i < n; ++i) {
    base[i] = slot;
    slot += (int64_t)hkv * nslots[i];
    for (int h = 0; h < hkv; ++h)
      out.merges.push_back(MergeItem{seqs[i].entry, h, (int32_t)(base[i] + (int64_t)h * nslots[i]), nslots[i]});
  }
  out.n_parts = slot;
  std::vector<DecodeItem> wide;
  for (size_t k = 0; k < streams.size(); ++k) {
    const Stream& st = streams[k];
    for (int h = 0; h < hkv; ++h)
      for (int p = 0; p < npieces[k]; ++p) {
        DecodeItem it{};
        it.kvh = h;
        it.t0 = st.first + p * plen[k];
        it.t1 = (int)std::min<int64_t>(st.first + st.len, (int64_t)it.t0 + plen[k]);
        it.n_rows = st.n_rows;
        for (int r = 0; r < kDecodeRows; ++r) {
          const int i = st.rows[std::min(r, st.n_rows - 1)];
          it.entry[r] = seqs[i].entry;
          it.part[r] = (int32_t)(base[i] + (int64_t)h * nslots[i] + st.slot_off + p);
        }
        out.kv_tokens += it.t1 - it.t0;
        (st.n_rows > R1 ? wide : out.items).push_back(it);
      }
  }
  // one-tile items first, then the wide ones, each longest first
  order_decode_items(out.items.data(), out.items.size());
  order_decode_items(wide.data(), wide.size());
  out.n_wide = (int64_t)wide.size();
  out.items.insert(out.items.end(), wide.begin(), wide.end());
}

void plan_prefill(const std::vector<PrefillEntry>& entries, int hkv, int qpi, PrefillPlan& out) {
  out.items.clear();
  out.merges.clear();
  out.n_parts = 0;
  out.tiles = 0;
  std::vector<PrefillItem> whole;
  for (const PrefillEntry& e : entries)
    for (int h = 0; h < hkv; ++h)
      for (int q0 = 0; q0 < e.n; q0 += qpi) {
        const int nq = std::min(qpi, e.n - q0);
        const int t1 = (e.pos0 + q0 + nq + 31) / 32;
        whole.push_back(PrefillItem{e.entry, h, q0, nq, 0, t1, -1, 0});
        out.tiles += t1;
      }
  // With fewer items than CUs some CUs would idle: items longer than the per-slot share
  // of one pass over the resident workgroups are cut into key ranges.  With more, they
  // are not: a CU's two resident workgroups share its matrix cores, so the one left
  // running a long item runs it faster, and cutting only adds partial writes and a merge.
  const int64_t share = std::max<int64_t>((out.tiles + kPrefillResident - 1) / kPrefillResident, kPrefillMinTiles);
  const bool split = (int64_t)whole.size() < kPrefillResident / 2;
  for (const PrefillItem& it : whole) {
    if (!split || it.t1 <= share) {
      out.items.push_back(it);
      continue;
    }
    const int np = (int)((it.t1 + share - 1) / share);
    const int len = (it.t1 + np - 1) / np;
    const int part0 = (int)out.n_parts;
    int k = 0;
    for (int t0 = 0; t0 < it.t1; t0 += len, ++k) {
      PrefillItem p = it;
      p.t0 = t0;
      p.t1 = std::min(it.t1, t0 + len);
      p.part = part0 + k;
      out.items.push_back(p);
    }
    out.n_parts += k;
    out.merges.push_back(PrefillMerge{it.entry, it.kvh, it.q0, it.nq, part0, k, 0, 0});
  }
  // Most tiles first; then, among the first resident workgroups, the second half in
  // reverse: workgroups w and w + kPrefillResident / 2 are placed on one CU, which so
  // gets one long and one short item (the causal items of a first chunk hold 1 to 64
  // tiles) instead of two long or two short ones.
  order_prefill_items(out.items.data(), out.items.size());
  const size_t half = kPrefillResident / 2, window = std::min<size_t>(out.items.size(), kPrefillResident);
  if (window > half) std::reverse(out.items.begin() + half, out.items.begin() + window);
}

}  // namespace hxf
