// Host-side work list of the paged decode-attention kernel.
#pragma once

#include <stdint.h>

#include <vector>

#include "kernels/kernels.hpp"

namespace hxf {

// One decoding sequence: batch entry, context length (the query attends to tokens
// [0, ctx)) and its block table on the host (at least ceil(ctx / 16) pages; null:
// the sequence is never grouped with others).
struct DecodeSeq {
  int entry;
  int ctx;
  const int32_t* pages;
};

struct DecodePlan {
  std::vector<DecodeItem> items;    // one-tile items, then the n_wide two-tile items (each longest first)
  int64_t n_wide = 0;
  std::vector<MergeItem> merges;    // one per (sequence, kv-head), in sequence order
  int64_t n_parts = 0;              // partial slots used
  int64_t kv_tokens = 0;            // (token, kv-head) pairs read: the sum of the item lengths
};

// Sequences whose block tables start with the same physical pages (forks of one
// retained parent share its full pages) form a group.  The shared full pages are
// attended by items that serve up to decode_rows_wide(G) of the group's sequences at
// once (two-tile items when more than decode_rows_narrow(G)), so each shared page is
// read once per such item instead of once per sequence; every sequence's own pages
// get items of their own.  All streams are
// cut into equal page-aligned partitions sized to fill the resident wavefronts
// (decode_target_tokens), and the partials of a (sequence, kv-head) occupy
// consecutive slots, merged by log-sum-exp.
void plan_decode(const std::vector<DecodeSeq>& seqs, int hkv, int G, DecodePlan& out);

// Chunked-prefill work list.  Each (prefill entry, kv-head, block of qpi queries) is
// one item over the key tiles its queries see.  With fewer items than CUs, an item
// longer than the per-slot share of one pass over the resident workgroups (at least
// kPrefillMinTiles) is cut into equal key ranges whose partials a merge job combines.
// Items are launched most tiles first, the long and short ones of the first pass
// paired on the CUs.
struct PrefillEntry {
  int entry, pos0, n;   // batch entry, position of its first query, queries
};
struct PrefillPlan {
  std::vector<PrefillItem> items;
  std::vector<PrefillMerge> merges;
  int64_t n_parts = 0;
  int64_t tiles = 0;    // key tiles over all items
};
void plan_prefill(const std::vector<PrefillEntry>& entries, int hkv, int qpi, PrefillPlan& out);
// Partial slots the prefill plan of n_items items can use (split items only).
inline int64_t prefill_parts_bound(int64_t n_items) { return n_items + kPrefillResident; }

// Upper bound of partial slots (and items) for n sequences of at most max_ctx tokens.
inline int64_t decode_parts_bound(int64_t n_seqs, int64_t hkv, int64_t max_ctx) {
  return n_seqs * hkv * ((max_ctx + kDecodeMinPartition - 1) / kDecodeMinPartition + 1);
}

}  // namespace hxf
