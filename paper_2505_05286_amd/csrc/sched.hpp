// Host-side scheduler of one serving instance: cost model, SLO budget,
// urgency-ordered local queue, continuous-batching batch former and the
// reference-counted KV page allocator.  Pure C++ (no HIP), integer time.
#pragma once

#include <cstdint>
#include <set>
#include <string>
#include <tuple>
#include <unordered_map>
#include <vector>

#include "hxf.h"

namespace hxf {

using i64 = int64_t;
using i128 = __int128;

// Floor division toward minus infinity (C++ '/' truncates toward zero).
inline i128 floor_div(i128 a, i128 b) {
  i128 q = a / b;
  if ((a % b != 0) && ((a < 0) != (b < 0))) --q;
  return q;
}

constexpr i64 kPsPerUs = 1000000;

// Compute-cost estimate, Section 4.1: t_prefill(L_in) + t_decode(L_out), here a
// polynomial in picoseconds floored to microseconds.
i64 t_comp_us(const i64 cost_ps[4], i64 l_in, i64 l_out);

// Per-request SLO budget, Section 4.2: the remaining end-to-end time shared in
// proportion to this request's (instance-average) cost among it and the later
// stages.  With one instance the average is the instance's own estimate.
i64 slo_budget_us(i64 slo_e2e, i64 elapsed, i64 c_j, const std::vector<i64>& rest_costs);

// Instance-average compute cost, Section 4.2: the mean over N instances of their
// t_comp estimates, given the N instances' cost coefficients summed (t_comp is
// linear in them): floor(sum of the unfloored estimates / N).  N = 1 with the
// instance's own coefficients is t_comp_us itself.
i64 t_comp_mean_us(const i64 cost_sum_ps[4], i64 n_instances, i64 l_in, i64 l_out);

// Iteration duration of the virtual clock.
i64 t_iter_us(const i64 iter_ps[5], i64 n_prefill, i64 n_decode, i64 sum_ctx_decode, i64 prefill_attn);

enum State : int32_t { QUEUED = 0, PREFILL = 1, DECODE = 2, DONE = 3, RELEASED = 4, CANCELLED = 5 };

struct Request {
  uint64_t id = 0, workflow = 0, parent = 0;
  int32_t stage = 0, max_new = 0;
  bool retain = false;
  i64 wf_arrival = 0, wf_slo = 0;
  std::vector<int32_t> context;     // full token sequence before generation (fork: parent's S ++ appended)
  std::vector<int32_t> pf_tokens;   // tokens this request prefills
  std::vector<int32_t> generated;   // sampled tokens
  std::vector<int32_t> forced;      // teacher-forced feedback tokens (empty: none)
  int32_t pf_pos0 = 0, n_pf_done = 0, n_kv = 0, n_shared = 0;
  i64 reserve = 0;
  i64 t_comp = 0, t_slo = 0, key = 0, enq = 0;
  i64 t_first_sched = -1, t_first_token = -1, t_finish = -1;
  std::vector<int32_t> bt;          // block table (shared pages first)
  State state = QUEUED;
};

// Lexicographic queue order; smaller is served first.
struct OrderKey {
  i64 a, b, c;
  uint64_t id;
  bool operator<(const OrderKey& o) const {
    return std::tie(a, b, c, id) < std::tie(o.a, o.b, o.c, o.id);
  }
};

class BlockAllocator {
 public:
  void init(i64 n);
  i64 n_free() const { return (i64)free_.size(); }
  i64 n_total() const { return (i64)ref_.size(); }
  bool alloc(i64 k, std::vector<int32_t>& out);   // lowest ids first; appends to out
  void share(const std::vector<int32_t>& b, size_t n);
  void release(const std::vector<int32_t>& b);
  int32_t ref(int32_t b) const { return ref_[b]; }

 private:
  std::vector<int32_t> ref_;
  std::set<int32_t> free_;
};

// One batch entry as seen by an executor.
struct BatchEntry {
  Request* r;
  bool decode;
  int32_t pos0;        // position of the first token
  int32_t n;           // tokens in this entry
  const int32_t* toks; // host token ids
  int32_t feed_tok;    // decode: the token fed (sampled or forced)
  bool logits;         // a token is sampled from its last row
};

class Executor {
 public:
  virtual ~Executor() = default;
  // Run one forward over the batch; write one sampled token per logits row (batch order).
  virtual int run(const std::vector<BatchEntry>& batch, std::vector<int32_t>& sampled, std::string& err) = 0;
  virtual int last_logits(uint64_t, float*, int32_t, std::string&) { return HXF_ENOTFOUND; }
};

class Scheduler {
 public:
  Scheduler(const hxf_model_cfg& m, const hxf_sched_cfg& s);

  // budget_cost_sum (may be null: this instance's own coefficients, N = 1): the cost
  // coefficients of the n_instances instances summed, for the SLO budget's
  // instance-average costs.  The urgency key always uses this instance's t_comp.
  int submit(const hxf_stage_req& q, i64 now, uint64_t* out_id, std::string& err,
             const i64* budget_cost_sum = nullptr, i64 n_instances = 1);
  // Sum of t_comp over the requests that have not finished (queued or running).
  i64 queue_cost() const { return queue_cost_; }
  // Batch formation at a batch boundary (admission in queue order).
  void form_batch(i64 now, std::vector<BatchEntry>& batch, std::vector<uint64_t>& admitted);
  // Apply sampled tokens, finish requests, free pages.
  void commit(std::vector<BatchEntry>& batch, const std::vector<int32_t>& sampled, i64 t_end,
              int32_t* n_finished);
  void batch_cost_terms(const std::vector<BatchEntry>& batch, i64* n_tok, i64* sum_ctx, i64* attn) const;

  int release(uint64_t id, std::string& err);
  int cancel(uint64_t id, std::string& err);
  Request* find(uint64_t id);
  std::vector<uint64_t> queue_order() const;

  std::vector<uint64_t> done_queue;
  BlockAllocator alloc;
  hxf_model_cfg mcfg;
  hxf_sched_cfg scfg;
  i64 iteration = 0;

 private:
  OrderKey order(const Request& r) const;
  std::unordered_map<uint64_t, Request> reqs_;
  std::set<OrderKey> queue_;
  std::vector<Request*> running_;   // admission order
  uint64_t next_id_ = 1;
  i64 queue_cost_ = 0;
};

}  // namespace hxf
