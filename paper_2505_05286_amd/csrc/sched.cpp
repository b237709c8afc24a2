// Host scheduler: Section 4.2 local priority queue inside a continuous-batching
// iteration with chunked prefill and eager page reservation.
#include "sched.hpp"

#include <algorithm>

namespace hxf {

i64 t_comp_us(const i64 c[4], i64 l_in, i64 l_out) {
  i128 ps = (i128)c[0] + (i128)c[1] * l_in + (i128)c[2] * l_in * l_in + (i128)c[3] * l_out;
  return (i64)floor_div(ps, kPsPerUs);
}

i64 t_comp_mean_us(const i64 sum[4], i64 n, i64 l_in, i64 l_out) {
  i128 ps = (i128)sum[0] + (i128)sum[1] * l_in + (i128)sum[2] * l_in * l_in + (i128)sum[3] * l_out;
  return (i64)floor_div(ps, (i128)n * kPsPerUs);
}

i64 slo_budget_us(i64 slo_e2e, i64 elapsed, i64 c_j, const std::vector<i64>& rest) {
  i128 remaining = (i128)slo_e2e - elapsed;
  i128 denom = c_j;
  for (i64 c : rest) denom += c;
  if (denom == 0) return (i64)remaining;
  return (i64)floor_div(remaining * c_j, denom);
}

i64 t_iter_us(const i64 it[5], i64 n_prefill, i64 n_decode, i64 sum_ctx, i64 attn) {
  i128 ps = (i128)it[0] + (i128)it[1] * n_prefill + (i128)it[2] * sum_ctx + (i128)it[3] * attn + (i128)it[4] * n_decode;
  return (i64)floor_div(ps, kPsPerUs);
}

// ---------------------------------------------------------------- allocator
void BlockAllocator::init(i64 n) {
  ref_.assign((size_t)n, 0);
  free_.clear();
  for (i64 b = 0; b < n; ++b) free_.insert(free_.end(), (int32_t)b);
}

bool BlockAllocator::alloc(i64 k, std::vector<int32_t>& out) {
  if ((i64)free_.size() < k) return false;
  for (i64 i = 0; i < k; ++i) {
    int32_t b = *free_.begin();
    free_.erase(free_.begin());
    ref_[b] = 1;
    out.push_back(b);
  }
  return true;
}

void BlockAllocator::share(const std::vector<int32_t>& b, size_t n) {
  for (size_t i = 0; i < n; ++i) ref_[b[i]] += 1;
}

void BlockAllocator::release(const std::vector<int32_t>& b) {
  for (int32_t x : b) {
    if (--ref_[x] == 0) free_.insert(x);
  }
}

// ---------------------------------------------------------------- scheduler
Scheduler::Scheduler(const hxf_model_cfg& m, const hxf_sched_cfg& s) : mcfg(m), scfg(s) {
  alloc.init(s.n_blocks);
}

OrderKey Scheduler::order(const Request& r) const {
  switch (scfg.policy) {
    case HXF_POLICY_FCFS: return OrderKey{r.enq, 0, 0, r.id};
    case HXF_POLICY_LLF: return OrderKey{r.key, r.enq, 0, r.id};
    default: return OrderKey{r.key, -(i64)r.stage, r.enq, r.id};
  }
}

static i64 pages_for(i64 n, i64 page) { return (n + page - 1) / page; }

int Scheduler::submit(const hxf_stage_req& q, i64 now, uint64_t* out_id, std::string& err, const i64* budget_cost_sum,
                      i64 n_instances) {
  if (n_instances < 1) {
    err = "submit: n_instances must be at least 1";
    return HXF_EINVAL;
  }
  if (q.max_new_tokens < 0 || (q.max_new_tokens == 0 && !q.retain_kv) || q.stage_index < 0) {
    err = "submit: bad output budget or stage index";
    return HXF_EINVAL;
  }
  if (q.prompt_len < 0 || (q.prompt_len > 0 && !q.prompt_ids) || q.n_rest < 0 || (q.n_rest > 0 && !q.rest)) {
    err = "submit: bad prompt or rest array";
    return HXF_EINVAL;
  }
  if (q.n_forced != 0 && (q.n_forced != q.max_new_tokens || !q.forced_ids)) {
    err = "submit: n_forced must be 0 or max_new_tokens";
    return HXF_EINVAL;
  }
  for (int32_t i = 0; i < q.prompt_len; ++i)
    if (q.prompt_ids[i] < 0 || q.prompt_ids[i] >= mcfg.vocab) {
      err = "submit: token id out of range";
      return HXF_EINVAL;
    }
  for (int32_t i = 0; i < q.n_forced; ++i)
    if (q.forced_ids[i] < 0 || q.forced_ids[i] >= mcfg.vocab) {
      err = "submit: forced token id out of range";
      return HXF_EINVAL;
    }
  const i64 page = mcfg.page_size;
  Request r;
  i64 n_shared = 0;
  const Request* par = nullptr;
  if (q.parent_id) {
    auto it = reqs_.find(q.parent_id);
    if (it == reqs_.end() || it->second.state == CANCELLED || it->second.state == RELEASED) {
      err = "submit: no such parent";
      return HXF_ENOTFOUND;
    }
    par = &it->second;
    if (par->state != DONE || !par->retain) {
      err = "submit: parent has not finished with retained KV";
      return HXF_ESTATE;
    }
    // the parent's sequence: its context and its tokens (under teacher forcing the forced
    // ones, which are what its sequence holds)
    const std::vector<int32_t>& ptoks = par->forced.empty() ? par->generated : par->forced;
    std::vector<int32_t> s(par->context);
    s.insert(s.end(), ptoks.begin(), ptoks.begin() + par->generated.size());
    const i64 n = (i64)s.size();
    n_shared = (n - 1) / page;
    r.context = s;
    r.context.insert(r.context.end(), q.prompt_ids, q.prompt_ids + q.prompt_len);
    r.pf_tokens.assign(s.begin() + n_shared * page, s.end());
    r.pf_tokens.insert(r.pf_tokens.end(), q.prompt_ids, q.prompt_ids + q.prompt_len);
    r.pf_pos0 = (int32_t)(n_shared * page);
  } else {
    if (q.prompt_len == 0) {
      err = "submit: empty prompt";
      return HXF_EINVAL;
    }
    r.context.assign(q.prompt_ids, q.prompt_ids + q.prompt_len);
    r.pf_tokens = r.context;
    r.pf_pos0 = 0;
  }
  const i64 total_kv = (i64)r.context.size() + std::max(q.max_new_tokens - 1, 0);
  if (total_kv > mcfg.max_context) {
    err = "submit: context exceeds max_context";
    return HXF_EINVAL;
  }
  r.reserve = pages_for(total_kv, page) - n_shared;
  if (r.reserve > scfg.n_blocks) {
    err = "submit: request can never fit the KV pool";
    return HXF_ENOMEM;
  }
  r.id = next_id_++;
  r.workflow = q.workflow_id;
  r.stage = q.stage_index;
  r.wf_arrival = q.workflow_arrival_us;
  r.wf_slo = q.workflow_slo_us;
  r.max_new = q.max_new_tokens;
  r.retain = q.retain_kv != 0;
  r.parent = q.parent_id;
  if (q.n_forced) r.forced.assign(q.forced_ids, q.forced_ids + q.n_forced);
  r.t_comp = t_comp_us(scfg.cost_ps, (i64)r.pf_tokens.size(), r.max_new);
  std::vector<i64> rest;
  for (int32_t i = 0; i < q.n_rest; ++i) rest.push_back(t_comp_us(scfg.cost_ps, q.rest[i].l_in, q.rest[i].l_out));
  if (budget_cost_sum) {
    // SLO budget from the instance-average costs of this and the later stages
    std::vector<i64> mean_rest;
    for (int32_t i = 0; i < q.n_rest; ++i)
      mean_rest.push_back(t_comp_mean_us(budget_cost_sum, n_instances, q.rest[i].l_in, q.rest[i].l_out));
    const i64 mean_j = t_comp_mean_us(budget_cost_sum, n_instances, (i64)r.pf_tokens.size(), r.max_new);
    r.t_slo = slo_budget_us(r.wf_slo, now - r.wf_arrival, mean_j, mean_rest);
  } else {
    r.t_slo = slo_budget_us(r.wf_slo, now - r.wf_arrival, r.t_comp, rest);
  }
  r.enq = now;
  if (scfg.policy == HXF_POLICY_LLF) {
    i64 s = r.t_comp;
    for (i64 c : rest) s += c;
    r.key = r.wf_arrival + r.wf_slo - s;
  } else {
    r.key = r.enq + r.t_slo - r.t_comp;
  }
  if (par) {
    r.bt.assign(par->bt.begin(), par->bt.begin() + n_shared);
    alloc.share(r.bt, (size_t)n_shared);
  }
  r.n_shared = (int32_t)n_shared;
  r.n_kv = r.pf_pos0;
  r.state = QUEUED;
  auto ins = reqs_.emplace(r.id, std::move(r));
  Request& rr = ins.first->second;
  queue_.insert(order(rr));
  queue_cost_ += rr.t_comp;
  *out_id = rr.id;
  return HXF_OK;
}

void Scheduler::form_batch(i64 now, std::vector<BatchEntry>& batch, std::vector<uint64_t>& admitted) {
  batch.clear();
  admitted.clear();
  for (Request* r : running_) {
    if (r->state != DECODE) continue;
    const size_t k = r->generated.size() - 1;
    const int32_t tok = r->forced.empty() ? r->generated[k] : r->forced[k];
    batch.push_back(BatchEntry{r, true, r->n_kv, 1, nullptr, tok, true});
  }
  i64 budget = scfg.chunk_tokens;   // prefill tokens; the decode tokens are not counted
  std::vector<Request*> pf;
  for (Request* r : running_)
    if (r->state == PREFILL) pf.push_back(r);
  std::sort(pf.begin(), pf.end(), [this](Request* a, Request* b) { return order(*a) < order(*b); });
  auto add_prefill = [&](Request* r) {
    const int32_t left = (int32_t)r->pf_tokens.size() - r->n_pf_done;
    const int32_t c = (int32_t)std::min<i64>(left, budget);
    const bool last = (c == left);
    batch.push_back(BatchEntry{r, false, r->n_kv, c, r->pf_tokens.data() + r->n_pf_done, 0,
                               last && r->max_new > 0});
    budget -= c;
  };
  for (Request* r : pf) {
    if (budget <= 0) break;
    add_prefill(r);
  }
  while (!queue_.empty() && budget > 0) {
    Request& r = reqs_.at(queue_.begin()->id);
    if ((i64)running_.size() >= scfg.max_seqs || alloc.n_free() < r.reserve) break;
    queue_.erase(queue_.begin());
    alloc.alloc(r.reserve, r.bt);
    r.state = PREFILL;
    r.t_first_sched = now;
    running_.push_back(&r);
    admitted.push_back(r.id);
    add_prefill(&r);
  }
  // decode entries point at their own fed token (stable once the vector is complete)
  for (auto& e : batch)
    if (e.decode) e.toks = &e.feed_tok;
}

void Scheduler::batch_cost_terms(const std::vector<BatchEntry>& batch, i64* n_tok, i64* sum_ctx, i64* attn) const {
  *n_tok = *sum_ctx = *attn = 0;
  for (const auto& e : batch) {
    *n_tok += e.n;
    if (e.decode) *sum_ctx += (i64)e.pos0 + 1;
    else *attn += (i64)e.n * ((i64)e.pos0 + e.n);
  }
}

void Scheduler::commit(std::vector<BatchEntry>& batch, const std::vector<int32_t>& sampled, i64 t_end,
                       int32_t* n_finished) {
  std::vector<Request*> fin;
  size_t k = 0;
  for (auto& e : batch) {
    Request* r = e.r;
    r->n_kv += e.n;
    if (!e.decode) {
      r->n_pf_done += e.n;
      if (r->n_pf_done == (int32_t)r->pf_tokens.size()) {
        r->state = DECODE;
        if (r->max_new == 0) fin.push_back(r);
      }
    }
    if (e.logits) {
      r->generated.push_back(sampled[k++]);
      if (r->generated.size() == 1) r->t_first_token = t_end;
      if ((int32_t)r->generated.size() == r->max_new) fin.push_back(r);
    }
  }
  for (Request* r : fin) {
    r->state = DONE;
    r->t_finish = t_end;
    queue_cost_ -= r->t_comp;
    running_.erase(std::find(running_.begin(), running_.end(), r));
    if (!r->retain) alloc.release(r->bt);
    done_queue.push_back(r->id);
  }
  *n_finished = (int32_t)fin.size();
  ++iteration;
}

Request* Scheduler::find(uint64_t id) {
  auto it = reqs_.find(id);
  return it == reqs_.end() ? nullptr : &it->second;
}

int Scheduler::release(uint64_t id, std::string& err) {
  Request* r = find(id);
  if (!r) { err = "release: unknown id"; return HXF_ENOTFOUND; }
  if (r->state != DONE || !r->retain) { err = "release: request is not finished with retained KV"; return HXF_ESTATE; }
  alloc.release(r->bt);
  r->state = RELEASED;
  return HXF_OK;
}

int Scheduler::cancel(uint64_t id, std::string& err) {
  Request* r = find(id);
  if (!r) { err = "cancel: unknown id"; return HXF_ENOTFOUND; }
  if (r->state == QUEUED) {
    queue_.erase(order(*r));
    alloc.release(r->bt);
  } else if (r->state == PREFILL || r->state == DECODE) {
    running_.erase(std::find(running_.begin(), running_.end(), r));
    alloc.release(r->bt);
  } else {
    err = "cancel: request is not queued or running";
    return HXF_ESTATE;
  }
  r->state = CANCELLED;
  queue_cost_ -= r->t_comp;
  return HXF_OK;
}

std::vector<uint64_t> Scheduler::queue_order() const {
  std::vector<uint64_t> out;
  for (const auto& k : queue_) out.push_back(k.id);
  return out;
}

}  // namespace hxf
