// C ABI of the serving instance (include/hxf.h).
#include <algorithm>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <memory>
#include <new>
#include <string>
#include <vector>

#include "executor.hpp"
#include "hxf.h"
#include "hxf_coord.h"
#include "sched.hpp"

using namespace hxf;

namespace {

// Scheduler-only stand-in for the forward pass: the sampled token is a fixed
// function of (request id, position of the new token); no device is touched.
class NullExecutor : public Executor {
 public:
  explicit NullExecutor(int32_t vocab) : vocab_(vocab) {}
  int run(const std::vector<BatchEntry>& batch, std::vector<int32_t>& sampled, std::string&) override {
    sampled.clear();
    for (const auto& e : batch) {
      if (!e.logits) continue;
      const int64_t pos = (int64_t)e.r->context.size() + (int64_t)e.r->generated.size();
      const __int128 v = (__int128)e.r->id * 1000003 + (__int128)pos * 7919 + 12345;
      sampled.push_back((int32_t)(v % vocab_));
    }
    return HXF_OK;
  }

 private:
  int32_t vocab_;
};

}  // namespace

struct hxf_instance {
  hxf_instance(const hxf_model_cfg& m, const hxf_sched_cfg& s) : sched(m, s) {}
  ~hxf_instance() {
    if (trace) std::fclose(trace);
  }
  Scheduler sched;
  std::FILE* trace = nullptr;   // HXF_TRACE: one JSON line per iteration
  std::unique_ptr<Executor> exec;
  std::string err;
  std::vector<BatchEntry> batch;
  std::vector<uint64_t> admitted, last_ids;
  std::vector<int32_t> sampled;
};

#define GUARD_BEGIN try {
#define GUARD_END                                        \
  }                                                      \
  catch (const std::bad_alloc&) {                        \
    if (inst) inst->err = "out of host memory";          \
    return HXF_ENOMEM;                                   \
  }                                                      \
  catch (const std::exception& ex) {                     \
    if (inst) inst->err = std::string("internal: ") + ex.what(); \
    return HXF_EINVAL;                                   \
  }

static int check_sched(const hxf_sched_cfg& s, std::string& err) {
  if (s.n_blocks <= 0 || s.n_blocks > (int64_t)1 << 31) { err = "sched: n_blocks out of range"; return HXF_EINVAL; }
  if (s.max_seqs <= 0 || s.chunk_tokens <= 0) { err = "sched: max_seqs and chunk_tokens must be positive"; return HXF_EINVAL; }
  if (s.policy < 0 || s.policy > 2 || s.clock < 0 || s.clock > 1 || s.executor < 0 || s.executor > 1) {
    err = "sched: bad policy, clock or executor";
    return HXF_EINVAL;
  }
  return HXF_OK;
}

extern "C" {

int hxf_create(const hxf_model_cfg* model, const hxf_sched_cfg* sched, hxf_instance** out) {
  if (!model || !sched || !out) return HXF_EINVAL;
  std::string err;
  if (validate_model(*model, err) || check_sched(*sched, err)) return HXF_EINVAL;
  hxf_instance* inst = nullptr;
  try {
    inst = new hxf_instance(*model, *sched);
    if (sched->executor == HXF_EXEC_NULL) inst->exec = std::make_unique<NullExecutor>(model->vocab);
    if (const char* path = std::getenv("HXF_TRACE"); path && path[0]) inst->trace = std::fopen(path, "a");
  } catch (...) {
    delete inst;
    return HXF_ENOMEM;
  }
  *out = inst;
  return HXF_OK;
}

void hxf_destroy(hxf_instance* inst) { delete inst; }

const char* hxf_last_error(const hxf_instance* inst) { return inst ? inst->err.c_str() : "null instance"; }

int64_t hxf_kv_pool_bytes(const hxf_model_cfg* model, int64_t n_blocks) {
  if (!model || n_blocks < 0) return -1;
  return kv_pool_bytes(*model, n_blocks);
}

int64_t hxf_workspace_bytes(const hxf_model_cfg* model, const hxf_sched_cfg* sched) {
  if (!model || !sched) return -1;
  std::string err;
  if (validate_model(*model, err) || check_sched(*sched, err)) return -1;
  return plan_workspace(*model, *sched).total;
}

int hxf_bind(hxf_instance* inst, const hxf_device_buffers* b, void* stream) {
  if (!inst || !b) return HXF_EINVAL;
  GUARD_BEGIN
  const auto& m = inst->sched.mcfg;
  const auto& s = inst->sched.scfg;
  if (s.executor != HXF_EXEC_HIP) { inst->err = "bind: instance uses the scheduler-only executor"; return HXF_ESTATE; }
  if (!b->embed || !b->final_norm || !b->lm_head || !b->layers || !b->kv_pool || !b->workspace) {
    inst->err = "bind: null buffer";
    return HXF_EINVAL;
  }
  for (int l = 0; l < m.n_layers; ++l) {
    const auto& L = b->layers[l];
    if (!L.attn_norm || !L.wqkv || !L.wo || !L.ffn_norm || !L.w_gate || !L.w_up || !L.w_down) {
      inst->err = "bind: null layer weight";
      return HXF_EINVAL;
    }
  }
  if (b->kv_pool_bytes < kv_pool_bytes(m, s.n_blocks)) { inst->err = "bind: KV pool too small"; return HXF_ENOMEM; }
  if (b->workspace_bytes < plan_workspace(m, s).total) { inst->err = "bind: workspace too small"; return HXF_ENOMEM; }
  if (((uintptr_t)b->kv_pool | (uintptr_t)b->workspace) & 255) {
    inst->err = "bind: KV pool and workspace must be 256-byte aligned";
    return HXF_EINVAL;
  }
  int rc = HXF_OK;
  auto ex = make_hip_executor(m, s, *b, stream, inst->err, &rc);
  if (rc) return rc;
  inst->exec = std::move(ex);
  return HXF_OK;
  GUARD_END
}

int hxf_submit(hxf_instance* inst, const hxf_stage_req* req, int64_t now_us, uint64_t* out_id) {
  if (!inst || !req || !out_id) return HXF_EINVAL;
  GUARD_BEGIN
  return inst->sched.submit(*req, now_us, out_id, inst->err);
  GUARD_END
}

int hxf_submit_shared(hxf_instance* inst, const hxf_stage_req* req, int64_t now_us, const int64_t* cost_sum_ps,
                      int32_t n_instances, uint64_t* out_id) {
  if (!inst || !req || !out_id || !cost_sum_ps || n_instances < 1) return HXF_EINVAL;
  GUARD_BEGIN
  return inst->sched.submit(*req, now_us, out_id, inst->err, cost_sum_ps, n_instances);
  GUARD_END
}

int hxf_queue_cost(hxf_instance* inst, int64_t* t_queue_us) {
  if (!inst || !t_queue_us) return HXF_EINVAL;
  *t_queue_us = inst->sched.queue_cost();
  return HXF_OK;
}

int hxf_request_cost(hxf_instance* inst, int32_t l_in, int32_t l_out, int64_t* out) {
  if (!inst || !out || l_in < 0 || l_out < 0) return HXF_EINVAL;
  *out = hxf::t_comp_us(inst->sched.scfg.cost_ps, l_in, l_out);
  return HXF_OK;
}

int hxf_step(hxf_instance* inst, int64_t now_us, hxf_step_info* out) {
  if (!inst) return HXF_EINVAL;
  GUARD_BEGIN
  if (!inst->exec) { inst->err = "step: instance is not bound to device buffers"; return HXF_ESTATE; }
  Scheduler& S = inst->sched;
  inst->last_ids.clear();
  S.form_batch(now_us, inst->batch, inst->admitted);
  hxf_step_info info{};
  info.iteration = S.iteration;
  if (inst->batch.empty()) {
    info.free_blocks = S.alloc.n_free();
    if (out) *out = info;
    return HXF_IDLE;
  }
  int64_t n_tok, sum_ctx, attn, n_dec = 0;
  S.batch_cost_terms(inst->batch, &n_tok, &sum_ctx, &attn);
  for (const auto& e : inst->batch) n_dec += e.decode ? 1 : 0;
  const auto t0 = std::chrono::steady_clock::now();
  int rc = inst->exec->run(inst->batch, inst->sampled, inst->err);
  if (rc) return rc;
  const auto t1 = std::chrono::steady_clock::now();
  int64_t dt = (S.scfg.clock == HXF_CLOCK_MEASURED)
                   ? std::chrono::duration_cast<std::chrono::microseconds>(t1 - t0).count()
                   : t_iter_us(S.scfg.iter_ps, n_tok - n_dec, n_dec, sum_ctx, attn);
  for (const auto& e : inst->batch) {
    info.n_decode += e.decode ? 1 : 0;
    info.n_prefill_tokens += e.decode ? 0 : e.n;
    info.n_logit_rows += e.logits ? 1 : 0;
    inst->last_ids.push_back(e.r->id);
  }
  std::sort(inst->last_ids.begin(), inst->last_ids.end());
  info.n_tokens = (int32_t)n_tok;
  info.sum_decode_ctx = sum_ctx;
  info.prefill_attn = attn;
  info.n_admitted = (int32_t)inst->admitted.size();
  info.t_iter_us = dt;
  S.commit(inst->batch, inst->sampled, now_us + dt, &info.n_finished);
  info.free_blocks = S.alloc.n_free();
  if (inst->trace) {
    std::fprintf(inst->trace,
                 "{\"instance\":\"%p\",\"iteration\":%lld,\"now_us\":%lld,\"t_iter_us\":%lld,\"n_tokens\":%d,"
                 "\"n_decode\":%d,\"n_prefill_tokens\":%d,\"n_logit_rows\":%d,\"sum_decode_ctx\":%lld,"
                 "\"prefill_attn\":%lld,\"n_finished\":%d,\"free_blocks\":%lld,\"admitted\":[",
                 (void*)inst, (long long)info.iteration, (long long)now_us, (long long)dt, info.n_tokens, info.n_decode,
                 info.n_prefill_tokens, info.n_logit_rows, (long long)sum_ctx, (long long)attn, info.n_finished,
                 (long long)info.free_blocks);
    for (size_t i = 0; i < inst->admitted.size(); ++i)
      std::fprintf(inst->trace, i ? ",%llu" : "%llu", (unsigned long long)inst->admitted[i]);
    std::fprintf(inst->trace, "]}\n");
    std::fflush(inst->trace);
  }
  if (out) *out = info;
  return HXF_OK;
  GUARD_END
}

int hxf_drain(hxf_instance* inst, hxf_completion* out, int32_t cap, int32_t* n) {
  if (!inst || !n || (cap > 0 && !out) || cap < 0) return HXF_EINVAL;
  GUARD_BEGIN
  Scheduler& S = inst->sched;
  const int32_t k = (int32_t)std::min<size_t>(cap, S.done_queue.size());
  for (int32_t i = 0; i < k; ++i) {
    const Request* r = S.find(S.done_queue[i]);
    hxf_completion& c = out[i];
    c = hxf_completion{};
    c.id = r->id;
    c.workflow_id = r->workflow;
    c.stage_index = r->stage;
    c.n_generated = (int32_t)r->generated.size();
    c.t_submit_us = r->enq;
    c.t_first_sched_us = r->t_first_sched;
    c.t_first_token_us = r->t_first_token;
    c.t_finish_us = r->t_finish;
    c.t_slo_us = r->t_slo;
    c.t_comp_us = r->t_comp;
    c.met_slo = (r->t_finish - r->enq) <= r->t_slo ? 1 : 0;
  }
  S.done_queue.erase(S.done_queue.begin(), S.done_queue.begin() + k);
  *n = k;
  return HXF_OK;
  GUARD_END
}

int hxf_completion_tokens(hxf_instance* inst, uint64_t id, int32_t* buf, int32_t cap, int32_t* n) {
  if (!inst || !n || cap < 0 || (cap > 0 && !buf)) return HXF_EINVAL;
  const Request* r = inst->sched.find(id);
  if (!r) { inst->err = "tokens: unknown id"; return HXF_ENOTFOUND; }
  *n = (int32_t)r->generated.size();
  if (*n > cap) { inst->err = "tokens: buffer too small"; return HXF_ENOMEM; }
  std::copy(r->generated.begin(), r->generated.end(), buf);
  return HXF_OK;
}

int hxf_release(hxf_instance* inst, uint64_t id) {
  if (!inst) return HXF_EINVAL;
  GUARD_BEGIN
  return inst->sched.release(id, inst->err);
  GUARD_END
}

int hxf_cancel(hxf_instance* inst, uint64_t id) {
  if (!inst) return HXF_EINVAL;
  GUARD_BEGIN
  return inst->sched.cancel(id, inst->err);
  GUARD_END
}

int hxf_queue_order(hxf_instance* inst, uint64_t* ids, int32_t cap, int32_t* n) {
  if (!inst || !n || cap < 0 || (cap > 0 && !ids)) return HXF_EINVAL;
  GUARD_BEGIN
  auto q = inst->sched.queue_order();
  *n = (int32_t)q.size();
  if (*n > cap) { inst->err = "queue_order: buffer too small"; return HXF_ENOMEM; }
  std::copy(q.begin(), q.end(), ids);
  return HXF_OK;
  GUARD_END
}

int hxf_block_table(hxf_instance* inst, uint64_t id, int32_t* blocks, int32_t cap, int32_t* n) {
  if (!inst || !n || cap < 0 || (cap > 0 && !blocks)) return HXF_EINVAL;
  const Request* r = inst->sched.find(id);
  if (!r) { inst->err = "block_table: unknown id"; return HXF_ENOTFOUND; }
  *n = (int32_t)r->bt.size();
  if (*n > cap) { inst->err = "block_table: buffer too small"; return HXF_ENOMEM; }
  std::copy(r->bt.begin(), r->bt.end(), blocks);
  return HXF_OK;
}

int hxf_request_state_get(hxf_instance* inst, uint64_t id, hxf_request_state* out) {
  if (!inst || !out) return HXF_EINVAL;
  const Request* r = inst->sched.find(id);
  if (!r) { inst->err = "request_state: unknown id"; return HXF_ENOTFOUND; }
  out->state = (int32_t)r->state;
  out->n_generated = (int32_t)r->generated.size();
  out->n_kv = r->n_kv;
  out->n_blocks = (int32_t)r->bt.size();
  out->t_comp_us = r->t_comp;
  out->t_slo_us = r->t_slo;
  out->key_us = r->key;
  out->t_submit_us = r->enq;
  return HXF_OK;
}

int hxf_last_batch(hxf_instance* inst, uint64_t* ids, int32_t cap, int32_t* n, uint64_t* admitted,
                   int32_t cap_admitted, int32_t* n_admitted) {
  if (!inst || !n || !n_admitted || cap < 0 || cap_admitted < 0) return HXF_EINVAL;
  *n = (int32_t)inst->last_ids.size();
  *n_admitted = (int32_t)inst->admitted.size();
  if (*n > cap || *n_admitted > cap_admitted) { inst->err = "last_batch: buffer too small"; return HXF_ENOMEM; }
  std::copy(inst->last_ids.begin(), inst->last_ids.end(), ids);
  std::copy(inst->admitted.begin(), inst->admitted.end(), admitted);
  return HXF_OK;
}

int hxf_last_logits(hxf_instance* inst, uint64_t id, float* dst, int32_t cap) {
  if (!inst || !dst) return HXF_EINVAL;
  GUARD_BEGIN
  if (!inst->exec) { inst->err = "last_logits: no executor"; return HXF_ESTATE; }
  return inst->exec->last_logits(id, dst, cap, inst->err);
  GUARD_END
}

int hxf_profile_enable(hxf_instance* inst, int32_t on) {
  if (!inst) return HXF_EINVAL;
  Profile* p = inst->exec ? executor_profile(inst->exec.get()) : nullptr;
  if (!p) { inst->err = "profile: instance has no HIP executor"; return HXF_ESTATE; }
  *p = Profile{};
  p->on = on != 0;
  return HXF_OK;
}

int hxf_profile_get(hxf_instance* inst, hxf_profile* out) {
  if (!inst || !out) return HXF_EINVAL;
  Profile* p = inst->exec ? executor_profile(inst->exec.get()) : nullptr;
  if (!p) { inst->err = "profile: instance has no HIP executor"; return HXF_ESTATE; }
  out->decode_attn_launches = p->decode_attn_launches;
  out->decode_attn_bytes = p->decode_attn_bytes;
  out->decode_attn_ms = p->decode_attn_ms;
  out->decode_merge_ms = p->decode_merge_ms;
  for (int i = 0; i < 5; ++i) {
    out->gemm_launches[i] = p->gemm_launches[i];
    out->gemm_flops[i] = p->gemm_flops[i];
    out->gemm_ms[i] = p->gemm_ms[i];
  }
  out->prefill_attn_launches = p->prefill_attn_launches;
  out->prefill_attn_flops = p->prefill_attn_flops;
  out->prefill_attn_ms = p->prefill_attn_ms;
  return HXF_OK;
}

}  // extern "C"
