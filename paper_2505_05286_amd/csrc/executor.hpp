// HIP forward executor: workspace plan, per-iteration metadata and the launch
// sequence of one continuous-batched decoder iteration.
#pragma once

#include <memory>
#include <string>
#include <vector>

#include "hxf.h"
#include "sched.hpp"

namespace hxf {

struct WsPlan {
  int64_t t_max = 0, r_max = 0, e_max = 0, bt_w = 0;
  int64_t dec_items_max = 0, merges_max = 0, pf_items_max = 0, pf_merges_max = 0, pf_parts_max = 0;
  // byte offsets into the workspace
  int64_t off_meta = 0, meta_bytes = 0;
  int64_t off_rope = 0, off_resid = 0, off_h = 0, off_qkv = 0, off_attn = 0, off_act = 0;
  int64_t off_part = 0, part_bytes = 0;
  int64_t off_attn_o = 0, off_attn_ml = 0, off_pf_o = 0, off_pf_ml = 0;
  int64_t off_logits = 0, off_hr = 0, off_sampled = 0;
  int64_t total = 0;
};

WsPlan plan_workspace(const hxf_model_cfg& m, const hxf_sched_cfg& s);
int64_t kv_pool_bytes(const hxf_model_cfg& m, int64_t n_blocks);
int validate_model(const hxf_model_cfg& m, std::string& err);

struct Profile {
  bool on = false;
  double decode_attn_ms = 0;     // decode attention kernel (split-K part) time
  int64_t decode_attn_launches = 0;
  int64_t decode_attn_bytes = 0; // algorithmic KV bytes read by those launches
  double decode_merge_ms = 0;    // log-sum-exp merge kernel time of the same iterations
  int64_t gemm_launches[5] = {};  // by projection: QKV, O, gate/up, down, LM head
  double gemm_flops[5] = {};      // 2*M*N*K
  double gemm_ms[5] = {};
  int64_t prefill_attn_launches = 0;
  double prefill_attn_flops = 0;  // 4*dh per (query, key, q-head) pair inside the causal mask
  double prefill_attn_ms = 0;
};

std::unique_ptr<Executor> make_hip_executor(const hxf_model_cfg& m, const hxf_sched_cfg& s,
                                            const hxf_device_buffers& b, void* stream, std::string& err, int* rc);

// Access to the profiling counters of a HIP executor (nullptr for other executors).
Profile* executor_profile(Executor* e);

// Host-built RoPE table: cs[p][i] = (cos, sin)(p * base^(-2i/dh)) computed in double.
void build_rope_table(std::vector<float>& out, int max_pos, int dh, float base);

}  // namespace hxf
