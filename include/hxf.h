/*
 * hxf.h -- C ABI of one continuous-batching serving instance on one MI355X.
 *
 * An instance owns a local request queue ordered by the urgency of the paper's
 * Section 4.2 (per-request SLO budget carved from the workflow's end-to-end
 * SLO, least-laxity urgency, argmax admission at every batch boundary), a
 * paged KV-cache allocator, and a HIP forward pass of a Llama-style decoder
 * (chunked prefill co-batched with paged decode, greedy sampling).
 *
 * Conventions
 *  - Every call returns int: HXF_OK (0), HXF_IDLE (1, hxf_step only) or a
 *    negative error code; hxf_last_error() gives the message.  No C++
 *    exception crosses this boundary.
 *  - All times are int64 microseconds supplied by the caller (virtual or
 *    measured clock).  The library never reads a clock except to report the
 *    measured duration of an iteration in HXF_CLOCK_MEASURED mode.
 *  - The library never allocates device memory.  The caller owns every device
 *    buffer (weights, KV pool, workspace) and the HIP stream; see hxf_bind.
 *    It allocates only host memory (request state, pinned metadata staging).
 *  - An instance is single-threaded: calls on one instance must not overlap.
 *  - Tracing: if the environment variable HXF_TRACE names a file when an instance is
 *    created, every hxf_step that runs an iteration appends one JSON line to it
 *    (instance, iteration, now_us, t_iter_us, batch token/row counts, cost-model terms,
 *    finished count, free pages, ids admitted).
 *  - Checked mode: with HXF_CHECK=1 in the environment when hxf_bind runs, every
 *    iteration's indices (token ids, positions, KV slots, block tables, attention work
 *    items) are validated on the host before any kernel is launched; a violation makes
 *    hxf_step return HXF_EINVAL with the reason in hxf_last_error.
 */
#ifndef HXF_H
#define HXF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  HXF_OK = 0,
  HXF_IDLE = 1,        /* hxf_step: nothing runnable (empty, or the queue head does not fit) */
  HXF_EINVAL = -1,     /* bad argument or configuration */
  HXF_ENOMEM = -2,     /* request can never fit the KV pool / a caller buffer is too small */
  HXF_ENOTFOUND = -3,  /* unknown request id */
  HXF_ESTATE = -4,     /* call not valid in the current state (unbound, parent still running, ...) */
  HXF_EDEVICE = -5     /* a HIP runtime call failed; the message names it */
};

/* Local queue policy.  PQ is the paper's (Section 4.2); FCFS and LLF are the
 * comparison policies of Section 5.1 ("Baseline"): arrival order, and least
 * laxity against the workflow's end-to-end deadline without per-stage budgets. */
enum { HXF_POLICY_PQ = 0, HXF_POLICY_FCFS = 1, HXF_POLICY_LLF = 2 };

/* Iteration duration reported by hxf_step: the integer iteration-cost model
 * (reproducible, for replays and parity) or the wall time of the iteration. */
enum { HXF_CLOCK_VIRTUAL = 0, HXF_CLOCK_MEASURED = 1 };

/* Forward executor: the HIP decoder, or a scheduler-only stand-in whose
 * "sampled" token is (id*1000003 + position*7919 + 12345) mod vocab and which
 * touches no device (used to test the host scheduler without a GPU). */
enum { HXF_EXEC_HIP = 0, HXF_EXEC_NULL = 1 };

typedef struct hxf_model_cfg {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_q_heads;
  int32_t n_kv_heads;     /* n_q_heads % n_kv_heads == 0; group size <= 16 */
  int32_t head_dim;       /* 64 or 128 */
  int32_t ffn_dim;        /* multiple of 16 */
  int32_t vocab;
  int32_t page_size;      /* tokens per KV page; must be 16 */
  int32_t max_context;    /* largest position + 1 any sequence may reach */
  float rms_eps;
  float rope_base;
} hxf_model_cfg;

typedef struct hxf_sched_cfg {
  int64_t n_blocks;       /* KV pages in the pool */
  int32_t max_seqs;       /* running sequences (prefill + decode) at most */
  int32_t chunk_tokens;   /* prefill tokens per iteration (every running decode comes on top) */
  int32_t policy;         /* HXF_POLICY_* */
  int32_t clock;          /* HXF_CLOCK_* */
  int32_t executor;       /* HXF_EXEC_* */
  int32_t reserved;
  /* Compute-cost estimate of a request, Section 4.1 (t_prefill(L_in) + t_decode(L_out)):
   * t_comp_us = floor((c0 + c1*L_in + c2*L_in^2 + d1*L_out) / 1e6), coefficients in ps. */
  int64_t cost_ps[4];     /* c0, c1, c2, d1 */
  /* Virtual iteration cost:
   * floor((i0 + i1*T_prefill + i2*sum_decode_ctx + i3*prefill_attn + i4*n_decode) / 1e6) us,
   * T_prefill = prefill tokens in the batch, n_decode = decode rows, sum_decode_ctx = sum of
   * the decode rows' context lengths, prefill_attn = sum over prefill chunks of
   * chunk_len * (chunk_start + chunk_len).  i4 = i1 charges every token alike. */
  int64_t iter_ps[5];
} hxf_sched_cfg;

/* (L_in, L_out) of one later stage on the workflow's critical path. */
typedef struct hxf_stage_shape {
  int32_t l_in;
  int32_t l_out;
} hxf_stage_shape;

typedef struct hxf_stage_req {
  uint64_t workflow_id;
  int32_t stage_index;          /* position of the stage in its workflow (later = preferred on ties) */
  int32_t prompt_len;           /* tokens in prompt_ids (may be 0 only for a fork) */
  int64_t workflow_arrival_us;  /* arrival of the workflow's query (start of tau_elapsed) */
  int64_t workflow_slo_us;      /* end-to-end SLO T^SLO of the query */
  const int32_t* prompt_ids;    /* host; copied.  For a fork: tokens appended to the parent's */
  int32_t max_new_tokens;       /* output budget = estimated L_out; 0 only with retain_kv */
  uint8_t retain_kv;            /* keep KV after finishing (until hxf_release) so it can be forked */
  uint8_t pad_[3];
  uint64_t parent_id;           /* 0, or a finished request submitted with retain_kv */
  const hxf_stage_shape* rest;  /* host; later stages of the workflow (budget denominator) */
  int32_t n_rest;
  int32_t n_forced;             /* 0, or max_new_tokens: teacher forcing */
  const int32_t* forced_ids;    /* host; token fed back after generated token k (k < n_forced):
                                   the request's sequence holds the forced tokens (a fork of it
                                   continues from them); the sampled argmax is still what
                                   hxf_completion_tokens returns */
} hxf_stage_req;

/* Device pointers of one decoder layer.  Every matrix is bf16, row-major
 * [out_features, in_features]. */
/* The projection matrices and the LM head are PACKED (hxf_op_pack_weight in
 * hxf_ops.h: 16x32 tiles in MFMA operand order); shapes below are the logical
 * row-major [rows, columns] before packing.  Norm gains and the embedding table
 * are plain row-major bf16. */
typedef struct hxf_layer_weights {
  const void* attn_norm;  /* bf16 [d] */
  const void* wqkv;       /* packed bf16 [(Hq + 2*Hkv)*dh, d]: rows of Wq, then Wk, then Wv */
  const void* wo;         /* packed bf16 [d, Hq*dh] */
  const void* ffn_norm;   /* bf16 [d] */
  const void* w_gate;     /* packed bf16 [F, d] */
  const void* w_up;       /* packed bf16 [F, d] */
  const void* w_down;     /* packed bf16 [d, F] */
} hxf_layer_weights;

typedef struct hxf_device_buffers {
  const void* embed;                 /* bf16 [V, d] */
  const void* final_norm;            /* bf16 [d] */
  const void* lm_head;               /* packed bf16 [V, d] */
  const hxf_layer_weights* layers;   /* host array of n_layers entries (copied by hxf_bind) */
  void* kv_pool;                     /* hxf_kv_pool_bytes(cfg, n_blocks) bytes, 256-byte aligned */
  int64_t kv_pool_bytes;
  void* workspace;                   /* hxf_workspace_bytes(...) bytes, 256-byte aligned */
  int64_t workspace_bytes;
} hxf_device_buffers;

typedef struct hxf_step_info {
  int32_t n_tokens;         /* tokens in the batch */
  int32_t n_decode;         /* decode rows */
  int32_t n_prefill_tokens; /* prefill tokens */
  int32_t n_logit_rows;     /* rows sampled this iteration */
  int32_t n_admitted;       /* requests admitted from the queue this iteration */
  int32_t n_finished;       /* requests that finished this iteration */
  int64_t t_iter_us;        /* virtual or measured duration of the iteration */
  int64_t free_blocks;      /* free KV pages after the iteration */
  int64_t iteration;        /* index of this iteration */
  int64_t sum_decode_ctx;   /* cost-model term: sum of the decode rows' context lengths */
  int64_t prefill_attn;     /* cost-model term: sum over prefill chunks of chunk_len * (chunk_start + chunk_len) */
} hxf_step_info;

typedef struct hxf_completion {
  uint64_t id;
  uint64_t workflow_id;
  int32_t stage_index;
  int32_t n_generated;
  int64_t t_submit_us;       /* enqueue time (the now of hxf_submit) */
  int64_t t_first_sched_us;  /* now of the iteration that admitted it */
  int64_t t_first_token_us;  /* end of the iteration that produced its first token (-1: none) */
  int64_t t_finish_us;       /* end of the iteration it finished in */
  int64_t t_slo_us;          /* per-request SLO budget (Section 4.2) */
  int64_t t_comp_us;         /* compute-cost estimate (Section 4.1) */
  int32_t met_slo;           /* t_finish - t_submit <= t_slo */
  int32_t pad_;
} hxf_completion;

typedef struct hxf_request_state {
  int32_t state;            /* 0 queued, 1 prefill, 2 decode, 3 finished, 4 released, 5 cancelled */
  int32_t n_generated;
  int32_t n_kv;             /* positions whose KV has been written */
  int32_t n_blocks;         /* block-table length */
  int64_t t_comp_us;
  int64_t t_slo_us;
  int64_t key_us;           /* static queue key (PQ: enqueue + t_slo - t_comp) */
  int64_t t_submit_us;
} hxf_request_state;

typedef struct hxf_instance hxf_instance;

/* Create an instance (host state only).  Validates both configurations. */
int hxf_create(const hxf_model_cfg* model, const hxf_sched_cfg* sched, hxf_instance** out);
void hxf_destroy(hxf_instance* inst);
const char* hxf_last_error(const hxf_instance* inst);

/* Bytes of a KV pool of n_blocks pages (all layers, K and V), and of the
 * workspace the forward pass needs for these configurations. */
int64_t hxf_kv_pool_bytes(const hxf_model_cfg* model, int64_t n_blocks);
int64_t hxf_workspace_bytes(const hxf_model_cfg* model, const hxf_sched_cfg* sched);

/* Attach caller-owned device buffers and the caller's HIP stream (hipStream_t,
 * may be 0).  Required before hxf_step with HXF_EXEC_HIP.  Builds the RoPE
 * table in the workspace (one host-to-device copy).  HXF_ENOMEM if a buffer is
 * smaller than required. */
int hxf_bind(hxf_instance* inst, const hxf_device_buffers* bufs, void* hip_stream);

/* Submit one workflow-stage request at time now_us (Section 4 problem formulation:
 * query i's request j with end-to-end SLO).  Computes t_comp and the fixed
 * per-request SLO budget, assigns an id (1, 2, ...), and queues it. */
int hxf_submit(hxf_instance* inst, const hxf_stage_req* req, int64_t now_us, uint64_t* out_id);

/* One batch boundary and one forward iteration.  The batch is formed by the
 * selection rule of Section 4.2: the queue is re-ranked at this boundary (the
 * urgency U = t_comp - (t_SLO - tau) of every queued request, taken in decreasing
 * order, i.e. the argmax over the local queue first, which the static key
 * enq + t_SLO - t_comp ranks identically); running decodes take one token each,
 * running prefills take chunk tokens in that order, then queued requests are
 * admitted in that order while a sequence slot, their page reservation and the
 * chunk budget allow, stopping at the first that does not fit.  now_us is the
 * caller's clock.  Synchronous: returns after the sampled token ids have reached
 * the host.  HXF_IDLE if nothing ran. */
int hxf_step(hxf_instance* inst, int64_t now_us, hxf_step_info* out);

/* Move up to cap completion records (in finishing order) to out.  A completion
 * frees its request's place in the queue, after which Section 4.2's selection
 * takes the next most urgent request at the next hxf_step; each record carries
 * the request's budget t_SLO and whether it finished within it. */
int hxf_drain(hxf_instance* inst, hxf_completion* out, int32_t cap, int32_t* n);
/* Generated (sampled) tokens of a request so far.  HXF_ENOMEM if cap is too small (n is set). */
int hxf_completion_tokens(hxf_instance* inst, uint64_t id, int32_t* buf, int32_t cap, int32_t* n);
/* Drop the retained KV of a finished request. */
int hxf_release(hxf_instance* inst, uint64_t id);
/* Remove a queued or running request and free its pages. */
int hxf_cancel(hxf_instance* inst, uint64_t id);

/* Introspection (parity tests). */
int hxf_queue_order(hxf_instance* inst, uint64_t* ids, int32_t cap, int32_t* n);
int hxf_block_table(hxf_instance* inst, uint64_t id, int32_t* blocks, int32_t cap, int32_t* n);
int hxf_request_state_get(hxf_instance* inst, uint64_t id, hxf_request_state* out);
/* Ids in the last iteration's batch (sorted) and the ids it admitted (in admission order). */
int hxf_last_batch(hxf_instance* inst, uint64_t* ids, int32_t cap, int32_t* n,
                   uint64_t* admitted, int32_t cap_admitted, int32_t* n_admitted);
/* fp32 logits (vocab floats) of the request's row in the last iteration; HXF_ENOTFOUND if it had none. */
int hxf_last_logits(hxf_instance* inst, uint64_t id, float* dst, int32_t cap);

/* Kernel timing for roofline reporting: HIP events stamped with the kernels' own
 * start and end on the bound stream.  While profiling is on, iterations launch
 * eagerly (no graph replay).  Enabling resets the counters. */
enum { HXF_PROF_QKV = 0, HXF_PROF_O = 1, HXF_PROF_GATE_UP = 2, HXF_PROF_DOWN = 3, HXF_PROF_LM_HEAD = 4 };
typedef struct hxf_profile {
  int64_t decode_attn_launches;  /* split-K attention kernel launches timed */
  int64_t decode_attn_bytes;     /* algorithmic K+V bytes those launches read (context tokens x 2 x dh x 2 B x kv-heads) */
  double decode_attn_ms;         /* summed split-K kernel time */
  double decode_merge_ms;        /* summed time of the log-sum-exp merge kernels that follow them */
  /* GEMMs by projection (HXF_PROF_*): launches, 2*M*N*K flops, time from the first
   * kernel's start to the last one's end (a split-K reduction pass included). */
  int64_t gemm_launches[5];
  double gemm_flops[5];
  double gemm_ms[5];
  /* chunked-prefill attention: launches, 4*dh flops per (query, key, q-head) inside the
   * causal mask, summed kernel time */
  int64_t prefill_attn_launches;
  double prefill_attn_flops;
  double prefill_attn_ms;
} hxf_profile;

int hxf_profile_enable(hxf_instance* inst, int32_t on);
int hxf_profile_get(hxf_instance* inst, hxf_profile* out);

#ifdef __cplusplus
}
#endif
#endif /* HXF_H */
