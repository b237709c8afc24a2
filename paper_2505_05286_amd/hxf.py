"""ctypes binding of libhxf.so (include/hxf.h and include/hxf_ops.h).

Argument marshalling only: every step of the serving iteration runs in the
library.  Device buffers are passed as integer addresses (e.g.
``tensor.data_ptr()``) and the stream as a ``hipStream_t`` address.
"""
import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# HXF_LIBRARY selects another build of the library (e.g. one with instrumented host code)
LIB_PATH = os.environ.get("HXF_LIBRARY") or os.path.join(_HERE, "libhxf.so")

OK, IDLE = 0, 1
EINVAL, ENOMEM, ENOTFOUND, ESTATE, EDEVICE = -1, -2, -3, -4, -5
POLICY_PQ, POLICY_FCFS, POLICY_LLF = 0, 1, 2
CLOCK_VIRTUAL, CLOCK_MEASURED = 0, 1
EXEC_HIP, EXEC_NULL = 0, 1
EPI_BF16, EPI_RESID, EPI_SWIGLU, EPI_F32 = 0, 1, 2, 3
GEMM_A_PACKED, GEMM_C_PACKED = 0x100, 0x200   # layout flags or-ed into the epilogue (include/hxf_ops.h)


class HxfError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"hxf error {code}: {msg}")
        self.code = code


class ModelCfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32),
                ("vocab", C.c_int32), ("page_size", C.c_int32), ("max_context", C.c_int32),
                ("rms_eps", C.c_float), ("rope_base", C.c_float)]


class SchedCfg(C.Structure):
    _fields_ = [("n_blocks", C.c_int64), ("max_seqs", C.c_int32), ("chunk_tokens", C.c_int32),
                ("policy", C.c_int32), ("clock", C.c_int32), ("executor", C.c_int32), ("reserved", C.c_int32),
                ("cost_ps", C.c_int64 * 4), ("iter_ps", C.c_int64 * 5)]


class StageShape(C.Structure):
    _fields_ = [("l_in", C.c_int32), ("l_out", C.c_int32)]


class StageReq(C.Structure):
    _fields_ = [("workflow_id", C.c_uint64), ("stage_index", C.c_int32), ("prompt_len", C.c_int32),
                ("workflow_arrival_us", C.c_int64), ("workflow_slo_us", C.c_int64),
                ("prompt_ids", C.POINTER(C.c_int32)), ("max_new_tokens", C.c_int32), ("retain_kv", C.c_uint8),
                ("pad_", C.c_uint8 * 3), ("parent_id", C.c_uint64), ("rest", C.POINTER(StageShape)),
                ("n_rest", C.c_int32), ("n_forced", C.c_int32), ("forced_ids", C.POINTER(C.c_int32))]


class LayerWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("attn_norm", "wqkv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")]


class DeviceBuffers(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("final_norm", C.c_void_p), ("lm_head", C.c_void_p),
                ("layers", C.POINTER(LayerWeights)), ("kv_pool", C.c_void_p), ("kv_pool_bytes", C.c_int64),
                ("workspace", C.c_void_p), ("workspace_bytes", C.c_int64)]


class StepInfo(C.Structure):
    _fields_ = [("n_tokens", C.c_int32), ("n_decode", C.c_int32), ("n_prefill_tokens", C.c_int32),
                ("n_logit_rows", C.c_int32), ("n_admitted", C.c_int32), ("n_finished", C.c_int32),
                ("t_iter_us", C.c_int64), ("free_blocks", C.c_int64), ("iteration", C.c_int64),
                ("sum_decode_ctx", C.c_int64), ("prefill_attn", C.c_int64)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class Completion(C.Structure):
    _fields_ = [("id", C.c_uint64), ("workflow_id", C.c_uint64), ("stage_index", C.c_int32),
                ("n_generated", C.c_int32), ("t_submit_us", C.c_int64), ("t_first_sched_us", C.c_int64),
                ("t_first_token_us", C.c_int64), ("t_finish_us", C.c_int64), ("t_slo_us", C.c_int64),
                ("t_comp_us", C.c_int64), ("met_slo", C.c_int32), ("pad_", C.c_int32)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_ if k != "pad_"}


class RequestState(C.Structure):
    _fields_ = [("state", C.c_int32), ("n_generated", C.c_int32), ("n_kv", C.c_int32), ("n_blocks", C.c_int32),
                ("t_comp_us", C.c_int64), ("t_slo_us", C.c_int64), ("key_us", C.c_int64),
                ("t_submit_us", C.c_int64)]


PROF_GEMMS = ("qkv", "o", "gate_up", "down", "lm_head")


class Profile(C.Structure):
    _fields_ = [("decode_attn_launches", C.c_int64), ("decode_attn_bytes", C.c_int64),
                ("decode_attn_ms", C.c_double), ("decode_merge_ms", C.c_double),
                ("gemm_launches", C.c_int64 * 5), ("gemm_flops", C.c_double * 5), ("gemm_ms", C.c_double * 5),
                ("prefill_attn_launches", C.c_int64), ("prefill_attn_flops", C.c_double),
                ("prefill_attn_ms", C.c_double)]


_lib = None

# name -> (restype, argtypes)
_SIGS = {
    "hxf_create": (C.c_int, [C.POINTER(ModelCfg), C.POINTER(SchedCfg), C.POINTER(C.c_void_p)]),
    "hxf_destroy": (None, [C.c_void_p]),
    "hxf_last_error": (C.c_char_p, [C.c_void_p]),
    "hxf_kv_pool_bytes": (C.c_int64, [C.POINTER(ModelCfg), C.c_int64]),
    "hxf_workspace_bytes": (C.c_int64, [C.POINTER(ModelCfg), C.POINTER(SchedCfg)]),
    "hxf_bind": (C.c_int, [C.c_void_p, C.POINTER(DeviceBuffers), C.c_void_p]),
    "hxf_submit": (C.c_int, [C.c_void_p, C.POINTER(StageReq), C.c_int64, C.POINTER(C.c_uint64)]),
    "hxf_step": (C.c_int, [C.c_void_p, C.c_int64, C.POINTER(StepInfo)]),
    "hxf_drain": (C.c_int, [C.c_void_p, C.POINTER(Completion), C.c_int32, C.POINTER(C.c_int32)]),
    "hxf_completion_tokens": (C.c_int, [C.c_void_p, C.c_uint64, C.POINTER(C.c_int32), C.c_int32,
                                        C.POINTER(C.c_int32)]),
    "hxf_release": (C.c_int, [C.c_void_p, C.c_uint64]),
    "hxf_cancel": (C.c_int, [C.c_void_p, C.c_uint64]),
    "hxf_queue_order": (C.c_int, [C.c_void_p, C.POINTER(C.c_uint64), C.c_int32, C.POINTER(C.c_int32)]),
    "hxf_block_table": (C.c_int, [C.c_void_p, C.c_uint64, C.POINTER(C.c_int32), C.c_int32, C.POINTER(C.c_int32)]),
    "hxf_request_state_get": (C.c_int, [C.c_void_p, C.c_uint64, C.POINTER(RequestState)]),
    "hxf_last_batch": (C.c_int, [C.c_void_p, C.POINTER(C.c_uint64), C.c_int32, C.POINTER(C.c_int32),
                                 C.POINTER(C.c_uint64), C.c_int32, C.POINTER(C.c_int32)]),
    "hxf_last_logits": (C.c_int, [C.c_void_p, C.c_uint64, C.POINTER(C.c_float), C.c_int32]),
    "hxf_profile_enable": (C.c_int, [C.c_void_p, C.c_int32]),
    "hxf_profile_get": (C.c_int, [C.c_void_p, C.POINTER(Profile)]),
    # coordinator decisions (hxf_coord.h)
    "hxf_queue_cost": (C.c_int, [C.c_void_p, C.POINTER(C.c_int64)]),
    "hxf_request_cost": (C.c_int, [C.c_void_p, C.c_int32, C.c_int32, C.POINTER(C.c_int64)]),
    "hxf_submit_shared": (C.c_int, [C.c_void_p, C.POINTER(StageReq), C.c_int64, C.POINTER(C.c_int64), C.c_int32,
                                    C.POINTER(C.c_uint64)]),
    "hxf_wb_select": (C.c_int, [C.c_int32, C.POINTER(C.c_int64), C.POINTER(C.c_int64), C.c_double, C.c_double,
                                C.POINTER(C.c_int32)]),
    "hxf_ttest_greater": (C.c_int, [C.POINTER(C.c_double), C.c_int32, C.POINTER(C.c_double), C.c_int32,
                                    C.POINTER(C.c_double), C.POINTER(C.c_double), C.POINTER(C.c_double)]),
    # ops
    "hxf_op_gemm_workspace_bytes": (C.c_int64, [C.c_int32, C.c_int32, C.c_int32]),
    "hxf_packed_weight_bytes": (C.c_int64, [C.c_int32, C.c_int32]),
    "hxf_op_pack_weight": (C.c_int, [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p]),
    "hxf_op_gemm": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32, C.c_int32,
                              C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_int64, C.c_void_p]),
    "hxf_op_gemm_noalloc": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32,
                                      C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_void_p]),
    "hxf_op_rmsnorm": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_float,
                                 C.c_void_p]),
    "hxf_op_embed_rmsnorm": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32,
                                       C.c_int32, C.c_float, C.c_void_p]),
    "hxf_op_rope_table": (C.c_int, [C.c_void_p, C.c_int32, C.c_int32, C.c_float, C.c_void_p]),
    "hxf_op_rope_kv_write": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                       C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_void_p]),
    "hxf_op_kv_scatter": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64,
                                    C.c_int32, C.c_int32, C.c_int32, C.c_void_p]),
    "hxf_op_decode_attention_workspace_bytes": (C.c_int64, [C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                                            C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.c_int32]),
    "hxf_op_decode_plan": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                     C.c_int32, C.POINTER(C.c_int32), C.c_int32, C.POINTER(C.c_int32),
                                     C.POINTER(C.c_int32), C.c_int32, C.POINTER(C.c_int32)]),
    "hxf_op_prefill_plan": (C.c_int, [C.c_int32, C.c_int32, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                      C.POINTER(C.c_int32), C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                      C.c_int32, C.POINTER(C.c_int32)]),
    "hxf_op_decode_attention": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p, C.c_int32,
                                          C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.c_void_p, C.c_int32,
                                          C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_int64, C.c_void_p]),
    "hxf_op_prefill_attention_workspace_bytes": (C.c_int64, [C.c_int32, C.c_int32, C.c_int32,
                                                             C.POINTER(C.c_int32)]),
    "hxf_op_prefill_attention": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p, C.c_int32,
                                           C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                           C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_void_p,
                                           C.c_int64, C.c_void_p]),
    "hxf_op_argmax": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_void_p]),
    "hxf_op_copy": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p]),
    "hxf_op_read": (C.c_int, [C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p]),
}

EXPORTED = tuple(_SIGS)


def lib():
    """Load libhxf.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2505_05286_amd.build`")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _i32(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(C.POINTER(C.c_int32))


def model_cfg(shape, max_context):
    return ModelCfg(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                    shape.ffn_dim, shape.vocab, shape.page_size, int(max_context), shape.rms_eps, shape.rope_base)


def sched_cfg(n_blocks, max_seqs, chunk_tokens, cost_ps, iter_ps, policy=POLICY_PQ, clock=CLOCK_VIRTUAL,
              executor=EXEC_HIP):
    s = SchedCfg()
    s.n_blocks, s.max_seqs, s.chunk_tokens = int(n_blocks), int(max_seqs), int(chunk_tokens)
    s.policy, s.clock, s.executor = policy, clock, executor
    for i in range(4):
        s.cost_ps[i] = int(cost_ps[i])
    # (i0, i1, i2, i3[, i4]): without i4 a decode row costs what a prefill token does
    it = tuple(iter_ps) if len(iter_ps) == 5 else tuple(iter_ps) + (iter_ps[1],)
    for i in range(5):
        s.iter_ps[i] = int(it[i])
    return s


def kv_pool_bytes(mcfg, n_blocks):
    return lib().hxf_kv_pool_bytes(C.byref(mcfg), int(n_blocks))


def workspace_bytes(mcfg, scfg):
    n = lib().hxf_workspace_bytes(C.byref(mcfg), C.byref(scfg))
    if n < 0:
        raise HxfError(EINVAL, "invalid configuration")
    return n


class Instance:
    """One serving instance (hxf_instance*)."""

    def __init__(self, mcfg, scfg):
        self.L = lib()
        self.mcfg, self.scfg = mcfg, scfg
        h = C.c_void_p()
        rc = self.L.hxf_create(C.byref(mcfg), C.byref(scfg), C.byref(h))
        if rc != OK:
            raise HxfError(rc, "hxf_create rejected the configuration")
        self.h = h
        self._keep = []

    def close(self):
        if self.h:
            self.L.hxf_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, rc, what):
        if rc < 0:
            raise HxfError(rc, f"{what}: {self.L.hxf_last_error(self.h).decode()}")
        return rc

    def bind(self, embed, final_norm, lm_head, layers, kv_pool, kv_pool_bytes, workspace, workspace_bytes, stream=0):
        arr = (LayerWeights * len(layers))()
        for i, lw in enumerate(layers):
            for k in ("attn_norm", "wqkv", "wo", "ffn_norm", "w_gate", "w_up", "w_down"):
                setattr(arr[i], k, int(lw[k]))
        b = DeviceBuffers(int(embed), int(final_norm), int(lm_head), arr, int(kv_pool), int(kv_pool_bytes),
                          int(workspace), int(workspace_bytes))
        self._check(self.L.hxf_bind(self.h, C.byref(b), C.c_void_p(int(stream))), "hxf_bind")

    def submit(self, now, workflow_id, stage_index, wf_arrival, wf_slo, prompt, max_new, parent=0, retain=False,
               rest=(), forced=None, cost_sum=None, n_instances=1):
        """Queue one stage request.  With cost_sum (the cost coefficients of n_instances
        instances summed) the SLO budget uses their average costs (hxf_submit_shared)."""
        p, pp = _i32(prompt)
        rs = (StageShape * max(1, len(rest)))()
        for i, (li, lo) in enumerate(rest):
            rs[i].l_in, rs[i].l_out = int(li), int(lo)
        q = StageReq()
        q.workflow_id, q.stage_index, q.prompt_len = int(workflow_id), int(stage_index), len(p)
        q.workflow_arrival_us, q.workflow_slo_us = int(wf_arrival), int(wf_slo)
        q.prompt_ids, q.max_new_tokens, q.retain_kv = pp, int(max_new), 1 if retain else 0
        q.parent_id, q.rest, q.n_rest = int(parent), rs, len(rest)
        if forced is not None:
            f, fp = _i32(forced)
            q.n_forced, q.forced_ids = len(f), fp
        out = C.c_uint64()
        if cost_sum is None:
            self._check(self.L.hxf_submit(self.h, C.byref(q), int(now), C.byref(out)), "hxf_submit")
        else:
            cs = (C.c_int64 * 4)(*[int(c) for c in cost_sum])
            self._check(self.L.hxf_submit_shared(self.h, C.byref(q), int(now), cs, int(n_instances), C.byref(out)),
                        "hxf_submit_shared")
        return out.value

    def queue_cost(self):
        """t_queue of Section 4.1: summed t_comp of the unfinished requests (us)."""
        v = C.c_int64()
        self._check(self.L.hxf_queue_cost(self.h, C.byref(v)), "hxf_queue_cost")
        return v.value

    def request_cost(self, l_in, l_out):
        """t_comp of Section 4.1 on this instance's cost model (us)."""
        v = C.c_int64()
        self._check(self.L.hxf_request_cost(self.h, int(l_in), int(l_out), C.byref(v)), "hxf_request_cost")
        return v.value

    def step(self, now):
        info = StepInfo()
        rc = self._check(self.L.hxf_step(self.h, int(now), C.byref(info)), "hxf_step")
        return rc, info.as_dict()

    def drain(self, cap=4096):
        buf = (Completion * cap)()
        n = C.c_int32()
        self._check(self.L.hxf_drain(self.h, buf, cap, C.byref(n)), "hxf_drain")
        return [buf[i].as_dict() for i in range(n.value)]

    def tokens(self, rid, cap=1 << 16):
        buf = (C.c_int32 * cap)()
        n = C.c_int32()
        self._check(self.L.hxf_completion_tokens(self.h, int(rid), buf, cap, C.byref(n)), "hxf_completion_tokens")
        return list(buf[:n.value])

    def release(self, rid):
        self._check(self.L.hxf_release(self.h, int(rid)), "hxf_release")

    def cancel(self, rid):
        self._check(self.L.hxf_cancel(self.h, int(rid)), "hxf_cancel")

    def queue_order(self, cap=1 << 16):
        buf = (C.c_uint64 * cap)()
        n = C.c_int32()
        self._check(self.L.hxf_queue_order(self.h, buf, cap, C.byref(n)), "hxf_queue_order")
        return list(buf[:n.value])

    def block_table(self, rid, cap=1 << 16):
        buf = (C.c_int32 * cap)()
        n = C.c_int32()
        self._check(self.L.hxf_block_table(self.h, int(rid), buf, cap, C.byref(n)), "hxf_block_table")
        return list(buf[:n.value])

    def request_state(self, rid):
        s = RequestState()
        self._check(self.L.hxf_request_state_get(self.h, int(rid), C.byref(s)), "hxf_request_state_get")
        return {k: getattr(s, k) for k, _ in s._fields_}

    def last_batch(self, cap=4096):
        ids = (C.c_uint64 * cap)()
        adm = (C.c_uint64 * cap)()
        n, na = C.c_int32(), C.c_int32()
        self._check(self.L.hxf_last_batch(self.h, ids, cap, C.byref(n), adm, cap, C.byref(na)), "hxf_last_batch")
        return list(ids[:n.value]), list(adm[:na.value])

    def last_logits(self, rid):
        v = self.mcfg.vocab
        out = np.empty(v, np.float32)
        self._check(self.L.hxf_last_logits(self.h, int(rid), out.ctypes.data_as(C.POINTER(C.c_float)), v),
                    "hxf_last_logits")
        return out

    def profile_enable(self, on=True):
        self._check(self.L.hxf_profile_enable(self.h, 1 if on else 0), "hxf_profile_enable")

    def profile(self):
        p = Profile()
        self._check(self.L.hxf_profile_get(self.h, C.byref(p)), "hxf_profile_get")
        out = {}
        for k, _ in p._fields_:
            v = getattr(p, k)
            out[k] = dict(zip(PROF_GEMMS, list(v))) if k.startswith("gemm_") else v
        return out


# ------------------------------------------------------------------ ops
def wb_select(t_comp_us, t_queue_us, alpha, beta):
    """Workload-balanced dispatch (Section 4.1): index of the best-scoring instance."""
    n = len(t_comp_us)
    c = (C.c_int64 * n)(*[int(v) for v in t_comp_us])
    q = (C.c_int64 * n)(*[int(v) for v in t_queue_us])
    out = C.c_int32()
    rc = lib().hxf_wb_select(n, c, q, float(alpha), float(beta), C.byref(out))
    if rc != OK:
        raise HxfError(rc, "hxf_wb_select: bad arguments")
    return out.value


def ttest_greater(x_new, x_ref):
    """One-sided Welch t-test of Section 4.3; returns (t, dof, p)."""
    a = np.ascontiguousarray(x_new, dtype=np.float64)
    b = np.ascontiguousarray(x_ref, dtype=np.float64)
    t, dof, p = C.c_double(), C.c_double(), C.c_double()
    rc = lib().hxf_ttest_greater(a.ctypes.data_as(C.POINTER(C.c_double)), len(a),
                                 b.ctypes.data_as(C.POINTER(C.c_double)), len(b), C.byref(t), C.byref(dof), C.byref(p))
    if rc != OK:
        raise HxfError(rc, "hxf_ttest_greater: bad arguments")
    return t.value, dof.value, p.value


def _op(rc, what):
    if rc != OK:
        raise HxfError(rc, what)


def op_gemm_workspace_bytes(M, N, K):
    return lib().hxf_op_gemm_workspace_bytes(M, N, K)


def op_gemm(A, lda, B, B2, Cp, ldc, M, N, K, epi, ws=0, ws_bytes=0, stream=0):
    _op(lib().hxf_op_gemm(A, lda, B, B2 or None, Cp, ldc, M, N, K, epi, ws or None, ws_bytes, stream or None),
        "hxf_op_gemm")


GEMM_NOALLOC_MAX_BYTES = 16 << 20


def op_gemm_noalloc(A, lda, B, B2, Cp, ldc, M, N, K, epi, stream=0):
    """hxf_op_gemm with its split-K partials in the library's own device array."""
    _op(lib().hxf_op_gemm_noalloc(A, lda, B, B2 or None, Cp, ldc, M, N, K, epi, stream or None),
        "hxf_op_gemm_noalloc")


def packed_weight_bytes(N, K):
    return lib().hxf_packed_weight_bytes(N, K)


def op_pack_weight(W, N, K, out, stream=0):
    _op(lib().hxf_op_pack_weight(W, N, K, out, stream or None), "hxf_op_pack_weight")


def op_rmsnorm(x, rows, g, out, n_rows, d, eps, stream=0):
    _op(lib().hxf_op_rmsnorm(x, rows or None, g, out, n_rows, d, eps, stream or None), "hxf_op_rmsnorm")


def op_embed_rmsnorm(ids, E, g, resid, out, T, d, eps, stream=0):
    _op(lib().hxf_op_embed_rmsnorm(ids, E, g, resid, out, T, d, eps, stream or None), "hxf_op_embed_rmsnorm")


def op_rope_table(dst, max_pos, dh, base, stream=0):
    _op(lib().hxf_op_rope_table(dst, max_pos, dh, base, stream or None), "hxf_op_rope_table")


def op_rope_kv_write(qkv, pos, slot, table, k_pool, v_pool, n_blocks, T, Hq, Hkv, dh, stream=0):
    _op(lib().hxf_op_rope_kv_write(qkv, pos, slot, table, k_pool, v_pool, n_blocks, T, Hq, Hkv, dh, stream or None),
        "hxf_op_rope_kv_write")


def op_kv_scatter(k, v, slot, k_pool, v_pool, n_blocks, T, Hkv, dh, stream=0):
    _op(lib().hxf_op_kv_scatter(k, v, slot, k_pool, v_pool, n_blocks, T, Hkv, dh, stream or None),
        "hxf_op_kv_scatter")


def op_decode_attention_workspace_bytes(B, Hq, Hkv, dh, ctx, bt_host=None, bt_stride=0):
    """bt_host: the block table [B, bt_stride] on the host (enables shared-prefix grouping) or None."""
    c, cp = _i32(ctx)
    b, bp = _i32(bt_host) if bt_host is not None else (None, None)
    return lib().hxf_op_decode_attention_workspace_bytes(B, Hq, Hkv, dh, cp, bp, bt_stride)


DECODE_ITEM_WORDS = 24
DECODE_ROWS = 8


def decode_rows_narrow(G):
    """Rows of a one-tile decode item (16 query columns) for GQA group size G."""
    return max(1, min(DECODE_ROWS, 16 // G))


def decode_rows_wide(G):
    """Rows of a two-tile (wide) decode item (32 query columns)."""
    return max(1, min(DECODE_ROWS, 32 // G))


def op_decode_plan(B, Hq, Hkv, ctx, bt_host=None, bt_stride=0):
    """The decode-attention work list: (items int32 [n, 24], merges int32 [m, 4]).  An item is
    {kvh, t0, t1, n_rows, entry[8], part[8], pad[4]}; one-tile items come first, then the
    two-tile (wide) items."""
    c, cp = _i32(ctx)
    b, bp = _i32(bt_host) if bt_host is not None else (None, None)
    ni, nm = C.c_int32(0), C.c_int32(0)
    rc = lib().hxf_op_decode_plan(B, Hq, Hkv, cp, bp, bt_stride, None, 0, C.byref(ni), None, 0, C.byref(nm))
    if rc not in (OK, ENOMEM):
        raise HxfError(rc, "hxf_op_decode_plan")
    items = np.zeros((ni.value, DECODE_ITEM_WORDS), np.int32)
    merges = np.zeros((nm.value, 4), np.int32)
    _op(lib().hxf_op_decode_plan(B, Hq, Hkv, cp, bp, bt_stride, items.ctypes.data_as(C.POINTER(C.c_int32)),
                                 ni.value, C.byref(ni), merges.ctypes.data_as(C.POINTER(C.c_int32)), nm.value,
                                 C.byref(nm)), "hxf_op_decode_plan")
    return items, merges


def op_prefill_plan(Hq, Hkv, pos0, n):
    """The prefill-attention work list for chunks of n[s] queries from position pos0[s]:
    (items int32 [k, 8] {entry, kvh, q0, nq, t0, t1, part, pad} in launch order, merges int32
    [m, 8] {entry, kvh, q0, nq, part0, n_part, pad, pad})."""
    S = len(n)
    p, pp = _i32(pos0)
    c, cp = _i32(n)
    ni, nm = C.c_int32(0), C.c_int32(0)
    rc = lib().hxf_op_prefill_plan(S, Hq, Hkv, pp, cp, None, 0, C.byref(ni), None, 0, C.byref(nm))
    if rc not in (OK, ENOMEM):
        raise HxfError(rc, "hxf_op_prefill_plan")
    items = np.zeros((ni.value, 8), np.int32)
    merges = np.zeros((nm.value, 8), np.int32)
    _op(lib().hxf_op_prefill_plan(S, Hq, Hkv, pp, cp, items.ctypes.data_as(C.POINTER(C.c_int32)), ni.value,
                                  C.byref(ni), merges.ctypes.data_as(C.POINTER(C.c_int32)), nm.value, C.byref(nm)),
        "hxf_op_prefill_plan")
    return items, merges


def op_decode_attention(q, k_pool, v_pool, n_blocks, bt, bt_stride, ctx, out, B, Hq, Hkv, dh, ws, ws_bytes, stream=0,
                        bt_host=None):
    c, cp = _i32(ctx)
    b, bp = _i32(bt_host) if bt_host is not None else (None, None)
    _op(lib().hxf_op_decode_attention(q, k_pool, v_pool, n_blocks, bt, bt_stride, cp, bp, out, B, Hq, Hkv, dh, ws,
                                      ws_bytes, stream or None), "hxf_op_decode_attention")


def op_prefill_attention_workspace_bytes(S, Hq, Hkv, n):
    a, ap = _i32(n)
    return lib().hxf_op_prefill_attention_workspace_bytes(S, Hq, Hkv, ap)


def op_prefill_attention(q, k_pool, v_pool, n_blocks, bt, bt_stride, row0, pos0, n, out, S, Hq, Hkv, dh, ws,
                         ws_bytes, stream=0):
    r, rp = _i32(row0)
    p, pp = _i32(pos0)
    m, mp = _i32(n)
    _op(lib().hxf_op_prefill_attention(q, k_pool, v_pool, n_blocks, bt, bt_stride, rp, pp, mp, out, S, Hq, Hkv, dh,
                                       ws, ws_bytes, stream or None), "hxf_op_prefill_attention")


def op_argmax(logits, out, R, V, stream=0):
    _op(lib().hxf_op_argmax(logits, out, R, V, stream or None), "hxf_op_argmax")


def op_copy(src, dst, nbytes, stream=0):
    _op(lib().hxf_op_copy(src, dst, nbytes, stream or None), "hxf_op_copy")


READ_SINK_WORDS = 4096 * 256


def op_read(src, nbytes, sink, stream=0):
    """HBM read probe: sink (READ_SINK_WORDS uint32) gets one XOR word per thread."""
    _op(lib().hxf_op_read(src, nbytes, sink, stream or None), "hxf_op_read")
