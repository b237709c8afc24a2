"""The C ABI: every function declared in include/*.h is exported by libhxf.so,
the binding declares the same set, and configuration checks run without a GPU."""
import ctypes
import glob
import os
import re

import pytest

import synth
from paper_2505_05286_amd import hxf

from ._lib import ensure_built

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        src = open(h).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        for m in re.finditer(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(hxf_[a-z_0-9]+)\s*\(", src, flags=re.M):
            names.add(m.group(1))
    return names


def test_every_declared_symbol_is_exported_and_bound():
    path = ensure_built()
    lib = ctypes.CDLL(path)
    names = declared()
    assert len(names) >= 30
    for n in sorted(names):
        assert hasattr(lib, n), n
    assert names == set(hxf.EXPORTED)


def test_config_validation_without_gpu():
    ensure_built()
    sh = synth.model_shape("llama8b")
    m = hxf.model_cfg(sh, 9280)
    s = hxf.sched_cfg(120_000, 256, 2048, (0,) * 4, (0,) * 4)
    ws = hxf.workspace_bytes(m, s)
    assert 0 < ws < 4 << 30
    assert hxf.kv_pool_bytes(m, 1) == 32 * 2 * 8 * 16 * 128 * 2   # 2 MiB per page across layers
    bad = hxf.model_cfg(sh.with_layers(2), 9280)
    bad.page_size = 32
    with pytest.raises(hxf.HxfError):
        hxf.Instance(bad, s)
    inst = hxf.Instance(m, s)   # HIP executor, not bound: stepping must refuse
    with pytest.raises(hxf.HxfError) as e:
        inst.step(0)
    assert e.value.code == hxf.ESTATE


def test_ops_reject_bad_arguments_without_launching():
    ensure_built()
    with pytest.raises(hxf.HxfError) as e:
        hxf.op_gemm(1, 7, 1, 0, 1, 8, 8, 8, 7, hxf.EPI_BF16)    # K % 8 != 0
    assert e.value.code == hxf.EINVAL
    with pytest.raises(hxf.HxfError):
        hxf.op_decode_attention(1, 1, 1, 8, 1, 1, [0], 1, 1, 4, 3, 128, 1, 1)   # Hq % Hkv


def test_iteration_trace_log(tmp_path, monkeypatch):
    """HXF_TRACE: one JSON line per iteration, matching what hxf_step returned."""
    import json

    import numpy as np
    ensure_built()
    path = tmp_path / "trace.jsonl"
    monkeypatch.setenv("HXF_TRACE", str(path))
    shape = synth.ModelShape("sched", 1, 64, 1, 1, 64, 64, 2048, 0)
    inst = hxf.Instance(hxf.model_cfg(shape, 4096),
                        hxf.sched_cfg(64, 4, 32, (1000 * 10**6, 10**6, 0, 10**6), (500 * 10**6, 10**6, 0, 0),
                                      executor=hxf.EXEC_NULL))
    ids = [inst.submit(0, k, 0, 0, 10**9, np.arange(20 + k, dtype=np.int32), 3) for k in range(3)]
    infos, now = [], 0
    while True:
        st, info = inst.step(now)
        if st == hxf.IDLE:
            break
        infos.append((now, info))
        now += info["t_iter_us"]
    inst.close()
    lines = [json.loads(l) for l in open(path)]
    assert len(lines) == len(infos) > 1
    for (t, info), rec in zip(infos, lines):
        assert rec["now_us"] == t
        for k in ("iteration", "t_iter_us", "n_tokens", "n_decode", "n_prefill_tokens", "n_logit_rows",
                  "sum_decode_ctx", "prefill_attn", "n_finished", "free_blocks"):
            assert rec[k] == info[k], k
    assert sorted(i for rec in lines for i in rec["admitted"]) == sorted(ids)
