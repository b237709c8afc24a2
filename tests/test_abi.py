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
