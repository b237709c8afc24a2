"""Helpers shared by the GPU tests: bf16 tensors in HBM, read-back, tolerances."""
import sys

import numpy as np

import synth


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def torch():
    import torch as t
    return t


def dev_bits(bits):
    """uint16 bf16 bits (numpy) -> int16 tensor on cuda:0."""
    t = torch()
    return t.from_numpy(np.ascontiguousarray(bits, np.uint16).view(np.int16)).to("cuda:0")


def dev_packed(bits):
    """uint16 bf16 bits [N, K] (numpy) -> the packed weight layout on cuda:0."""
    from paper_2505_05286_amd import hxf
    t = torch()
    n, k = bits.shape
    src = dev_bits(bits)
    out = t.empty(hxf.packed_weight_bytes(n, k) // 2, dtype=t.int16, device="cuda:0")
    hxf.op_pack_weight(src.data_ptr(), n, k, out.data_ptr())
    t.cuda.synchronize()
    return out


def host_f64(tensor_i16):
    """int16 bf16-bit tensor -> float64 numpy."""
    b = tensor_i16.detach().cpu().numpy().view(np.uint16)
    return synth.bf16_bits_to_f32(b).astype(np.float64)


def rand_bf16(rng, shape, scale=1.0):
    """Random bf16 bits and their exact float64 values."""
    x = (rng.standard_normal(shape) * scale).astype(np.float32)
    b = synth.f32_to_bf16_bits(x)
    return b.reshape(shape), synth.bf16_bits_to_f32(b).astype(np.float64).reshape(shape)


def empty_i16(n):
    t = torch()
    return t.empty(n, dtype=t.int16, device="cuda:0")


def i32(a):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(a, np.int32)).to("cuda:0")


def rel_max_err(got, ref):
    """max |got - ref| / max |ref| (the logits metric, per row when 2-D)."""
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    if got.ndim == 1:
        return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-30))
    return max(rel_max_err(g, r) for g, r in zip(got, ref))


# Attention parity bound, relative to the output's own scale: for every (row, head),
# max_d |got - ref| / max_d |ref| <= ATTN_TOL.  The kernels take bf16 Q, K, V exactly,
# accumulate in fp32, round the probabilities to bf16 for the PV product (relative
# error <= 2^-9 per probability, independent signs, so about 2^-9/sqrt(3) of the
# output's RMS) and round the output to bf16 (<= 2^-9 of each element): a few 1e-3
# of max|ref| at worst.  One mis-addressed 16-token page at the workloads' context
# lengths moves a head's output by several percent of max|ref|
# (tests/test_attention_tolerance.py checks both on the CPU).
ATTN_TOL = 1e-2


def attn_rel_err(got, ref):
    """Largest over (row, head) of max_d |got - ref| / max_d |ref|; got, ref [n, H, dh]."""
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    num = np.max(np.abs(got - ref), axis=-1)
    den = np.maximum(np.max(np.abs(ref), axis=-1), 1e-30)
    return float(np.max(num / den))


def assert_attn_close(got, ref, what=""):
    err = attn_rel_err(got, ref)
    assert err <= ATTN_TOL, f"{what}: attention rel err {err:.3e} > {ATTN_TOL}"
    return err
