"""hxf_op_gemm_noalloc (split-K partials in the library's own device array, no
workspace) against hxf_op_gemm (partials in a caller workspace) through the C
ABI: the same kernels and plans, so the outputs must be bit-identical.  Two
calls in a row on the array, the second with a smaller input, then a shape
whose partials exceed the array, which must be refused with nothing written."""
import numpy as np
import pytest

from paper_2505_05286_amd import hxf

from .gpu_util import dev_packed, log, rand_bf16, torch

pytestmark = pytest.mark.gpu


def _operands(rng, M, N, K, epi):
    t = torch()
    rows = N // 2 if epi == hxf.EPI_SWIGLU else N
    a_bits, _ = rand_bf16(rng, (M, K), 0.5)
    A = t.from_numpy(a_bits.view(np.int16)).to("cuda:0")
    Bs = [dev_packed(rand_bf16(rng, (rows, K), 0.05)[0]) for _ in range(2 if epi == hxf.EPI_SWIGLU else 1)]
    f32 = epi in (hxf.EPI_RESID, hxf.EPI_F32)
    C0 = (t.from_numpy(rng.standard_normal((M, rows)).astype(np.float32)).to("cuda:0") if f32
          else t.zeros(M * rows, dtype=t.int16, device="cuda:0"))
    return A, Bs, C0, rows


def _both(M, N, K, epi, seed):
    """(noalloc output, workspace output) for one GEMM on the same operands."""
    t = torch()
    rng = np.random.default_rng(seed)
    A, Bs, C0, rows = _operands(rng, M, N, K, epi)
    B2 = Bs[-1].data_ptr() if len(Bs) > 1 else 0
    got = C0.clone()
    hxf.op_gemm_noalloc(A.data_ptr(), K, Bs[0].data_ptr(), B2, got.data_ptr(), rows, M, N, K, epi)
    ref = C0.clone()
    wsn = hxf.op_gemm_workspace_bytes(M, N, K)
    ws = t.empty(max(wsn, 256), dtype=t.uint8, device="cuda:0")
    hxf.op_gemm(A.data_ptr(), K, Bs[0].data_ptr(), B2, ref.data_ptr(), rows, M, N, K, epi, ws.data_ptr(), wsn)
    t.cuda.synchronize()
    return got.cpu().numpy(), ref.cpu().numpy(), wsn


@pytest.mark.parametrize("first,second", [
    ((64, 4096, 4096, "RESID"), (16, 4096, 4096, "RESID")),        # 8 splits, then a smaller M
    ((128, 4096, 4096, "F32"), (40, 6144, 4096, "BF16")),          # 16 MiB of partials, then 5 splits
    ((96, 4096, 14336, "RESID"), (33, 2 * 1024, 4096, "SWIGLU")),  # ragged M, then SwiGLU
])
def test_noalloc_matches_the_workspace_entry_point_twice(first, second):
    for k, (M, N, K, e) in enumerate((first, second)):
        epi = getattr(hxf, f"EPI_{e}")
        log(f"noalloc gemm call {k}: M={M} N={N} K={K} {e}")
        got, ref, wsn = _both(M, N, K, epi, seed=M * 7 + k)
        assert wsn <= hxf.GEMM_NOALLOC_MAX_BYTES
        np.testing.assert_array_equal(got, ref)


def test_noalloc_refuses_partials_beyond_its_array():
    t = torch()
    M, N, K = 256, 4096, 14336                      # a down projection at 256 rows: split-K partials of 32 MiB
    assert hxf.op_gemm_workspace_bytes(M, N, K) > hxf.GEMM_NOALLOC_MAX_BYTES
    rng = np.random.default_rng(3)
    A, Bs, C0, rows = _operands(rng, M, N, K, hxf.EPI_RESID)
    out = C0.clone()
    with pytest.raises(hxf.HxfError) as e:
        hxf.op_gemm_noalloc(A.data_ptr(), K, Bs[0].data_ptr(), 0, out.data_ptr(), rows, M, N, K, hxf.EPI_RESID)
    assert e.value.code == hxf.ENOMEM
    t.cuda.synchronize()
    assert t.equal(out, C0)
    # a smaller call afterwards still works
    got, ref, _ = _both(64, 4096, 4096, hxf.EPI_RESID, seed=9)
    np.testing.assert_array_equal(got, ref)
