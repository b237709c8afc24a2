"""Kernel-level parity through the C ABI (include/hxf_ops.h) against the oracle.

Inputs are seeded bf16 values; references are float64 (oracle functions, or a
plain matmul for the GEMM).  Tolerances follow from bf16 storage of the
outputs (relative rounding 2^-9) and of the attention probabilities fed to
the PV product.
"""
import numpy as np
import pytest

import synth
from oracle import model as M
from oracle import paged as P
from paper_2505_05286_amd import hxf

from .gpu_util import assert_attn_close, dev_bits, dev_packed, empty_i16, host_f64, i32, log, rand_bf16, torch

pytestmark = pytest.mark.gpu


def _gemm_case(M_, N, K, epi, seed, rows=None):
    """rows: compare only these output rows (the reference is computed for them alone)."""
    t = torch()
    rng = np.random.default_rng(seed)
    ab, af = rand_bf16(rng, (M_, K))
    bb, bf = rand_bf16(rng, (N if epi != hxf.EPI_SWIGLU else N // 2, K), 0.05)
    A, B = dev_bits(ab), dev_packed(bb)
    B2 = None
    if epi == hxf.EPI_SWIGLU:
        b2b, b2f = rand_bf16(rng, (N // 2, K), 0.05)
        B2 = dev_packed(b2b)
    ws_n = hxf.op_gemm_workspace_bytes(M_, N, K)
    ws = t.empty(max(ws_n, 256), dtype=t.uint8, device="cuda:0")
    n_out = N // 2 if epi == hxf.EPI_SWIGLU else N
    if epi in (hxf.EPI_BF16, hxf.EPI_SWIGLU):
        C = empty_i16(M_ * n_out)
    else:
        base = rng.standard_normal((M_, n_out)).astype(np.float32)
        C = t.from_numpy(base.copy()).to("cuda:0") if epi == hxf.EPI_RESID else t.empty(M_ * n_out, dtype=t.float32,
                                                                                         device="cuda:0")
    log(f"gemm M={M_} N={N} K={K} epi={epi} ws={ws_n}")
    hxf.op_gemm(A.data_ptr(), K, B.data_ptr(), B2.data_ptr() if B2 is not None else 0, C.data_ptr(), n_out, M_, N, K,
                epi, ws.data_ptr(), ws.numel())
    t.cuda.synchronize()
    sel = np.arange(M_) if rows is None else np.asarray(rows)
    a_s = af[sel]
    if epi == hxf.EPI_SWIGLU:
        ref = M.silu(a_s @ bf.T) * (a_s @ b2f.T)
        got = host_f64(C).reshape(M_, n_out)[sel]
    elif epi == hxf.EPI_BF16:
        ref = a_s @ bf.T
        got = host_f64(C).reshape(M_, n_out)[sel]
    else:
        ref = a_s @ bf.T + (base[sel].astype(np.float64) if epi == hxf.EPI_RESID else 0.0)
        got = C.cpu().numpy().astype(np.float64).reshape(M_, n_out)[sel]
    scale = np.max(np.abs(ref))
    rtol = 2 ** -7 if epi in (hxf.EPI_BF16, hxf.EPI_SWIGLU) else 1e-5
    np.testing.assert_allclose(got, ref, rtol=rtol, atol=2e-4 * scale)


@pytest.mark.parametrize("M_,N,K", [(1, 64, 64), (37, 200, 136), (64, 6144, 4096), (48, 1000, 4096),
                                    (64, 4096, 14336), (3, 520, 1384), (16, 4096, 4096), (64, 256, 8192),
                                    (32, 136, 160), (17, 8192, 1024), (65, 4096, 4096),
                                    (256, 1024, 688), (300, 1000, 688),
                                    (2080, 384, 512), (600, 1000, 688), (2080, 6144, 1024), (1031, 4096, 1384),
                                    (2048, 4096, 256), (2080, 4096, 264), (2048, 6144, 96), (200, 32768, 512),
                                    (96, 20000, 256), (250, 6144, 1024), (2300, 6144, 72), (960, 11008, 72),
                                    (64, 10240, 8192), (64, 8192, 28672), (2080, 10240, 1024),
                                    (256, 6144, 4096), (256, 4096, 14336), (512, 4096, 4096), (129, 4096, 4096),
                                    (500, 1000, 4096), (384, 6144, 1000), (200, 8192, 2056),
                                    (600, 256, 8), (1030, 320, 24)])
@pytest.mark.parametrize("epi", [hxf.EPI_BF16, hxf.EPI_RESID, hxf.EPI_F32])
def test_gemm(M_, N, K, epi):
    _gemm_case(M_, N, K, epi, seed=M_ * 7 + N + K + epi)


@pytest.mark.parametrize("M_,N,K", [(5, 64, 256), (64, 2 * 688, 256), (33, 2 * 688, 2048), (64, 2 * 14336, 4096),
                                    (20, 2 * 4096, 4096), (64, 2 * 96, 8192), (2080, 2 * 4096, 200),
                                    (300, 2 * 1376, 512), (128, 2 * 14336, 4096), (700, 2 * 688, 256),
                                    (2080, 2 * 2080, 512), (1040, 2 * 5504, 72), (520, 2 * 3584, 72),
                                    (64, 2 * 28672, 8192), (1024, 2 * 5632, 1000), (2080, 2 * 7168, 1000),
                                    (256, 2 * 14336, 4096), (512, 2 * 14336, 4096), (200, 2 * 1376, 1000)])
def test_gemm_swiglu(M_, N, K):
    _gemm_case(M_, N, K, hxf.EPI_SWIGLU, seed=M_ + N + K)


@pytest.mark.parametrize("name,M_,N,K,epi", [
    ("8B qkv", 2080, 6144, 4096, hxf.EPI_BF16), ("8B o", 2080, 4096, 4096, hxf.EPI_RESID),
    ("8B gate/up", 2080, 2 * 14336, 4096, hxf.EPI_SWIGLU), ("8B down", 2080, 4096, 14336, hxf.EPI_RESID),
    ("70B qkv", 2080, 10240, 8192, hxf.EPI_BF16), ("70B down", 2080, 8192, 28672, hxf.EPI_RESID),
    ("8B lm head", 64, 128256, 4096, hxf.EPI_F32)])
def test_gemm_full_size_sampled(name, M_, N, K, epi):
    """Mixed-iteration projections at their full sizes (2048 prefill + 32 decode rows) in the
    launch configuration the forward uses; the reference is computed for sampled rows: the
    first and last of every 32-row tile boundary region and the ragged tail."""
    rows = sorted(r for r in set(list(range(0, M_, 97)) + [31, 32, 255, 256, M_ - 33, M_ - 32, M_ - 1]) if r < M_)
    log(f"gemm full size {name}: {len(rows)} sampled rows")
    _gemm_case(M_, N, K, epi, seed=M_ + N + K, rows=rows)


def _unpack_rows(packed_i16, M_, K):
    """A packed-layout bf16 matrix (16 x 32 tiles, [k%32 / 8][r%16][k%8] inside) -> [M_, K] bits."""
    kt = -(-K // 32)
    m16 = -(-M_ // 16) * 16
    a = packed_i16.detach().cpu().numpy().view(np.uint16)[:m16 * kt * 32]
    return a.reshape(m16 // 16, kt, 4, 16, 8).transpose(0, 3, 1, 2, 4).reshape(m16, kt * 32)[:M_, :K]


@pytest.mark.parametrize("M_,N,K,epi", [(2080, 6144, 4096, hxf.EPI_BF16), (2080, 4096, 4096, hxf.EPI_RESID),
                                        (1031, 1000, 1408, hxf.EPI_F32), (600, 4096, 14336, hxf.EPI_RESID),
                                        (513, 320, 32, hxf.EPI_BF16), (2080, 2 * 14336, 4096, hxf.EPI_SWIGLU),
                                        (700, 2 * 1376, 512, hxf.EPI_SWIGLU), (64, 6144, 4096, hxf.EPI_BF16),
                                        (64, 4096, 14336, hxf.EPI_RESID), (17, 1000, 1024, hxf.EPI_F32),
                                        (64, 2 * 14336, 4096, hxf.EPI_SWIGLU), (33, 2 * 2048, 4096, hxf.EPI_SWIGLU),
                                        (256, 6144, 4096, hxf.EPI_BF16), (256, 4096, 14336, hxf.EPI_RESID),
                                        (256, 2 * 14336, 4096, hxf.EPI_SWIGLU), (129, 4096, 4096, hxf.EPI_F32),
                                        (96, 20000, 256, hxf.EPI_F32)])
def test_gemm_packed_activations(M_, N, K, epi):
    """GEMMs reading the activations in the packed tile layout (the streaming kernel at decode
    sizes, the big-tile kernel with or without split K above) give the row-major call's result
    bit for bit; a SwiGLU output written packed holds the same values."""
    t = torch()
    rng = np.random.default_rng(M_ + N + K)
    ab, _ = rand_bf16(rng, (M_, K))
    rows = N // 2 if epi == hxf.EPI_SWIGLU else N
    A = dev_bits(ab)
    Ap = dev_packed(ab)                        # the activations through the weight packing kernel
    Bs = [dev_packed(rand_bf16(rng, (rows, K), 0.05)[0]) for _ in range(2 if epi == hxf.EPI_SWIGLU else 1)]
    B2 = Bs[-1].data_ptr() if len(Bs) > 1 else 0
    f32 = epi in (hxf.EPI_RESID, hxf.EPI_F32)
    base = rng.standard_normal((M_, rows)).astype(np.float32)

    def out():
        return (t.from_numpy(base.copy()).to("cuda:0") if f32 else t.zeros(M_ * rows, dtype=t.int16, device="cuda:0"))
    log(f"gemm packed activations M={M_} N={N} K={K} epi={epi}")
    ref, got = out(), out()
    wsn = hxf.op_gemm_workspace_bytes(M_, N, K)
    ws = t.empty(max(wsn, 256), dtype=t.uint8, device="cuda:0")
    hxf.op_gemm(A.data_ptr(), K, Bs[0].data_ptr(), B2, ref.data_ptr(), rows, M_, N, K, epi, ws.data_ptr(), wsn)
    hxf.op_gemm(Ap.data_ptr(), 0, Bs[0].data_ptr(), B2, got.data_ptr(), rows, M_, N, K, epi | hxf.GEMM_A_PACKED,
                ws.data_ptr(), wsn)
    t.cuda.synchronize()
    assert t.equal(ref, got)
    if epi == hxf.EPI_SWIGLU:
        cp = t.zeros(-(-M_ // 16) * 16 * rows, dtype=t.int16, device="cuda:0")
        hxf.op_gemm(Ap.data_ptr(), 0, Bs[0].data_ptr(), B2, cp.data_ptr(), 0, M_, N, K,
                    epi | hxf.GEMM_A_PACKED | hxf.GEMM_C_PACKED, ws.data_ptr(), wsn)
        t.cuda.synchronize()
        np.testing.assert_array_equal(_unpack_rows(cp, M_, rows), ref.cpu().numpy().view(np.uint16).reshape(M_, rows))


def test_gemm_packed_flags_refused_off_their_shapes():
    """The layout flags need K % 32 == 0 (packed activations), SwiGLU with F % 32 == 0 (packed output)."""
    for M_, N, K, flags in ((64, 256, 72, hxf.EPI_BF16 | hxf.GEMM_A_PACKED),
                            (1024, 256, 72, hxf.EPI_BF16 | hxf.GEMM_A_PACKED),
                            (64, 2 * 688, 256, hxf.EPI_SWIGLU | hxf.GEMM_A_PACKED),
                            (1024, 256, 256, hxf.EPI_BF16 | hxf.GEMM_C_PACKED),
                            (1024, 2 * 688, 256, hxf.EPI_SWIGLU | hxf.GEMM_C_PACKED),
                            (1024, 256, 256, hxf.EPI_BF16 | 0x400)):
        with pytest.raises(hxf.HxfError) as e:
            hxf.op_gemm(1, K, 1, 1, 1, N, M_, N, K, flags)
        assert e.value.code == hxf.EINVAL


@pytest.mark.parametrize("M_", [64, 256])
def test_gemm_split_repeatable(M_):
    """Repeated split-K calls on one workspace give bit-identical results (the weight-
    streaming kernel at 64 rows, the big-tile kernel at 256)."""
    t = torch()
    rng = np.random.default_rng(77)
    N, K = 6144, 4096
    ab, _ = rand_bf16(rng, (M_, K))
    bb, _ = rand_bf16(rng, (N, K), 0.05)
    A, B = dev_bits(ab), dev_packed(bb)
    ws = t.empty(hxf.op_gemm_workspace_bytes(M_, N, K), dtype=t.uint8, device="cuda:0")
    outs = []
    for _ in range(3):
        C = t.empty(M_ * N, dtype=t.float32, device="cuda:0")
        hxf.op_gemm(A.data_ptr(), K, B.data_ptr(), 0, C.data_ptr(), N, M_, N, K, hxf.EPI_F32, ws.data_ptr(), ws.numel())
        outs.append(C)
    t.cuda.synchronize()
    assert t.equal(outs[0], outs[1]) and t.equal(outs[0], outs[2])


# rows // 2 + 1 rows are normed: up to 256 one workgroup per row, above that one wavefront per
# row for d / 256 in {4, 8, 16, 20, 24, 32} (3072: the per-workgroup kernel at 301 rows)
@pytest.mark.parametrize("d,rows", [(256, 7), (4096, 64), (5120, 33), (4096, 600), (5120, 520), (8192, 1040),
                                    (1024, 1000), (3072, 600)])
def test_rmsnorm_and_embed(d, rows):
    t = torch()
    rng = np.random.default_rng(d + rows)
    x = (rng.standard_normal((rows, d)) * 3).astype(np.float32)
    gb, gf = rand_bf16(rng, d)
    xs = t.from_numpy(x).to("cuda:0")
    G = dev_bits(gb)
    sel = rng.permutation(rows)[: rows // 2 + 1].astype(np.int32)
    out = empty_i16(len(sel) * d)
    sel_d = i32(sel)
    hxf.op_rmsnorm(xs.data_ptr(), sel_d.data_ptr(), G.data_ptr(), out.data_ptr(), len(sel), d, 1e-5)
    t.cuda.synchronize()
    ref = M.rmsnorm(x[sel].astype(np.float64), gf, 1e-5)
    np.testing.assert_allclose(host_f64(out).reshape(len(sel), d), ref, rtol=2 ** -7, atol=1e-6)
    # embedding gather + norm
    V = 300
    eb, ef = rand_bf16(rng, (V, d), 0.02)
    ids = rng.integers(0, V, rows).astype(np.int32)
    resid = t.empty(rows * d, dtype=t.float32, device="cuda:0")
    out2 = empty_i16(rows * d)
    ids_d, E = i32(ids), dev_bits(eb)
    hxf.op_embed_rmsnorm(ids_d.data_ptr(), E.data_ptr(), G.data_ptr(), resid.data_ptr(), out2.data_ptr(), rows, d,
                         1e-5)
    t.cuda.synchronize()
    np.testing.assert_array_equal(resid.cpu().numpy().reshape(rows, d), ef[ids].astype(np.float32))
    np.testing.assert_allclose(host_f64(out2).reshape(rows, d), M.rmsnorm(ef[ids], gf, 1e-5), rtol=2 ** -7,
                               atol=1e-6)


def _make_pools(nb, hkv, dh):
    t = torch()
    kp = t.zeros(nb * hkv * 16 * dh, dtype=t.int16, device="cuda:0")
    vp = t.zeros(nb * hkv * 16 * dh, dtype=t.int16, device="cuda:0")
    return kp, vp


# token t of a V page row is stored at position t with bits 2 and 3 swapped
V_POS = np.array([(t & 3) | ((t >> 1) & 4) | ((t << 1) & 8) for t in range(16)])


def _logical_pool(kp, vp, nb, hkv, dh):
    """Read the physical pools back into the oracle's logical [nb, 16, Hkv, dh] layout."""
    k = host_f64(kp).reshape(hkv, nb, dh // 8, 16, 8).transpose(1, 3, 0, 2, 4).reshape(nb, 16, hkv, dh)
    v = host_f64(vp).reshape(hkv, nb, dh, 16)[..., V_POS].transpose(1, 3, 0, 2)
    return k, v


@pytest.mark.parametrize("hq,hkv,dh", [(4, 2, 64), (32, 8, 128), (40, 8, 128), (64, 8, 128), (8, 1, 128)])
def test_rope_kv_write(hq, hkv, dh):
    t = torch()
    rng = np.random.default_rng(hq + dh)
    T, nb, maxpos = 50, 20, 9000
    qkvb, qkvf = rand_bf16(rng, (T, (hq + 2 * hkv) * dh))
    pos = rng.integers(0, maxpos, T).astype(np.int32)
    slots = rng.permutation(nb * 16)[:T].astype(np.int32)
    table = t.empty(maxpos * dh // 2 * 2, dtype=t.float32, device="cuda:0")
    hxf.op_rope_table(table.data_ptr(), maxpos, dh, 10000.0)
    qkv = dev_bits(qkvb)
    kp, vp = _make_pools(nb, hkv, dh)
    pos_d, slots_d = i32(pos), i32(slots)
    hxf.op_rope_kv_write(qkv.data_ptr(), pos_d.data_ptr(), slots_d.data_ptr(), table.data_ptr(), kp.data_ptr(),
                         vp.data_ptr(), nb, T, hq, hkv, dh)
    t.cuda.synchronize()
    q = qkvf[:, : hq * dh].reshape(T, hq, dh)
    k = qkvf[:, hq * dh:(hq + hkv) * dh].reshape(T, hkv, dh)
    v = qkvf[:, (hq + hkv) * dh:].reshape(T, hkv, dh)
    got_q = host_f64(qkv).reshape(T, -1)[:, : hq * dh].reshape(T, hq, dh)
    np.testing.assert_allclose(got_q, M.apply_rope(q, pos, 1e4), rtol=2 ** -7, atol=2e-3)
    K, V = _logical_pool(kp, vp, nb, hkv, dh)
    flatk = K.reshape(nb * 16, hkv, dh)
    flatv = V.reshape(nb * 16, hkv, dh)
    np.testing.assert_allclose(flatk[slots], M.apply_rope(k, pos, 1e4), rtol=2 ** -7, atol=2e-3)
    np.testing.assert_array_equal(flatv[slots], v)


@pytest.mark.parametrize("hq,hkv,dh", [(32, 8, 128), (4, 2, 64), (40, 8, 128)])
def test_rope_kv_write_prefill_rows(hq, hkv, dh):
    """A prefill-sized batch (V rows staged per 16 tokens and written as whole page rows):
    12 whole pages in order, 32 tokens from the middle of a page on, a 16-token group whose
    slots run in order but start mid-page, then 90 tokens in scattered slots."""
    t = torch()
    rng = np.random.default_rng(7 * hq + dh)
    nb, maxpos = 80, 9000
    perm = rng.permutation(nb)
    whole = [int(b) * 16 + j for b in perm[:12] for j in range(16)]
    mid = [int(perm[12]) * 16 + 5 + j for j in range(11)] + [int(perm[13]) * 16 + j for j in range(16)] + \
          [int(perm[14]) * 16 + j for j in range(5)]
    shifted = [int(perm[15]) * 16 + 3 + j for j in range(13)] + [int(perm[16]) * 16 + j for j in range(3)]
    free = np.array([int(b) * 16 + j for b in perm[17:] for j in range(16)])
    rest = [int(x) for x in rng.permutation(free)[:90]]
    slots = np.array(whole + mid + shifted + rest, np.int32)
    assert len(set(slots.tolist())) == len(slots)
    T = len(slots)
    qkvb, qkvf = rand_bf16(rng, (T, (hq + 2 * hkv) * dh))
    pos = rng.integers(0, maxpos, T).astype(np.int32)
    table = t.empty(maxpos * dh // 2 * 2, dtype=t.float32, device="cuda:0")
    hxf.op_rope_table(table.data_ptr(), maxpos, dh, 10000.0)
    qkv = dev_bits(qkvb)
    kp, vp = _make_pools(nb, hkv, dh)
    pos_d, slots_d = i32(pos), i32(slots)
    log(f"rope/kv write prefill rows T={T} hq={hq} hkv={hkv} dh={dh}")
    hxf.op_rope_kv_write(qkv.data_ptr(), pos_d.data_ptr(), slots_d.data_ptr(), table.data_ptr(), kp.data_ptr(),
                         vp.data_ptr(), nb, T, hq, hkv, dh)
    t.cuda.synchronize()
    q = qkvf[:, : hq * dh].reshape(T, hq, dh)
    k = qkvf[:, hq * dh:(hq + hkv) * dh].reshape(T, hkv, dh)
    v = qkvf[:, (hq + hkv) * dh:].reshape(T, hkv, dh)
    got_q = host_f64(qkv).reshape(T, -1)[:, : hq * dh].reshape(T, hq, dh)
    np.testing.assert_allclose(got_q, M.apply_rope(q, pos, 1e4), rtol=2 ** -7, atol=2e-3)
    K, V = _logical_pool(kp, vp, nb, hkv, dh)
    np.testing.assert_allclose(K.reshape(nb * 16, hkv, dh)[slots], M.apply_rope(k, pos, 1e4), rtol=2 ** -7,
                               atol=2e-3)
    np.testing.assert_array_equal(V.reshape(nb * 16, hkv, dh)[slots], v)
    # slots nobody wrote stay zero
    untouched = np.setdiff1d(np.arange(nb * 16), slots)
    assert not V.reshape(nb * 16, hkv, dh)[untouched].any()


def _fill_paged(rng, ctxs, hkv, dh, extra_blocks=3):
    """Random K/V for sequences of the given lengths written through the library's
    scatter op into randomly permuted pages.  Returns pools, block tables and the
    logical copies the oracle reads."""
    t = torch()
    pages = [P.pages_for(c) for c in ctxs]
    nb = sum(pages) + extra_blocks
    perm = rng.permutation(nb)
    bts, o = [], 0
    for n in pages:
        bts.append(list(perm[o:o + n]))
        o += n
    width = max(pages)
    bt = np.zeros((len(ctxs), width), np.int32)
    for i, b in enumerate(bts):
        bt[i, : len(b)] = b
    kp, vp = _make_pools(nb, hkv, dh)
    # poison the unused tail of every last page with NaN bit patterns
    kp.fill_(0x7FC0)
    vp.fill_(0x7FC0)
    tot = sum(ctxs)
    kb, kf = rand_bf16(rng, (tot, hkv, dh))
    vb, vf = rand_bf16(rng, (tot, hkv, dh))
    slots = np.concatenate([[P.slot(b, p) for p in range(c)] for b, c in zip(bts, ctxs)]).astype(np.int32)
    k_d, v_d, slots_d = dev_bits(kb), dev_bits(vb), i32(slots)
    hxf.op_kv_scatter(k_d.data_ptr(), v_d.data_ptr(), slots_d.data_ptr(), kp.data_ptr(), vp.data_ptr(), nb, tot, hkv,
                      dh)
    t.cuda.synchronize()
    Kl = np.zeros((nb, 16, hkv, dh))
    Vl = np.zeros((nb, 16, hkv, dh))
    o = 0
    for b, c in zip(bts, ctxs):
        P.scatter(Kl, b, 0, kf[o:o + c])
        P.scatter(Vl, b, 0, vf[o:o + c])
        o += c
    return kp, vp, nb, bt, bts, Kl, Vl


def _decode_case(ctxs, hq, hkv, dh, seed, sample=None):
    t = torch()
    rng = np.random.default_rng(seed)
    B = len(ctxs)
    log(f"decode attention B={B} hq={hq} hkv={hkv} dh={dh} sum_ctx={sum(ctxs)}")
    kp, vp, nb, bt, bts, Kl, Vl = _fill_paged(rng, ctxs, hkv, dh)
    qb, qf = rand_bf16(rng, (B, hq, dh))
    out = empty_i16(B * hq * dh)
    wsn = hxf.op_decode_attention_workspace_bytes(B, hq, hkv, dh, ctxs)
    ws = t.empty(wsn, dtype=t.uint8, device="cuda:0")
    q_d, bt_d = dev_bits(qb), i32(bt)
    hxf.op_decode_attention(q_d.data_ptr(), kp.data_ptr(), vp.data_ptr(), nb, bt_d.data_ptr(), bt.shape[1], ctxs,
                            out.data_ptr(), B, hq, hkv, dh, ws.data_ptr(), wsn)
    t.cuda.synchronize()
    got = host_f64(out).reshape(B, hq, dh)
    seqs = range(B) if sample is None else sample
    for b in seqs:
        c = ctxs[b]
        ref = P.paged_attention(qf[b:b + 1], np.array([c - 1]), Kl, Vl, bts[b], c)[0]
        assert_attn_close(got[b:b + 1], ref[None], f"seq {b} ctx {c}")


@pytest.mark.parametrize("hq,hkv,dh", [(4, 2, 64), (32, 8, 128), (40, 8, 128), (64, 8, 128), (8, 1, 128)])
def test_decode_attention_ragged(hq, hkv, dh):
    ctxs = [1, 15, 16, 17, 31, 32, 33, 255, 256, 257, 511, 700, 1500]
    _decode_case(ctxs, hq, hkv, dh, seed=hq)


def test_decode_attention_cfg2_full_size_sampled():
    """Config-2 shape: 64 sequences with lognormal contexts (median 3000, clipped to
    [1024, 8192]), 32 q-heads / 8 kv-heads of 128; oracle on 12 sampled sequences."""
    ctxs, _ = synth.workloads.cfg2_contexts()
    ctxs = [int(c) for c in ctxs]
    order = np.argsort(ctxs)
    sample = sorted(set(list(order[:4]) + list(order[-4:]) + list(order[30:34])))
    _decode_case(ctxs, 32, 8, 128, seed=2, sample=sample)


def test_decode_attention_one_item_per_pair():
    """260 sequences x 8 kv-heads: at least as many (sequence, kv-head) pairs as the
    chip holds wavefronts, so every pair is one work item (no split)."""
    rng = np.random.default_rng(260)
    ctxs = [int(c) for c in rng.integers(1, 300, 260)]
    sample = list(range(0, 260, 13)) + [259]
    _decode_case(ctxs, 32, 8, 128, seed=260, sample=sample)


@pytest.mark.parametrize("hq,hkv,dh", [(4, 2, 64), (32, 8, 128), (40, 8, 128), (64, 8, 128), (8, 1, 128)])
def test_decode_attention_shared_prefix(hq, hkv, dh):
    """Forks of two parents (255 and 40 shared full pages) decoding together with an
    unrelated sequence: the shared pages are read once per group of rows, and every
    fork's output equals attention over its whole context."""
    t = torch()
    rng = np.random.default_rng(hq * 3 + dh)
    parents = [255 * 16, 40 * 16]
    own = [[int(k) for k in rng.integers(1, 300, 8)], [int(k) for k in rng.integers(1, 40, 5)]]
    lone = 1234
    phys = parents + [k for o in own for k in o] + [lone]       # sequences that own pages
    kp, vp, nb, bt0, bts, Kl, Vl = _fill_paged(rng, phys, hkv, dh)
    seqs, o = [], len(parents)
    for g, plen in enumerate(parents):
        for k in own[g]:
            seqs.append((plen + k, list(bts[g]) + list(bts[o])))
            o += 1
    seqs.append((lone, list(bts[o])))
    ctxs = [c for c, _ in seqs]
    B = len(seqs)
    width = max(len(b) for _, b in seqs)
    bt = np.zeros((B, width), np.int32)
    for i, (_, b) in enumerate(seqs):
        bt[i, :len(b)] = b
    items, _ = hxf.op_decode_plan(B, hq, hkv, ctxs, bt, width)
    assert (items[:, 3] > 1).any()
    log(f"decode attention shared prefix B={B} hq={hq} hkv={hkv} dh={dh} items={len(items)}")
    qb, qf = rand_bf16(rng, (B, hq, dh))
    out = empty_i16(B * hq * dh)
    wsn = hxf.op_decode_attention_workspace_bytes(B, hq, hkv, dh, ctxs, bt, width)
    ws = t.empty(wsn, dtype=t.uint8, device="cuda:0")
    q_d, bt_d = dev_bits(qb), i32(bt)
    hxf.op_decode_attention(q_d.data_ptr(), kp.data_ptr(), vp.data_ptr(), nb, bt_d.data_ptr(), width, ctxs,
                            out.data_ptr(), B, hq, hkv, dh, ws.data_ptr(), wsn, bt_host=bt)
    t.cuda.synchronize()
    got = host_f64(out).reshape(B, hq, dh)
    for b, (c, pages) in enumerate(seqs):
        ref = P.paged_attention(qf[b:b + 1], np.array([c - 1]), Kl, Vl, pages, c)[0]
        assert_attn_close(got[b:b + 1], ref[None], f"seq {b} ctx {c}")


def _prefill_case(chunks, hq, hkv, dh, seed):
    """chunks: list of (pos0, n): n new queries at positions pos0.. over a context of pos0+n."""
    t = torch()
    rng = np.random.default_rng(seed)
    ctxs = [p0 + n for p0, n in chunks]
    log(f"prefill attention chunks={chunks} hq={hq} hkv={hkv} dh={dh}")
    kp, vp, nb, bt, bts, Kl, Vl = _fill_paged(rng, ctxs, hkv, dh)
    ns = [n for _, n in chunks]
    row0 = np.concatenate([[0], np.cumsum(ns)[:-1]]).astype(np.int32)
    T = sum(ns)
    qb, qf = rand_bf16(rng, (T, hq, dh))
    out = empty_i16(T * hq * dh)
    S = len(chunks)
    wsn = hxf.op_prefill_attention_workspace_bytes(S, hq, hkv, ns)
    ws = t.empty(max(wsn, 256), dtype=t.uint8, device="cuda:0")
    q_d, bt_d = dev_bits(qb), i32(bt)
    hxf.op_prefill_attention(q_d.data_ptr(), kp.data_ptr(), vp.data_ptr(), nb, bt_d.data_ptr(), bt.shape[1], row0,
                             [p for p, _ in chunks], ns, out.data_ptr(), S, hq, hkv, dh, ws.data_ptr(), ws.numel())
    t.cuda.synchronize()
    got = host_f64(out).reshape(T, hq, dh)
    for s, (p0, n) in enumerate(chunks):
        ref = P.paged_attention(qf[row0[s]:row0[s] + n], np.arange(p0, p0 + n), Kl, Vl, bts[s], p0 + n)
        assert_attn_close(got[row0[s]:row0[s] + n], ref, f"chunk {s} at {p0}")


def test_prefill_attention_cfg3_full_size():
    """Workload-3 chunks at full size, 8B heads: the first 2048-token chunk of a prompt
    and the last chunk of an 8192-token prompt (queries at 6144-8191), in one launch."""
    _prefill_case([(0, 2048), (6144, 2048)], 32, 8, 128, seed=3)


@pytest.mark.parametrize("hq,hkv,dh,chunks", [(32, 8, 128, [(4352, 512)]), (32, 8, 128, [(4080, 16)]),
                                               (40, 8, 128, [(0, 300), (2000, 40)]),
                                               (4, 2, 64, [(0, 2048), (16, 33)]), (64, 8, 128, [(3000, 200)])])
def test_prefill_attention_key_range_splits(hq, hkv, dh, chunks):
    """Chunks with fewer work items than CUs (a short chunk deep into a prompt, a fork's
    re-prefilled partial page): the items are cut into key ranges whose partials are
    merged by log-sum-exp, up to ~20 parts per item (merged four at a time)."""
    _prefill_case(chunks, hq, hkv, dh, seed=hq + dh + len(chunks))


@pytest.mark.parametrize("hq,hkv,dh", [(4, 2, 64), (32, 8, 128), (40, 8, 128), (64, 8, 128), (8, 1, 128)])
def test_prefill_attention_chunks(hq, hkv, dh):
    chunks = [(0, 1), (0, 17), (0, 64), (16, 16), (40, 9), (100, 77), (0, 300), (513, 130)]
    _prefill_case(chunks, hq, hkv, dh, seed=dh + hq)


def test_argmax_ties_and_lowest_index():
    t = torch()
    rng = np.random.default_rng(5)
    R, V = 9, 128256
    x = rng.standard_normal((R, V)).astype(np.float32)
    x[0, [5, 77, 100000]] = 50.0          # tie: lowest index 5
    x[1, :] = 1.0                          # all equal: index 0
    x[2, V - 1] = 99.0                     # last element
    x[3, [7, 8]] = -np.inf
    out = t.empty(R, dtype=t.int32, device="cuda:0")
    xs = t.from_numpy(x).to("cuda:0")
    hxf.op_argmax(xs.data_ptr(), out.data_ptr(), R, V)
    t.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy(), M.argmax_lowest(x))


def test_copy_probe():
    t = torch()
    a = t.arange(1 << 20, dtype=t.int32, device="cuda:0")
    b = t.zeros_like(a)
    hxf.op_copy(a.data_ptr(), b.data_ptr(), a.numel() * 4)
    t.cuda.synchronize()
    assert t.equal(a, b)


@pytest.mark.parametrize("nbytes", [0, 16, 4096 + 48, 64 << 20])
def test_read_probe(nbytes):
    """Every 32-bit word of src is read exactly once: the XOR over the (zeroed) sink is
    the XOR of all words, which a dropped or repeated load would change."""
    t = torch()
    rng = np.random.default_rng(nbytes % 1000)
    words = rng.integers(0, 2 ** 32, nbytes // 4, dtype=np.uint64).astype(np.uint32)
    src = t.from_numpy(words.view(np.int32).copy()).to("cuda:0") if nbytes else t.zeros(4, dtype=t.int32,
                                                                                         device="cuda:0")
    sink = t.zeros(hxf.READ_SINK_WORDS, dtype=t.int32, device="cuda:0")
    hxf.op_read(src.data_ptr(), nbytes, sink.data_ptr())
    t.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    want = np.bitwise_xor.reduce(words) if nbytes else np.uint32(0)
    assert got == want


@pytest.mark.parametrize("N,K", [(37, 72), (64, 4096), (1, 8), (200, 136)])
def test_pack_weight_layout(N, K):
    """The packed weight layout is the row-major matrix, zero padded to 16 x 32
    multiples, cut into 16 x 32 tiles (row-tiles outermost) stored [k/8][row][8]."""
    rng = np.random.default_rng(N * 131 + K)
    bits, _ = rand_bf16(rng, (N, K))
    got = dev_packed(bits).cpu().numpy().view(np.uint16)
    np_, kp = -(-N // 16) * 16, -(-K // 32) * 32
    pad = np.zeros((np_, kp), np.uint16)
    pad[:N, :K] = bits
    want = pad.reshape(np_ // 16, 16, kp // 32, 4, 8).transpose(0, 2, 3, 1, 4).reshape(-1)
    assert got.shape == want.shape and np.array_equal(got, want)
