"""The decode-attention work list (host logic, no GPU): every (sequence, kv-head)
attends to each of its context tokens exactly once, its partials fill a block of
consecutive slots, shared-prefix items only cover pages the rows really share, and
the items fill the resident wavefronts without exceeding them."""
import numpy as np
import pytest

from paper_2505_05286_amd import hxf

from ._lib import ensure_built

RESIDENT = 2048


@pytest.fixture(scope="module", autouse=True)
def _built():
    ensure_built()


def _tables(rng, ctxs, groups=()):
    """Block tables: distinct pages per sequence, except that each group (list of
    sequence indices) shares the first `shared` pages of its first member."""
    width = max(-(-c // 16) for c in ctxs)
    bt = np.full((len(ctxs), width), -1, np.int32)
    nxt = 0
    for i, c in enumerate(ctxs):
        n = -(-c // 16)
        bt[i, :n] = np.arange(nxt, nxt + n)
        nxt += n
    for members, shared in groups:
        for m in members[1:]:
            bt[m, :shared] = bt[members[0], :shared]
    return bt


def _check(ctxs, hq, hkv, bt=None):
    B = len(ctxs)
    G = hq // hkv
    items, merges = hxf.op_decode_plan(B, hq, hkv, ctxs, bt, bt.shape[1] if bt is not None else 0)
    assert merges.shape == (B * hkv, 4)
    narrow, wide = hxf.decode_rows_narrow(G), hxf.decode_rows_wide(G)
    n_wide = int(np.sum(items[:, 3] > narrow))
    assert (items[:len(items) - n_wide, 3] <= narrow).all()      # one-tile items first, then the wide ones
    cover = {}          # (seq, kvh) -> list of (t0, t1)
    slot_owner = {}
    for it in items:
        kvh, t0, t1, n_rows = it[:4]
        ents, parts = it[4:12], it[12:20]
        assert 1 <= n_rows <= wide and 0 <= t0 < t1
        assert t0 % 16 == 0
        for r in range(n_rows):
            e = int(ents[r])
            assert t1 <= ctxs[e]
            if r > 0 and bt is not None:   # rows read entry[0]'s pages: they must be theirs too
                p0, p1 = t0 // 16, -(-t1 // 16)
                assert np.array_equal(bt[e, p0:p1], bt[ents[0], p0:p1])
                assert t1 % 16 == 0 and t1 <= (ctxs[e] // 16) * 16     # only full pages are shared
            cover.setdefault((e, int(kvh)), []).append((int(t0), int(t1)))
            assert int(parts[r]) not in slot_owner
            slot_owner[int(parts[r])] = (e, int(kvh))
    for e, kvh, part0, n_part in merges:
        ranges = sorted(cover[(int(e), int(kvh))])
        assert ranges[0][0] == 0 and ranges[-1][1] == ctxs[e]
        assert all(a[1] == b[0] for a, b in zip(ranges, ranges[1:]))
        assert len(ranges) == n_part
        assert all(slot_owner[s] == (e, kvh) for s in range(part0, part0 + n_part))
    assert len(slot_owner) == sum(int(m[3]) for m in merges)
    for part in (items[:len(items) - n_wide], items[len(items) - n_wide:]):
        lengths = [int(t1 - t0) for t0, t1 in part[:, 1:3]]
        assert lengths == sorted(lengths, reverse=True)       # longest first within each kind
    return items, merges


@pytest.mark.parametrize("hq,hkv", [(4, 2), (32, 8), (40, 8)])
def test_plan_covers_every_token_once_without_tables(hq, hkv):
    rng = np.random.default_rng(hq)
    ctxs = [1, 15, 16, 17, 255, 256, 257, 1000, 4096, 8191] + [int(c) for c in rng.integers(1, 9000, 40)]
    items, _ = _check(ctxs, hq, hkv)
    assert (items[:, 3] == 1).all()


def test_plan_fills_but_does_not_exceed_the_resident_wavefronts():
    rng = np.random.default_rng(2)
    ctxs = [int(c) for c in np.clip(rng.lognormal(np.log(3000), 0.5, 64), 1024, 8192)]
    items, _ = _check(ctxs, 32, 8)
    assert 0.8 * RESIDENT <= len(items) <= RESIDENT
    # at least as many (sequence, kv-head) pairs as resident wavefronts: every pair has an
    # item, and the streams longer than an even share of all tokens are cut to that share
    ctxs = [int(c) for c in rng.integers(1, 5000, 260)]
    items, _ = _check(ctxs, 32, 8)
    share = max(-(-sum(ctxs) * 8 // RESIDENT), 256)
    assert 260 * 8 < len(items) <= 260 * 8 + RESIDENT
    assert (items[:, 2] - items[:, 1]).max() <= -(-share // 16) * 16
    # uniform lengths: the share is the length itself, one item per pair
    items, _ = _check([3000] * 260, 32, 8)
    assert len(items) == 260 * 8


def test_plan_cuts_a_shared_prefix_longer_than_the_even_share():
    """32 groups of 8 forks of 4096-token parents (each fork 1-255 tokens past the
    shared 256 pages): 288 streams x 8 kv-heads exceed the resident wavefronts, yet
    the shared-prefix streams are cut to the even share instead of one 4096-token item
    each."""
    rng = np.random.default_rng(6)
    ctxs = [4096 + int(k) for k in rng.integers(1, 256, 256)]
    bt = _tables(rng, ctxs, groups=[(list(range(8 * g, 8 * g + 8)), 256) for g in range(32)])
    items, _ = _check(ctxs, 32, 8, bt)
    wide = items[items[:, 3] == 8]
    share = -(-sum(ctxs) * 8 // RESIDENT)
    assert len(wide) > 32 * 8 and (wide[:, 2] - wide[:, 1]).max() <= -(-share // 16) * 16


@pytest.mark.parametrize("hq,hkv,per_item", [(32, 8, 8), (40, 8, 6), (64, 8, 4), (16, 8, 8)])
def test_plan_shares_fork_prefixes(hq, hkv, per_item):
    """Two groups of 8 forks sharing 255 pages (4096-token parents), plus unrelated
    sequences: the shared pages are read by items of min(8, 32/G) rows (two query tiles
    when more than 16/G), i.e. once per group of eight forks at G <= 4."""
    rng = np.random.default_rng(4)
    ctxs = [4096 + 16 + int(k) for k in rng.integers(1, 256, 16)] + [3000, 5000]
    bt = _tables(rng, ctxs, groups=[(list(range(8)), 255), (list(range(8, 16)), 255)])
    items, _ = _check(ctxs, hq, hkv, bt)
    shared = items[items[:, 3] > 1]
    assert len(shared) > 0 and shared[:, 3].max() == per_item
    assert (shared[:, 2] <= 255 * 16).all()
    # every fork reads the 4080 shared tokens through shared items only
    tok = {}
    for it in shared:
        for r in range(it[3]):
            tok[int(it[4 + r]), int(it[0])] = tok.get((int(it[4 + r]), int(it[0])), 0) + int(it[2] - it[1])
    assert all(tok[(e, h)] == 255 * 16 for e in range(16) for h in range(hkv))
    # the (token, kv-head) pairs read drop by the sharing factor on the shared part
    read = int((items[:, 2] - items[:, 1]).sum())
    logical = sum(ctxs) * hkv
    items_per_group = -(-8 // per_item)
    assert read == logical - 16 * hkv * 4080 + 2 * items_per_group * hkv * 4080


def test_plan_groups_need_a_common_full_page():
    """Equal first pages with a partial first page (context < 16) or nested forks with
    different shared lengths: the group shares only what all members share."""
    rng = np.random.default_rng(5)
    ctxs = [700, 800, 900, 40]
    bt = _tables(rng, ctxs, groups=[([0, 1, 2], 30)])
    bt[2, 20:30] = 10_000 + np.arange(10)          # the third fork diverges after 20 pages
    items, _ = _check(ctxs, 32, 8, bt)
    shared = items[items[:, 3] > 1]
    assert (shared[:, 2] <= 20 * 16).all() and (shared[:, 3] == 3).all()
    ctxs = [10, 12]
    bt = _tables(rng, ctxs, groups=[([0, 1], 1)])
    items, _ = _check(ctxs, 32, 8, bt)
    assert (items[:, 3] == 1).all()


def test_plans_reused_across_iterations_carry_nothing_over(tmp_path):
    """The executor plans every iteration into the same plan objects: after an
    iteration with two-tile fork items, an iteration with no decoding sequence must
    report no items of either kind (a stale two-tile count sent the wide kernel to
    items before the start of an empty list).  Host code only, built with g++."""
    import os
    import subprocess
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    csrc = os.path.join(root, "paper_2505_05286_amd", "csrc")
    exe = str(tmp_path / "plan_reuse")
    subprocess.run(["g++", "-std=c++17", "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I" + csrc,
                    os.path.join(root, "tests", "plan_reuse.cpp"), os.path.join(csrc, "decode_plan.cpp"), "-o", exe],
                   check=True, capture_output=True, timeout=300)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr


# ------------------------------------------------------------------ prefill work list

PF_PAIRS, PF_RESIDENT = 128, 512


def _check_prefill(pos0, n, hq, hkv):
    """Every (chunk, kv-head, query block) attends to its key tiles exactly once, either as
    one whole item or as the consecutive parts of one merge; returns (items, merges, share)."""
    items, merges = hxf.op_prefill_plan(hq, hkv, pos0, n)
    G = hq // hkv
    qpi = PF_PAIRS // G
    whole = {}
    for s, (p0, ns) in enumerate(zip(pos0, n)):
        for h in range(hkv):
            for q0 in range(0, ns, qpi):
                nq = min(qpi, ns - q0)
                whole[(s, h, q0)] = (nq, -(-(p0 + q0 + nq) // 32))
    tiles = sum(t for _, t in whole.values())
    share = max(-(-tiles // PF_RESIDENT), 8)
    assert len(items) <= len(whole) + PF_RESIDENT
    got = {}
    for e, h, q0, nq, t0, t1, part, _ in items:
        assert (e, h, q0) in whole and whole[(e, h, q0)][0] == nq
        assert 0 <= t0 < t1 <= whole[(e, h, q0)][1]
        got.setdefault((e, h, q0), []).append((t0, t1, part))
    assert set(got) == set(whole)
    parts_seen = set()
    merged = {(m[0], m[1], m[2]): m for m in merges}
    for key, ranges in got.items():
        ranges.sort()
        assert ranges[0][0] == 0 and ranges[-1][1] == whole[key][1]
        for (a0, a1, _), (b0, b1, _) in zip(ranges, ranges[1:]):
            assert a1 == b0                                  # no gap, no overlap
        if len(ranges) == 1:
            assert ranges[0][2] == -1 and key not in merged
        else:
            m = merged[key]
            assert m[3] == whole[key][0] and m[5] == len(ranges)
            assert [r[2] for r in ranges] == list(range(m[4], m[4] + m[5]))
            parts_seen.update(r[2] for r in ranges)
    assert len(parts_seen) == sum(m[5] for m in merges) <= len(whole) + PF_RESIDENT
    return items, merges, share, whole


def test_prefill_plan_full_chunks_are_not_cut():
    """With at least one item per CU nothing is cut: a prompt's first 2048-token chunk at the
    8B heads (512 causal items of 1 to 64 key tiles), its second, one deep into the prompt, and
    a 1024-token first chunk (256 items)."""
    for p0, n in ((0, 2048), (2048, 2048), (6144, 2048), (0, 1024)):
        items, merges, share, whole = _check_prefill([p0], [n], 32, 8)
        assert len(merges) == 0 and len(items) == len(whole) == n // 4
        assert (items[:, 6] == -1).all()


@pytest.mark.parametrize("p0,n", [(4352, 512), (4080, 16), (0, 960)])
def test_prefill_plan_few_items_cut_to_the_share(p0, n):
    """Fewer items than CUs: every item longer than the share is cut."""
    items, merges, share, whole = _check_prefill([p0], [n], 32, 8)
    assert len(whole) < PF_RESIDENT // 2
    assert max(t1 - t0 for *_, t0, t1, _p, _pad in items) <= share
    assert len(merges) == sum(1 for nq, t in whole.values() if t > share)


@pytest.mark.parametrize("pos0,n,hq,hkv", [
    ([0, 100, 5000], [700, 33, 2048], 32, 8), ([0], [1], 4, 2), ([4080], [16], 40, 8), ([0, 0], [2048, 2048], 64, 8),
    ([17, 0, 3000], [2300, 5, 640], 4, 2)])
def test_prefill_plan_covers_every_key_tile_once(pos0, n, hq, hkv):
    _check_prefill(pos0, n, hq, hkv)
