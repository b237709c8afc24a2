"""Oracle paged KV-cache semantics -- TEST INFRASTRUCTURE ONLY.

The paper serves requests with a paged-attention engine (Section 5.1,
"Runtime") but does not restate its rules; the rules below are the plain
definition this instance implements:

* KV of (sequence s, position p) lives in slot ``bt[s][p // P] * P + p % P``
  of the pool, P = page size (16).
* Pages are reserved eagerly at admission, lowest free block id first, page by
  page in logical order; the reservation covers every token whose KV will be
  written: the context plus ``max(max_new_tokens - 1, 0)`` generated tokens
  (the last sampled token is never fed back).
* A fork of a retained parent whose token sequence S has n tokens shares the
  parent's first ``floor((n - 1) / P)`` pages (all full, read-only) and
  re-prefills the rest of S plus its appended tokens; no page is copied.
* A page returns to the free set when its reference count reaches zero.

The oracle's pool is logical: K and V arrays [n_blocks, P, Hkv, dh].
"""
import numpy as np

from .model import attention


def slot(bt, p, page=16):
    return int(bt[p // page]) * page + p % page


def pages_for(n_tokens, page=16):
    return -(-int(n_tokens) // page)


def reservation(ctx_total, max_new_tokens, shared_pages=0, page=16):
    """Pages to reserve at admission (C-2)."""
    return pages_for(ctx_total + max(max_new_tokens - 1, 0), page) - shared_pages


def fork_shared_pages(parent_tokens, page=16):
    """Full pages of a retained parent that a fork shares: floor((n-1)/P)."""
    return (int(parent_tokens) - 1) // page


def gather(pool, bt, ctx, page=16):
    """Dense [ctx, H, dh] view of a sequence's KV through its block table."""
    idx = [slot(bt, p, page) for p in range(ctx)]
    flat = pool.reshape(-1, *pool.shape[2:])
    return flat[idx]


def scatter(pool, bt, start, kv, page=16):
    """Write kv [n, H, dh] at positions start.. through the block table."""
    flat = pool.reshape(-1, *pool.shape[2:])
    for i in range(kv.shape[0]):
        flat[slot(bt, start + i, page)] = kv[i]


def paged_attention(q, q_pos, k_pool, v_pool, bt, ctx, page=16):
    """Causal GQA attention of q [n, Hq, dh] (at positions q_pos) over the
    first ``ctx`` positions of a paged sequence."""
    k = gather(k_pool, bt, ctx, page)
    v = gather(v_pool, bt, ctx, page)
    return attention(q, k, v, q_pos, np.arange(ctx))


class BlockAllocator:
    """Reference-counted block pool, lowest free id first."""

    def __init__(self, n_blocks):
        self.n = int(n_blocks)
        self.ref = [0] * self.n

    def n_free(self):
        return sum(1 for r in self.ref if r == 0)

    def alloc(self, k):
        """k fresh blocks, lowest ids first; None if fewer are free."""
        out = []
        for b in range(self.n):
            if len(out) == k:
                break
            if self.ref[b] == 0:
                out.append(b)
        if len(out) < k:
            return None
        for b in out:
            self.ref[b] = 1
        return out

    def share(self, blocks):
        for b in blocks:
            assert self.ref[b] > 0
            self.ref[b] += 1

    def release(self, blocks):
        for b in blocks:
            assert self.ref[b] > 0
            self.ref[b] -= 1
