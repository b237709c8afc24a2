"""Oracle serving loop: the oracle scheduler driving the oracle decoder.
TEST INFRASTRUCTURE ONLY.

Each request keeps a dense float64 KV history (``model.Sequence``).  A forked
request starts from a copy of its parent's history truncated to the shared
full pages, which is exactly what sharing those pages means; it then
re-prefills the remaining tokens like any chunk.
"""
import numpy as np

from . import model as M


class DecoderExecutor:
    def __init__(self, weights, forced=None, keep_logits=True):
        self.w = weights
        self.seqs = {}
        self.logits = {}            # request id -> list of float64 logit rows
        self.forced = forced or {}  # request id -> tokens to feed back instead of the sampled ones
        self.keep = keep_logits
        self.sched = None

    def _seq(self, r):
        s = self.seqs.get(r.id)
        if s is None:
            s = M.Sequence(self.w.shape.n_layers)
            if r.parent:
                ps = self.seqs[r.parent]
                n = r.pf_pos0
                for l in range(self.w.shape.n_layers):
                    s.k[l] = ps.k[l][:n].copy()
                    s.v[l] = ps.v[l][:n].copy()
                s.n = n
            self.seqs[r.id] = s
        assert s.n == r.n_kv
        return s

    def __call__(self, batch, rows):
        seqs, chunks, want = [], [], []
        row_ids = {id(r) for r in rows}
        for r, kind, toks, p0 in batch:
            s = self._seq(r)
            feed = list(toks)
            if kind == "d" and r.id in self.forced:
                feed = [self.forced[r.id][len(r.generated) - 1]]
            seqs.append(s)
            chunks.append(np.asarray(feed))
            want.append(id(r) in row_ids)
        lg = M.forward(self.w, seqs, chunks)
        out = {}
        for (r, _, _, _), l, w in zip(batch, lg, want):
            if w:
                out[r.id] = l[0]
                if self.keep:
                    self.logits.setdefault(r.id, []).append(l[0])
        return [int(M.argmax_lowest(out[r.id])) for r in rows]

    def drop(self, rid):
        self.seqs.pop(rid, None)
