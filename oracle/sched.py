"""Oracle of one instance's scheduler -- TEST INFRASTRUCTURE ONLY.

Exact integer (microsecond) restatement of the paper's local priority queue
(Section 4.2) inside a continuous-batching iteration:

* compute cost, Section 4.1 equation for t_comp: t_prefill(L_in) + t_decode(L_out),
  here ``(c0 + c1*L_in + c2*L_in^2 + d1*L_out) // 10^6`` with picosecond
  coefficients (the paper only says the estimates come from empirical
  profiles); L_out is the request's declared output budget;
* instance-average cost, Section 4.2: with one instance it is t_comp itself;
* SLO budget, Section 4.2:
  ``t_SLO = (T_SLO - tau_elapsed) * c_j / (c_j + sum of the later stages' costs)``,
  floored toward minus infinity, fixed when the request is submitted;
* urgency, Section 4.2: ``U = t_comp - (t_SLO - tau)`` with tau the time spent
  in the local queue.  At one instant U ranks requests exactly as the static key
  ``K = enq + t_SLO - t_comp`` (U = now - K), so the queue is a heap on K;
* selection, Section 4.2: the most urgent queued request is taken whenever a
  batch is formed; ties go to the later workflow stage, then the earlier
  arrival, then the lower id.

Iteration rules (the paper only says batches are formed by continuous
batching): running decodes get one token each; running prefills get chunk
tokens in queue order from a budget of ``chunk_tokens`` (decode tokens are not
counted); then queued requests are admitted in queue order while a sequence
slot, the page reservation and budget are all available, stopping at the
first that does not fit.

Baseline policies for comparison: FCFS (order by arrival in the queue) and
LLF (laxity against the workflow's end-to-end deadline, no per-stage budget,
Section 5.1 "Baseline").

Token ids come from an executor callback, so the scheduler can be checked on
its own (``fake_token``) or driven by the oracle decoder.
"""
import heapq

from .paged import BlockAllocator, fork_shared_pages, pages_for

PS = 10 ** 6          # picoseconds per microsecond

POLICY_PQ, POLICY_FCFS, POLICY_LLF = 0, 1, 2
CLOCK_VIRTUAL, CLOCK_MEASURED = 0, 1

OK, IDLE = 0, 1
EINVAL, ENOMEM, ENOTFOUND, ESTATE = -1, -2, -3, -4

QUEUED, PREFILL, DECODE, DONE, RELEASED, CANCELLED = range(6)


class SchedError(Exception):
    def __init__(self, code, msg=""):
        super().__init__(msg)
        self.code = code


def floor_div(a, b):
    return a // b          # Python floors toward minus infinity


def t_comp(cost, l_in, l_out):
    """Compute-cost estimate (Section 4.1, t_comp = t_prefill + t_decode), in us."""
    c0, c1, c2, d1 = cost
    return floor_div(c0 + c1 * l_in + c2 * l_in * l_in + d1 * l_out, PS)


def t_comp_mean(cost_sum, n_inst, l_in, l_out):
    """Instance-average compute cost (Section 4.2): the mean of the N instances'
    unfloored estimates, floored; cost_sum is their coefficients added up."""
    c0, c1, c2, d1 = cost_sum
    return floor_div(c0 + c1 * l_in + c2 * l_in * l_in + d1 * l_out, n_inst * PS)


def slo_budget(t_slo_e2e, elapsed, c_j, rest_costs):
    """Per-request SLO budget (Section 4.2): remaining end-to-end time shared
    in proportion to this request's cost among it and the later stages."""
    remaining = t_slo_e2e - elapsed
    denom = c_j + sum(rest_costs)
    if denom == 0:
        return remaining
    return floor_div(remaining * c_j, denom)


def urgency(t_comp_us, t_slo_us, tau_us):
    """Urgency (Section 4.2): estimated cost minus remaining SLO margin."""
    return t_comp_us - (t_slo_us - tau_us)


def t_iter(it, n_prefill, n_decode, sum_ctx_decode, attn_pf):
    """Virtual-clock duration of one iteration (us): a fixed part, prefill tokens,
    decode rows, the decode rows' context and the prefill attention pairs, each with
    its own coefficient (ps).  A 4-coefficient model charges a decode row like a
    prefill token."""
    i0, i1, i2, i3 = it[:4]
    i4 = it[4] if len(it) == 5 else i1
    return floor_div(i0 + i1 * n_prefill + i2 * sum_ctx_decode + i3 * attn_pf + i4 * n_decode, PS)


def fake_token(req_id, pos, vocab):
    """Token id of the scheduler-only executor: a fixed function of (id, position)."""
    return (req_id * 1000003 + pos * 7919 + 12345) % vocab


class Req:
    pass


class Scheduler:
    def __init__(self, n_blocks, max_seqs, chunk_tokens, cost, iter_cost, page=16,
                 policy=POLICY_PQ, vocab=2048):
        self.alloc = BlockAllocator(n_blocks)
        self.n_blocks = n_blocks
        self.max_seqs = max_seqs
        self.chunk = chunk_tokens
        self.cost = tuple(cost)
        self.iter_cost = tuple(iter_cost)
        self.page = page
        self.policy = policy
        self.vocab = vocab
        self.reqs = {}
        self.heap = []
        self.running = []            # admission order
        self.done_queue = []
        self.next_id = 1
        self.iteration = 0

    # ------------------------------------------------------------ ordering
    def order(self, r):
        if self.policy == POLICY_PQ:
            return (r.key, -r.stage, r.enq, r.id)
        if self.policy == POLICY_FCFS:
            return (r.enq, r.id)
        return (r.key, r.enq, r.id)

    # ------------------------------------------------------------ submit
    def submit(self, now, workflow, stage, wf_arrival, wf_slo, prompt, max_new, parent=0,
               retain=False, rest=(), budget_cost_sum=None, n_inst=1):
        """Queue a request.  With ``budget_cost_sum`` (N instances' cost coefficients
        summed) its SLO budget is shared out by the instance-average costs of
        Section 4.2 instead of this instance's own estimates."""
        prompt = [int(t) for t in prompt]
        if max_new < 0 or (max_new == 0 and not retain) or stage < 0:
            raise SchedError(EINVAL, "bad output budget")
        if any(t < 0 or t >= self.vocab for t in prompt):
            raise SchedError(EINVAL, "token id out of range")
        r = Req()
        shared = []
        if parent:
            p = self.reqs.get(parent)
            if p is None or p.state in (CANCELLED, RELEASED):
                raise SchedError(ENOTFOUND, "no such parent")
            if p.state != DONE or not p.retain:
                raise SchedError(ESTATE, "parent not finished with retained KV")
            s_tokens = p.context + p.generated
            n = len(s_tokens)
            s = fork_shared_pages(n, self.page)
            shared = p.bt[:s]
            r.context = s_tokens + prompt
            r.pf_tokens = s_tokens[s * self.page:] + prompt
            r.pf_pos0 = s * self.page
        else:
            if len(prompt) == 0:
                raise SchedError(EINVAL, "empty prompt")
            r.context = prompt
            r.pf_tokens = prompt
            r.pf_pos0 = 0
        r.reserve = pages_for(len(r.context) + max(max_new - 1, 0), self.page) - len(shared)
        if r.reserve > self.n_blocks:
            raise SchedError(ENOMEM, "request can never fit the pool")
        r.id = self.next_id
        self.next_id += 1
        r.workflow, r.stage = workflow, stage
        r.wf_arrival, r.wf_slo = wf_arrival, wf_slo
        r.max_new, r.retain, r.parent = max_new, bool(retain), parent
        r.t_comp = t_comp(self.cost, len(r.pf_tokens), max_new)
        rest_costs = [t_comp(self.cost, li, lo) for li, lo in rest]
        if budget_cost_sum is None:
            r.t_slo = slo_budget(wf_slo, now - wf_arrival, r.t_comp, rest_costs)
        else:
            mean_j = t_comp_mean(budget_cost_sum, n_inst, len(r.pf_tokens), max_new)
            mean_rest = [t_comp_mean(budget_cost_sum, n_inst, li, lo) for li, lo in rest]
            r.t_slo = slo_budget(wf_slo, now - wf_arrival, mean_j, mean_rest)
        r.enq = now
        if self.policy == POLICY_LLF:
            r.key = wf_arrival + wf_slo - (r.t_comp + sum(rest_costs))
        else:
            r.key = r.enq + r.t_slo - r.t_comp
        self.alloc.share(shared)
        r.bt = list(shared)
        r.n_shared = len(shared)
        r.state = QUEUED
        r.n_pf_done = 0
        r.n_kv = r.pf_pos0
        r.generated = []
        r.t_first_sched = r.t_first_token = r.t_finish = -1
        self.reqs[r.id] = r
        heapq.heappush(self.heap, (self.order(r), r.id))
        return r.id

    # ------------------------------------------------------------ introspection
    def queue_cost(self):
        """Queueing cost (Section 4.1): t_comp summed over the requests that are
        queued or running."""
        return sum(r.t_comp for r in self.reqs.values() if r.state in (QUEUED, PREFILL, DECODE))

    def queue_order(self):
        return [rid for _, rid in sorted(self.heap)]

    def block_table(self, rid):
        return list(self.reqs[rid].bt)

    # ------------------------------------------------------------ step
    def form_batch(self, now):
        """Return the batch as a list of (req, kind, tokens, pos0) and the admitted ids."""
        batch = []
        for r in self.running:
            if r.state == DECODE:
                batch.append((r, "d", [r.generated[-1]], r.n_kv))
        budget = self.chunk
        pf = sorted((r for r in self.running if r.state == PREFILL), key=self.order)
        for r in pf:
            if budget <= 0:
                break
            c = min(len(r.pf_tokens) - r.n_pf_done, budget)
            batch.append((r, "p", r.pf_tokens[r.n_pf_done:r.n_pf_done + c], r.n_kv))
            budget -= c
        admitted = []
        while self.heap and budget > 0:
            _, rid = self.heap[0]
            r = self.reqs[rid]
            if len(self.running) >= self.max_seqs or self.alloc.n_free() < r.reserve:
                break
            heapq.heappop(self.heap)
            own = self.alloc.alloc(r.reserve)
            r.bt = r.bt + own
            r.state = PREFILL
            r.t_first_sched = now
            self.running.append(r)
            admitted.append(r.id)
            c = min(len(r.pf_tokens), budget)
            batch.append((r, "p", r.pf_tokens[:c], r.n_kv))
            budget -= c
        return batch, admitted

    def step(self, now, executor=None, measured_us=None):
        """One batch boundary plus one forward.  ``executor(batch, rows)`` returns
        the sampled token per logit row; default is ``fake_token``."""
        batch, admitted = self.form_batch(now)
        if not batch:
            return IDLE, None
        rows = []
        n_tok = sum_ctx = attn = 0
        for r, kind, toks, p0 in batch:
            n_tok += len(toks)
            if kind == "d":
                sum_ctx += p0 + 1
                rows.append(r)
            else:
                attn += len(toks) * (p0 + len(toks))
                if r.n_pf_done + len(toks) == len(r.pf_tokens) and r.max_new > 0:
                    rows.append(r)
        if executor is None:
            sampled = [fake_token(r.id, len(r.context) + len(r.generated), self.vocab) for r in rows]
        else:
            sampled = executor(batch, rows)
        n_dec = sum(1 for b in batch if b[1] == "d")
        dt = t_iter(self.iter_cost, n_tok - n_dec, n_dec, sum_ctx, attn) if measured_us is None else measured_us
        t_end = now + dt
        finished = []
        k = 0
        for r, kind, toks, p0 in batch:
            r.n_kv += len(toks)
            has_row = kind == "d"
            if kind == "p":
                r.n_pf_done += len(toks)
                if r.n_pf_done == len(r.pf_tokens):
                    r.state = DECODE
                    has_row = r.max_new > 0
                    if r.max_new == 0:
                        finished.append(r)
            if has_row:
                r.generated.append(int(sampled[k]))
                k += 1
                if len(r.generated) == 1:
                    r.t_first_token = t_end
                if len(r.generated) == r.max_new:
                    finished.append(r)
        for r in finished:
            r.state = DONE
            r.t_finish = t_end
            self.running.remove(r)
            if not r.retain:
                self._free(r)
            self.done_queue.append(r.id)
        self.iteration += 1
        info = dict(n_tokens=n_tok, n_decode=sum(1 for b in batch if b[1] == "d"),
                    n_prefill_tokens=sum(len(b[2]) for b in batch if b[1] == "p"),
                    n_logit_rows=len(rows), t_iter_us=dt, n_admitted=len(admitted),
                    n_finished=len(finished), free_blocks=self.alloc.n_free(),
                    sum_decode_ctx=sum_ctx, prefill_attn=attn,
                    admitted=admitted, batch_ids=sorted(b[0].id for b in batch))
        return OK, info

    def _free(self, r):
        self.alloc.release(r.bt)

    # ------------------------------------------------------------ completion
    def drain(self):
        out = []
        for rid in self.done_queue:
            r = self.reqs[rid]
            out.append(dict(id=r.id, workflow=r.workflow, stage=r.stage, t_submit=r.enq,
                            t_first_sched=r.t_first_sched, t_first_token=r.t_first_token,
                            t_finish=r.t_finish, t_slo=r.t_slo, t_comp=r.t_comp,
                            n_generated=len(r.generated),
                            met_slo=int(r.t_finish - r.enq <= r.t_slo)))
        self.done_queue = []
        return out

    def tokens(self, rid):
        return list(self.reqs[rid].generated)

    def release(self, rid):
        r = self.reqs.get(rid)
        if r is None:
            raise SchedError(ENOTFOUND)
        if r.state != DONE or not r.retain:
            raise SchedError(ESTATE)
        self._free(r)
        r.state = RELEASED

    def cancel(self, rid):
        r = self.reqs.get(rid)
        if r is None:
            raise SchedError(ENOTFOUND)
        if r.state == QUEUED:
            self.heap = [e for e in self.heap if e[1] != rid]
            heapq.heapify(self.heap)
            self._free(r)
        elif r.state in (PREFILL, DECODE):
            self.running.remove(r)
            self._free(r)
        else:
            raise SchedError(ESTATE)
        r.state = CANCELLED
