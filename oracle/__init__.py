"""CPU oracle -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 (floating point) / exact-integer (scheduling) restatement
of what one serving instance computes:

* ``oracle.model``  -- the Llama-style decoder forward and greedy decoding;
* ``oracle.paged``  -- paged KV-cache semantics (slots, block tables, reservation);
* ``oracle.sched``  -- the local priority queue of the paper's Section 4.2
  (per-request SLO budget, urgency, argmax admission) wrapped in a
  continuous-batching iteration with chunked prefill and a page allocator.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library
and never imports it; both take their inputs from ``synth``.
"""
