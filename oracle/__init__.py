"""Oracle for the mixed prefill/decode iteration of Decode-Latency Feedback Prefill.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call, link
or execute anything in this package; only the test suite, the package's smoke
check and the CPU-baseline leg of the benchmark use it.  It shares no code
with the HIP library or its Python binding: the two are independent
implementations of the same definitions, and only the seeded input generator
(which holds none of the method's arithmetic) feeds both.

Contents, each written from the definition it cites:

* ``attention``  -- masked softmax attention over the logical (unpaged)
  sequences of one mixed iteration (Eq. 1's decode and prefill shares,
  Sec. 2.1; chunked prefill over a cached prefix, Sec. 2.1; attention math left
  unchanged by the controller, Sec. 3.2): ``attention_rows`` for query rows at
  given absolute positions, ``attention_sequence`` for a sequence's new
  tokens.  float64, plain PyTorch CPU ops.
* ``paging``     -- the gather twin: reads a sequence back out of the paged KV
  pool through its block table (PagedAttention layout, Sec. 2.1), token by
  token (``gather_sequence``) or page by page (``gather_pages``).
* ``meta``       -- the varlen-metadata twin (cumulative query offsets, query
  positions, slot mapping) and a validity checker for work lists.
* ``controller`` -- the proportional chunk controller, Eq. 2 (Sec. 3.1), with
  its guard and reset rules.
* ``stats``      -- paired Student-t confidence intervals (Sec. 4.3, Table 1).

Parity status: every function here is pinned by ``tests/test_oracle_*.py``
against values the paper prints, closed forms, brute force on tiny inputs,
library routines, or invariants.  Nothing here is "parity unpinned".
"""
