"""CPU oracle for suffix-prefill attention over a paged, prefix-cached KV store.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call, link or
execute anything in this package: only the test suite, the smoke check and the
bench's CPU-baseline leg use it. It shares no code with the HIP library or its
Python binding; both sides only receive the same seeded input arrays.

Modules
  attention  fp64 attention of the uncached suffix rows over prefix + suffix keys
             (the computation that prefix reuse shortens; paper Sec. 1 and 2.1).
  paged      chained block hashes, a block-pool simulation with prefix lookup,
             and the expected KV-cache image after appending suffix K/V
             (APC over fixed 16-token blocks; paper Sec. 2.1, Fig. 1).
  ordering   the knowledge tree by its definition, reusable prefix depth l(O, T),
             Algorithm 1, the exhaustive argmax over all orders (paper Sec. 3.3,
             Eq. 1) and the baseline orders (Sec. 4).
  projection the suffix QKV projection with rotary position embedding (the
             per-layer work that feeds the cache append and attention).

Every function is a plain, slow, obviously correct statement of its definition.
The only blocking anywhere is the independent-row chunking in `attention`, which
bounds memory and does not change any row's arithmetic.

Parity status: every function here is pinned by tests/test_oracle_pins.py,
tests/test_ordering.py and tests/test_projection.py (brute force, closed forms, a library routine, published test vectors, the
paper's worked examples). No function is "parity unpinned".
"""
