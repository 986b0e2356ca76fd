"""CPU oracle for the dynamic-batching hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct implementation in NumPy fp64 of what the
batched GPU path must reproduce:

  * ``schedule``  -- the validator and the reference scheduler (depth, stable
    sort by (depth, op), edge labels), written as the plain definitions of
    Section 2 of the paper (the five scheduling steps);
  * ``cells``     -- the per-node operations (embedding lookup, TreeRNN cell,
    binary Tree-LSTM, LSTM step, projection) and their hand-derived
    gradients;
  * ``evaluate``  -- forward by memoised recursion, one node at a time and
    unbatched, and backward in reverse topological order;
  * ``compare``   -- the error metric the parity tests use.

Dynamic batching is a rewrite: its result equals evaluating every graph on its
own (Section 2: batching plus identity pass-throughs, differentiable
gather/concat), so the oracle never batches anything.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline
leg may import this package.  The product path never does, and this package
imports nothing from the product package.
"""
