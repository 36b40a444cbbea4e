"""CPU oracle of the co-located instances' batched transformer forward pass.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or run anything in this package.
The product library (``paper_2503_05130_amd``) never imports, links or calls it,
and this package imports nothing from the product.

Contents:
* ``init_spec`` -- the seeded random-init spec (pure-Python reference + a C fast path).
* ``forward``   -- plain NumPy fp64 forward pass (the oracle proper).
* ``scalar``    -- an independent pure-Python loop implementation for tiny shapes.

The paper (Dilu, Sec. 3-5) treats the forward pass as the workload each
serverless DL instance runs and states none of its arithmetic; the definitions
here are the standard post-LN (BERT-style) and pre-LN causal (GPT-style)
transformer, with each point the paper leaves open written down where it is used.

Parity status: the arithmetic is pinned by closed forms, invariants, textbook
values and brute force (tests/test_oracle_*.py).  Agreement with numbers printed
in the paper: parity unpinned -- the paper prints no forward-pass values.
"""
