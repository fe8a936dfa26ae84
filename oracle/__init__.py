"""Plain, slow, float64 CPU oracle for Stream-CQSA (arxiv 2604.20819).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the C-ABI library
and its Python binding) imports, calls, links or executes anything here.
Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU
baseline leg use it.  It shares no code with the HIP path: inputs come in
as plain arrays produced by the seeded generators, results go out as
numpy float64 arrays.

Modules
-------
dense       dense softmax attention forward and its analytic gradients,
            the definition that CQS decomposition reproduces exactly
            (Section 3.1, Eqs. 2-3; Section 3.2, Eqs. 4-6; App. D).
planner     an independent CPU CQS planner: interest sets (App. C,
            Table "interest_set"), BuildSubseq semantics (Alg. 3), the CQS
            mask (Section 3.3), runs, 64-token block summaries and the
            128x128 tile census (App. A.2).
decomposed  the decomposed forward (Alg. 1 in Num/Den form and the
            max-shifted merge of App. A.1, Eq. "merge") and backward (Alg. 2
            and the global-LSE form of App. A.1, Eq. "globallse").

Parity status: every function here is pinned by a ``-m "not gpu"`` test
(tests/test_oracle_*.py) against values the paper prints, closed forms,
an independent library routine (torch float64 attention and autograd) or
finite differences.  No function is "parity unpinned".
"""
