"""fp64 CPU oracle for streaming variable-width beam search.

TEST INFRASTRUCTURE ONLY. This package is the plain, slow, obviously-correct
definition that the HIP path is checked against. Only the test suite, the
smoke check and the benchmark's CPU-baseline leg may import it; the product
path never calls it, and it imports nothing from the HIP package.

Contents (each function cites the passage of Yang et al., "A Streaming
Approach For Efficient Batched Beam Search", EMNLP 2020, that it follows):
  decoder  -- the synthetic decoder D(e_i, y) and its log-softmax (Sec. 2)
  beam     -- one beam-search step: expansion, top-k, EOS termination with
              no-op expansions, pruning heuristics H (Sec. 2, Sec. 4, App. A.1)
  search   -- Alg. 1 (Var-Stream) and its settings Fixed / Var-Batch (Sec. 3)
  brute    -- exhaustive enumeration and teacher-forced scoring for pins
  compare  -- GPU-vs-oracle comparison with near-tie excuses

Every function is pinned by tests in tests/test_oracle_*.py against closed
forms, brute force, the greedy special case and the paper's invariants.
"""
