"""CPU oracle for the GreedyLore compression path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product (the HIP library and its
Python binding) imports, calls or links this package; only the tests,
``__graft_entry__.smoke()`` and the bench's CPU-baseline leg use it.

It is a plain, slow, fp64 restatement of the method in the paper
(arXiv 2507.08784): error feedback (Section V-A, eq-ef), the Semi-Lazy SVD
operator (Section V-B, eq-SVD-P1 / eq:new_sub_problem / eq-semi-lazy-svd-2),
Approx-Top-r (Algorithm 2, eq:random-v, eq:lambda-bar, eq-semi-lazy-svd-3),
GreedyLore (Algorithm 3) and its arbitrary-shape form (Algorithm 4,
Appendix D), and the MSGD / Adam updates (Section III, eq-msgd, eq-adam).
It shares no code with the GPU path.

Modules:
  philox  -- Philox4x32-10 counter-based generator and Box-Muller normals
  svd     -- complete left singular basis by one-sided (Hestenes) Jacobi
  subspace -- top-r left singular block by subspace iteration with
             Gram-Schmidt-twice half steps and a Rayleigh-Ritz step (the
             refresh route when every step is a refresh, tau = 1)
  method  -- compressor, selection, optimizers and the per-step driver

Parity-pin status of each function is recorded in its docstring; every
function here is pinned by a ``-m "not gpu"`` test in tests/test_oracle_*.py.
"""
