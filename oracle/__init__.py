"""CPU oracle for the Spectral-LSH hot path: a plain, slow, fp64 NumPy
implementation of what the paper defines, used to check the HIP path.

TEST INFRASTRUCTURE. Only tests/, __graft_entry__.smoke() and the CPU-baseline
leg of bench.py may import, call or run anything in this package. The product
(paper_2607_19368_amd) never imports it, and this package imports nothing from
the product: the two share no code.

Parity status of each function (how it is pinned; see tests/test_oracle_pins.py):
  philox4x32_10       published known-answer vectors (tests/golden/philox4x32_10_kat.txt)
  bf16_round (and the W draw's rounding)
                      hand-worked round-to-nearest-even ties (tests/golden/bf16_round_hand.txt);
                      torch's float32 -> bfloat16 cast on random finite bit patterns
  feature_map         Monte-Carlo convergence to exp(x.y/sqrt(D)) at rate m^-1/2;
                      diagonal limit; reduces to the printed Eq. 3 with kernel="gauss"
  lanczos + ritz      dense eigendecomposition of the explicit Phi Phi^T; exact
                      spectrum and breakdown on a low-rank operator with known
                      eigenvalues; orthonormality and the Lanczos relation;
                      interlacing; Toeplitz closed form for the tridiagonal solve
  simhash             hand-worked example (tests/golden/simhash_hand.txt); positive
                      row scaling invariance; collision law (Eq. 6) by Monte Carlo
  merge               hand-worked example (tests/golden/merge_hand.txt); bucket sizes
                      sum to N; causal, strictly increasing positions; singleton
                      identity; renormalised norms
  merge_groups        the same hand example given as groups (offset positions:
                      the max member, not the min); equals merge() on merge()'s groups
  redundancy_score    identical rows give 1; orthonormal equal-norm rows give 1/sqrt(L)
  chunk_pool          brute-force segmented mean
  adjust_to_target, target_budgets
                      parity unpinned: the paper names the exact-length adjustment and
                      per-window budgets without an algorithm; the reading (R20) is
                      pinned by hand-worked examples and invariants only
"""
