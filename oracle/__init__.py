"""CPU oracle for the subgraph GCN training step (GraphACT, FPGA '20).

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package. The product path (the HIP library
and its Python binding) never imports, calls or links anything here, and this
package imports nothing from the product path.

Plain, slow, float64 NumPy/SciPy code written from the paper:
  * graph.py      - subgraph construction (Section 2.1, Section 3.1)
  * reduction.py  - redundancy reduction, Algorithms 1-3 repeated in rounds,
                    Theorem 1 and the gamma ratios (Section 3.2)
  * gcn.py        - aggregation (Eq. 1, Section 4.2), layer forward (Eq. 1),
                    classifier, loss, backward (Eq. 2a-2c) and the
                    gradient-descent update (Section 2.1)
  * precision.py  - bfloat16 operand rounding of the bf16 variant of the
                    dense products
  * optim.py      - the momentum and Adam weight updates (Section 4.1 names
                    their state; the rules are the cited methods')
  * sample.py     - frontier sampling of a minibatch's vertex set and the
                    induced subgraph (Section 3.1 names the cited
                    multi-dimensional random walk as its sampler)

Pins (tests/test_oracle_*.py): the worked examples of Fig. 1 and Fig. 2,
Theorem 1's exact accounting, brute force on tiny graphs, an independent
sparse-matrix form of Algorithm 1, the greedy matching's 1/2-approximation
against an exact maximum-weight matching, constant-feature and closed-form
loss cases, central finite differences of the loss, and closed forms of the
optimisers under a constant gradient, the sampler's published generator
outputs, a closed-form step share between two regular components, its
steady state (visits in proportion to degree) and a dense-matrix induced
subgraph.

Parity unpinned (no printed value or closed form fixes it): the greedy
matching's order among equal weights. The paper leaves it open; the oracle
takes (-weight, smaller id, larger id) ascending, and only the matching's
validity, maximality and approximation bound are pinned.
"""
