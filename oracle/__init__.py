"""CPU oracle for OrderMoE's per-layer hot path (arXiv 2607.17154).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, deliberately
unoptimised CPU implementation written from the paper, used to check the HIP
library.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
may import it; the library never does, and it shares no code, header, table or
constant generator with the library.  Inputs come from the seeded generators
in ``workloads`` (random draws only) or from the tests themselves.

Modules and the passages they follow:
  route       -- router logits (eq 3 per token), gate, top-k, logit margin
  similarity  -- H, Sim, activation counts (eq 3-5), greedy grouping (eq 24-26),
                 representativeness and importance (eq 27-28); Alg. 1 part 1
  placement   -- mandatory and redundant deployment (eq 29-35); Alg. 1 parts 2-3
  tables      -- theta_l (eq 6), substitutes (eq 7-8), loss (eq 18), static
                 per-step cost (eq 37-38), transitions and look-ahead (eq 41-42)
  layer       -- per-token selection (eq 36-44, Alg. 2 for one layer, in
                 select.c), dispatch list (eq 13-14), one server's output
Precision: fp64 for every real-valued quantity, except the selection's
decision arithmetic, which is fp32 as the runtime tables are fp32.

Pins (tests/test_oracle_*.py): brute-force cosine and textbook top-k;
a cosine limit for Gaussian calibration inputs; exact MoE when substitution is
off; all-local deployments giving no remote slots; Properties 1 and 2 of the
paper; hand-traced placements; exhaustive enumeration of eq 43 on tiny layers;
H = 1 giving Phi = 0 and a closed form of Phi for all-local deployments;
hand-traced look-ahead values where a budget-free substitute or an unpinned
remote copy is the future minimum; a literal path expansion of eq 42 and the
expected realized cost of the trajectory it induces (Property 3) on tiny
random stacks with every selection mode.
Parity unpinned: the paper prints no worked numeric example (no Sim values,
groups, placements or per-token decisions), so no value here is checked
against a number printed in the paper.
"""
from . import layer, placement, route, similarity, tables  # noqa: F401
