"""CPU oracle for memoized DNN mutation testing -- TEST INFRASTRUCTURE ONLY.

This package is the plain, slow reference the GPU library is checked against.
Only the test-suite, the smoke check and the CPU-baseline leg of the benchmark
may import it; the product path never does.

Contents
  numerics   -- bfloat16 round-to-nearest-even and the rounding points
  layers     -- the layer functions Phi(v) and the activation recursion a_v
                (Section 4) with float64 accumulation
  mutate     -- the four neuron-level operators (Section 3.1)
  vanilla    -- exhaustive ("vanilla") mutation testing, the kill predicate,
                killingLabels and the mutation score (Section 5.2), margins
                and the ambiguous-pair set
  memoized   -- Algorithms 1-4 (dependence graph, memoization boundary,
                clustering, instrumentation, chopping) taken step by step,
                used to check the soundness theorem (Theorem 1) by brute force
  ledger     -- the additive MAC cost model of Section 4.2 (axioms C1-C3,
                Lemma 4)

Every function is pinned by the CPU tests (tests/test_oracle_*.py) to
something outside itself: library routines in float64, brute-force loops on
tiny inputs, closed forms on the output layer, Table 1's parameter counts and
hand-worked kill/score fixtures.  Logit values of the five synthetic workloads
have no printed counterpart in the paper: beyond those pins they are "parity
unpinned".
"""
from .numerics import rne_bf16, bf16_bits_to_f32
from .layers import OracleModel, forward, forward_all
from .mutate import apply_records
from .vanilla import VanillaResult, run_vanilla, kill_and_score, margins, pack_bits
from .memoized import get_dep_graph, boundary, mure, instrument, chop_mutant
from .ledger import node_macs, cluster_costs

__all__ = [
    "rne_bf16", "bf16_bits_to_f32", "OracleModel", "forward", "forward_all",
    "apply_records", "VanillaResult", "run_vanilla", "kill_and_score", "margins",
    "pack_bits", "get_dep_graph", "boundary", "mure", "instrument", "chop_mutant",
    "node_macs", "cluster_costs",
]
