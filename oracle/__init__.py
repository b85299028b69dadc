"""CPU oracle for the residual workload predictor and the budgeted expert-swap planner.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously-correct restatement of what the
paper's method computes; it exists to check the HIP implementation.  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may import it.  The product
path (the ``paper_2608_14205_amd`` package and its C ABI library) never imports, links or calls it,
and it shares no code with that path.

Modules
-------
``predictor``  Sec. "Residual Workload Prediction": early router invocation (Eq. 2) of the linear
               router (Eq. 4), the model's own top-k rule, the predicted workload (Eq. 5), the rank
               aggregation of Alg. 1 and the max-to-mean metric of Sec. "Metrics".  float64 GEMM,
               logits rounded to float32.
``planner``    Sec. "Budgeted Expert-Swap Planning": pairwise-swap load update (Eq. 6-7), the load
               objective Phi (Eq. 8) evaluated literally with exact rationals, the deterministic greedy
               ordering and acceptance rule, the frontier restriction and the Alg. 1 loop.
``replicas``   Replicated placements: replica shares of an expert's tokens and the rank loads they
               give (the reading of the "EPLB + Ours" setting).
``cost``       Swap cost (Eq. 9) and attention-window budget (Eq. 10) as a swap count.
``exact``      Micro-oracle for tiny inputs: exact rational dot products rounded once to float32,
               brute-force selections with ``sorted``.

Readings of points the paper leaves open are listed in each function's docstring.
"""
from . import cost, exact, planner, predictor, replicas  # noqa: F401
