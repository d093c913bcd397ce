"""Plain, slow CPU oracle of KnapSpec's self-speculative decode step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product package imports, calls or
executes anything here; only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` do.  It shares no code with the HIP path:
its only input dependency is the seeded generator module ``workloads``.

Arithmetic is float64 throughout.  For bf16 models the weights are the
generator's bf16 values and keys/values are rounded to bf16 when stored in the
cache, because that is the storage format of the workload; all other values
stay float64.

Modules
-------
``model``     decoder forward, skip masks, greedy AR, the greedy speculative round
              and generation loop (Section 2 and 2.1 of the paper).
``select``    cosine similarity, the model-mode knapsack DP (Algorithm 1 /
              Eq. h_candidates, dp_main), stage 2 (Algorithm 2, Eq. acceptance,
              Eq. TPT), brute force over skip masks.
``latency``   latency model fit and integer weight normalisation (Section 3.4,
              Appendix C).
``additive``  the isolated integer knapsack (additive log-loss surrogate of the
              per-budget problem, Eq. objective_knapsack) and its brute force.

Parity status per function is stated in each module header.
"""
