"""CPU oracle for the Ripples P-Reduce hot path -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct numpy statement of what the
hot path computes, written from the paper ("Heterogeneity-Aware Asynchronous
Decentralized Training", arXiv 1909.08029).  It exists to check the HIP path.
Only the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg
of ``bench.py`` may import or run it.  The product path (the C-ABI library and
its Python binding) never imports it and has no CPU fallback.

It shares no code with the HIP path: not the arithmetic, not the scheduler,
not the random-number generator of the scheduler.  Inputs (parameters,
gradients) are passed in as arrays; they come from the separate ``seedgen``
module.

Modules
  preduce  -- one step of the algorithm of Fig. 4 (local update, Step 2;
              P-Reduce of each scheduled group, Step 4; the matrix F^G of
              Sec. 3.2) on replicas stored as fp32 or bf16, fp32 arithmetic.
  sched    -- group generation (Step 3): static periodic schedules (Sec. 4.2,
              Fig. 8), the rule table of Fig. 9, the centralized Group
              Generator with per-worker Group Buffers (Sec. 4.1, Sec. 5.1),
              Global Division and the slowdown filter (Sec. 5.1, Sec. 5.3).
  splitmix -- the oracle's own SplitMix64, used only by ``sched``.
"""
