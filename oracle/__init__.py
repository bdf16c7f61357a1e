"""CPU oracle for the DARTS rollout hot path -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously-correct numpy code that states what the rollout path
computes: Philox-seeded random-init weights, a pre-norm decoder forward in
float64, the Gumbel-max sampler with token log-probability and entropy, the
exogenous termination rule, the distribution-aware selection of Alg. 2
(dual-end length sampling, shortest-only tail pruning with proactive early
stopping), and KV page accounting.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path;
the only module both use is ``workload`` (seeded input draws).

Precision: float64 for every model quantity (the paper fixes no precision).
Two places are float32 on purpose because a floating-point value decides an
integer there and both sides must decide in the same precision as the kernel:
the Gumbel perturbed scores whose argmax is the sampled token, and the
accumulated/mean log-probability used as the selection tie-break.

Parity status per function is listed in each module's header.
"""
