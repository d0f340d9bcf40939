"""Oracle for the DASH rollout hot path — TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct CPU implementation of what the GPU path
computes, written from the paper (arXiv 2505.17218, "Effective Reinforcement
Learning for Reasoning in Language Models") and from the decoder definition
the rollouts use:

* :mod:`oracle.model`     — the policy LM forward pass (float64, full causal
  recompute, teacher-forced) that the rollout samples from (Sec. 3, Eq. (1):
  trajectories are drawn from pi_theta).
* :mod:`oracle.sampler`   — temperature sampling by Gumbel-max with
  counter-based Philox4x32-10 noise (float32, bit-exact contract).
* :mod:`oracle.advantage` — the GRPO group advantage (Sec. 3.3, Eq. (4)) and
  the gradient filter (Sec. 3.5), float32, bit-exact contract.
* :mod:`oracle.pg`        — teacher-forced log-probs of sampled completions and
  the policy-gradient loss over the kept samples (Sec. 3.2, Eq. (2)).
* :mod:`oracle.policy`    — the KL regulariser D_KL(pi_base || pi_theta) and the
  clipped PPO surrogate with sequence ratios (Sec. 3.2), float64.
* :mod:`oracle.rollout`   — a whole preemptive-sampling rollout with per-sample
  completion lengths (Sec. 3.4, App. A maximum completion length): the live-row
  schedule, row compaction, page accounting of the group fork, and the tokens.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path
(``paper_2505_17218_amd``) and imports nothing from it; the two meet only in
the seeded input generators, which the callers pass in as plain arrays.

Parity status: every function here is pinned by ``-m "not gpu"`` tests against
closed forms, invariants, library routines or brute force (see each module's
header).  Values for the Qwen2.5-sized random-init shapes beyond those pins are
checked only through the same code that the tiny-shape pins cover.
"""
