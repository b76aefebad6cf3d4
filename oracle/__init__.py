"""CPU oracle for the cached N-candidate DiT rollout.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, float64 numpy
implementation written from the paper's definitions, used to check the GPU
path.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
may import it; the library and its binding never do, and the oracle never
imports them.

Modules:
  dit      -- the transformer velocity model (parity unpinned by the paper:
              its internals are this project's Wan-shaped spec; primitives
              are pinned against library routines and identities)
  rollout  -- cache rule, Euler/CFG update, scorer (Sec. Method, Eqs.
              euler, cfg, delta, skip, indicator; Alg. 1)
  rank     -- ranking and Spearman correlation (Sec. Experiments,
              definitions and protocol)
"""
