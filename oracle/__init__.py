"""CPU oracle for one speculative verification round -- TEST INFRASTRUCTURE.

Plain, slow, fp64 numpy restatements of what the round computes:

* ``gather``    -- KV-state preparation of arriving requests (Prepare(B, w) in
                   Algorithm 1; HostKV extents, Appendix E.1; copy plans, E.4).
* ``attention`` -- target verification of the anchor plus K proposal tokens
                   over the paged KV cache (Sections 1 and 3; Appendix H).
* ``accept``    -- speculative acceptance with residual resampling, the rule
                   of the speculative-decoding works the paper builds on
                   (Leviathan et al. 2023; Chen et al. 2023; cited in
                   Sections 1 and 2; the paper does not restate it).
* ``commit``    -- closing the round: appending the window's K/V to the paged
                   cache, committed lengths, and the suffix written back to the
                   host arena (Section 3; Section 5; Appendix E.1).
* ``draft``     -- the draft stage before verification (Eq. 1): K single-query
                   decode steps over the draft cache and inverse-CDF sampling
                   of each proposal.
* ``schedule``  -- worker-triggered batch reconstruction (Algorithm 1,
                   Eqs. 4-8) and the profiling-driven discrete-event
                   simulator with ideal migration (Appendix H).

Only the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP library
and imports nothing from it; its inputs come from the seeded ``workload``
generator, never from the GPU path.

Every function is pinned by ``tests/test_oracle_*.py`` against a library
routine, closed forms, invariants or a sampling theorem; none is "parity
unpinned".
"""
from . import gather, attention, accept, commit, draft, schedule

__all__ = ["gather", "attention", "accept", "commit", "draft", "schedule"]
