"""Plain fp64 CPU oracle for the BiCache shared-prefix denoising step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product library imports, links or
calls this package; only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
path: every function here is written from the paper's definitions, in NumPy
float64, with no blocking, fusion or reordering beyond what those definitions
state.

Modules
-------
attention     Eq. 2 bidirectional (unmasked) softmax attention, and the
              shared-prefix form used by the shallow layers (Eq. 4).
transformer   The per-layer forward, the prefix-only populate (Sec. 5.2,
              "on a miss ... computes the KVs for p at the first step for all
              layers"), the step at reuse depth d (Eq. 4 and the refresh case of
              Eq. 5) and the un-cached full forward ("no caching").
xxh64         The 64-bit xxHash used as the prefix key (Appendix C), from the
              published algorithm.
cache_table   A Python model of the FIFO-evicting KV store H (Appendix C).

Parity status: every function has a pin in ``tests/test_oracle_*.py``.  The
one reading the paper leaves open -- which prefix hidden state enters the first
deep layer -- is pinned only by the invariants it implies (see
``transformer.step``); the paper prints no reference values for the forward.
"""
