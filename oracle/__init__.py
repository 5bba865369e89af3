"""CPU oracle for the tiered-memory (HBM + host) decode path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(the HIP library and its Python binding) never calls it and shares no code with
it: the only common module is ``synth`` (seeded input generators).

Every function here is plain and slow on purpose: NumPy (fp64 unless stated),
written from the paper (BOOST: Concurrent Access to Host Memory and HBM to
Accelerate LLM Inference), each citing the passage it follows.

Modules
  placement  -- C1 modulus from the bandwidth ratio, C2 modulo page placement
                (MPP) with superpages, C3 modulus from an HBM budget, and the
                contrast placements (random BAPP-R, linear).
  kvpool     -- C4 KV pool geometry (linear page placement + heads-outermost
                layout), C5 the wave-aware block allocator (DSR).
  gemv       -- C6 y = W x with fp32 / fp64 accumulation, bf16 encode/decode.
  attention  -- C7 GQA decode attention over logical K/V.
  waves      -- C9 per-wave host fraction of a unit schedule.

Pins: every function is checked by ``tests/test_oracle_*.py`` against values the
paper prints, closed forms, invariants and brute force.  Functions whose exact
output the paper does not fix (allocator tie-breaks) say "parity unpinned" in
their docstring; their invariants are still pinned.
"""
