"""CPU oracle for the acoustic-to-text streaming KV step — TEST INFRASTRUCTURE ONLY.

This package is the slow, plain, float64 reference that the GPU library is
checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run it; the product path
(the HIP library and its Python binding) never does, and it shares no code,
constants or helpers with that path.  Its only shared dependency is the
seeded input generator in ``synth/``, which holds none of the method's
arithmetic.

What it computes, following the paper:

* ``rope``      rotary position encoding of keys and queries at their original
                position ids (Sec. 3.3: kept keys keep their rotary positions
                and are never re-encoded).  Rotate-half convention, theta a
                parameter (the paper names neither; see the readings list).
* ``attention`` causal grouped-query softmax attention of a step's new rows
                over the resident cache — the plain definition, written out.
* ``policy``    the online budgeted eviction rule of Sec. 3.3, step by step
                in the paper's order, plus the stable compaction indices.
* ``cache``     a per-stream cache that appends, attends and evicts.
* ``replay``    metadata-only policy passes and state reconstruction
                (resume at any unit).

Parity status: every function here is pinned by ``tests/test_oracle_*.py``
against closed forms, invariants, a brute-force re-derivation of the policy
and a library routine (torch CPU float64 attention).  The RoPE variant and
theta are a reading, not a paper value: their parity is internal only.
"""
