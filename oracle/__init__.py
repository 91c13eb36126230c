"""CPU oracle for the LibraSpec verification step -- TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 reference of what the GPU library computes, written from the
paper (LibraSpec, arXiv 2608.08721):

* ``selector``  -- the length-selection rule: the simplified speedup objective
  (Sec. 3.2, Eq. 2), single beneficial adjustments (Def. 3.1), the unimodality
  criterion (Thm. 3.5) and Algorithm 1;
* ``accept``    -- greedy and speculative-rejection acceptance of a drafted block
  (Sec. 3.1: the verification step compares q_v and p_v and keeps the target's
  output distribution unchanged);
* ``forward``   -- the single target forward pass over the drafted positions that
  yields p_v (Sec. 3.1), for a pre-norm Llama-style decoder;
* ``philox``    -- Philox4x64-10 (Salmon et al., SC'11), the counter-based RNG that
  the sampling acceptance draws from.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the GPU library
(``paper_2608_08721_amd``) and never imports it; the only common dependency is
the seeded input generator ``synth``, which holds none of the method's
arithmetic.
"""
