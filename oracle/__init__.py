"""CPU oracle for the MOSAIC hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, deliberately unoptimised implementation of what the GPU path
computes, written from the paper's definitions (arxiv 2607.29221):

* ``philox``    -- the counter-based generator (Salmon et al., SC'11) that both
                   sides use for the random mask material;
* ``sampling``  -- uniform ring elements, the discrete Gaussian of Section 4.1
                   ("Bounded protocol error"), LPN sparse noise of rate mu
                   (Background) and of fixed row weight t (Example 4.1);
* ``ring``      -- Z_{2^32} matrix arithmetic and the signed-digit encoding
                   used by the 8-bit emulation (Section 6.1, "Emulation
                   approach");
* ``protocol``  -- Pi_Sec-Approx-MatMul of Section 4.2 (protocol box): Init W,
                   Init X, the server product, unmasking;
* ``hadamard``  -- the random Hadamard rotation of Section 5 and Fino's fast
                   Walsh-Hadamard transform;
* ``quant``     -- the per-row fixed-point quantisation of Pi_Sec-Linear.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. It shares no code with the HIP path and
imports nothing from it; the only shared module is ``synthetic_inputs`` (seeded
input generators, no arithmetic of the method).
"""
