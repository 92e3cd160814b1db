"""CPU oracle for the VSD EM path-scoring hot path -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, deliberately unoptimised restatement of what the
paper's EM step computes (Appendix "Algorithm Detail": Alg. 1, Alg. 2,
Eqs. beta_update, zeta_update, basic, advance; Sec. "Preliminary", Eq. acc;
Sec. "Theoretical Analysis", Eqs. survival_def, accepted_len_cond, EA_def).
It exists to check the HIP implementation and is used only by the tests, by
``__graft_entry__.smoke()`` and by the ``cpu_baseline`` leg of ``bench.py``.
The product path never imports it, and it imports nothing from the product
package: the two share no code.

Precision: all path mathematics in float64; the sampler keys in float32 exactly
as the library's normative sampler definition fixes them (the paper names no
sampler).

Modules
  sampler     Philox4x32-10, the normative log, Gumbel keys, token draws.
  paths       fp64 row statistics, acceptance, survival, oracle gate,
              correction, ARW, CAR, loss, coefficients, gradient.
  bruteforce  exhaustive enumeration over tiny vocabularies (pins only).
"""
