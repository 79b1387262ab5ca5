"""CPU oracle for the MixFP4 quantizer, dequantizer and GEMM.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct
restatement of the MixFP4 method (Algorithm 1, Sec. 3.1-3.2, App. B.1-B.3,
with App. D's stochastic rounding and the Hadamard rotation of Sec. 3.2) in
NumPy / Python ``fractions``.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it.  The HIP library never
calls, links or imports anything here, and nothing here imports the HIP
library: the two share no code apart from the seeded input generators in
``workloads``.

Modules
  formats  codebooks built from the value equation, nearest-value rounding
  quant    Algorithm 1 (vectorised over 16-element blocks), packing, dequant
  exact    brute-force rational quantizer (scan all codes, exact squared error)
  gemm     fp64 GEMM of exactly dequantized operands and its tolerance bound
  philox   Philox4x32-10 and the per-element draws of stochastic rounding
  hadamard block-diagonal (random) Hadamard transform, exact then rounded

Every function pinned by a ``-m "not gpu"`` test; see each module's header
for the passages it follows.
"""
