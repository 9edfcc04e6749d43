"""Plain, slow, fp64 CPU oracle of one FastTPS token-phase decoder layer.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call, link
or execute anything in this package: only the test suite, the smoke check of
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` use it. It shares
no code with the HIP library; the two meet only in the seeded input bits.

Modules:
  ref           -- the layer as the paper defines it, in fp64 (numpy)
  formulations  -- the paper's unfused formulations (Alg. 1, Alg. 2) and the
                   interlaced gate/up layout (Alg. 4, Eq. 29-32), kept apart
                   so the equivalence the paper claims (Section 3) can be
                   checked in fp64
  brute         -- the same layer again in pure Python scalars (math.fsum,
                   exact Fraction rounding), for tiny shapes
  kvquant       -- 8-bit KV cache formats (FP8 E4M3, INT8 with per-head
                   scales) for the layer with a quantized cache

Parity status of each function is stated in its module header.
"""
