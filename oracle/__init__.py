"""CPU oracle for DKM forward/backward — TEST INFRASTRUCTURE ONLY.

Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import or execute anything in this package.  The product path
(the HIP library and its Python binding) never touches it, and the two share no
code: the only module both sides use is the seeded input generator, which holds
none of the method's arithmetic.

Two oracles live here:

* ``dense``  — the definition: DKM over the full N x k attention map in fp64
  (plain C, ``dkm_dense.c``), forward and reverse-mode backward.
* ``table``  — the uniquified form of the same computation in fp64 numpy, one
  row per distinct fp16 bit pattern weighted by its count (the paper's
  Sec. 2.2 attention table + index list).  It is a second oracle, trusted only
  because the tests pin it to ``dense`` at sizes both can run; it is used for
  spot checks at sizes where the dense oracle is too slow.
"""
