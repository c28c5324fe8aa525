"""CPU oracle for nested-Winograd convolution -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import anything from this package.  The product (the HIP
library and its Python binding) never imports, links or calls it, and this
package never imports the product.

Contents
--------
direct   -- the plain definition: stride-1 2D correlation in fp64
            (Sec. II.A), as shifted GEMMs, plus a brute-force loop version.
nested   -- a slow, plain CPU nested-Winograd reference (Sec. III.B,
            eqs. 2.1-2.3, Alg. 1 read as a chain of n identical bases) in
            fp64 or exact rationals, used to check the GPU's intermediate
            stages and to count multiplications.
lindecomp-- the linear-decomposition Winograd algorithm (Sec. II.B) on the
            CPU, used for the multiplication-count comparison of Sec. III.C.
counts   -- closed-form multiplication complexities (eqs. 3.2, 3.3).

Every function is pinned by ``tests/test_oracle_*.py`` to facts that do not
come from this package: brute-force sums, library routines
(scipy.signal.correlate, torch.nn.functional.conv2d in float64), exact
rational identities, and the numbers the paper prints.
"""
