"""CPU oracle for the NVFP4 Root Newton-Schulz orthogonalisation.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import, call or run anything in this
package.  The product (the HIP library and its Python binding) never does, and
this package imports nothing from the product except the seeded input
generators, which hold none of the method's arithmetic.

Plain, slow, obviously-correct NumPy code written from the paper:

* ``formats``  - the NVFP4 element (E2M1) and block-scale (E4M3) number formats
                 (Section 2, "NVFP4 format"; OCP 8-bit / 4-bit float definitions).
* ``rht``      - the fresh 16x16 random Hadamard transform (Sections 2 "Others",
                 3.2 and 3.4 display equation).
* ``quantize`` - the NVFP4 quantiser Q_1x16 / Q_16x1 with RTN and adaptive 4/6
                 block scaling (Sections 2 and 3.4).
* ``quantile`` - the p99 outlier threshold (Section 3.4, Table 8 "Root quantile
                 ratio 0.99").
* ``ns``       - Frobenius normalisation and the quantised / unquantised
                 Newton-Schulz recurrence (Section 2 "Root optimizer", Section 3.4
                 display equation).
* ``momentum`` - the first moment kept in NVFP4 with Hadamard mixing, stochastic
                 rounding and adaptive 4/6 (Section 3.3 storage recipe, Section 2
                 "AdamW optimizer" update), the input of the NS orthogonalisation.
* ``root_step`` - the parameter update around the orthogonalised momentum
                 (decoupled weight decay, update scale, BF16 master weights).
* ``qadamw``   - quantized-state AdamW: the first-moment recipe plus the second
                 moment's square-root / BF16 tile-mean / Hadamard pipeline with
                 BF16 block scales (Section 3.3), and the AdamW update.

Floating point: the quantiser is emulated exactly in binary32 (NumPy float32
arithmetic, which rounds each operation to nearest-even and never fuses), the
4/6 block errors and every matrix product are evaluated in binary64.

Pins: ``tests/test_oracle_*.py`` check every function against brute force,
closed forms, library routines and invariants.  Parity of the absolute
quantised Newton-Schulz output values is unpinned beyond this oracle (the paper
prints no such values); see each function's docstring.
"""
