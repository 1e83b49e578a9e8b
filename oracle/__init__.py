"""CPU reference implementation of LM-GC (arXiv 2409.17836) -- TEST INFRASTRUCTURE.

This package is the oracle against which the GPU library is checked.  It is
plain and slow on purpose: NumPy float64 for the decoder forward pass
(forward.py), plain C for serialisation, table quantisation and arithmetic
coding (coder.c), and a straightforward codec driver (pipeline.py).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import it.  The GPU library never does, and this package never imports the
GPU library.  Inputs come from the seeded generators in `synth`, which hold
none of the method's arithmetic.

Every function is pinned by tests under tests/ against closed forms, the
paper's worked arithmetic-coding example, brute force on tiny inputs and
library routines; none is "parity unpinned".
"""
