"""CPU oracle for IsoQuant compressed-space decode attention.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, fp64 NumPy
restatement of what the method computes, written to check the GPU library
against.  Only the test suite, the smoke check and the CPU-baseline leg of the
benchmark may import it.  The product path (the C-ABI library and its Python
binding) never imports, links or calls anything here, and this package never
imports the product path: the two share no code, tables or constants.  The
only thing both sides consume is the seeded input generator, which lives in a
module of its own and holds none of the method's arithmetic.

Modules (each function cites the passage of the paper it follows):

* ``codebook``  - Lloyd-Max scalar quantizer levels for the post-rotation
  marginal (Sec. 3.2, Step 3).
* ``rotation``  - seeded unit quaternions, the normalized Walsh-Hadamard
  matrix H_d, the SO(4) block maps v -> q_L v conj(q_R) and the composed
  rotation R = R_SO(4) H_d (Sec. 3.2 Step 2, Eq. 2; Sec. 3.3; App. B).
* ``compress``  - Algorithm 1: normalize, rotate, quantize, bit-pack, at the
  bit width b of the codebook given (b = 3 in the paper's experiments; 2
  and 4 through the same steps with C_2, C_4).
* ``attention`` - decode attention in the compressed space (App. A, Table 2)
  and the reconstruct-then-compute path it replaces (Sec. 1, Fig. 1 top).
* ``rotation_study`` - distortion, coordinate energy and attention error of
  the rotation designs of the ablation (Sec. 4.6) on seeded synthetic K/V.

Parity status: every function is pinned by tests under ``tests/`` against
closed forms, textbook tables, invariants or brute force, except where a
function's docstring says "parity unpinned".
"""


