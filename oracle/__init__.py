"""fp64 CPU oracle for the finite-difference Hessian-vector product and
Lanczos / stochastic Lanczos quadrature.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
(the HIP library and its Python binding) never imports, links or calls it, and
this package never imports the product.  The two share nothing except the
seeded input generator in ``synth``, which holds none of the method's
arithmetic.

Contents (each function names the passage of the paper it follows):

* ``model``   - decoder-only LM loss and hand-written reverse pass in float64
                (GPT-2-like and Llama-like families), parameter layout;
* ``hvp``     - central finite-difference HVP (section 3.1, Eq. grad-fd-hvp;
                Algorithm 1) and the quadratic-diagonal test operator;
* ``lanczos`` - Lanczos three-term recurrence with full / windowed / no
                reorthogonalisation (section 4; Appendix C), SLQ nodes and
                weights (section 4), trace estimate;
* ``block``   - the block-diagonal hypothesis statistics (section 6, Exp I).

Parity status: every function here is pinned by ``tests/test_oracle_*.py``
against closed forms, invariants or brute force.  The windowed
reorthogonalisation (Appendix C's window of r stored vectors) is pinned by the
orthogonality pattern it must leave: each new Lanczos vector orthogonal to
rounding level against exactly the r most recent vectors, and measurably not
against the one just outside the window, on a spectrum whose Ritz values
converge early.
"""
