"""Float64 CPU oracle for log-linear attention (Guo et al., "Log-Linear Attention").

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports, calls or links this
package: only the test-suite, the smoke check and the benchmark's CPU-baseline leg
do.  It shares no code with the HIP library: it is plain NumPy/SciPy in float64,
written from the paper's definitions, slow and obviously correct.

Modules
-------
fenwick   Fenwick bucket partition and the level function l(t, s)   (Sec. 3.1 footnote)
mamba2    log-linear Mamba-2: quadratic masked form, per-level recurrent form,
          brute force, and the special cases it must reduce to        (Eqs. 1-4, Sec. 3.2, 3.4)
mamba2_grad  gradients of log-linear Mamba-2 with respect to q, k, v, log alpha and lambda,
          from the quadratic form by the chain rule (full and sampled rows/columns)
gdn       log-linear Gated DeltaNet: the same three forms              (Sec. 2 delta rule, Sec. 3.4)
matrix_lambda  log-linear Mamba-2 with matrix-valued level weights Lambda_t^(l) (the 4D-tensor
          view of App. A): quadratic, recurrent and brute-force forms

Every function works on arrays laid out as [B, T, H, ...] (batch, time, head, feature),
the layout of the paper's own PyTorch listing (App. C), and returns float64.
"""

from . import fenwick, mamba2, mamba2_grad, gdn, matrix_lambda  # noqa: F401
