"""Reference oracle for the chunkwise preconditioned delta rule (PDN / PGDN /
PKDA).  TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, float64 CPU implementation of what the paper
"Preconditioned DeltaNet: Curvature-aware Sequence Modeling for Linear
Recurrences" (arXiv 2604.21100) defines.  It exists to check the HIP kernels;
only the tests, the smoke check and the benchmark's CPU-baseline leg may
import it.  The product path (the HIP library and its Python binding) never
imports, calls or falls back to anything here, and nothing here imports the
product path.

Modules
    recurrent   token-by-token recurrences (Eq. precond_end2end and its gated
                forms; identity and external write keys; exact-Gram, diagonal
                Sherman-Morrison and apply-to-query modes of Sec. 3)
    chunkwise   the chunkwise-parallel algebra of App. D, in float64, with every
                per-chunk intermediate exposed
    adjoint     the reverse-mode derivative of the token recurrence
    lsq         brute-force ridge least squares (Sec. 2.3, Eq. normal_eqs)
    abi         conversions between the C-ABI tensor layout and the per-head
                layout used here, plus a per-head process pool

Orientation: the paper's state S_t has shape (d_v, d_k) and o_t = S_t q_t.
The C ABI stores the transpose; `abi` converts at the boundary.
"""
from . import recurrent, chunkwise, adjoint, lsq, abi  # noqa: F401
