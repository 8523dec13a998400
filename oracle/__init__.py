"""Float64 CPU oracle for exact attention backward-over-backward (BoB).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this package: only the test suite, the smoke check and the CPU
baseline leg of the benchmark use it.  It shares no code with the HIP
library and never consumes a value produced by it.

Every function takes plain NumPy arrays, works in float64 and materialises
the full (or row-slab) N x N attention matrices, following the paper's
definitions directly (Sec. 2 eqs. 1-3, Sec. 3.1 eqs. 4-5, Sec. 3.2 eqs. 6-8,
App. A "Final assembled identities", App. B proof of Prop. 3.1, and the three-pass control schedule of App.
"Three-pass versus two-pass"), plus grouped key/value heads, the extension the
paper names in its limitations.
"""
from .bob_oracle import (  # noqa: F401
    forward_head,
    first_backward_head,
    bob_head,
    bob_affine_head,
    bob_threepass_head,
    first_backward_rowloop,
    phi_rowloop,
    forward,
    first_backward,
    bob,
    bob_rows,
    bob_affine,
    bob_threepass,
    row_scalars,
    row_scalars_slab,
    bob_cols,
    bob_gqa,
    expand_kv,
    group_sum,
)
