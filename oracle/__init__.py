"""fp64 CPU oracle for the MemFine chunked MoE expert layer.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import anything from this
package.  The product path (the HIP library and its Python binding) never
imports, links or calls it, and this package imports nothing from the
product path: the two share no code.

Contents
--------
``moe``          dispatch (stable permutation by expert), the expert SwiGLU
                 FFN, the gate-weighted combine, and the chunked forward /
                 chunked-recompute backward of the paper's FCDA
                 (Section 4.1, Eq. (4)-(7)), in float64 NumPy.
``memory_model`` the paper's memory cost model (Section 3: Eq. (1), Table 2,
                 Eq. (2), Eq. (3)) and the MACT chunk choice (Section 4.2:
                 Eq. (8), Eq. (9), bins), in exact rational arithmetic.

Pins (what each function is checked against, other than itself) are listed
in the module docstrings.  Functions with no independent pin say
"parity unpinned" there.
"""
from . import memory_model, moe  # noqa: F401
