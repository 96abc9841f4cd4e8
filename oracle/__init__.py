"""CPU oracle for SparseInfer (arXiv 2411.12692) -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  The product path (the HIP library and its Python
binding) never does.
"""

from .sparseinfer_ref import *  # noqa: F401,F403
from .sparseinfer_ref import __all__  # noqa: F401
