"""CPU oracle of SMAT's simulate / backward-accumulate / storage-switch path.

Test infrastructure, not product code: only `tests/`, the package's
`smoke()` check and the benchmark's CPU-baseline leg may import it.  It
shares no code with the HIP path (no kernels, headers, helpers or tables) and
imports nothing from it.  Every function is pinned by CPU tests to facts the
paper or the mathematics fix (known-answer vectors, closed forms, moments,
finite differences, library routines); none is "parity unpinned".
"""
from . import smat_oracle
from .smat_oracle import *  # noqa: F401,F403
