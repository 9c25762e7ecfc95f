"""CPU oracle (test infrastructure): see simplicial_oracle.py (the trilinear
form of Section 4) and determinant_oracle.py (the determinant form of
Section 5, imported as `oracle.determinant_oracle`).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg import this
package. Every function of both modules is pinned (none is "parity unpinned"):
tests/test_oracle_pins.py, tests/test_oracle_mutations.py and
tests/test_determinant_oracle.py.
"""

from .simplicial_oracle import *  # noqa: F401,F403
from .simplicial_oracle import __all__  # noqa: F401
