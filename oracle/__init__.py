"""CPU oracle (test infrastructure): see simplicial_oracle.py.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg import this
package. Parity status of every function is listed in simplicial_oracle.py's
header; all are pinned (none is "parity unpinned").
"""

from .simplicial_oracle import *  # noqa: F401,F403
from .simplicial_oracle import __all__  # noqa: F401
