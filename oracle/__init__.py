"""CPU oracle for the BITCOS ternary GEMV.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call, link
or execute anything in this package: only the test suite, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` use it.  It
shares no code with the HIP library (no kernels, headers, tables, constant
generators, pre- or post-processing); the two meet only through the seeded
synthetic inputs in ``workloads``.

See ``oracle/bitcos_oracle.py`` for what each function follows in the paper
("Breaking the 1.58-bit Barrier for Ternary LLMs") and how it is pinned.
"""

from .bitcos_oracle import *  # noqa: F401,F403
from .bitcos_oracle import __all__  # noqa: F401
