"""CPU oracle (test infrastructure only; see ``qlin_ref`` for what it computes).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s cpu_baseline leg
may import this package.  It never imports the product package.
"""
from . import qlin_ref  # noqa: F401
