"""CPU oracle for (post-)local SGD: test infrastructure only.

Importable by ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg
of ``bench.py``; never by the product package.
"""
from .lsgd_oracle import *  # noqa: F401,F403
from . import lsgd_oracle  # noqa: F401
