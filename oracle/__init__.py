"""CPU oracle for GRACE's wide-beam decode attention (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The HIP library never calls it.
"""
from .grace_oracle import *  # noqa: F401,F403
from .grace_oracle import __all__  # noqa: F401
from . import beam_oracle  # noqa: F401,E402
from . import gtm_oracle  # noqa: F401,E402
