"""CPU oracle for the expert-server forward step (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's cpu_baseline
leg may import this package.  The product path never calls it.
"""
from .eaas_oracle import *  # noqa: F401,F403
from .segments_oracle import *  # noqa: F401,F403
from .server_oracle import *  # noqa: F401,F403
from .w8a8_oracle import *  # noqa: F401,F403
