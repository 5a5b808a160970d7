"""CPU oracle of the X-Cache cached chunk forward (test infrastructure only).

Imported by ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg; never by the product path.
"""
from .xcache_oracle import *  # noqa: F401,F403
from .xcache_oracle import XCacheOracle, rollout  # noqa: F401
