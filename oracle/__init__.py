"""CPU oracle for the simulated-ring AllReduce -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import anything from this package.  The HIP product path never
imports, links or executes it, and it shares no code with that path.

``ring_oracle`` is the numpy oracle; ``c_oracle`` builds and calls the
equivalent plain-C oracle used for CPU timing.
"""
from . import ring_oracle  # noqa: F401
