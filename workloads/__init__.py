"""Seeded synthetic inputs shared by the oracle tests, the GPU parity tests and
the benchmark: the stack-bytecode format and assembler, the five workload
programs, and their observation/parameter generators.  Nothing here performs
the method's arithmetic (tracing, replay or reverse sweep)."""
from . import bytecode, randtree, configs  # noqa: F401
from .configs import Workload, build, ORDER  # noqa: F401
