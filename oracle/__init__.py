"""CPU oracle for Dynamic Memory Sparsification (DMS) inference.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  The GPU library never
calls it and shares no code with it.
"""
from .dms_oracle import *  # noqa: F401,F403
from .latency_model import *  # noqa: F401,F403
from .train_oracle import *  # noqa: F401,F403
from .kv_fp8 import *  # noqa: F401,F403
from .quest import *  # noqa: F401,F403
