"""Oracle package — TEST INFRASTRUCTURE ONLY.

Plain CPU implementations (numpy float64 and pure-Python loops) of what the
bounded KV-window recomputation path computes.  Only the tests, the smoke check
and the benchmark's CPU-baseline leg may import anything here; the HIP library
and its Python binding never do, and this package imports neither of them.

Parity status: every function is pinned by `-m "not gpu"` tests against
closed forms, invariants the paper states, brute force on tiny inputs and
independent library routines (torch, and the transformers Qwen2 decoder layer).
"""
from . import oracle, brute  # noqa: F401
