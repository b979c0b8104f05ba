"""Float64 CPU oracle for one FP32 GPT-2 training step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package; only the test-suite, the smoke check and the CPU
baseline leg of the benchmark use it.  It shares no code with the HIP path:
it is a plain, slow, obviously-correct transcription of the definitions of
each operation, accumulated in float64.

Every function cites the passage of the paper it follows (section, figure,
table or algorithm).  Where the paper is silent the reading taken is stated
in the function's docstring.

Parity status: every function is pinned by tests against closed forms,
invariants, brute force or an independent library routine (see the
``tests/test_oracle_*.py`` suites); the full 124M step is pinned only through
its parts plus the zero-embedding ln(V) loss.
"""
from . import ops, gpt2, context_parallel  # noqa: F401
