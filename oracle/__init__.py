"""CPU oracle (test infrastructure only): a plain float64 NumPy statement of
the Decode-Branch Transformer's inference path.  Only the tests, the smoke
check and the benchmark's CPU-baseline leg may import it."""
from .dbt_oracle import *  # noqa: F401,F403
from .dbt_oracle import expert_assignments  # noqa: F401
