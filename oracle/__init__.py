"""Float64 CPU oracle of the DLA layer forward (arXiv 2606.10650).

TEST INFRASTRUCTURE: only tests/, the smoke check and the benchmark's CPU
baseline leg may import this package.  It shares no code with the HIP path.
"""
from .oracle import OracleCache, build_oracle, oracle_forward, oracle_threads  # noqa: F401
