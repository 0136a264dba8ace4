"""CPU oracle of the TReVS pruning path (test infrastructure only).

Only tests, the smoke check and the benchmark's CPU-baseline leg may import
this package; the HIP library and its binding never do."""

from .trevs_oracle import *  # noqa: F401,F403
