"""fp64 CPU oracle of the TNT memory layer.  Test infrastructure only: used by
tests/, the smoke check and the benchmark's CPU baseline, never by the product
path."""
from .tnt_oracle import *  # noqa: F401,F403
