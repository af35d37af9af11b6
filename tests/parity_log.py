"""Record of the per-tensor errors measured by the GPU parity tests.

Every GPU parity check calls ``check_err`` (or ``record``), which keeps the
measured max relative error beside its bound; at the end of the session
``tests/conftest.py`` writes the table to ``gpurun_out/parity_margins.tsv`` so
the margins of each run are on record.
"""
import math

_ROWS = []


def record(case: str, tensor: str, err: float, tol: float) -> None:
    _ROWS.append((case, tensor, float(err), float(tol)))


def check_err(case: str, tensor: str, err: float, tol: float) -> bool:
    """Record and return whether ``err`` is finite and within ``tol``."""
    record(case, tensor, err, tol)
    return math.isfinite(err) and err <= tol


def rows():
    return list(_ROWS)
