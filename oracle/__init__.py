"""CPU oracle for the fixpoint engine (test infrastructure only; see datalog.py)."""
from .datalog import ConvergenceFailure, OracleResult, evaluate, parse  # noqa: F401
