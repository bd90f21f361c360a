"""CPU oracle (test infrastructure only; see adadsf_oracle for the contract)."""
from . import adadsf_oracle  # noqa: F401
