"""CPU oracle (test infrastructure only; never imported by the library)."""
from . import fbdt_oracle  # noqa: F401
