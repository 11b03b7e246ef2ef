"""CPU oracle (test infrastructure only; see saga_oracle)."""
from . import saga_oracle  # noqa: F401
