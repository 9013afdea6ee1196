"""CPU oracle of the Rift hot path: test infrastructure only (see rift_oracle)."""
from . import rift_oracle  # noqa: F401
