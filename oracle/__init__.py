"""AWSRC reference oracle (test infrastructure only; see awsrc_oracle)."""
from . import awsrc_oracle  # noqa: F401
