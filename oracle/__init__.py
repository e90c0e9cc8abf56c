"""fp64 CPU oracle for SSBA -- test infrastructure only (tests, smoke check,
benchmark CPU baseline).  Never imported by the product path."""
from . import ssba_oracle  # noqa: F401
