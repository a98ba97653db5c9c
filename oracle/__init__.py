"""Float64 CPU oracle of SelKV (test infrastructure only; see selkv_oracle)."""
from . import selkv_oracle  # noqa: F401
