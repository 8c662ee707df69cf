"""Float64 CPU oracle (test infrastructure; never used by the product path)."""

from .gradlev_oracle import EXCLUSIVE, INCLUSIVE, decode_step, scan_bwd, scan_fwd

__all__ = ["EXCLUSIVE", "INCLUSIVE", "scan_fwd", "scan_bwd", "decode_step"]
