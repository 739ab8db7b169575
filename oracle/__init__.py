"""fp64 CPU oracle for the DiTFastAttn attention hot path (test infrastructure only)."""
