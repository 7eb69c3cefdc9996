"""fp64 CPU oracle for the STAR-KV decode path (test infrastructure only)."""
