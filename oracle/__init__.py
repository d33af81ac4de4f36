"""fp64 CPU oracle of the TransX serving path (test infrastructure only)."""
