"""fp64 CPU oracle of the mixed-task batched forward (test infrastructure only)."""
