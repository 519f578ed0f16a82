"""CPU float64 reference of the matching step (test infrastructure only)."""
