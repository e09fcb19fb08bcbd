"""CPU oracle for the vector-index output head (test infrastructure only)."""
