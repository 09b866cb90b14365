"""CPU oracle of the decode path (test infrastructure only)."""
