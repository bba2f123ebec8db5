"""CPU oracle of the tree-verification step (test infrastructure only)."""
