"""CPU oracle of the region-sparse DiT step (test infrastructure only)."""
