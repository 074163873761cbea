"""CPU oracle of the resident-expert MoE layer (test infrastructure only)."""
