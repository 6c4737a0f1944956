"""CPU oracle of the LampAttention forward pass (test infrastructure only)."""
