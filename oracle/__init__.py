"""CPU oracle of the PARK forward -- test infrastructure only (see park_oracle)."""
