"""CPU oracle (test infrastructure only; see grinqh_oracle)."""
