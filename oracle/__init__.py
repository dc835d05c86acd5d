"""CPU oracle (test infrastructure only; see ot_oracle)."""
