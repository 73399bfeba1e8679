"""CPU oracle (test infrastructure only; see pblock_oracle)."""
