"""CPU oracle (test infrastructure only): see ``partir_oracle``."""
