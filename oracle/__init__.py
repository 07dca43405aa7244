"""CPU oracle (test infrastructure only): see ``oracle.stmoe_oracle``."""
