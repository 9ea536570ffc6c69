"""CPU oracle for the BFLA hot path -- test infrastructure only (see bfla_oracle)."""
