"""CPU oracle (test infrastructure only; see ntc_oracle.h)."""
