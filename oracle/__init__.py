"""CPU oracle (test infrastructure only; see fw_oracle.py)."""
