"""CPU oracle (test infrastructure only): see ssq_oracle.py."""
