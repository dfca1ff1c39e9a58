"""fp64 CPU oracle of CCQ (test infrastructure; see ccq_oracle.py)."""
