"""Kernel K-means oracle (test infrastructure only; see kkm_oracle.py)."""
