"""CIERA reference oracle: test infrastructure only (see oracle.py)."""
