"""CPU oracle for the W4A4 path -- test infrastructure only (see oracle.py)."""
