"""CPU oracle for the SAEF round -- test infrastructure only (see oracle.py)."""
