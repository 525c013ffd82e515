"""CPU oracle for the MoEBlaze layer: test infrastructure only (see oracle.py)."""
