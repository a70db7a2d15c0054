"""fp64 CPU oracle for the GCN training path (test infrastructure only; see oracle.py)."""
