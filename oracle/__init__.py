"""CPU oracle for dense GEMM (test infrastructure only; see oracle.py)."""
