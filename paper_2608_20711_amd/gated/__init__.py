"""Gated verification harness (AsmEvo section 3.7, Algorithm 1; Eq. 2)
around a kernel K0 built from source in this directory."""
