"""Test infrastructure: the CPU oracle of the QSVD hot path (see qsvd_oracle)."""
