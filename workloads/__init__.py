"""Workload definitions shared by tests and the benchmark: model parameter
tables and seeded synthetic round inputs.  Nothing here computes any part of a
synchronisation round."""
