"""Seeded synthetic workload inputs (no simulator arithmetic lives here)."""
