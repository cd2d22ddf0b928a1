"""Seeded synthetic inputs (execution graphs and what-if scenarios)."""
