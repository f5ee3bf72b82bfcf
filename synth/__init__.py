"""Seeded synthetic input generators shared by tests, bench and smoke."""
