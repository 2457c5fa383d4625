"""Seeded synthetic instance generators (no schedule arithmetic)."""
