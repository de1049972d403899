"""Seeded synthetic inputs for the re-batched decode step (input generation only)."""
