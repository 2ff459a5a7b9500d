"""Seeded synthetic inputs shared by the oracle and the HIP path."""
