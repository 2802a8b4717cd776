"""Seeded synthetic inputs (values and conversation traces). Holds none of the method's arithmetic."""
