"""Seeded synthetic models, inputs and the model-file writer (test and benchmark input generation)."""
