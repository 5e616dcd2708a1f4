"""Offline construction of the gfx950 plan table (profiling and compilation)."""
