"""Nested-ancestry routing and aggregation on AMD Instinct MI355X (gfx950)."""
