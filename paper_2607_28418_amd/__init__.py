"""WIDE token-level dynamic-width masked projections on MI355X (gfx950)."""
