"""Memory-efficient exact attention for MI355X (gfx950)."""
