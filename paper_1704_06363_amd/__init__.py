"""Hard mixture-of-experts hot path for MI355X (gfx950)."""
