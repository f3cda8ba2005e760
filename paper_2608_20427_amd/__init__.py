"""BF1 causal dyadic block-sparse attention for MI355X (gfx950)."""
