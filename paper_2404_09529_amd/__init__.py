"""Packed prefill (Prepacking) for AMD Instinct MI355X (gfx950)."""
