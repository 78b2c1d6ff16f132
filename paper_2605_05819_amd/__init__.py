"""Error-compensated quantized linear layers on MI355X (gfx950)."""
