"""ID Balancing router step and bias controller for AMD MI355X (gfx950)."""
