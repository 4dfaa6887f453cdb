"""AcceptMoE verify-block MoE layer for MI355X (gfx950)."""
