"""W4A8 MoE hot path for MI355X (binding filled in below)."""
