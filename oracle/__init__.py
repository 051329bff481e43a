"""CPU oracle of the MoE expert-FFN layer: test infrastructure, never part of the library's
compute path (see moe_oracle's header)."""
