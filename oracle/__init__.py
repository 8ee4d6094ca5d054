"""CPU oracle (test infrastructure only; never used by the product path)."""

from .moe import combine, expert_ffn, layer, layout, local_map, permute, route, router_logits, token_output

__all__ = ["router_logits", "route", "local_map", "layout", "permute", "expert_ffn", "combine", "layer", "token_output"]
