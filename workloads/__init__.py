"""Seeded synthetic workloads for the MLA-Online step (no method arithmetic)."""
from .configs import (Geometry, Workload, make_workload, make_custom, f32_to_bf16_bits,
                      bf16_bits_to_f32, round_bf16, ROW_CHUNK, BASE_SEED)
from .router import router_weights, wb_inputs

__all__ = ["Geometry", "Workload", "make_workload", "make_custom", "f32_to_bf16_bits",
           "bf16_bits_to_f32", "round_bf16", "ROW_CHUNK", "BASE_SEED", "router_weights", "wb_inputs"]
