"""CPU oracle (test infrastructure only; never on the product path)."""
from .rosa_oracle import (OracleModel, attention, gelu_tanh, modulate, rms_norm, silu,
                          softmax_rows, tau_grid, timestep_embedding)
from .prefill import prefill, prefill_context
from .homogeneous import schedule_homogeneous
from .s1_batching import rank_percentile, select_batch, simulate_worker

__all__ = ["OracleModel", "attention", "gelu_tanh", "modulate", "rms_norm", "silu",
           "softmax_rows", "tau_grid", "timestep_embedding", "rank_percentile", "select_batch", "simulate_worker", "prefill",
           "schedule_homogeneous", "prefill_context"]
