"""Plain, slow CPU oracle of the MoE-layer hot path of ExpertFlow (arXiv 2410.17954).

This package is TEST INFRASTRUCTURE. It exists to define, in the most direct
form available, what every GPU step must compute, so that the HIP path can be
checked against it element by element. Only the test suite, the smoke check of
the entry module and the CPU-baseline leg of the benchmark may import it; the
product path (the C-ABI library and its Python binding) never does.

Arithmetic: float64 for every floating-point quantity, int64 for every integer.
Inputs are the exact (already bf16- or fp32-rounded) values the GPU receives.
The oracle shares no code with the GPU path: no kernels, headers, helpers or
tables. It imports nothing but NumPy.

Modules and the passages they follow:
  gating    -- softmax gating and top-k expert selection (Sec. 2.1)
  permute   -- expert-major grouping of (token, choice) pairs (implied by the
               batched expert evaluation of Sec. 2.1)
  ffn       -- the SwiGLU expert E_i(x) of Sec. 2.1 (the paper leaves the form
               of E_i open; the models of Table 1 use gated SiLU experts)
  combine   -- the weighted sum y = sum_i G_i(x) E_i(x) of Sec. 2.1, restricted
               to experts resident in the cache (Sec. 3.4, real-time correction)
  schedule  -- routing paths (Sec. 3.2), the rebatching objective (Sec. 3.3.1,
               Eq. 2) and its K-means-style approximation (Sec. 3.3.2)
  slots     -- per-layer resident-set rule from predicted demand (Sec. 3.4.1)
  cache     -- cross-layer slot planning, real-time correction and the LRU
               baseline of the expert cache engine (Sec. 3.4)
  layer     -- the composed MoE layer, the dense-FFN identity used as a pin, and
               a residual stack of pre-normalised layers
  kv        -- KV-cache Merge and Reindex of Sec. 3.3.3
  rpp       -- forward pass of the routing path predictor of Sec. 3.2
"""
from .gating import router_logits, topk_select, softmax, gate_weights, route
from .permute import permute
from .ffn import silu, swiglu, swiglu_loops, expert_ffn
from .combine import combine
from .schedule import (route_bits, eq2_objective, signature_rank, hamming_to,
                       cluster_distance_sums, schedule, batch_accuracy, multi_batch_offsets,
                       schedule_multi)
from .slots import plan_slots
from .cache import plec_order, plec_run, lru_run
from .layer import moe_layer, dense_ffn, moe_stack, round_bf16, rms_norm
from .kv import kv_merge, kv_gather, kv_reindex
from . import rpp

__all__ = [
    "router_logits", "topk_select", "softmax", "gate_weights", "route",
    "permute", "silu", "swiglu", "swiglu_loops", "expert_ffn", "combine",
    "route_bits", "eq2_objective", "signature_rank", "hamming_to",
    "cluster_distance_sums", "schedule", "batch_accuracy", "multi_batch_offsets",
    "schedule_multi", "plan_slots",
    "plec_order", "plec_run", "lru_run",
    "moe_layer", "dense_ffn", "moe_stack", "round_bf16", "rms_norm",
    "kv_merge", "kv_gather", "kv_reindex", "rpp",
]
