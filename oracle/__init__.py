"""CPU oracle of BAG's budget-aware cached DiT sampler -- TEST INFRASTRUCTURE.

This package is a plain, slow, float64 NumPy statement of what the sampler
computes.  It exists only to check the HIP implementation: tests, the smoke
check and the CPU-baseline leg of the benchmark may import it; the product
path (the C-ABI library and its Python binding) never does, and this
package imports nothing from that path.

Modules
  numerics  rounding to the storage precision (bf16 / f32)
  dit       the random-init DiT blocks (double-stream, single-stream,
            video cross-attention), embeddings and the final layer
  gate      the gate MLP read from its self-describing blob (Eq. 1)
  sampler   Alg. 2 (budget-exact inference) with the Eq. 3 state,
            plain residual reuse (Sec. 3.1, App. A.1), guidance and the
            Euler flow-matching update

Parity status of each function is stated in its docstring; the only part
without an external pin is the bf16 end-to-end latent of the large
workloads, which the paper does not print (parity unpinned there: it is
checked against this oracle only).
"""
from .numerics import round_bf16, round_f32, round_storage
from .gate import Gate, parse_gate_blob
from .sampler import sample, sigma_schedule, static_schedule, SampleResult, decide, budget_features
from . import dit

__all__ = ["round_bf16", "round_f32", "round_storage", "Gate", "parse_gate_blob",
           "sample", "sigma_schedule", "static_schedule", "SampleResult", "decide", "budget_features", "dit"]
