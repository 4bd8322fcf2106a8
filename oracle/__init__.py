"""CPU oracle of the Cross-Request State Packed Forward (ActionFlow, arXiv 2512.20276).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call, link or
execute anything in this package: only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library (no kernels, headers, helpers, tables or constant generators); the two
meet only through the seeded inputs of the ``workload`` module.

It is a plain, slow NumPy implementation in float64.  Where the GPU stores a
tensor in a narrower type (bf16 or fp32), the oracle rounds the same tensor to that
type at the same point (``storage=``), so a comparison measures only the order of
accumulation, not the storage format; ``storage=None`` gives the unrounded model.

Contents
  model.py     per-row math of one decoder layer and the packed forward (Alg. 2,
               Eq. (1)), the final norm, LM head and greedy argmax (Alg. 1)
  ring.py      slot bookkeeping of the Unified KV Ring Buffer (Sec. 3.3), as a
               plain Python state machine
  pipeline.py  the cross-request pipeline (Alg. 1) and the plain per-request
               definition it must reproduce (one prefill, then single-row decodes)

Pins (tests/test_oracle_*.py) tie each function to something other than itself:
closed forms of RMSNorm and RoPE, brute-force float64 attention, the HF Llama
decoder run on the same weights, packed == sequential (the paper's losslessness
claim, Sec. 4.4), ring == linear cache, and the round-robin slot closed form.
"""
from .model import (OracleModel, round_storage, rmsnorm, rope, silu, attend_segment,
                    Segment, OracleRingKV)
from .ring import RingModel, RingError
from .pipeline import PipelineOracle, sequential_generate

__all__ = [
    "OracleModel", "round_storage", "rmsnorm", "rope", "silu", "attend_segment", "Segment",
    "OracleRingKV", "RingModel", "RingError", "PipelineOracle", "sequential_generate",
]
