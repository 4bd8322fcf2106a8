"""Seeded synthetic inputs for the packed forward: weights, prefill rows, ring contents.

This module is shared by the CPU oracle and the HIP path and therefore holds none
of the method's arithmetic: only random draws, tensor shapes, the storage-dtype
cast of each draw (torch's round-to-nearest-even), and the packing recipes of the
workloads (which request sits in which rows and slots).

Every draw is keyed: ``draw(key, ...)`` seeds a fresh torch generator on the
target device from a stable hash of ``key``, so a tensor does not depend on the
order in which others were drawn.  Values drawn on ``cpu`` and on ``cuda`` differ
(different generators); a test always hands the same bits to both sides by
copying one set.

Model shapes follow the paper's setting (a Llama-2-7B-class decoder, MHA,
RMSNorm, rotary positions, SwiGLU MLP); see the "ActionFlow Pipeline Design"
section for the prefill composition (vision rows followed by instruction rows).
"""
from __future__ import annotations

import dataclasses
import hashlib
from dataclasses import dataclass
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import torch

__all__ = [
    "ModelShape", "TINY", "LLAMA7B", "draw", "draw_ids", "layer_weights",
    "global_weights", "model_weights", "SegmentSpec", "pipeline_prefill_inputs",
    "WEIGHT_STD", "LAYER_TENSORS", "SWEEP_PREFILL", "SWEEP_DECODE", "SWEEP_RING", "sweep_point_specs",
    "STRESS",
]

WEIGHT_STD = 0.02  # linear and embedding weights ~ N(0, 0.02)

# Per-layer tensors, HF [out, in] layout for the projections.
LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")


@dataclass(frozen=True)
class ModelShape:
    """Decoder shape.  ``dtype`` is the storage type of weights and activations."""

    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0
    dtype: str = "bf16"  # "bf16" | "f32"

    @property
    def n_kv_heads(self) -> int:  # multi-head attention throughout
        return self.n_heads

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def with_layers(self, n: int) -> "ModelShape":
        return dataclasses.replace(self, n_layers=n)


# Tiny fp32 decoder: 2 layers, d 256, 4 heads x 64, SwiGLU 688, vocab 512.
TINY = ModelShape(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ff=688, vocab=512, dtype="f32")
# Llama-2-7B shape: 32 layers, d 4096, 32 heads x 128, SwiGLU 11008, vocab 32000.
LLAMA7B = ModelShape(n_layers=32, d_model=4096, n_heads=32, head_dim=128, d_ff=11008, vocab=32000, dtype="bf16")


def _seed(key: Sequence) -> int:
    h = hashlib.sha256(repr(tuple(key)).encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def draw(key: Sequence, shape: Tuple[int, ...], std: float = 1.0, mean: float = 0.0,
         dtype: torch.dtype = torch.bfloat16, device: str | torch.device = "cpu") -> torch.Tensor:
    """N(mean, std^2) draw of ``shape``, cast to ``dtype`` (RNE), from a generator keyed by ``key``."""
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(_seed(key))
    x = torch.randn(shape, generator=g, device=dev, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    if mean != 0.0:
        x.add_(mean)
    return x.to(dtype)


def draw_ids(key: Sequence, n: int, vocab: int, device: str | torch.device = "cpu") -> torch.Tensor:
    """``n`` token ids uniform in [0, vocab), int32."""
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(_seed(key))
    return torch.randint(0, vocab, (n,), generator=g, device=dev, dtype=torch.int64).to(torch.int32)


def layer_weights(shape: ModelShape, layer: int, seed: int = 0, device="cpu",
                  random_gains: bool = False) -> Dict[str, torch.Tensor]:
    """Weights of one decoder layer.  Norm gains are 1 unless ``random_gains``."""
    D, F, Hd = shape.d_model, shape.d_ff, shape.n_kv_heads * shape.head_dim
    dt = shape.torch_dtype
    w = {}
    for name, shp in (("wq", (D, D)), ("wk", (Hd, D)), ("wv", (Hd, D)), ("wo", (D, D)),
                      ("w_gate", (F, D)), ("w_up", (F, D)), ("w_down", (D, F))):
        w[name] = draw(("w", seed, layer, name), shp, std=WEIGHT_STD, dtype=dt, device=device)
    for name in ("attn_norm", "mlp_norm"):
        if random_gains:
            w[name] = draw(("g", seed, layer, name), (D,), std=0.25, mean=1.0, dtype=dt, device=device)
        else:
            w[name] = torch.ones(D, dtype=dt, device=device)
    return w


def global_weights(shape: ModelShape, seed: int = 0, device="cpu",
                   random_gains: bool = False) -> Dict[str, torch.Tensor]:
    """Embedding table, final norm gain and LM head."""
    D, V = shape.d_model, shape.vocab
    dt = shape.torch_dtype
    w = {
        "embed": draw(("w", seed, "embed"), (V, D), std=WEIGHT_STD, dtype=dt, device=device),
        "lm_head": draw(("w", seed, "lm_head"), (V, D), std=WEIGHT_STD, dtype=dt, device=device),
    }
    if random_gains:
        w["final_norm"] = draw(("g", seed, "final_norm"), (D,), std=0.25, mean=1.0, dtype=dt, device=device)
    else:
        w["final_norm"] = torch.ones(D, dtype=dt, device=device)
    return w


def model_weights(shape: ModelShape, seed: int = 0, device="cpu", random_gains: bool = False):
    """(global weights, [layer weights]) for every layer of ``shape``."""
    return (global_weights(shape, seed, device, random_gains),
            [layer_weights(shape, l, seed, device, random_gains) for l in range(shape.n_layers)])


@dataclass
class SegmentSpec:
    """One request's rows in a packed step (host-side description used to build inputs)."""

    request_id: int
    q_len: int
    slot: int
    pos0: int
    emit: bool = True


def pipeline_prefill_inputs(shape: ModelShape, request: int, n_vision: int, text_ids: Optional[torch.Tensor],
                            seed: int = 0, device="cpu") -> Tuple[torch.Tensor, torch.Tensor]:
    """Prefill input of one request: ``n_vision`` N(0,1) embedding rows followed by the
    instruction token ids.  Returns (ids int32 [L_P] with -1 for embedding rows,
    embeds [L_P, D] with zero rows where an id is given)."""
    D = shape.d_model
    n_text = 0 if text_ids is None else int(text_ids.numel())
    L_P = n_vision + n_text
    ids = torch.full((L_P,), -1, dtype=torch.int32, device=device)
    emb = torch.zeros((L_P, D), dtype=shape.torch_dtype, device=device)
    if n_vision:
        emb[:n_vision] = draw(("vision", seed, request), (n_vision, D), dtype=shape.torch_dtype, device=device)
    if n_text:
        ids[n_vision:] = text_ids.to(device=device, dtype=torch.int32)
    return ids, emb


# ----------------------------------------------------------------------------- packed-mix sweep
# One 7B-shape layer over every combination of a prefill of P rows and d single decode rows;
# ring of 16 slots x 544 positions with N(0, 1) history.
SWEEP_PREFILL = (0, 128, 276, 512)
SWEEP_DECODE = (1, 3, 7, 15)
SWEEP_RING = (16, 544)


def sweep_point_specs(P: int, d: int, seed: int = 0) -> List[Tuple[int, int, int]]:
    """(request_id, pos0, q_len) in packing order for sweep point (P, d): the prefill (if any)
    as request 100 at positions 0..P-1, then decode rows of requests 200..200+d-1 whose context
    (kv_len, the new row included) is uniform in {max(1, P), .., P + 7}."""
    g = torch.Generator()
    g.manual_seed(_seed(("sweep kv_len", seed, P, d)))
    lo, hi = max(1, P), P + 7
    kv = torch.randint(lo, hi + 1, (d,), generator=g).tolist()
    specs = [(100, 0, P)] if P > 0 else []
    return specs + [(200 + i, kv[i] - 1, 1) for i in range(d)]


# ----------------------------------------------------------------------------- stress workload
# Eight independent pipelines of depth 8 (a prefill of 256 vision + 20 instruction rows and the
# decode rows of stages 1..7) packed into each forward of the 32-layer 7B shape: M = 8 x 283 =
# 2264 rows in steady state, one ring slot per live request (64 slots x 288 positions).
STRESS = dict(n_pipes=8, K=8, n_vision=256, n_text=20, n_slots=64, max_pos=288)
