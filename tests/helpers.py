"""Test-side glue: hands the same seeded bits to the oracle and to the HIP path."""
from __future__ import annotations

import numpy as np
import torch

import workload as wl


def to_np(t: torch.Tensor) -> np.ndarray:
    """Exact float64 copy of a (bf16/fp32) tensor."""
    return t.detach().to("cpu", torch.float64).numpy()


def weights_np(globals_, layers):
    g = {k: to_np(v) for k, v in globals_.items()}
    ls = [{k: to_np(v) for k, v in lw.items()} for lw in layers]
    return g, ls


def oracle_model(shape, globals_, layers, storage="match"):
    import oracle
    if storage == "match":
        storage = "bf16" if shape.dtype == "bf16" else "f32"
    g, ls = weights_np(globals_, layers)
    return oracle.OracleModel(shape, g, ls, storage=storage)


def tiny_prefill_fn(shape, L_P, seed=0, n_vision=None, device="cpu"):
    """Prefill of request t for the tiny config: token ids uniform in [0, V) (all rows
    are ids unless ``n_vision`` rows of N(0,1) embeddings lead)."""
    nv = 0 if n_vision is None else n_vision

    def fn(t):
        text = wl.draw_ids(("prompt", seed, t), L_P - nv, shape.vocab, device=device)
        ids, emb = wl.pipeline_prefill_inputs(shape, t, nv, text, seed=seed, device=device)
        return ids.cpu().numpy().astype(np.int64), to_np(emb)

    return fn


def allclose_report(got, ref, atol, rtol):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = np.abs(got - ref)
    bound = atol + rtol * np.abs(ref)
    bad = err > bound
    return dict(ok=not bad.any(), n_bad=int(bad.sum()), max_abs=float(err.max(initial=0.0)),
                max_rel=float((err / np.maximum(np.abs(ref), 1e-30)).max(initial=0.0)),
                rms=float(np.sqrt(np.mean(err ** 2))) if err.size else 0.0)
