"""Oracle: the cross-request pipeline (Alg. 1) and the per-request definition it must equal.

TEST INFRASTRUCTURE ONLY (see the package docstring).

``sequential_generate`` is the plain definition: one request alone, with its own
linear KV cache, a causal prefill over its L_P rows, then one single-row decode per
further token (standard autoregressive inference, the paper's Baseline).

``PipelineOracle`` is the method: at step t it packs the prefill of request t with
the single decode row of every request t-s (s = 1..K-1) still in flight, in the
order of Eq. (1) (prefill rows first, then stages 1..K-1), runs one packed forward,
appends each segment's greedy token to its request's partial action sequence and
emits the request that now holds K tokens (Alg. 1).  Readings:
  * the last row of every segment emits a token, the prefill's included (Alg. 1
    applies the LM head to each of the K stages);
  * during warm-up only live requests are packed (no dummy rows);
  * a finished request's slot is released after its step (index-rotation form of
    InPlaceKVShift, see ring.py).
"""
from __future__ import annotations

from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

from .model import F64, OracleModel, OracleRingKV, Segment, linear, rmsnorm, rope, silu
from .ring import RingModel


def _block_linear_cache(model: OracleModel, l: int, x, positions, ck, cv):
    """Textbook decoder block over rows at ``positions`` with a linear cache ck/cv
    [T, H, hd]: write the rows' keys/values at their positions, then attend keys
    0..position with an explicit causal mask."""
    lw, H, hd, eps, rs = model.layers[l], model.H, model.hd, model.shape.rms_eps, model.rs
    n_rows = x.shape[0]
    positions = np.asarray(positions)
    n = rs(rmsnorm(x, lw["attn_norm"], eps))
    q = rs(rope(linear(n, lw["wq"]).reshape(n_rows, H, hd), positions, model.shape.rope_theta))
    k = rs(rope(linear(n, lw["wk"]).reshape(n_rows, H, hd), positions, model.shape.rope_theta))
    v = rs(linear(n, lw["wv"]).reshape(n_rows, H, hd))
    ck[positions] = k
    cv[positions] = v
    T = int(positions.max()) + 1
    mask = np.arange(T)[None, :] <= positions[:, None]          # [n_rows, T]
    o = np.empty((n_rows, H, hd), dtype=F64)
    for h in range(H):
        s = (q[:, h] @ ck[:T, h].T) * model.scale
        s = np.where(mask, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        o[:, h] = (p / p.sum(axis=1, keepdims=True)) @ cv[:T, h]
    o = rs(o.reshape(n_rows, H * hd))
    x = rs(x + linear(o, lw["wo"]))
    m = rs(rmsnorm(x, lw["mlp_norm"], eps))
    a = rs(silu(linear(m, lw["w_gate"])) * linear(m, lw["w_up"]))
    return rs(x + linear(a, lw["w_down"]))


def sequential_generate(model: OracleModel, ids, embeds, n_tokens: int, forced: Optional[Sequence[int]] = None):
    """Generate ``n_tokens`` greedy tokens for one request alone (linear cache).

    ``ids``/``embeds`` are the prefill rows (id -1 takes the embeds row).  With
    ``forced``, token j fed back to the next decode is forced[j] instead of the argmax.
    Returns dict(tokens, logits [n_tokens, V], hidden [L_P + n_tokens - 1, D] (state after
    the last layer of every processed row), cache_k/cache_v [L, T, H, hd]).
    """
    shp = model.shape
    L_P = len(ids)
    T = L_P + n_tokens - 1
    ck = np.zeros((shp.n_layers, T, model.H, model.hd), dtype=F64)
    cv = np.zeros_like(ck)
    hidden = np.zeros((T, shp.d_model), dtype=F64)
    x = model.embed(ids, embeds)
    pos = np.arange(L_P)
    for l in range(shp.n_layers):
        x = _block_linear_cache(model, l, x, pos, ck[l], cv[l])
    hidden[:L_P] = x
    tokens, logits = [], []
    z = model.logits(x[-1:])
    for j in range(n_tokens):
        logits.append(z[0])
        tok = int(model.argmax(z)[0])
        tokens.append(tok)
        if j == n_tokens - 1:
            break
        feed = tok if forced is None else int(forced[j])
        p = L_P + j
        x = model.embed(np.array([feed]), None)
        for l in range(shp.n_layers):
            x = _block_linear_cache(model, l, x, np.array([p]), ck[l], cv[l])
        hidden[p] = x[0]
        z = model.logits(x)
    return dict(tokens=tokens, logits=np.stack(logits), hidden=hidden, cache_k=ck, cache_v=cv)


def top2_margin(z) -> np.ndarray:
    """Gap between the largest and second-largest logit of each row."""
    z = np.sort(np.asarray(z, dtype=F64), axis=-1)
    return z[..., -1] - z[..., -2]


class PipelineOracle:
    """Alg. 1 over the oracle's packed forward.

    ``prefill_fn(t)`` returns (ids [L_P], embeds [L_P, D]) of request t's prefill.
    """

    def __init__(self, model: OracleModel, K: int, n_slots: int, max_pos: int,
                 prefill_fn: Callable[[int], Tuple[np.ndarray, np.ndarray]]):
        if K < 1:
            raise ValueError("K >= 1")
        self.model, self.K = model, K
        shp = model.shape
        self.ring = RingModel(n_slots, max_pos)
        self.kv = OracleRingKV(shp.n_layers, n_slots, max_pos, model.H, model.hd)
        self.prefill_fn = prefill_fn
        self.seqs: Dict[int, List[int]] = {}
        self.t = 0

    def plan(self, t: int) -> List[Tuple[int, int]]:
        """(request, n_rows) of step t in packing order: request t's prefill (n_rows -1 =
        its L_P rows), then the decode row of request t-s for s = 1..K-1 (those that exist)."""
        return [(t - s, -1 if s == 0 else 1) for s in range(self.K) if t - s >= 0]

    def step(self, forced: Optional[Sequence[int]] = None, trace: Optional[list] = None):
        """Run one packed step.  Returns dict(t, segments, ids, embeds, hidden, logits,
        tokens (oracle argmax), used (tokens fed back), margins, done {request: K tokens}).
        With ``trace`` (a list), each layer appends its input, intermediates and output."""
        t, K, D = self.t, self.K, self.model.shape.d_model
        ids_rows, emb_rows, segs = [], [], []
        row = 0
        for (r, n) in self.plan(t):
            if n < 0:
                pids, pemb = self.prefill_fn(r)
                pids = np.asarray(pids)
                n = len(pids)
                ids_rows.append(pids)
                emb_rows.append(np.asarray(pemb, dtype=F64))
                self.seqs[r] = []
            else:
                ids_rows.append(np.array([self.seqs[r][-1]]))
                emb_rows.append(np.zeros((1, D)))
            slot, pos0 = self.ring.append(r, n)
            segs.append(Segment(q_start=row, q_len=n, slot=slot, pos0=pos0, request_id=r, emit=True))
            row += n
        ids = np.concatenate(ids_rows)
        embeds = np.concatenate(emb_rows)
        hidden, z, toks = self.model.forward_packed(ids, embeds, segs, self.kv, trace)
        used = list(toks) if forced is None else [int(v) for v in forced]
        done = {}
        for sg, tok in zip(segs, used):
            self.seqs[sg.request_id].append(int(tok))
            if len(self.seqs[sg.request_id]) == K:
                done[sg.request_id] = self.seqs.pop(sg.request_id)
        for r in done:
            self.ring.release(r)
        self.t += 1
        return dict(t=t, segments=segs, ids=ids, embeds=embeds, hidden=hidden, logits=z,
                    tokens=[int(v) for v in toks], used=used, margins=top2_margin(z), done=done)
