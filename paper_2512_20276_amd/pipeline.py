"""Cross-request pipeline driver (Alg. 1) over the library's packed forward.

Step t packs request t's prefill (L_P rows) with the single decode row of each request
t-s, s = 1..K-1, still in flight (Eq. (1) order: prefill rows, then stages 1..K-1).  Slots
come from the ring's rotation (af_ring_append); a request is released once it holds K
tokens (the index-rotation form of InPlaceKVShift).

Token feedback stays on the device: the step's greedy tokens are written by the library
straight into the next step's id buffer.  Segment j of step t (stage j) feeds stage j+1
of step t+1, so ``out_tokens`` of step t is the slice ids_next[L_P : L_P + n_seg]; the
entry at L_P + K - 1 (if any) is the final token of the request that completes.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional

import torch

from . import AF_SEG_EMIT, Ring, Weights, packed_forward, segments_array


@dataclass
class StepResult:
    t: int
    M: int
    segments: list
    tokens: torch.Tensor            # device int32 [n_seg], segment order
    hidden: torch.Tensor            # device [M, D] residual stream after the last layer
    logits: Optional[torch.Tensor]  # device fp32 [n_seg, V] if requested
    done: Optional[int] = None      # request completed by this step


class Pipeline:
    """Alg. 1 on one GPU.

    ``prefill_embeds(t)`` returns a device tensor [L_P + K - 1, D] (or at least L_P rows
    plus K - 1 spare rows) whose first rows are request t's embedding-input rows; rows with
    a token id (instruction tokens, decode rows) are ignored.  ``prefill_ids`` is the device
    int32 [L_P] id pattern of every prefill (-1 for embedding rows)."""

    def __init__(self, weights: Weights, ring: Ring, K: int, prefill_ids: torch.Tensor,
                 prefill_embeds: Callable[[int], torch.Tensor], keep_logits: bool = False,
                 keep_history: bool = True, stream=None):
        if K < 1:
            raise ValueError("K >= 1")
        self.w, self.ring, self.K = weights, ring, K
        self.L_P = int(prefill_ids.numel())
        self.prefill_embeds = prefill_embeds
        self.keep_logits, self.keep_history = keep_logits, keep_history
        self.stream = stream
        dev = prefill_ids.device
        D = weights.shape.d_model
        self.M_max = self.L_P + K - 1
        self.ids = [torch.zeros(self.L_P + K, dtype=torch.int32, device=dev) for _ in range(2)]
        for b in self.ids:
            b[:self.L_P] = prefill_ids
        self.hidden = torch.empty((self.M_max, D), dtype=weights.dtype, device=dev)
        self.logits = torch.empty((K, weights.shape.vocab), dtype=torch.float32, device=dev) if keep_logits else None
        self.t = 0
        self.counts: Dict[int, int] = {}
        self.history: List[torch.Tensor] = []  # per step: device copy of its tokens

    def plan(self, t: int):
        return [(t - s, self.L_P if s == 0 else 1) for s in range(self.K) if t - s >= 0]

    def step(self) -> StepResult:
        t = self.t
        segs, row = [], 0
        for rid, n in self.plan(t):
            s = self.ring.append(rid, n)
            s.q_start = row
            s.flags = AF_SEG_EMIT
            segs.append(s)
            row += n
        M = row
        n_seg = len(segs)
        cur, nxt = self.ids[t % 2], self.ids[(t + 1) % 2]
        out_tokens = nxt[self.L_P:self.L_P + n_seg]
        emb = self.prefill_embeds(t)
        arr = segments_array(segs)
        packed_forward(self.w, cur[:M], emb[:M], arr, self.ring, self.hidden[:M],
                       self.logits[:n_seg] if self.keep_logits else None, out_tokens, self.stream)
        done = None
        for s in segs:
            c = self.counts.get(s.request_id, 0) + 1
            if c == self.K:
                done = s.request_id
                self.counts.pop(s.request_id, None)
            else:
                self.counts[s.request_id] = c
        if done is not None:
            self.ring.release(done)
        if self.keep_history:
            self.history.append(out_tokens.clone())
        self.t += 1
        return StepResult(t=t, M=M, segments=[s.astuple() for s in segs], tokens=out_tokens,
                          hidden=self.hidden[:M], logits=self.logits[:n_seg] if self.keep_logits else None,
                          done=done)

    def request_tokens(self, r: int) -> List[int]:
        """Tokens generated so far for request r (host copy; synchronizes)."""
        out = []
        for s in range(self.K):
            t = r + s
            if t >= len(self.history):
                break
            out.append(int(self.history[t][s].item()))
        return out
