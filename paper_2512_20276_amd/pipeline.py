"""Cross-request pipeline driver (Alg. 1) over the library's packed forward.

Step t packs request t's prefill (L_P rows) with the single decode row of each request
t-s, s = 1..K-1, still in flight (Eq. (1) order: prefill rows, then stages 1..K-1).  Slots
come from the ring's rotation (af_ring_append); a request is released once it holds K
tokens (the index-rotation form of InPlaceKVShift).

Several independent pipelines (``n_pipes`` = P) can share one forward: step t then packs
the P prefills first and then stage 1 of every pipeline, stage 2 of every pipeline, and so
on (Eq. (1) with each stage widened to P rows).  Request ids are t * P + p.

With ``shift="copy"`` (one pipeline) the stage regions move instead, as the paper's
InPlaceKVShift copy does: stage s always sits in slot s, and after each step the ring
copies every live request's keys and values one slot along (af_ring_shift_stages).  The
attention inputs, and so every output, are the same as with the rotation; only bytes move.

Token feedback stays on the device: the step's greedy tokens are written by the library
straight into the next step's id buffer.  Stage s of step t feeds stage s+1 of step t+1,
and in this row order the stages' tokens (segment order: stage-major) are exactly the next
step's decode ids: ``out_tokens`` of step t is the slice ids_next[P L_P : P L_P + n_seg];
the last P entries of a full step are the final tokens of the requests that complete.
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
    done: object = None             # request completed by this step (a list of them for P > 1)


class Pipeline:
    """Alg. 1 on one GPU, for ``n_pipes`` independent pipelines packed into each forward.

    ``prefill_embeds(t)`` returns a device tensor of at least P (L_P + K - 1) rows whose
    first P L_P rows are the embedding-input rows of the step's P prefills (pipeline p's at
    rows [p L_P, (p + 1) L_P)); rows with a token id (instruction tokens, decode rows) are
    ignored.  ``prefill_ids`` is the device int32 [L_P] id pattern of every prefill (-1 for
    embedding rows)."""

    def __init__(self, weights: Weights, ring: Ring, K: int, prefill_ids: torch.Tensor,
                 prefill_embeds: Callable[[int], torch.Tensor], keep_logits: bool = False,
                 keep_history: bool = True, stream=None, n_pipes: int = 1, shift: str = "rotate"):
        if K < 1 or n_pipes < 1:
            raise ValueError("K >= 1 and n_pipes >= 1")
        if shift not in ("rotate", "copy") or (shift == "copy" and (n_pipes != 1 or K < 2)):
            raise ValueError("shift is 'rotate', or 'copy' for one pipeline with K >= 2")
        self.shift = shift
        self.w, self.ring, self.K, self.P = weights, ring, K, n_pipes
        self.L_P = int(prefill_ids.numel())
        self.prefill_embeds = prefill_embeds
        self.keep_logits, self.keep_history = keep_logits, keep_history
        self.stream = stream
        dev = prefill_ids.device
        D = weights.shape.d_model
        P = n_pipes
        self.M_max = P * (self.L_P + K - 1)
        self.ids = [torch.zeros(P * (self.L_P + K), dtype=torch.int32, device=dev) for _ in range(2)]
        for b in self.ids:
            b[:P * self.L_P] = prefill_ids.repeat(P)
        self.hidden = torch.empty((self.M_max, D), dtype=weights.dtype, device=dev)
        self.logits = (torch.empty((P * K, weights.shape.vocab), dtype=torch.float32, device=dev)
                       if keep_logits else None)
        self.t = 0
        self.counts: Dict[int, int] = {}
        self.history: List[torch.Tensor] = []  # per step: device copy of its tokens

    def request_id(self, t: int, p: int = 0) -> int:
        return t * self.P + p

    def plan(self, t: int):
        """(request id, rows) of step t's segments in packing order."""
        return [(self.request_id(t - s, p), self.L_P if s == 0 else 1)
                for s in range(self.K) if t - s >= 0 for p in range(self.P)]

    def reserve(self, t: int):
        """Appends step t's rows to the ring; returns its segment table (Segment objects)."""
        segs, row = [], 0
        for rid, n in self.plan(t):
            s = self.ring.append(rid, n)
            s.q_start = row
            s.flags = AF_SEG_EMIT
            segs.append(s)
            row += n
        return segs, row

    def finish(self, segs):
        """Counts each request's tokens and releases the slots of the requests that hold K."""
        done = []
        for s in segs:
            c = self.counts.get(s.request_id, 0) + 1
            if c == self.K:
                done.append(s.request_id)
                self.counts.pop(s.request_id, None)
            else:
                self.counts[s.request_id] = c
        for rid in done:
            self.ring.release(rid)
        if self.shift == "copy":
            self.ring.shift_stages(self.K, self.stream)
        return done

    def step(self) -> StepResult:
        t = self.t
        segs, M = self.reserve(t)
        n_seg = len(segs)
        base = self.P * self.L_P
        cur, nxt = self.ids[t % 2], self.ids[(t + 1) % 2]
        out_tokens = nxt[base:base + n_seg]
        emb = self.prefill_embeds(t)
        arr = segments_array(segs)
        packed_forward(self.w, cur[:M], emb[:M], arr, self.ring, self.hidden[:M],
                       self.logits[:n_seg] if self.keep_logits else None, out_tokens, self.stream)
        done = self.finish(segs)
        if self.keep_history:
            self.history.append(out_tokens.clone())
        self.t += 1
        return StepResult(t=t, M=M, segments=[s.astuple() for s in segs], tokens=out_tokens,
                          hidden=self.hidden[:M], logits=self.logits[:n_seg] if self.keep_logits else None,
                          done=done if self.P > 1 else (done[0] if done else None))

    def request_tokens(self, r: int, p: int = 0) -> List[int]:
        """Tokens generated so far for request r of pipeline p (host copy; synchronizes)."""
        out = []
        for s in range(self.K):
            t = r + s
            if t >= len(self.history):
                break
            out.append(int(self.history[t][s * self.P + p].item()))
        return out
