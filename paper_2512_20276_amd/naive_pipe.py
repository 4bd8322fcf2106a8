"""The cross-request pipeline without the unified ring: the "Naive Pipe" ablation of the
paper's evaluation (Sec. 4, Table 1), motivated in Sec. 3.1 and Sec. 3.3.

Same schedule and packing as Alg. 1 (``pipeline.Pipeline``: step t packs request t's prefill
and the decode rows of stages 1..K-1, Eq. (1) order), the same kernels per layer, but the
keys and values are kept the way a stock varlen-attention stack keeps them:

* every request owns a separate KV cache (its own device allocation, all layers, linear in
  position); a pool of K caches is allocated up front and request r uses cache r mod K, the
  steady state of a caching allocator;
* the varlen attention wants the step's histories side by side in one buffer, so before each
  layer the host gathers every decode request's history of that layer (positions 0..pos0-1)
  from its cache into a contiguous one-layer buffer, the layer runs against that buffer (its
  new keys and values land there), and the new rows are copied back to the caches;
* the host coordinates the batch: it waits for the device after every layer before it
  issues the next gather (``sync_per_layer``), and the greedy tokens go through host memory
  to build the next step's input ids.

The outputs are those of ``Pipeline`` (the attention sees the same keys in the same order);
only copies and host round trips are added.
"""
from __future__ import annotations

from typing import Callable, Dict, List

import torch

from . import AF_SEG_EMIT, Ring, Segment, Weights, op_embed, op_lm_head_argmax, packed_layer_forward, \
    segments_array
from .pipeline import StepResult


class NaivePipeline:
    """Alg. 1 for one pipeline with per-request caches and per-layer gather/scatter.

    ``prefill_ids`` (device int32 [L_P], -1 for embedding rows) and ``prefill_embeds(t)``
    (device rows, the first L_P are step t's prefill embedding inputs) are as for
    ``Pipeline``."""

    def __init__(self, weights: Weights, K: int, prefill_ids: torch.Tensor,
                 prefill_embeds: Callable[[int], torch.Tensor], sync_per_layer: bool = True,
                 keep_logits: bool = False, stream=None):
        if K < 1:
            raise ValueError("K >= 1")
        sh = weights.shape
        self.w, self.K, self.sync_per_layer, self.stream = weights, K, sync_per_layer, stream
        self.L_P = int(prefill_ids.numel())
        self.max_pos = self.L_P + K - 1
        self.prefill_ids_host = prefill_ids.cpu()
        self.prefill_embeds = prefill_embeds
        dev = prefill_ids.device
        self.caches = [Ring(sh.n_layers, 1, self.max_pos, sh.n_kv_heads, sh.head_dim, weights.dtype, stream)
                       for _ in range(K)]
        self.staging = Ring(1, K, self.max_pos, sh.n_kv_heads, sh.head_dim, weights.dtype, stream)
        self.hidden = torch.empty((self.L_P + K - 1, sh.d_model), dtype=weights.dtype, device=dev)
        self.tokens = torch.empty(K, dtype=torch.int32, device=dev)
        self.logits = (torch.empty((K, sh.vocab), dtype=torch.float32, device=dev) if keep_logits else None)
        self.counts: Dict[int, int] = {}   # rows cached so far per live request
        self.last: Dict[int, int] = {}     # last generated token per live request (host)
        self.history: List[List[int]] = []
        self.t = 0
        self.copy_bytes = 0                # gather + scatter bytes of the last step (read = written)

    def close(self):
        for r in self.caches:
            r.close()
        self.staging.close()

    def plan(self, t: int):
        return [(t - s, self.L_P if s == 0 else 1) for s in range(self.K) if t - s >= 0]

    def _sync(self):
        (self.stream or torch.cuda.current_stream()).synchronize()

    def step(self) -> StepResult:
        t, K, L_P = self.t, self.K, self.L_P
        sh = self.w.shape
        plan = self.plan(t)
        # host-built batch: segment table over the one-layer gather buffer and the input ids
        self.staging.reset()
        segs, ids, row = [], [], 0
        for rid, n in plan:
            pos0 = self.counts.get(rid, 0)
            s = self.staging.append(rid, pos0 + n)  # region of the buffer: slot s.slot, length pos0 + n
            seg = Segment(row, n, s.slot, pos0, rid, AF_SEG_EMIT, 0)
            segs.append(seg)
            ids.append(self.prefill_ids_host if pos0 == 0 else torch.tensor([self.last[rid]], dtype=torch.int32))
            row += n
        M = row
        arr = segments_array(segs)
        ids_dev = torch.cat(ids).to(self.hidden.device)
        emb = self.prefill_embeds(t)
        hidden = self.hidden[:M]
        op_embed(self.w, ids_dev, emb[:M], hidden, self.stream)
        es = torch.empty((), dtype=self.w.dtype).element_size()
        row_bytes = 2 * sh.n_kv_heads * sh.head_dim * es
        moved = 0
        for l in range(sh.n_layers):
            for seg in segs:  # gather: histories into the contiguous buffer
                if seg.pos0 > 0:
                    self.caches[seg.request_id % K].copy_kv_to(l, 0, self.staging, 0, seg.slot, 0, seg.pos0,
                                                               self.stream)
                    moved += seg.pos0 * row_bytes
            packed_layer_forward(self.w, l, hidden, arr, self.staging, self.stream, ring_layer=0)
            for seg in segs:  # scatter: the new rows back to each request's cache
                self.staging.copy_kv_to(0, seg.slot, self.caches[seg.request_id % K], l, 0, seg.pos0, seg.q_len,
                                        self.stream)
                moved += seg.q_len * row_bytes
            if self.sync_per_layer:
                self._sync()
        n_seg = len(segs)
        op_lm_head_argmax(self.w, hidden, arr, self.logits[:n_seg] if self.logits is not None else None,
                          self.tokens[:n_seg], self.stream)
        toks = self.tokens[:n_seg].cpu().tolist()  # synchronizes: the host builds the next batch
        done = None
        for seg, tok in zip(segs, toks):
            self.counts[seg.request_id] = seg.pos0 + seg.q_len
            self.last[seg.request_id] = tok
        # request t - (K - 1) emitted its K-th token (stage K - 1) and is complete
        if t - (K - 1) >= 0:
            done = t - (K - 1)
            self.counts.pop(done, None)
            self.last.pop(done, None)
        self.history.append(toks)
        self.copy_bytes = moved
        self.t += 1
        return StepResult(t=t, M=M, segments=[s.astuple() for s in segs], tokens=self.tokens[:n_seg],
                          hidden=hidden, logits=self.logits[:n_seg] if self.logits is not None else None, done=done)

    def request_tokens(self, r: int) -> List[int]:
        """Tokens generated so far for request r."""
        return [self.history[r + s][s] for s in range(self.K) if r + s < len(self.history)]
