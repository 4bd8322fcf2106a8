"""Oracle: one decoder layer over a packed Cross-Request State, and the model around it.

TEST INFRASTRUCTURE ONLY (see the package docstring): float64 NumPy, no blocking,
no fusion.  Each function names the passage of the paper it follows.

Readings of the paper used here (the paper leaves these open or garbles them):
  * The block is the standard sequential pre-norm Llama block: attention residual
    first, then the MLP residual on the norm of the updated stream.  The printed
    Alg. 2 update line reads as if the MLP consumed the pre-projection attention
    output; the paper runs the unmodified OpenVLA/Llama-2 backbone and claims the
    method is lossless against it (Sec. 4.4), so the textbook block is the definition.
  * Norm = RMSNorm with gain, eps from the model (1e-6); the paper says "LayerNorm"
    only in passing.
  * RoPE pairs dimension j with j + hd/2 ("rotate half"), theta = 10000, at the
    0-based absolute position of the row inside its own request (Sec. 3.3: the
    rotary position is the logical position within the original request).  A decode
    row of stage s has position L_P + s - 1, i.e. its KV length minus one.
  * New keys/values are written to the ring before attention, so a row sees its own
    key (Alg. 2: the write precedes the varlen attention).
  * Softmax scale 1/sqrt(hd), multi-head attention (no grouping), no biases.
  * Greedy token = the lowest index attaining the maximum logit over the full vocab.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np

F64 = np.float64


# ----------------------------------------------------------------------------- storage
def round_storage(x, storage: Optional[str]):
    """Round float64 values to the storage type the GPU keeps them in.

    ``storage`` is None (no rounding), "f32" (IEEE single, round-to-nearest-even)
    or "bf16" (the float64 value rounded to single, then the single rounded to
    bfloat16 by round-to-nearest-even on its upper 16 bits; the GPU rounds its fp32
    accumulators the same way).
    """
    x = np.asarray(x, dtype=F64)
    if storage is None:
        return x
    f = np.ascontiguousarray(x.astype(np.float32))
    if storage == "f32":
        return f.astype(F64)
    if storage != "bf16":
        raise ValueError(f"unknown storage {storage!r}")
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)).astype(np.uint32)
    return r.view(np.float32).astype(F64)


# ----------------------------------------------------------------------------- per-row math
def rmsnorm(x, g, eps):
    """RMSNorm over the last axis: g * x / sqrt(mean(x^2) + eps).  (Alg. 2 "Norm".)"""
    x = np.asarray(x, dtype=F64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(g, dtype=F64)


def rope(u, pos, theta):
    """Rotary embedding of head vectors ``u`` [..., n_heads, hd] at absolute positions
    ``pos`` (broadcast over u.shape[:-2]).  Pair (j, j + hd/2) is rotated by the angle
    pos * theta^(-2j/hd).  (Sec. 3.3, FusedRoPEAndWriteKV.)"""
    u = np.asarray(u, dtype=F64)
    hd = u.shape[-1]
    half = hd // 2
    j = np.arange(half, dtype=F64)
    omega = np.power(F64(theta), -2.0 * j / hd)
    phi = np.asarray(pos, dtype=F64)[..., None, None] * omega  # [..., 1, half]
    c, s = np.cos(phi), np.sin(phi)
    a, b = u[..., :half], u[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(z):
    """SiLU(z) = z / (1 + exp(-z))."""
    z = np.asarray(z, dtype=F64)
    return z / (1.0 + np.exp(-z))


def linear(x, w):
    """x @ w.T with w in [out, in] layout (library matmul, float64)."""
    return np.asarray(x, dtype=F64) @ np.asarray(w, dtype=F64).T


def attend_segment(q, pos, keys, values, scale):
    """Attention of the query rows of one segment and one head over that request's keys.

    q [n, hd] are rows at absolute positions pos [n]; keys/values [kv, hd] hold the
    request's history at positions 0..kv-1.  Row i sees keys 0..pos[i] (causal inside a
    prefill segment, the full history for a decode row).  Softmax subtracts the row max.
    (Alg. 2 VarlenAttention; Sec. 3.2: each segment attends only its own history.)
    """
    q = np.asarray(q, dtype=F64)
    k = np.asarray(keys, dtype=F64)
    v = np.asarray(values, dtype=F64)
    pos = np.asarray(pos)
    s = (q @ k.T) * scale                                        # [n, kv]
    visible = np.arange(k.shape[0])[None, :] <= pos[:, None]
    if not np.all(visible.any(axis=1)):
        raise ValueError("a query row sees no key")
    s = np.where(visible, s, -np.inf)
    s = s - np.max(s, axis=1, keepdims=True)
    p = np.exp(s)
    p = p / np.sum(p, axis=1, keepdims=True)
    return p @ v


# ----------------------------------------------------------------------------- packed state
@dataclass
class Segment:
    """Rows [q_start, q_start + q_len) of the packed state belong to one request whose
    KV lives in ring slot ``slot``; the first row sits at absolute position ``pos0``."""

    q_start: int
    q_len: int
    slot: int
    pos0: int
    request_id: int = -1
    emit: bool = True

    @property
    def kv_len(self) -> int:
        return self.pos0 + self.q_len


class OracleRingKV:
    """Contents of the Unified KV Ring Buffer in logical form: per layer,
    k/v [n_slots, max_pos, n_heads, hd] (Sec. 3.3: one region, logically partitioned
    per request).  Slot bookkeeping lives in ``ring.RingModel``."""

    def __init__(self, n_layers, n_slots, max_pos, n_heads, head_dim):
        shp = (n_layers, n_slots, max_pos, n_heads, head_dim)
        self.k = np.zeros(shp, dtype=F64)
        self.v = np.zeros(shp, dtype=F64)
        self.n_slots, self.max_pos = n_slots, max_pos


class OracleModel:
    """The decoder of the paper's setting (Llama-style, Sec. 3.1), float64.

    ``globals_`` holds "embed" [V, D], "final_norm" [D], "lm_head" [V, D];
    ``layers`` is a list of dicts with "attn_norm", "wq", "wk", "wv", "wo",
    "mlp_norm", "w_gate", "w_up", "w_down" in [out, in] layout.  Values may be any
    float array type; they are held as float64.
    """

    def __init__(self, shape, globals_: Dict, layers: Sequence[Dict], storage: Optional[str] = "bf16"):
        self.shape = shape
        self.storage = storage
        self.g = {k: np.asarray(v, dtype=F64) for k, v in globals_.items()}
        self.layers = [{k: np.asarray(v, dtype=F64) for k, v in lw.items()} for lw in layers]
        self.H, self.hd = shape.n_heads, shape.head_dim
        self.scale = 1.0 / np.sqrt(F64(shape.head_dim))

    def rs(self, x):
        return round_storage(x, self.storage)

    # Alg. 1 Embed: an id >= 0 selects an embedding-table row; -1 takes the given row.
    def embed(self, ids, embeds):
        ids = np.asarray(ids)
        out = np.zeros((ids.shape[0], self.shape.d_model), dtype=F64)
        for r, t in enumerate(ids):
            out[r] = self.g["embed"][t] if t >= 0 else np.asarray(embeds[r], dtype=F64)
        return self.rs(out)

    # ------------------------------------------------------------------ Alg. 2, one layer
    def layer_packed(self, l: int, x, segs: Sequence[Segment], ring: OracleRingKV, trace=None):
        """One layer over the packed state ``x`` [M, D] (Alg. 2), writing the new keys and
        values of every row into its request's ring slot.  Returns the updated state."""
        lw, H, hd, eps = self.layers[l], self.H, self.hd, self.shape.rms_eps
        M = x.shape[0]
        x_in = x
        pos = np.empty(M, dtype=np.int64)
        for sg in segs:
            pos[sg.q_start:sg.q_start + sg.q_len] = sg.pos0 + np.arange(sg.q_len)
        # Norm, QKVProj
        n = self.rs(rmsnorm(x, lw["attn_norm"], eps))
        q = linear(n, lw["wq"]).reshape(M, H, hd)
        k = linear(n, lw["wk"]).reshape(M, H, hd)
        v = linear(n, lw["wv"]).reshape(M, H, hd)
        # FusedRoPEAndWriteKV: rotate at each row's own absolute position, store in the ring
        q = self.rs(rope(q, pos, self.shape.rope_theta))
        k = self.rs(rope(k, pos, self.shape.rope_theta))
        v = self.rs(v)
        for sg in segs:
            rows = slice(sg.q_start, sg.q_start + sg.q_len)
            ring.k[l, sg.slot, sg.pos0:sg.kv_len] = k[rows]
            ring.v[l, sg.slot, sg.pos0:sg.kv_len] = v[rows]
        # VarlenAttention: each segment reads only its own slot, keys 0..pos of each row
        o = np.zeros((M, H, hd), dtype=F64)
        for sg in segs:
            rows = slice(sg.q_start, sg.q_start + sg.q_len)
            for h in range(H):
                o[rows, h] = attend_segment(q[rows, h], pos[rows], ring.k[l, sg.slot, :sg.kv_len, h],
                                            ring.v[l, sg.slot, :sg.kv_len, h], self.scale)
        o = self.rs(o.reshape(M, H * hd))
        # (InPlaceShiftKV moves no data here: slots are recycled by the bookkeeping.)
        # OutputProj + residual, then the MLP residual (standard Llama block)
        x = self.rs(x + linear(o, lw["wo"]))
        x_mid = x
        m = self.rs(rmsnorm(x, lw["mlp_norm"], eps))
        a = self.rs(silu(linear(m, lw["w_gate"])) * linear(m, lw["w_up"]))
        x = self.rs(x + linear(a, lw["w_down"]))
        if trace is not None:
            trace.append(dict(x_in=x_in, n=n, q=q, k=k, v=v, o=o, x_mid=x_mid, a=a, x=x))
        return x

    # ------------------------------------------------------------------ head
    def logits(self, rows):
        """Final norm and LM head of the given rows (Alg. 1: LMHead(Norm(.))), rounded to
        fp32 when the model stores anything narrower than float64."""
        n = self.rs(rmsnorm(rows, self.g["final_norm"], self.shape.rms_eps))
        z = linear(n, self.g["lm_head"])
        return z if self.storage is None else round_storage(z, "f32")

    @staticmethod
    def argmax(z):
        """Greedy token: the lowest index attaining the row maximum (Alg. 1 ArgMax)."""
        z = np.asarray(z)
        return np.argmax(z, axis=-1).astype(np.int64)  # numpy returns the first maximum

    # ------------------------------------------------------------------ whole forward
    def forward_packed(self, ids, embeds, segs: Sequence[Segment], ring: OracleRingKV, trace=None):
        """Embed, every layer of Alg. 2, then logits and tokens of the last row of each
        emitting segment (ordered as the segments).  Returns (hidden [M, D], logits
        [n_emit, V], tokens [n_emit])."""
        M = len(ids)
        covered = np.zeros(M, dtype=np.int64)
        for sg in segs:
            covered[sg.q_start:sg.q_start + sg.q_len] += 1
        if not np.all(covered == 1):
            raise ValueError("segments must tile the packed rows exactly once")
        x = self.embed(ids, embeds)
        for l in range(self.shape.n_layers):
            x = self.layer_packed(l, x, segs, ring, trace)
        last = [sg.q_start + sg.q_len - 1 for sg in segs if sg.emit]
        if not last:
            return x, np.zeros((0, self.shape.vocab)), np.zeros((0,), dtype=np.int64)
        z = self.logits(x[last])
        return x, z, self.argmax(z)
