"""Python binding of libactionflow (the MI355X Cross-Request State Packed Forward).

Argument marshalling only: every step of the path runs in the library's HIP kernels.
Device buffers are passed as torch tensors (their data pointers); PyTorch provides
device memory and streams.  Importing this module loads the in-tree shared library and
raises if it has not been built (``python paper_2512_20276_amd/build.py``); there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, List, Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("AF_LIBRARY_PATH") or os.path.join(_HERE, "libactionflow.so")

AF_OK, AF_ERR_INVALID_ARG, AF_ERR_OUT_OF_RANGE, AF_ERR_SLOT_BUSY = 0, -1, -2, -3
AF_ERR_UNKNOWN_REQUEST, AF_ERR_DEVICE, AF_ERR_OOM, AF_ERR_UNSUPPORTED = -4, -5, -6, -7
AF_F32, AF_BF16 = 0, 1
AF_SEG_EMIT = 1
AF_OPT_NO_SPLIT_K = 1
KERNEL_CLASSES = ["embed", "rmsnorm", "gemm_qkv", "attention", "gemm_o", "gemm_gateup", "gemm_down",
                  "lm_head", "argmax"]
AF_K_COUNT = len(KERNEL_CLASSES)


class AFError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class ModelDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_ff", C.c_int32), ("vocab", C.c_int32),
                ("rms_eps", C.c_float), ("rope_theta", C.c_float), ("dtype", C.c_int32)]


class RingDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("n_slots", C.c_int32), ("max_pos", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("dtype", C.c_int32)]


class Segment(C.Structure):
    _fields_ = [("q_start", C.c_int32), ("q_len", C.c_int32), ("slot", C.c_int32), ("pos0", C.c_int32),
                ("request_id", C.c_int64), ("flags", C.c_int32), ("reserved", C.c_int32)]

    def astuple(self):
        return (self.q_start, self.q_len, self.slot, self.pos0, self.request_id, self.flags)

    def __repr__(self):
        return (f"Segment(q_start={self.q_start}, q_len={self.q_len}, slot={self.slot}, pos0={self.pos0}, "
                f"request_id={self.request_id}, flags={self.flags})")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2512_20276_amd/build.py` "
                          "(the HIP library is required: there is no fallback)")
    lib = C.CDLL(LIB_PATH)
    P, I32, I64, U32, F32 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_float
    PP = C.POINTER(C.c_void_p)
    SEG = C.POINTER(Segment)
    sigs = {
        "af_last_error": (C.c_char_p, []),
        "af_ring_create": (I32, [C.POINTER(RingDesc), P, PP]),
        "af_ring_destroy": (I32, [P]),
        "af_ring_reset": (I32, [P]),
        "af_ring_append": (I32, [P, I64, I32, SEG]),
        "af_ring_release": (I32, [P, I64]),
        "af_ring_state": (I32, [P, C.POINTER(I64), C.POINTER(I32), C.POINTER(I32)]),
        "af_ring_shift_stages": (I32, [P, I32, P]),
        "af_ring_write_kv": (I32, [P, I32, I32, I32, I32, P, P, P]),
        "af_ring_read_kv": (I32, [P, I32, I32, I32, I32, P, P, P]),
        "af_ring_copy_kv": (I32, [P, I32, I32, P, I32, I32, I32, I32, P]),
        "af_weights_tensor_count": (I32, [I32]),
        "af_weights_create": (I32, [C.POINTER(ModelDesc), PP, I32, P, PP]),
        "af_weights_destroy": (I32, [P]),
        "af_packed_forward": (I32, [P, P, P, I32, SEG, I32, P, P, P, P, P]),
        "af_packed_forward_noalloc": (I32, [P, P, P, I32, SEG, I32, P, P, P, P, P]),
        "af_packed_layer_forward": (I32, [P, I32, P, I32, SEG, I32, P, P]),
        "af_packed_layer_forward_kv": (I32, [P, I32, P, I32, SEG, I32, P, I32, P]),
        "af_weights_device_errors": (I32, [P, P, C.POINTER(I32)]),
        "af_op_embed": (I32, [P, P, P, I32, P, P]),
        "af_op_rmsnorm": (I32, [I32, P, P, P, I32, I32, F32, P]),
        "af_op_linear": (I32, [I32, P, P, P, I32, I32, I32, P]),
        "af_op_qkv_rope_write": (I32, [P, I32, P, I32, SEG, I32, P, P, P]),
        "af_op_attention": (I32, [P, I32, P, I32, SEG, I32, P, P]),
        "af_op_o_proj_residual": (I32, [P, I32, P, P, I32, P]),
        "af_op_gate_up_swiglu": (I32, [P, I32, P, P, I32, P]),
        "af_op_down_residual": (I32, [P, I32, P, P, I32, P]),
        "af_op_lm_head_argmax": (I32, [P, P, I32, SEG, I32, P, P, P]),
        "af_weights_set_options": (I32, [P, U32]),
        "af_timing_enable": (I32, [P, U32]),
        "af_timing_read": (I32, [P, C.POINTER(C.c_double), C.POINTER(I64)]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


def _check(code: int):
    if code != AF_OK:
        raise AFError(code, lib.af_last_error().decode())


def last_error() -> str:
    return lib.af_last_error().decode()


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    return C.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        if not torch.cuda.is_available():
            return None
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def dtype_code(dt) -> int:
    if dt in (torch.bfloat16, "bf16"):
        return AF_BF16
    if dt in (torch.float32, "f32"):
        return AF_F32
    raise ValueError(f"unsupported dtype {dt}")


def segments_array(segs: Sequence) -> "C.Array[Segment]":
    """Builds a host segment table from Segment objects or tuples
    (q_start, q_len, slot, pos0, request_id[, flags])."""
    arr = (Segment * len(segs))()
    for i, s in enumerate(segs):
        if isinstance(s, Segment):
            arr[i] = s
        else:
            t = tuple(s)
            flags = t[5] if len(t) > 5 else AF_SEG_EMIT
            arr[i] = Segment(t[0], t[1], t[2], t[3], t[4], flags, 0)
    return arr


# ----------------------------------------------------------------------------- ring
class Ring:
    """Unified KV Ring Buffer handle (device KV + slot bookkeeping)."""

    def __init__(self, n_layers: int, n_slots: int, max_pos: int, n_kv_heads: int = 0, head_dim: int = 0,
                 dtype=torch.bfloat16, stream=None):
        self.desc = RingDesc(n_layers, n_slots, max_pos, n_kv_heads, head_dim,
                             dtype_code(dtype) if n_layers > 0 else AF_BF16)
        self.dtype = dtype
        h = C.c_void_p()
        _check(lib.af_ring_create(C.byref(self.desc), _stream(stream) if n_layers > 0 else None, C.byref(h)))
        self.h = h

    def close(self):
        if getattr(self, "h", None) and self.h.value:
            _check(lib.af_ring_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def reset(self):
        _check(lib.af_ring_reset(self.h))

    def append(self, request_id: int, n_new: int) -> Segment:
        s = Segment()
        _check(lib.af_ring_append(self.h, request_id, n_new, C.byref(s)))
        return s

    def release(self, request_id: int):
        _check(lib.af_ring_release(self.h, request_id))

    def shift_stages(self, n_stages: int, stream=None):
        """InPlaceKVShift by physical copy: slot s -> s + 1 for s < n_stages - 1 (see the header)."""
        _check(lib.af_ring_shift_stages(self.h, n_stages, _stream(stream) if self.desc.n_layers > 0 else None))

    def state(self):
        n = self.desc.n_slots
        owners, lens, head = (C.c_int64 * n)(), (C.c_int32 * n)(), C.c_int32()
        _check(lib.af_ring_state(self.h, owners, lens, C.byref(head)))
        return list(owners), list(lens), head.value

    def write_kv(self, layer, slot, pos0, k: torch.Tensor, v: torch.Tensor, stream=None):
        _check(lib.af_ring_write_kv(self.h, layer, slot, pos0, k.shape[0], _ptr(k), _ptr(v), _stream(stream)))

    def copy_kv_to(self, layer, slot, dst: "Ring", dst_layer, dst_slot, pos0, n, stream=None):
        """Keys and values of positions [pos0, pos0 + n) of (layer, slot) into dst's (dst_layer, dst_slot)."""
        _check(lib.af_ring_copy_kv(self.h, layer, slot, dst.h, dst_layer, dst_slot, pos0, n, _stream(stream)))

    def read_kv(self, layer, slot, pos0, n, stream=None):
        d = self.desc
        k = torch.empty((n, d.n_kv_heads, d.head_dim), dtype=self.dtype, device="cuda")
        v = torch.empty_like(k)
        _check(lib.af_ring_read_kv(self.h, layer, slot, pos0, n, _ptr(k), _ptr(v), _stream(stream)))
        return k, v


# ----------------------------------------------------------------------------- weights
LAYER_ORDER = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")


class Weights:
    """Library-owned, repacked copy of the model (plus the forward's scratch activations)."""

    def __init__(self, shape, globals_: Dict[str, torch.Tensor], layers: List[Dict[str, torch.Tensor]],
                 stream=None):
        self.shape = shape
        self.dtype = shape.torch_dtype
        self.desc = ModelDesc(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                              shape.d_ff, shape.vocab, shape.rms_eps, shape.rope_theta, dtype_code(shape.dtype))
        tensors = [globals_["embed"], globals_["final_norm"], globals_["lm_head"]]
        for lw in layers:
            tensors += [lw[k] for k in LAYER_ORDER]
        for t in tensors:
            if not t.is_cuda or t.dtype != self.dtype or not t.is_contiguous():
                raise ValueError("weights must be contiguous device tensors of the model dtype")
        arr = (C.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])
        h = C.c_void_p()
        _check(lib.af_weights_create(C.byref(self.desc), arr, len(tensors), _stream(stream), C.byref(h)))
        self.h = h

    def close(self):
        if getattr(self, "h", None) and self.h.value:
            _check(lib.af_weights_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def device_errors(self, stream=None) -> int:
        c = C.c_int32()
        _check(lib.af_weights_device_errors(self.h, _stream(stream), C.byref(c)))
        return c.value

    def set_options(self, flags: int):
        _check(lib.af_weights_set_options(self.h, flags))

    def timing_enable(self, mask: int):
        _check(lib.af_timing_enable(self.h, mask))

    def timing_read(self):
        ms, n = (C.c_double * AF_K_COUNT)(), (C.c_int64 * AF_K_COUNT)()
        _check(lib.af_timing_read(self.h, ms, n))
        return {k: (ms[i], n[i]) for i, k in enumerate(KERNEL_CLASSES)}


# ----------------------------------------------------------------------------- calls
def packed_forward(w: Weights, token_ids: torch.Tensor, embeds: Optional[torch.Tensor], segs, ring: Ring,
                   out_hidden: torch.Tensor, out_logits: Optional[torch.Tensor] = None,
                   out_tokens: Optional[torch.Tensor] = None, stream=None):
    sa = segs if isinstance(segs, C.Array) else segments_array(segs)
    _check(lib.af_packed_forward(w.h, _ptr(token_ids), _ptr(embeds), token_ids.shape[0], sa, len(sa), ring.h,
                                 _ptr(out_hidden), _ptr(out_logits), _ptr(out_tokens), _stream(stream)))


def packed_forward_noalloc(w: Weights, token_ids: torch.Tensor, embeds: Optional[torch.Tensor], segs, ring: Ring,
                           out_hidden: torch.Tensor, out_logits: Optional[torch.Tensor] = None,
                           out_tokens: Optional[torch.Tensor] = None, stream=None):
    """packed_forward with the library's fixed per-GPU scratch array instead of allocations."""
    sa = segs if isinstance(segs, C.Array) else segments_array(segs)
    _check(lib.af_packed_forward_noalloc(w.h, _ptr(token_ids), _ptr(embeds), token_ids.shape[0], sa, len(sa), ring.h,
                                         _ptr(out_hidden), _ptr(out_logits), _ptr(out_tokens), _stream(stream)))


def packed_layer_forward(w: Weights, layer: int, hidden: torch.Tensor, segs, ring: Ring, stream=None,
                         ring_layer: Optional[int] = None):
    """One layer in place on hidden; its keys and values in ring layer ``ring_layer`` (default ``layer``)."""
    sa = segs if isinstance(segs, C.Array) else segments_array(segs)
    if ring_layer is None:
        _check(lib.af_packed_layer_forward(w.h, layer, _ptr(hidden), hidden.shape[0], sa, len(sa), ring.h,
                                           _stream(stream)))
    else:
        _check(lib.af_packed_layer_forward_kv(w.h, layer, _ptr(hidden), hidden.shape[0], sa, len(sa), ring.h,
                                              ring_layer, _stream(stream)))


def op_embed(w: Weights, token_ids, embeds, out, stream=None):
    _check(lib.af_op_embed(w.h, _ptr(token_ids), _ptr(embeds), token_ids.shape[0], _ptr(out), _stream(stream)))


def op_rmsnorm(x: torch.Tensor, g: torch.Tensor, y: torch.Tensor, eps: float, stream=None):
    M, D = x.shape
    _check(lib.af_op_rmsnorm(dtype_code(x.dtype), _ptr(x), _ptr(g), _ptr(y), M, D, eps, _stream(stream)))


def op_linear(x: torch.Tensor, wt: torch.Tensor, y: torch.Tensor, stream=None):
    M, K = x.shape
    N = wt.shape[0]
    _check(lib.af_op_linear(dtype_code(x.dtype), _ptr(x), _ptr(wt), _ptr(y), M, N, K, _stream(stream)))


def op_qkv_rope_write(w: Weights, layer, xn, segs, ring: Ring, q_out, stream=None):
    sa = segments_array(segs)
    _check(lib.af_op_qkv_rope_write(w.h, layer, _ptr(xn), xn.shape[0], sa, len(sa), ring.h, _ptr(q_out),
                                    _stream(stream)))


def op_attention(ring: Ring, layer, q, segs, o, stream=None):
    sa = segments_array(segs)
    _check(lib.af_op_attention(ring.h, layer, _ptr(q), q.shape[0], sa, len(sa), _ptr(o), _stream(stream)))


def op_o_proj_residual(w: Weights, layer, o, hidden, stream=None):
    _check(lib.af_op_o_proj_residual(w.h, layer, _ptr(o), _ptr(hidden), hidden.shape[0], _stream(stream)))


def op_gate_up_swiglu(w: Weights, layer, xn, act, stream=None):
    _check(lib.af_op_gate_up_swiglu(w.h, layer, _ptr(xn), _ptr(act), xn.shape[0], _stream(stream)))


def op_down_residual(w: Weights, layer, act, hidden, stream=None):
    _check(lib.af_op_down_residual(w.h, layer, _ptr(act), _ptr(hidden), hidden.shape[0], _stream(stream)))


def op_lm_head_argmax(w: Weights, hidden, segs, out_logits=None, out_tokens=None, stream=None):
    sa = segments_array(segs)
    _check(lib.af_op_lm_head_argmax(w.h, _ptr(hidden), hidden.shape[0], sa, len(sa), _ptr(out_logits),
                                    _ptr(out_tokens), _stream(stream)))
