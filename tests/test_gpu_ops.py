"""GPU parity of each step of the packed forward against the oracle, through the C ABI.

Inputs are seeded draws handed as identical bits to both sides.  Tolerances: values the
GPU stores in bf16 must lie within |gpu - ref| <= atol + rtol |ref| of the oracle rounded
at the same storage points (fp32 accumulation vs float64 moves a result across at most a
couple of bf16 rounding boundaries); fp32 results within 1e-4-level bounds.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workload as wl
from oracle.model import attend_segment, linear, rmsnorm, rope, round_storage, silu
from tests.helpers import (advance_head, allclose_report, exact_fraction, gpu_shape_weights, oracle_segments,
                           reserve_step, to_np)

pytestmark = pytest.mark.gpu

af = pytest.importorskip("paper_2512_20276_amd")

TOL = {"bf16": dict(atol=2e-2, rtol=1e-2), "f32": dict(atol=1e-4, rtol=1e-4)}
DT = {"bf16": torch.bfloat16, "f32": torch.float32}


def _assert_close(got, ref, storage, what, min_exact=None, **kw):
    """Elementwise bound with no outliers; for bf16 results optionally also the fraction of
    bit-identical elements (a systematic rounding or indexing error shows up there first)."""
    tol = dict(TOL[storage])
    tol.update(kw)
    got = to_np(got) if isinstance(got, torch.Tensor) else got
    rep = allclose_report(got, ref, **tol)
    assert rep["ok"], (what, rep)
    if min_exact is not None and storage == "bf16":
        ex = exact_fraction(got, ref)
        assert ex >= min_exact, (what, "bit-identical fraction", ex)
    return rep


# ----------------------------------------------------------------------------- RMSNorm
@pytest.mark.parametrize("storage", ["bf16", "f32"])
@pytest.mark.parametrize("M,D", [(1, 256), (34, 256), (282, 4096), (7, 4096), (1027, 4096), (2264, 256)])
def test_rmsnorm(storage, M, D):
    dt = DT[storage]
    x = wl.draw(("t_norm_x", M, D), (M, D), dtype=dt, device="cuda")
    g = wl.draw(("t_norm_g", D), (D,), std=0.3, mean=1.0, dtype=dt, device="cuda")
    y = torch.empty_like(x)
    af.op_rmsnorm(x, g, y, 1e-6)
    torch.cuda.synchronize()
    ref = round_storage(rmsnorm(to_np(x), to_np(g), 1e-6), storage)
    _assert_close(y, ref, storage, "rmsnorm", min_exact=0.999, atol=1e-5 if storage == "f32" else 1e-3)


@pytest.mark.parametrize("M,D", [(1024, 4096), (2264, 4096), (1031, 256)])
def test_rmsnorm_many_rows_equals_few_rows(M, D):
    """From 1024 rows the norm runs one row per wave; every row must equal, bit for bit, the
    same row normalised in a launch of a few rows (one row per workgroup), including the
    rows of a last, partly filled workgroup."""
    x = wl.draw(("t_norm_x", M, D), (M, D), device="cuda")
    g = wl.draw(("t_norm_g", D), (D,), std=0.3, mean=1.0, device="cuda")
    y = torch.empty_like(x)
    af.op_rmsnorm(x, g, y, 1e-6)
    for r0 in (0, 300, M - 7):
        part = x[r0:r0 + 7].contiguous()
        yp = torch.empty_like(part)
        af.op_rmsnorm(part, g, yp, 1e-6)
        torch.cuda.synchronize()
        assert torch.equal(yp, y[r0:r0 + 7]), r0


# ----------------------------------------------------------------------------- GEMM core
@pytest.mark.parametrize("storage", ["bf16", "f32"])
@pytest.mark.parametrize("M", [1, 7, 15, 33, 96, 97, 282, 291, 527])
@pytest.mark.parametrize("N,K", [(256, 256), (1376, 256), (256, 688), (4096, 4096)])
def test_linear(storage, M, N, K):
    if storage == "f32" and K == 4096 and M > 100:
        pytest.skip("covered by the smaller fp32 shapes")
    dt = DT[storage]
    x = wl.draw(("t_lin_x", M, K), (M, K), dtype=dt, device="cuda")
    w = wl.draw(("t_lin_w", N, K), (N, K), std=0.02, dtype=dt, device="cuda")
    y = torch.full((M, N), float("nan"), dtype=dt, device="cuda")
    af.op_linear(x, w, y)
    torch.cuda.synchronize()
    ref = round_storage(linear(to_np(x), to_np(w)), storage)
    _assert_close(y, ref, storage, "linear", min_exact=0.99, atol=1e-3 if storage == "bf16" else 1e-5,
                  rtol=8e-3 if storage == "bf16" else 1e-5)


@pytest.mark.parametrize("M", [161, 200, 282, 291, 320, 326, 351, 384])
def test_linear_qkv_width_split_k(M):
    """N = 12288, K = 4096 (the QKV projection's width) at 161..384 rows: a two-way K split on the
    six-wave 160 x 192 tile (192 x 192 from 321 rows), two row tiles, ragged rows; partial sums
    and reduce against fp64."""
    N, K = 12288, 4096
    x = wl.draw(("t_lin_x", M, K), (M, K), device="cuda")
    w = wl.draw(("t_lin_w", N, K), (N, K), std=0.02, device="cuda")
    y = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    af.op_linear(x, w, y)
    torch.cuda.synchronize()
    ref = round_storage(linear(to_np(x), to_np(w)), "bf16")
    _assert_close(y, ref, "bf16", "linear", min_exact=0.99, atol=1e-3, rtol=8e-3)


@pytest.mark.parametrize("M", [161, 282, 320, 326, 384])
@pytest.mark.parametrize("K", [4096, 11008])
def test_linear_narrow_split_k(M, K):
    """N = 4096 (the output and down projections' width) at 161..384 rows: the four-wave
    160 x 128 tile (192 x 128 from 321 rows) split four ways over K (K = 11008: splits of 11
    and 10 k units), two row tiles with a ragged second one; partial sums and reduce against
    fp64."""
    N = 4096
    x = wl.draw(("t_lin_x", M, K), (M, K), device="cuda")
    w = wl.draw(("t_lin_w", N, K), (N, K), std=0.02, device="cuda")
    y = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    af.op_linear(x, w, y)
    torch.cuda.synchronize()
    ref = round_storage(linear(to_np(x), to_np(w)), "bf16")
    _assert_close(y, ref, "bf16", "linear", min_exact=0.99, atol=1e-3, rtol=8e-3)


def test_linear_large_m():
    """M = 2264 (eight 283-row pipelines), several M tiles and a ragged tail."""
    M, N, K = 2264, 512, 4096
    x = wl.draw(("t_lin_x", M, K), (M, K), device="cuda")
    w = wl.draw(("t_lin_w", N, K), (N, K), std=0.02, device="cuda")
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    af.op_linear(x, w, y)
    torch.cuda.synchronize()
    ref = round_storage(linear(to_np(x), to_np(w)), "bf16")
    _assert_close(y, ref, "bf16", "linear", min_exact=0.99, atol=1e-3, rtol=8e-3)


@pytest.mark.parametrize("M,N,K", [(400, 22016, 4096), (2264, 4672, 4096), (2264, 12288, 512)])
def test_linear_wide_tile(M, N, K):
    """Shapes that take the 288 x 256 tile (two row tiles of gate/up width; eight row tiles with
    a last column tile half past N; QKV width at 2264 rows, one pass of wide tiles over the
    first 8192 columns and 288 x 128 tiles for the rest), against fp64."""
    x = wl.draw(("t_lin_x", M, K), (M, K), device="cuda")
    w = wl.draw(("t_lin_w", N, K), (N, K), std=0.02, device="cuda")
    y = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    af.op_linear(x, w, y)
    torch.cuda.synchronize()
    ref = round_storage(linear(to_np(x), to_np(w)), "bf16")
    _assert_close(y, ref, "bf16", "linear", min_exact=0.99, atol=1e-3, rtol=8e-3)


# ----------------------------------------------------------------------------- attention
def _fill_ring(ring, layer, n_slots, max_pos, H, hd, dt, key):
    """N(0,1) K/V in every position of every slot; returns oracle-side copies [slot, pos, H, hd]."""
    ks, vs = [], []
    for s in range(n_slots):
        k = wl.draw((key, "k", layer, s), (max_pos, H, hd), dtype=dt, device="cuda")
        v = wl.draw((key, "v", layer, s), (max_pos, H, hd), dtype=dt, device="cuda")
        ring.write_kv(layer, s, 0, k, v)
        ks.append(to_np(k))
        vs.append(to_np(v))
    torch.cuda.synchronize()
    return np.stack(ks), np.stack(vs)


ATTN_CASES = {
    # (request, pos0, q_len) in packing order
    "prefill_only": [(1, 0, 130)],
    "decode_only": [(1, 40, 1), (2, 7, 1), (3, 0, 1), (4, 63, 1)],
    "mixed_7b_step": [(10, 0, 276)] + [(10 - s, 276 + s - 1, 1) for s in range(1, 7)],
    "chunked_prefill": [(1, 100, 70), (2, 0, 1), (3, 5, 64), (4, 200, 1)],
    "single_key": [(1, 0, 1)],
    # the ring's last position (max_pos = 288): a decode row at 287 and a prefill ending there
    "ring_end": [(1, 287, 1), (2, 200, 88), (3, 255, 1)],
    # query-tile and key-chunk edges: 64 and 65 prefill rows, decode rows at 31, 32, 64, 95
    "tile_edges": [(1, 0, 64), (2, 0, 65), (3, 31, 1), (4, 32, 1), (5, 64, 1), (6, 95, 1)],
    # more than 16 decode rows beside a prefill at 32 heads: the query tiles and the decode
    # rows take one launch of four-wave workgroups (the K = 32 step of the K sweep, and the
    # stress step's mix)
    "k32_step": [(40, 0, 276)] + [(40 - s, 276 + s - 1, 1) for s in range(1, 32)],
    "stress_mix": [(1000 + p, 0, 276) for p in range(8)] +
                  [(1000 + 8 * s + p, 276 + s - 1, 1) for s in range(1, 8) for p in range(8)],
    # four prefills beside 17 decode rows: the four-wave launch, with more query-tile blocks
    # (640) than decode blocks (544), so query tiles are left over once the two kinds stop
    # alternating
    "tiles_exceed_decode": [(2000 + p, 0, 276) for p in range(4)] + [(2100 + i, 100 + 10 * i, 1) for i in range(17)],
}
# cases that need a larger ring than 8 slots x 288, and run only at 32 heads x 128
ATTN_RING = {"k32_step": (33, 320), "stress_mix": (64, 288), "tiles_exceed_decode": (24, 288)}


@pytest.mark.parametrize("storage,H,hd", [("bf16", 32, 128), ("bf16", 4, 64), ("f32", 4, 64), ("f32", 2, 128)])
@pytest.mark.parametrize("case", sorted(ATTN_CASES))
def test_attention(storage, H, hd, case):
    dt = DT[storage]
    n_slots, max_pos = ATTN_RING.get(case, (8, 288))
    if case in ATTN_RING and (storage, H, hd) != ("bf16", 32, 128):
        pytest.skip("four-wave launch cases run at the 7B head shape")
    ring = af.Ring(1, n_slots, max_pos, H, hd, dtype=dt)
    advance_head(ring, 3)  # start the rotation mid-ring so slots wrap
    K, V = _fill_ring(ring, 0, n_slots, max_pos, H, hd, dt, ("t_attn", storage, H, hd))
    segs = reserve_step(ring, ATTN_CASES[case])
    M = sum(s[1] for s in segs)
    q = wl.draw(("t_attn_q", case, H, hd), (M, H * hd), dtype=dt, device="cuda")
    o = torch.full((M, H * hd), float("nan"), dtype=dt, device="cuda")
    af.op_attention(ring, 0, q, segs, o)
    torch.cuda.synchronize()
    qn = to_np(q).reshape(M, H, hd)
    ref = np.zeros((M, H, hd))
    for sg in oracle_segments(segs):
        rows = slice(sg.q_start, sg.q_start + sg.q_len)
        pos = sg.pos0 + np.arange(sg.q_len)
        for h in range(H):
            ref[rows, h] = attend_segment(qn[rows, h], pos, K[sg.slot, :sg.kv_len, h], V[sg.slot, :sg.kv_len, h],
                                          1 / math.sqrt(hd))
    ref = round_storage(ref.reshape(M, H * hd), storage)
    _assert_close(o, ref, storage, case, min_exact=0.97, **({"atol": 1e-2, "rtol": 1e-2} if storage == "bf16" else {}))
    ring.close()


# ----------------------------------------------------------------------------- fused steps with weights
def _layer_setup(shape, M_specs, seed=0, random_gains=True):
    dt = shape.torch_dtype
    g, layers = gpu_shape_weights(shape, seed=seed, random_gains=random_gains)
    w = af.Weights(shape, g, layers)
    return g, layers, w


@pytest.mark.parametrize("shape_name", ["tiny", "7b"])
def test_qkv_rope_write_and_untouched_ring(shape_name):
    """Queries rotated at each row's position; rotated keys and values land at exactly the
    (slot, position) cells of the step; every other ring cell keeps its sentinel bits."""
    shape = (wl.TINY if shape_name == "tiny" else wl.LLAMA7B).with_layers(1)
    storage = shape.dtype
    dt = shape.torch_dtype
    H, hd, D = shape.n_heads, shape.head_dim, shape.d_model
    g, layers, w = _layer_setup(shape, None)
    n_slots, max_pos = 8, 288
    ring = af.Ring(1, n_slots, max_pos, H, hd, dtype=dt)
    sentinel = torch.full((max_pos, H, hd), 7.0, dtype=dt, device="cuda")
    for s in range(n_slots):
        ring.write_kv(0, s, 0, sentinel, sentinel)
    advance_head(ring, 2)
    specs = [(10, 0, 276)] + [(10 - s, 276 + s - 1, 1) for s in range(1, 7)] if shape_name == "7b" else \
        [(5, 0, 32), (4, 32, 1), (3, 33, 1)]
    segs = reserve_step(ring, specs)
    M = sum(s[1] for s in segs)
    xn = wl.draw(("t_qkv_x", shape_name), (M, D), dtype=dt, device="cuda")
    q = torch.full((M, D), float("nan"), dtype=dt, device="cuda")
    af.op_qkv_rope_write(w, 0, xn, segs, ring, q)
    torch.cuda.synchronize()
    lw = {k: to_np(v) for k, v in layers[0].items()}
    x = to_np(xn)
    pos = np.concatenate([s[3] + np.arange(s[1]) for s in segs])
    qr = round_storage(rope(linear(x, lw["wq"]).reshape(M, H, hd), pos, shape.rope_theta), storage)
    kr = round_storage(rope(linear(x, lw["wk"]).reshape(M, H, hd), pos, shape.rope_theta), storage)
    vr = round_storage(linear(x, lw["wv"]).reshape(M, H, hd), storage)
    _assert_close(q, qr.reshape(M, D), storage, "q", min_exact=0.99)
    written = np.zeros((n_slots, max_pos), dtype=bool)
    for s in segs:
        written[s[2], s[3]:s[3] + s[1]] = True
    for slot in range(n_slots):
        k, v = ring.read_kv(0, slot, 0, max_pos)
        k, v = to_np(k), to_np(v)
        rows = [s for s in segs if s[2] == slot]
        for s in rows:
            r = slice(s[0], s[0] + s[1])
            _assert_close(k[s[3]:s[3] + s[1]], kr[r], storage, f"k slot {slot}")
            _assert_close(v[s[3]:s[3] + s[1]], vr[r], storage, f"v slot {slot}")
        untouched = ~written[slot]
        assert np.all(k[untouched] == 7.0) and np.all(v[untouched] == 7.0), f"stray write in slot {slot}"
    ring.close()
    w.close()


@pytest.mark.parametrize("shape_name", ["tiny", "7b"])
@pytest.mark.parametrize("M", [1, 34, 282, 343])
def test_mlp_and_residual_steps(shape_name, M):
    shape = (wl.TINY if shape_name == "tiny" else wl.LLAMA7B).with_layers(1)
    storage, dt, D, F = shape.dtype, shape.torch_dtype, shape.d_model, shape.d_ff
    g, layers, w = _layer_setup(shape, None)
    lw = {k: to_np(v) for k, v in layers[0].items()}
    xn = wl.draw(("t_mlp_x", shape_name, M), (M, D), dtype=dt, device="cuda")
    act = torch.full((M, F), float("nan"), dtype=dt, device="cuda")
    af.op_gate_up_swiglu(w, 0, xn, act)
    x = to_np(xn)
    ref_act = round_storage(silu(linear(x, lw["w_gate"])) * linear(x, lw["w_up"]), storage)
    hid = wl.draw(("t_mlp_h", shape_name, M), (M, D), dtype=dt, device="cuda")
    h0 = to_np(hid)
    af.op_down_residual(w, 0, act, hid)
    torch.cuda.synchronize()
    _assert_close(act, ref_act, storage, "swiglu", min_exact=0.99)
    ref_h = round_storage(h0 + linear(to_np(act), lw["w_down"]), storage)
    _assert_close(hid, ref_h, storage, "down+residual", min_exact=0.99)
    o = wl.draw(("t_o", shape_name, M), (M, D), dtype=dt, device="cuda")
    h1 = to_np(hid)
    af.op_o_proj_residual(w, 0, o, hid)
    torch.cuda.synchronize()
    _assert_close(hid, round_storage(h1 + linear(to_np(o), lw["wo"]), storage), storage, "o+residual")
    w.close()


@pytest.mark.parametrize("shape_name", ["tiny", "7b"])
def test_embed_and_lm_head_argmax(shape_name):
    shape = (wl.TINY if shape_name == "tiny" else wl.LLAMA7B).with_layers(1)
    storage, dt, D, V = shape.dtype, shape.torch_dtype, shape.d_model, shape.vocab
    g, layers, w = _layer_setup(shape, None)
    M = 40
    ids = wl.draw_ids(("t_ids", shape_name), M, V, device="cuda")
    ids[::3] = -1
    emb = wl.draw(("t_emb", shape_name), (M, D), dtype=dt, device="cuda")
    out = torch.empty((M, D), dtype=dt, device="cuda")
    af.op_embed(w, ids, emb, out)
    torch.cuda.synchronize()
    idn = ids.cpu().numpy()
    ref = np.where(idn[:, None] >= 0, to_np(g["embed"])[np.maximum(idn, 0)], to_np(emb))
    assert np.array_equal(to_np(out), ref)
    assert w.device_errors() == 0
    bad = ids.clone()
    bad[0] = V + 5
    af.op_embed(w, bad, emb, out)
    assert w.device_errors() == 1
    # LM head on the last row of each emitting segment
    hidden = wl.draw(("t_hid", shape_name), (M, D), dtype=dt, device="cuda")
    segs = [(0, 10, 0, 0, 1, 1), (10, 1, 1, 0, 2, 0), (11, 29, 2, 0, 3, 1)]
    logits = torch.empty((2, V), dtype=torch.float32, device="cuda")
    toks = torch.empty(2, dtype=torch.int32, device="cuda")
    af.op_lm_head_argmax(w, hidden, segs, logits, toks)
    torch.cuda.synchronize()
    model = oracle.OracleModel(shape, {k: to_np(v) for k, v in g.items()}, [], storage=storage)
    z = model.logits(to_np(hidden)[[9, 39]])
    _assert_close(logits, z, "f32", "logits", atol=2e-3 if storage == "bf16" else 1e-4, rtol=1e-3)
    zs = np.sort(z, axis=1)
    for i, t in enumerate(toks.cpu().numpy()):
        if zs[i, -1] - zs[i, -2] > 1e-2:
            assert t == int(np.argmax(z[i]))
    w.close()


def test_argmax_ties_take_lowest_index():
    shape = wl.TINY.with_layers(1)
    g, layers, w = _layer_setup(shape, None)
    D = shape.d_model
    hidden = torch.zeros((2, D), dtype=torch.float32, device="cuda")  # all-zero rows -> all logits 0
    toks = torch.full((2,), -7, dtype=torch.int32, device="cuda")
    af.op_lm_head_argmax(w, hidden, [(0, 1, 0, 0, 1, 1), (1, 1, 1, 0, 2, 1)], None, toks)
    torch.cuda.synchronize()
    assert toks.tolist() == [0, 0]
    w.close()
