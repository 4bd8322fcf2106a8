"""GPU parity on the packed-mix sweep and the multi-pipeline stress workload.

* Sweep (one 7B-shape layer, bf16): a prefill of P in {0, 128, 276, 512} rows packed with
  d in {1, 3, 7, 15} decode rows whose contexts are uniform in {max(1, P), .., P + 7}, on a
  ring of 16 slots x 544 positions pre-filled with N(0, 1) keys/values whose slots wrap:
  hidden states against the oracle's packed layer, every written ring cell against the
  oracle's, every other cell bit-for-bit untouched.
* Stress step (one 7B-shape layer): 8 pipelines x (276 prefill + 7 decode rows), M = 2264,
  ring 64 x 288, against the oracle.
* Stress pipeline (32 layers, the full size): the 8 pipelines packed into each forward give
  every pipeline exactly the rows, logits and tokens it gets when run alone on the same
  kernels (split-K off: a row's result does not depend on what it is packed with).  The
  oracle cannot run 32 layers at M = 2264 in test time; this property holds at any size.
"""
import numpy as np
import pytest
import torch

import oracle
import workload as wl
from tests.helpers import (advance_head, allclose_report, bf16_layer_parity, oracle_model, oracle_segments,
                           reserve_step, to_np)

pytestmark = pytest.mark.gpu
af = pytest.importorskip("paper_2512_20276_amd")
from paper_2512_20276_amd.pipeline import Pipeline  # noqa: E402

TOL = dict(atol=2e-2, rtol=1e-2)


@pytest.fixture(scope="module")
def layer7b():
    shape = wl.LLAMA7B.with_layers(1)
    g, layers = wl.model_weights(shape, seed=0, device="cuda")
    w = af.Weights(shape, g, layers)
    model = oracle_model(shape, g, layers)
    yield shape, w, model
    w.close()


def _history(key, n_slots, max_pos, H, hd):
    k = wl.draw((key, "k"), (n_slots, max_pos, H, hd), device="cuda")
    v = wl.draw((key, "v"), (n_slots, max_pos, H, hd), device="cuda")
    return k, v, to_np(k), to_np(v)


@pytest.fixture(scope="module")
def sweep_history(layer7b):
    shape = layer7b[0]
    n_slots, max_pos = wl.SWEEP_RING
    return _history("sweep history", n_slots, max_pos, shape.n_heads, shape.head_dim)


def _run_layer(shape, w, model, hist, n_slots, max_pos, specs, head_shift, key):
    kd, vd, kh, vh = hist
    H, hd, D = shape.n_heads, shape.head_dim, shape.d_model
    ring = af.Ring(1, n_slots, max_pos, H, hd, dtype=torch.bfloat16)
    for s in range(n_slots):
        ring.write_kv(0, s, 0, kd[s], vd[s])
    advance_head(ring, head_shift)
    segs = reserve_step(ring, specs)
    M = sum(s[1] for s in segs)
    x = wl.draw(key, (M, D), device="cuda")
    x0 = to_np(x)
    af.packed_layer_forward(w, 0, x, segs, ring)
    torch.cuda.synchronize()
    okv = oracle.OracleRingKV(1, n_slots, max_pos, H, hd)
    okv.k[0], okv.v[0] = kh, vh
    ref = model.layer_packed(0, x0, oracle_segments(segs), okv)
    rep = bf16_layer_parity(to_np(x), ref)
    print(specs[:2], "...", len(specs), "segments, M", M, rep)
    assert rep["ok"], rep
    for slot in sorted({s[2] for s in segs}):
        k, v = ring.read_kv(0, slot, 0, max_pos)
        k, v = to_np(k), to_np(v)
        touched = np.zeros(max_pos, bool)
        for s in segs:
            if s[2] == slot:
                touched[s[3]:s[3] + s[1]] = True
        assert allclose_report(k[touched], okv.k[0, slot][touched], **TOL)["ok"], slot
        assert allclose_report(v[touched], okv.v[0, slot][touched], **TOL)["ok"], slot
        assert np.array_equal(k[~touched], kh[slot][~touched]) and np.array_equal(v[~touched], vh[slot][~touched])
    ring.close()
    return segs


@pytest.mark.parametrize("d", wl.SWEEP_DECODE)
@pytest.mark.parametrize("P", wl.SWEEP_PREFILL)
def test_sweep_point_matches_oracle(layer7b, sweep_history, P, d):
    shape, w, model = layer7b
    n_slots, max_pos = wl.SWEEP_RING
    specs = wl.sweep_point_specs(P, d)
    segs = _run_layer(shape, w, model, sweep_history, n_slots, max_pos, specs, head_shift=(7 * P + d) % n_slots,
                      key=("sweep rows", P, d))
    assert len(segs) == d + (P > 0)


def test_stress_step_layer_matches_oracle(layer7b):
    """One layer of the steady-state stress step: 8 pipelines, each a 276-row prefill and
    the decode rows of stages 1..7 (contexts 277..283), stage-major rows, 64 slots."""
    shape, w, model = layer7b
    st = wl.STRESS
    P, K, n_slots, max_pos = st["n_pipes"], st["K"], st["n_slots"], st["max_pos"]
    L_P = st["n_vision"] + st["n_text"]
    specs = [(1000 + p, 0, L_P) for p in range(P)]
    specs += [(1000 + 8 * s + p, L_P + s - 1, 1) for s in range(1, K) for p in range(P)]
    hist = _history("stress history", n_slots, max_pos, shape.n_heads, shape.head_dim)
    segs = _run_layer(shape, w, model, hist, n_slots, max_pos, specs, head_shift=5, key=("stress rows",))
    assert sum(s[1] for s in segs) == P * (L_P + K - 1) == 2264


@pytest.mark.timeout(900)
def test_stress_pipelines_pack_independently_32_layers():
    shape = wl.LLAMA7B
    st = wl.STRESS
    P, K, n_slots, max_pos = st["n_pipes"], st["K"], st["n_slots"], st["max_pos"]
    L_V, L_T = st["n_vision"], st["n_text"]
    L_P, D = L_V + L_T, shape.d_model
    g, layers = wl.model_weights(shape, seed=0, device="cuda")
    w = af.Weights(shape, g, layers)
    del g, layers
    w.set_options(af.AF_OPT_NO_SPLIT_K)
    text = wl.draw_ids(("instruction", 0), L_T, shape.vocab, device="cuda")
    pids = torch.cat([torch.full((L_V,), -1, dtype=torch.int32, device="cuda"), text])

    def vision(t, p):
        return wl.draw(("stress vision", t, p), (L_V, D), device="cuda")

    def packed_embeds(t):
        e = torch.zeros((P * (L_P + K - 1), D), dtype=torch.bfloat16, device="cuda")
        for p in range(P):
            e[p * L_P:p * L_P + L_V] = vision(t, p)
        return e

    steps = K + 1
    ring = af.Ring(shape.n_layers, n_slots, max_pos, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
    pipe = Pipeline(w, ring, K, pids, packed_embeds, keep_logits=True, n_pipes=P)
    got = {}   # (t0, p, stage) -> (rows, logits)
    for t in range(steps):
        res = pipe.step()
        assert res.M == P * L_P + P * min(t, K - 1)
        for j, sg in enumerate(res.segments):
            t0, p = divmod(sg[4], P)
            got[(t0, p, t - t0)] = (to_np(res.hidden[sg[0]:sg[0] + sg[1]]), to_np(res.logits[j]))
    toks = {(t0, p): pipe.request_tokens(t0, p) for t0 in range(2) for p in range(P)}
    ring.close()
    for p in (0, 3, 7):
        sring = af.Ring(shape.n_layers, 8, max_pos, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)

        def alone_embeds(t, p=p):
            e = torch.zeros((L_P + K - 1, D), dtype=torch.bfloat16, device="cuda")
            e[:L_V] = vision(t, p)
            return e

        alone = Pipeline(w, sring, K, pids, alone_embeds, keep_logits=True)
        for t in range(steps):
            res = alone.step()
            for j, sg in enumerate(res.segments):
                t0 = sg[4]
                rows, z = got[(t0, p, t - t0)]
                assert np.array_equal(to_np(res.hidden[sg[0]:sg[0] + sg[1]]), rows), (p, t0, t)
                assert np.array_equal(to_np(res.logits[j]), z), (p, t0, t)
        for t0 in range(2):
            assert alone.request_tokens(t0) == toks[(t0, p)], (p, t0)
        assert len(toks[(0, p)]) == K
        sring.close()
    w.close()


# ----------------------------------------------------------------------------- physical-copy shift
def test_shift_stages_moves_ring_contents():
    """af_ring_shift_stages copies each live stage's keys and values (every layer, positions
    0 .. len - 1) one slot along, bit for bit, and leaves slots past the stages untouched."""
    H, hd, L, n_slots, max_pos, K = 4, 64, 3, 6, 40, 4
    ring = af.Ring(L, n_slots, max_pos, H, hd, dtype=torch.bfloat16)
    lens = {0: 9, 1: 21, 2: 33}                 # stages 0..2 live, slot 3 (the last stage) free
    for slot, n in lens.items():
        ring.append(100 + slot, n)
    ring.append(999, 5)                         # slot 3, then released: the finished request
    ring.release(999)
    before = {}
    for l in range(L):
        for slot in range(n_slots):
            kv = wl.draw(("shift", l, slot), (2, max_pos, H, hd), device="cuda")
            ring.write_kv(l, slot, 0, kv[0], kv[1])
            before[(l, slot)] = (to_np(kv[0]), to_np(kv[1]))
    ring.shift_stages(K)
    torch.cuda.synchronize()
    owners, lengths, head = ring.state()
    assert owners[:4] == [-1, 100, 101, 102] and lengths[:4] == [0, 9, 21, 33] and head == 0
    for l in range(L):
        for slot, n in lens.items():
            k, v = ring.read_kv(l, slot + 1, 0, n)
            assert np.array_equal(to_np(k), before[(l, slot)][0][:n]), (l, slot)
            assert np.array_equal(to_np(v), before[(l, slot)][1][:n]), (l, slot)
        for slot in (4, 5):
            k, v = ring.read_kv(l, slot, 0, max_pos)
            assert np.array_equal(to_np(k), before[(l, slot)][0]) and np.array_equal(to_np(v), before[(l, slot)][1])
    ring.close()


@pytest.mark.timeout(600)
def test_copy_shift_pipeline_equals_rotation_32_layers():
    """The paper's physical-copy InPlaceKVShift and this build's index rotation give attention
    the same keys and values, so the whole 32-layer pipeline produces identical rows, logits
    and tokens (K = 7, through the first full step and beyond)."""
    shape = wl.LLAMA7B
    K, L_V, L_T = 7, 256, 20
    L_P, D = L_V + L_T, shape.d_model
    g, layers = wl.model_weights(shape, seed=0, device="cuda")
    w = af.Weights(shape, g, layers)
    del g, layers
    text = wl.draw_ids(("instruction", 0), L_T, shape.vocab, device="cuda")
    pids = torch.cat([torch.full((L_V,), -1, dtype=torch.int32, device="cuda"), text])
    pool = {}

    def embeds(t):
        if t not in pool:
            e = torch.zeros((L_P + K - 1, D), dtype=torch.bfloat16, device="cuda")
            e[:L_V] = wl.draw(("vision", 0, t), (L_V, D), device="cuda")
            pool[t] = e
        return pool[t]

    out = {}
    for mode, n_slots in (("rotate", 8), ("copy", 7)):
        ring = af.Ring(shape.n_layers, n_slots, 288, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
        pipe = Pipeline(w, ring, K, pids, embeds, keep_logits=True, shift=mode)
        rows = []
        for t in range(K + 2):
            res = pipe.step()
            rows.append((to_np(res.hidden), to_np(res.logits), res.tokens.cpu().tolist()))
            if mode == "copy":
                assert [sg[2] for sg in res.segments] == list(range(len(res.segments)))
        out[mode] = rows
        ring.close()
    for t, (a, b) in enumerate(zip(out["rotate"], out["copy"])):
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[2] == b[2], t
    w.close()
