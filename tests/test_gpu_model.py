"""GPU parity of the whole packed forward and the Alg. 1 pipeline against the oracle.

* Tiny fp32 decoder (2 layers, d 256, 4 x 64, SwiGLU 688, vocab 512), K = 3, L_P = 32, ring
  4 slots x 64: every step of a cold-start pipeline (step 2 is the 34-row packed step), hidden
  states and logits to fp32 tolerance, tokens exactly.
* One 7B-shape layer in bf16 on a pre-filled ring whose slots wrap: 276 prefill rows + 6
  decode rows at contexts 277..282 (M = 282); hidden to max-abs 2e-2 / rel 1e-2, ring cells.
* 32-layer 7B-shape pipeline, K = 7, steps 0..6 against the oracle pipeline forced with the
  GPU's tokens: each layer of the first full step (M = 282) run from the oracle's input and
  ring history and held elementwise to 2e-2 + 1e-2 |ref|; error growth per layer; every
  step's hidden rows, logits and tokens.
Greedy tokens are compared exactly wherever the oracle's top-2 margin exceeds twice the
largest logit deviation of that row, capped at 0.05; rows inside that window are near-ties.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
import workload as wl
from oracle.pipeline import PipelineOracle
from tests.helpers import (advance_head, allclose_report, bf16_layer_parity, check_tokens, oracle_model,
                           oracle_segments, reserve_step, tiny_prefill_fn, to_np)

pytestmark = pytest.mark.gpu
af = pytest.importorskip("paper_2512_20276_amd")
from paper_2512_20276_amd.pipeline import Pipeline  # noqa: E402

HID_TOL_BF16 = dict(atol=2e-2, rtol=1e-2)
HID_TOL_F32 = dict(atol=1e-4, rtol=1e-4)


def _weights(shape, device="cuda", random_gains=False):
    g, layers = wl.model_weights(shape, seed=0, device=device, random_gains=random_gains)
    return g, layers, af.Weights(shape, g, layers)


# ----------------------------------------------------------------------------- tiny fp32 pipeline
@pytest.mark.parametrize("K", [3, 8, 16])
def test_tiny_fp32_pipeline_matches_oracle(K):
    """K = 3 is the tiny configuration (step 2 packs 32 + 1 + 1 = 34 rows); K = 8 packs seven
    decode rows beside each prefill (an odd number: the last pair of decode rows is half idle)
    and wraps a 9-slot ring; K = 16 (the K sweep's second point) packs fifteen and wraps 17."""
    shape = wl.TINY
    L_P = 32
    n_slots, max_pos = (4, 64) if K == 3 else (K + 1, L_P + K)
    n_steps = 7 if K == 3 else 2 * K + 2
    g, layers, w = _weights(shape, random_gains=True)
    ring = af.Ring(shape.n_layers, n_slots, max_pos, shape.n_heads, shape.head_dim, dtype=torch.float32)
    fn = tiny_prefill_fn(shape, L_P, seed=0)   # token ids uniform in [0, 512)
    ids0, _ = fn(0)
    # all prefill rows are token ids here; each request draws its own prompt
    prompts = {}

    def prefill_embeds(t):
        return torch.zeros((L_P + K - 1, shape.d_model), dtype=torch.float32, device="cuda")

    model = oracle_model(shape, g, layers)
    opipe = PipelineOracle(model, K, n_slots, max_pos, fn)
    pipe = Pipeline(w, ring, K, torch.full((L_P,), -1, dtype=torch.int32, device="cuda"), prefill_embeds,
                    keep_logits=True)
    for t in range(n_steps):
        ids_t, _ = fn(t)
        pipe.ids[t % 2][:L_P] = torch.from_numpy(ids_t).to(torch.int32).cuda()
        res = pipe.step()
        torch.cuda.synchronize()
        got_tokens = res.tokens.cpu().tolist()
        ost = opipe.step(forced=got_tokens)
        assert res.segments == [(s.q_start, s.q_len, s.slot, s.pos0, s.request_id, 1) for s in ost["segments"]]
        rep = allclose_report(to_np(res.hidden), ost["hidden"], **HID_TOL_F32)
        assert rep["ok"], (t, rep)
        rep = allclose_report(to_np(res.logits), ost["logits"], atol=1e-4, rtol=1e-4)
        assert rep["ok"], (t, rep)
        check_tokens(got_tokens, ost["logits"], to_np(res.logits))
        if K == 3 and t == 2:
            assert res.M == 34
    # GPU ring == oracle ring for the live requests
    owners, lens, _ = ring.state()
    for slot, (rid, n) in enumerate(zip(owners, lens)):
        if rid < 0:
            continue
        for l in range(shape.n_layers):
            k, v = ring.read_kv(l, slot, 0, n)
            assert allclose_report(to_np(k), opipe.kv.k[l, slot, :n], **HID_TOL_F32)["ok"]
            assert allclose_report(to_np(v), opipe.kv.v[l, slot, :n], **HID_TOL_F32)["ok"]
    w.close()
    ring.close()


# ----------------------------------------------------------------------------- one 7B layer
def _prefilled_7b_layer_step(shape):
    n_slots, max_pos, H, hd = 8, 288, shape.n_heads, shape.head_dim
    ring = af.Ring(1, n_slots, max_pos, H, hd, dtype=torch.bfloat16)
    K_hist, V_hist = [], []
    for s in range(n_slots):
        k = wl.draw(("ring_k", 0, s), (max_pos, H, hd), device="cuda")
        v = wl.draw(("ring_v", 0, s), (max_pos, H, hd), device="cuda")
        ring.write_kv(0, s, 0, k, v)
        K_hist.append(to_np(k))
        V_hist.append(to_np(v))
    # requests 4..10 occupy slots 4,5,6,7,0,1,2: prefill slot 2, decodes slots 1,0,7,6,5,4
    advance_head(ring, 4)
    for r in range(4, 10):          # in-flight requests arrived earlier, oldest first
        ring.append(r, 276 + (10 - r) - 1)
    specs = [(10, 0, 276)] + [(10 - s, 276 + s - 1, 1) for s in range(1, 7)]
    segs = reserve_step(ring, specs)
    return ring, segs, np.stack(K_hist), np.stack(V_hist)


def test_7b_layer_packed_step_matches_oracle():
    shape = wl.LLAMA7B.with_layers(1)
    g, layers, w = _weights(shape)
    ring, segs, Kh, Vh = _prefilled_7b_layer_step(shape)
    assert [s[2] for s in segs] == [2, 1, 0, 7, 6, 5, 4]
    M = 282
    x = torch.cat([wl.draw(("vision", 0, 10), (256, shape.d_model), device="cuda"),
                   wl.draw(("text_rows", 0, 10), (20, shape.d_model), device="cuda"),
                   wl.draw(("decode_rows", 0), (6, shape.d_model), device="cuda")])
    x0 = to_np(x)
    af.packed_layer_forward(w, 0, x, segs, ring)
    torch.cuda.synchronize()
    model = oracle_model(shape, g, layers)
    okv = oracle.OracleRingKV(1, 8, 288, shape.n_heads, shape.head_dim)
    okv.k[0], okv.v[0] = Kh, Vh
    ref = model.layer_packed(0, x0, oracle_segments(segs), okv)
    rep = bf16_layer_parity(to_np(x), ref)
    print("7b layer hidden parity", rep)
    assert rep["ok"], rep
    for slot in range(8):
        k, v = ring.read_kv(0, slot, 0, 288)
        k, v = to_np(k), to_np(v)
        assert allclose_report(k, okv.k[0, slot], **HID_TOL_BF16)["ok"], slot
        assert allclose_report(v, okv.v[0, slot], **HID_TOL_BF16)["ok"], slot
        touched = np.zeros(288, bool)
        for s in segs:
            if s[2] == slot:
                touched[s[3]:s[3] + s[1]] = True
        assert np.array_equal(k[~touched], Kh[slot][~touched]) and np.array_equal(v[~touched], Vh[slot][~touched])
    w.close()
    ring.close()


def test_7b_layer_segment_order_and_slot_invariance():
    """Permuting the packing order permutes the rows; moving requests to other slots changes
    nothing (each row sees only its own request)."""
    shape = wl.LLAMA7B.with_layers(1)
    g, layers, w = _weights(shape)
    D = shape.d_model

    def run(order, head_shift):
        ring = af.Ring(1, 8, 288, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
        advance_head(ring, head_shift)
        base = [(10, 0, 100), (9, 150, 1), (8, 40, 1), (7, 0, 30)]
        specs = [base[i] for i in order]
        segs = reserve_step(ring, specs)
        # history: per request, deterministic K/V independent of the slot
        for (rid, pos0, q_len), s in zip(specs, segs):
            if pos0:
                k = wl.draw(("hist_k", rid), (pos0, shape.n_heads, shape.head_dim), device="cuda")
                v = wl.draw(("hist_v", rid), (pos0, shape.n_heads, shape.head_dim), device="cuda")
                ring.write_kv(0, s[2], 0, k, v)
        rows = {rid: wl.draw(("rows", rid), (q_len, D), device="cuda") for rid, _, q_len in specs}
        x = torch.cat([rows[rid] for rid, _, _ in specs])
        af.packed_layer_forward(w, 0, x, segs, ring)
        torch.cuda.synchronize()
        out, r = {}, 0
        for rid, _, q_len in specs:
            out[rid] = to_np(x[r:r + q_len])
            r += q_len
        ring.close()
        return out

    a = run([0, 1, 2, 3], 0)
    b = run([3, 1, 0, 2], 5)
    for rid in a:
        assert np.array_equal(a[rid], b[rid]) or allclose_report(a[rid], b[rid], atol=1e-2, rtol=1e-2)["ok"], rid
    w.close()


# ----------------------------------------------------------------------------- 32 layers
def _layer_report(got, ref, tr=None):
    """Layer-gate report; with the oracle's trace of the layer, also the number of elements
    outside 2e-2 + 1e-2 x the residual stream's magnitude at that element (the largest of the
    layer's input, its state after the attention residual and its output: the scale at which
    the two residual adds round)."""
    rep = bf16_layer_parity(got, ref)
    out = {k: rep[k] for k in ("ok", "max_abs", "max_rel", "rms", "norm_rel", "row_norm_rel", "n_bad", "worst_ratio")}
    if tr is not None:
        scale = np.maximum(np.maximum(np.abs(ref), np.abs(tr["x_in"])), np.abs(tr["x_mid"]))
        out["n_bad_stream_scale"] = int(np.sum(~(np.abs(np.asarray(got) - ref) <= 2e-2 + 1e-2 * scale)))
    return out


def _logits_report(got, ref):
    rep = allclose_report(got, ref, atol=2e-2, rtol=1e-2)
    rep["norm_rel"] = float(np.linalg.norm(np.asarray(got) - ref) / np.linalg.norm(ref))
    return rep


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("K", [7, 16, pytest.param(32, marks=pytest.mark.skipif(
    os.environ.get("AF_LONG_TESTS") != "1",
    reason="32 oracle pipeline steps take about 200 s with no output; set AF_LONG_TESTS=1 to run"))])
def test_7b_32_layer_pipeline_matches_oracle(monkeypatch, K):
    """The benchmark workload (32 layers, K = 7, 8 slots) and the K sweep's K = 16 and K = 32
    points (K + 1 slots; at K = 32 the 31 decode rows and the query tiles take the four-wave
    attention launch) against the oracle pipeline.

    The GPU pipeline runs steps 0..K-1 on its own greedy tokens; the oracle pipeline (Alg. 1
    over the float64 packed forward with bf16 storage) runs the same steps forced with the
    GPU's tokens, so the two trajectories never part.  Step K-1 is the first full step: a
    276-row prefill and K-1 decode rows at contexts 277..276+K-1 (M = 282 at K = 7, 291 at
    K = 16, 307 at K = 32).
      * Per layer (the gate): each of the 32 layers of step K-1 runs on the GPU from the
        oracle's input to that layer, with the oracle's ring history of that layer, and is held
        to the layer gate (max-abs 2e-2 / rel 1e-2 elementwise, normwise and per row).
      * Head: the final norm, LM head and argmax run on the oracle's last hidden rows of every
        step, and the last layer plus the head on the oracle's input to the last layer at step
        K-1: logits elementwise to 2e-2 + 1e-2 |ref|; greedy tokens equal wherever the oracle's
        top-2 margin exceeds min(2 x the row's largest logit deviation, 0.05) (near-ties inside
        that window are counted and bounded: at most 2, or a tenth of the tokens checked).
      * Growth: the 32 layers of step K-1 chained on the GPU's own outputs from the oracle's
        layer-0 input (error growth per layer inside one step), reported.
      * End to end: every step's hidden rows and logits of the free-running pipeline.  Both
        sides store bf16 after every layer, and a summation order that differs (fp32 MFMA against
        float64) flips roundings that later layers mix into every element, so 32 layers drift.
        The drift allowed is set by a second implementation of the same definition: the oracle
        with its matrix products accumulated in float32 instead of float64, run over the same
        32 layers of step K-1.  The GPU's hidden rows and logits may drift from the float64 oracle
        at most twice as far (normwise) as that float32 oracle does; tokens must agree outside
        twice the observed logit deviation, and the capped-window count is reported.
    """
    shape = wl.LLAMA7B
    L_V, L_T = 256, 20
    n_slots, max_pos = (8, 288) if K == 7 else (K + 1, L_V + L_T + K)
    L_P, H, hd, V = L_V + L_T, shape.n_heads, shape.head_dim, shape.vocab
    g, layers, w = _weights(shape)
    text = wl.draw_ids(("instruction", 0), L_T, shape.vocab, device="cuda")
    pids = torch.cat([torch.full((L_V,), -1, dtype=torch.int32, device="cuda"), text])
    pool = {}

    def prefill_embeds(t):
        if t not in pool:
            e = torch.zeros((L_P + K - 1, shape.d_model), dtype=torch.bfloat16, device="cuda")
            e[:L_V] = wl.draw(("vision", 0, t), (L_V, shape.d_model), device="cuda")
            pool[t] = e
        return pool[t]

    ring = af.Ring(shape.n_layers, n_slots, max_pos, H, hd, dtype=torch.bfloat16)
    pipe = Pipeline(w, ring, K, pids, prefill_embeds, keep_logits=True)
    gpu = []
    for t in range(K):
        res = pipe.step()
        gpu.append(dict(segments=res.segments, hidden=to_np(res.hidden), logits=to_np(res.logits),
                        tokens=res.tokens.cpu().tolist()))
    ring.close()
    assert gpu[-1]["hidden"].shape[0] == L_P + K - 1
    emb = {t: to_np(prefill_embeds(t)[:L_P]) for t in range(K)}
    ids = pids.cpu().numpy().astype(np.int64)
    del pool
    gh = {k: to_np(v) for k, v in g.items()}
    lh = [{k: to_np(v) for k, v in lw.items()} for lw in layers]
    del g, layers
    torch.cuda.empty_cache()
    model = oracle.OracleModel(shape, gh, lh, storage="bf16")
    del gh, lh
    opipe = PipelineOracle(model, K, n_slots, max_pos, lambda t: (ids, emb[t]))

    def gpu_head(hidden_np, segs):
        """Final norm + LM head + argmax of the GPU on the given bf16 rows."""
        hid = torch.from_numpy(hidden_np).to(torch.bfloat16).cuda()
        assert np.array_equal(to_np(hid), hidden_np)
        z = torch.empty((len(segs), V), dtype=torch.float32, device="cuda")
        tok = torch.empty(len(segs), dtype=torch.int32, device="cuda")
        af.op_lm_head_argmax(w, hid, segs, z, tok)
        return to_np(z), tok.cpu().tolist()

    # ---- end to end, every step; the head on the oracle's hidden rows
    trace, e2e, head = [], [], []
    ties_head = n_head = capped_flips = 0
    for t in range(K):
        ost = opipe.step(forced=gpu[t]["tokens"], trace=trace if t == K - 1 else None)
        assert gpu[t]["segments"] == [(s.q_start, s.q_len, s.slot, s.pos0, s.request_id, 1)
                                      for s in ost["segments"]], t
        hrep = _layer_report(gpu[t]["hidden"], ost["hidden"])
        zrep = _logits_report(gpu[t]["logits"], ost["logits"])
        # free-running tokens: exact outside twice the observed deviation
        check_tokens(gpu[t]["tokens"], ost["logits"], gpu[t]["logits"], cap=np.inf)
        try:
            check_tokens(gpu[t]["tokens"], ost["logits"], gpu[t]["logits"])
        except AssertionError:
            capped_flips += 1
        e2e.append(dict(t=t, hidden=hrep, logits={k: zrep[k] for k in ("max_abs", "rms", "norm_rel", "n_bad")},
                        oracle_tokens=ost["tokens"], gpu_tokens=gpu[t]["tokens"]))
        print("end-to-end step", t, e2e[-1], flush=True)
        z, tok = gpu_head(ost["hidden"], gpu[t]["segments"])
        hz = _logits_report(z, ost["logits"])
        ties_head += check_tokens(tok, ost["logits"], z)
        n_head += len(tok)
        head.append(dict(t=t, ok=hz["ok"], max_abs=hz["max_abs"], rms=hz["rms"], n_bad=hz["n_bad"]))
        print("head on the oracle's hidden, step", t, head[-1], flush=True)
    print("head near-ties", ties_head, "of", n_head, "; free-running steps with a flip outside the capped window",
          capped_flips, flush=True)
    assert len(trace) == shape.n_layers

    # ---- per layer, from the oracle's input and ring history (step K - 1)
    segs_last = gpu[K - 1]["segments"]
    lring = af.Ring(shape.n_layers, n_slots, max_pos, H, hd, dtype=torch.bfloat16)
    for sg in sorted(segs_last, key=lambda s: s[4]):      # request r holds slot r, as in the pipeline
        if sg[3] > 0:
            lring.append(sg[4], sg[3])
    segs = reserve_step(lring, [(sg[4], sg[3], sg[1]) for sg in segs_last])
    assert [s[:4] for s in segs] == [s[:4] for s in segs_last]
    per_layer, growth = [], []
    for l in range(shape.n_layers):
        for sg in segs:
            if sg[3] > 0:
                kk = torch.from_numpy(opipe.kv.k[l, sg[2], :sg[3]]).to(torch.bfloat16).cuda()
                vv = torch.from_numpy(opipe.kv.v[l, sg[2], :sg[3]]).to(torch.bfloat16).cuda()
                lring.write_kv(l, sg[2], 0, kk, vv)
        x = torch.from_numpy(trace[l]["x_in"]).to(torch.bfloat16).cuda()
        assert np.array_equal(to_np(x), trace[l]["x_in"])
        af.packed_layer_forward(w, l, x, segs, lring)
        xl = to_np(x)
        per_layer.append(_layer_report(xl, trace[l]["x"], trace[l]))
        print("layer", l, "from the oracle's input", per_layer[-1], flush=True)
    # last layer + head from the oracle's input to the last layer
    z, tok = gpu_head(xl, segs_last)
    ost_z = opipe.model.logits(trace[-1]["x"][[s[0] + s[1] - 1 for s in segs_last]])
    last = _logits_report(z, ost_z)
    ties_last = check_tokens(tok, ost_z, z)
    print("last layer + head from the oracle's input", {k: last[k] for k in ("ok", "max_abs", "rms", "n_bad")},
          "near-ties", ties_last, flush=True)
    x = torch.from_numpy(trace[0]["x_in"]).to(torch.bfloat16).cuda()
    for l in range(shape.n_layers):
        af.packed_layer_forward(w, l, x, segs, lring)
        growth.append(_layer_report(to_np(x), trace[l]["x"]))
        print("layer", l, "chained on the GPU", growth[-1], flush=True)
    lring.close()
    w.close()

    # the drift of a float32-accumulating oracle over the same step (same input and history)
    import oracle.model as om

    def linear_f32(x, wt):
        return (np.asarray(x, np.float32) @ np.asarray(wt, np.float32).T).astype(np.float64)

    monkeypatch.setattr(om, "linear", linear_f32)
    osegs = oracle_segments(segs_last)
    x = trace[0]["x_in"]
    floor = []
    for l in range(shape.n_layers):
        x = opipe.model.layer_packed(l, x, osegs, opipe.kv)
        floor.append(_layer_report(x, trace[l]["x"]))
        print("layer", l, "float32-accumulating oracle", floor[-1], flush=True)
    z32 = opipe.model.logits(x[[s[0] + s[1] - 1 for s in segs_last]])
    monkeypatch.undo()
    floor_z = _logits_report(z32, ost_z)
    print("float32-accumulating oracle logits", {k: floor_z[k] for k in ("max_abs", "rms", "norm_rel", "n_bad")},
          flush=True)

    bad = [(l, r) for l, r in enumerate(per_layer) if not r["ok"]]
    assert not bad, bad
    assert last["ok"], last
    assert all(h["ok"] for h in head), head
    assert ties_head + ties_last <= max(2, (n_head + len(segs_last)) // 10), (ties_head, ties_last, n_head)
    h_floor, z_floor = floor[-1]["norm_rel"], floor_z["norm_rel"]
    for r in e2e:
        assert r["hidden"]["norm_rel"] <= 2 * h_floor and r["logits"]["norm_rel"] <= 2 * z_floor, (r, h_floor, z_floor)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("split_k", [False, True])
def test_7b_32_layer_packed_equals_sequential_on_gpu(split_k):
    """The paper's losslessness claim on the GPU at full size: the packed pipeline (K = 7, 8
    slots, run until the slots have wrapped) and the plain per-request run on the same kernels
    (a 276-row prefill alone, then single-row decodes, each request in its own ring), for
    requests 0, 1 and 9 (in a recycled slot).  Every kernel computes a row independently of the
    rows packed with it.  With split-K off (AF_OPT_NO_SPLIT_K) every row, logit and token is
    bit-identical.  With the default split-K the prefill rows still are (their GEMMs pick the
    same split factors in both runs); a decode row alone (M = 1) picks other factors, i.e.
    another fp32 summation order, which 32 layers of bf16 storage turn into a drift bounded
    normwise by 10%; its token must then agree outside the near-tie window."""
    shape = wl.LLAMA7B
    K, L_V, L_T = 7, 256, 20
    L_P = L_V + L_T
    g, layers, w = _weights(shape)
    if not split_k:
        w.set_options(af.AF_OPT_NO_SPLIT_K)
    text = wl.draw_ids(("instruction", 0), L_T, shape.vocab, device="cuda")
    pids = torch.cat([torch.full((L_V,), -1, dtype=torch.int32, device="cuda"), text])
    pool = {}

    def prefill_embeds(t):
        if t not in pool:
            e = torch.zeros((L_P + K - 1, shape.d_model), dtype=torch.bfloat16, device="cuda")
            e[:L_V] = wl.draw(("vision", 0, t), (L_V, shape.d_model), device="cuda")
            pool[t] = e
        return pool[t]

    ring = af.Ring(shape.n_layers, 8, 288, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
    pipe = Pipeline(w, ring, K, pids, prefill_embeds, keep_logits=True)
    # requests 0 and 1, and request 9, which reuses request 1's slot once the ring has wrapped
    rows, logits, slots = {0: {}, 1: {}, 9: {}}, {0: {}, 1: {}, 9: {}}, {}
    for t in range(9 + K):
        res = pipe.step()
        for j, sg in enumerate(res.segments):
            if sg[4] in rows:
                rows[sg[4]][sg[3]] = to_np(res.hidden[sg[0]:sg[0] + sg[1]])
                logits[sg[4]][sg[3]] = to_np(res.logits[j])
                slots[sg[4]] = sg[2]
    assert slots[9] == slots[1]
    packed_tokens = {r: pipe.request_tokens(r) for r in rows}
    ring.close()
    D, V = shape.d_model, shape.vocab
    for r in rows:
        sring = af.Ring(shape.n_layers, 1, 288, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
        hid = torch.empty((L_P, D), dtype=torch.bfloat16, device="cuda")
        tok = torch.empty(1, dtype=torch.int32, device="cuda")
        z = torch.empty((1, V), dtype=torch.float32, device="cuda")
        s = sring.append(r, L_P)
        af.packed_forward(w, pids.clone(), prefill_embeds(r)[:L_P], [(0, L_P, s.slot, 0, r, 1)], sring, hid, z, tok)
        assert np.array_equal(to_np(hid), rows[r][0]), f"request {r}: prefill rows differ"
        assert np.array_equal(to_np(z)[0], logits[r][0])
        assert int(tok.item()) == packed_tokens[r][0]
        seq_z, pk_z, seq_tok = [], [], []
        for j in range(1, K):
            s = sring.append(r, 1)
            assert s.pos0 == L_P + j - 1
            feed = torch.tensor([packed_tokens[r][j - 1]], dtype=torch.int32, device="cuda")
            h1 = torch.empty((1, D), dtype=torch.bfloat16, device="cuda")
            af.packed_forward(w, feed, None, [(0, 1, s.slot, s.pos0, r, 1)], sring, h1, z, tok)
            if split_k:
                rep = bf16_layer_parity(to_np(h1), rows[r][s.pos0], norm_rel=0.1, row_norm_rel=0.1,
                                        outlier_frac=1.0, outlier_cap=np.inf)
                assert rep["ok"], (r, j, rep)
            else:
                assert np.array_equal(to_np(h1), rows[r][s.pos0]), f"request {r}: decode {j} differs"
                assert np.array_equal(to_np(z)[0], logits[r][s.pos0])
            seq_z.append(to_np(z)[0])
            pk_z.append(logits[r][s.pos0])
            seq_tok.append(int(tok.item()))
        if split_k:
            # GPU against GPU with another fp32 summation order: the window is twice the
            # observed deviation, not capped (the capped window is for oracle comparisons)
            check_tokens(packed_tokens[r][1:], np.stack(pk_z), np.stack(seq_z), cap=np.inf)
        else:
            assert seq_tok == packed_tokens[r][1:]
        sring.close()
    w.close()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("K,L_T", [(16, 20), (24, 64), (32, 20), (7, 256)])
def test_7b_k_sweep_packed_equals_sequential_4_layers(K, L_T):
    """The K sweep's points beyond the benchmark's (a prefill of 256 vision rows and L_T
    instruction rows packed with K - 1 decode rows; at K = 24 and 32 the decode rows and the
    query tiles take the four-wave attention launch; K = 24 with the 64-row instruction of a
    longer prefill, 326..343 rows
    on 192-row tiles; L_T = 256, 518 rows, gate/up on the 288 x 256 tile): with split-K off
    every row, logit and token of requests 0 and 1 equals the plain per-request run on the same
    kernels, bit for bit (a 4-layer model of the 7B shape)."""
    shape = wl.LLAMA7B.with_layers(4)
    L_V = 256
    L_P, D, V = L_V + L_T, shape.d_model, shape.vocab
    g, layers, w = _weights(shape)
    del g, layers
    w.set_options(af.AF_OPT_NO_SPLIT_K)
    text = wl.draw_ids(("instruction", 0), L_T, V, device="cuda")
    pids = torch.cat([torch.full((L_V,), -1, dtype=torch.int32, device="cuda"), text])
    pool = {}

    def prefill_embeds(t):
        if t not in pool:
            e = torch.zeros((L_P + K - 1, D), dtype=torch.bfloat16, device="cuda")
            e[:L_V] = wl.draw(("vision", 0, t), (L_V, D), device="cuda")
            pool[t] = e
        return pool[t]

    ring = af.Ring(shape.n_layers, K + 1, L_P + K, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
    pipe = Pipeline(w, ring, K, pids, prefill_embeds, keep_logits=True)
    rows, logits, Ms = {0: {}, 1: {}}, {0: {}, 1: {}}, []
    for t in range(K + 1):
        res = pipe.step()
        Ms.append(res.M)
        for j, sg in enumerate(res.segments):
            if sg[4] in rows:
                rows[sg[4]][sg[3]] = to_np(res.hidden[sg[0]:sg[0] + sg[1]])
                logits[sg[4]][sg[3]] = to_np(res.logits[j])
    assert max(Ms) == L_P + K - 1
    packed_tokens = {r: pipe.request_tokens(r) for r in rows}
    ring.close()
    for r in rows:
        sring = af.Ring(shape.n_layers, 1, L_P + K, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
        hid = torch.empty((L_P, D), dtype=torch.bfloat16, device="cuda")
        tok = torch.empty(1, dtype=torch.int32, device="cuda")
        z = torch.empty((1, V), dtype=torch.float32, device="cuda")
        s = sring.append(r, L_P)
        af.packed_forward(w, pids.clone(), prefill_embeds(r)[:L_P], [(0, L_P, s.slot, 0, r, 1)], sring, hid, z, tok)
        assert np.array_equal(to_np(hid), rows[r][0]), f"request {r}: prefill rows differ"
        assert np.array_equal(to_np(z)[0], logits[r][0]) and int(tok.item()) == packed_tokens[r][0]
        for j in range(1, K):
            s = sring.append(r, 1)
            feed = torch.tensor([packed_tokens[r][j - 1]], dtype=torch.int32, device="cuda")
            h1 = torch.empty((1, D), dtype=torch.bfloat16, device="cuda")
            af.packed_forward(w, feed, None, [(0, 1, s.slot, s.pos0, r, 1)], sring, h1, z, tok)
            assert np.array_equal(to_np(h1), rows[r][s.pos0]), f"request {r}: decode {j} differs"
            assert np.array_equal(to_np(z)[0], logits[r][s.pos0]) and int(tok.item()) == packed_tokens[r][j]
        sring.close()
    w.close()
