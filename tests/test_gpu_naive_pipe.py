"""GPU tests of the pipeline without the unified ring (per-request caches, a per-layer gather
into one contiguous buffer and a scatter back, host-coordinated batching).

* af_ring_copy_kv moves exactly the named region between rings of different shapes, bit for
  bit, and leaves every other cell untouched; mismatched rings are rejected before any launch.
* af_packed_layer_forward_kv (a layer whose keys and values live in another ring layer) gives
  the same hidden rows and written keys/values, bit for bit, as the plain per-layer call.
* The naive pipeline reproduces the ring pipeline's hidden rows, logits and tokens exactly,
  on the tiny fp32 decoder and on the 32-layer 7B shape (the attention sees the same keys in
  the same order; only copies and host round trips differ).  The ring pipeline is held to
  the oracle by the model tests, so this carries that parity over.
"""
import dataclasses

import numpy as np
import pytest
import torch

import workload as wl
from tests.helpers import advance_head, reserve_step, tiny_prefill_fn, to_np

pytestmark = pytest.mark.gpu
af = pytest.importorskip("paper_2512_20276_amd")
from paper_2512_20276_amd.naive_pipe import NaivePipeline  # noqa: E402
from paper_2512_20276_amd.pipeline import Pipeline  # noqa: E402


def _fill(ring, L, n_slots, max_pos, H, hd, key, dtype=torch.bfloat16):
    cells = {}
    for l in range(L):
        for s in range(n_slots):
            kv = wl.draw((key, l, s), (2, max_pos, H, hd), dtype=dtype, device="cuda")
            ring.write_kv(l, s, 0, kv[0], kv[1])
            cells[(l, s)] = (to_np(kv[0]), to_np(kv[1]))
    return cells


def test_ring_copy_kv_between_rings():
    H, hd = 4, 64
    a = af.Ring(3, 5, 40, H, hd, dtype=torch.bfloat16)
    b = af.Ring(1, 3, 24, H, hd, dtype=torch.bfloat16)
    ca = _fill(a, 3, 5, 40, H, hd, "copy a")
    cb = _fill(b, 1, 3, 24, H, hd, "copy b")
    a.copy_kv_to(2, 4, b, 0, 1, 3, 17)      # a[2][4][3:20] -> b[0][1][3:20]
    b.copy_kv_to(0, 2, a, 1, 0, 0, 24)      # b[0][2][0:24] -> a[1][0][0:24]
    a.copy_kv_to(0, 1, a, 0, 3, 5, 11)      # within one ring: a[0][1][5:16] -> a[0][3][5:16]
    a.copy_kv_to(1, 1, a, 1, 1, 0, 40)      # onto itself: no-op
    torch.cuda.synchronize()
    want_b = {k: (v[0].copy(), v[1].copy()) for k, v in cb.items()}
    want_b[(0, 1)][0][3:20] = ca[(2, 4)][0][3:20]
    want_b[(0, 1)][1][3:20] = ca[(2, 4)][1][3:20]
    want_a = {k: (v[0].copy(), v[1].copy()) for k, v in ca.items()}
    want_a[(1, 0)][0][:24] = cb[(0, 2)][0]
    want_a[(1, 0)][1][:24] = cb[(0, 2)][1]
    want_a[(0, 3)][0][5:16] = ca[(0, 1)][0][5:16]
    want_a[(0, 3)][1][5:16] = ca[(0, 1)][1][5:16]
    for ring, want, (L, n_slots, max_pos) in ((a, want_a, (3, 5, 40)), (b, want_b, (1, 3, 24))):
        for l in range(L):
            for s in range(n_slots):
                k, v = ring.read_kv(l, s, 0, max_pos)
                assert np.array_equal(to_np(k), want[(l, s)][0]), (l, s)
                assert np.array_equal(to_np(v), want[(l, s)][1]), (l, s)
    c = af.Ring(1, 2, 24, H, 128, dtype=torch.bfloat16)
    with pytest.raises(af.AFError) as e:
        b.copy_kv_to(0, 0, c, 0, 0, 0, 4)   # head_dim differs
    assert e.value.code == -1
    with pytest.raises(af.AFError) as e:
        a.copy_kv_to(0, 0, b, 0, 0, 20, 8)  # past b's max_pos
    assert e.value.code == -2
    for r in (a, b, c):
        r.close()


@pytest.mark.parametrize("storage", ["f32", "bf16"])
def test_layer_forward_kv_equals_plain_layer(storage):
    """Layer 1 of a 2-layer model against ring layer 1 of a full ring, and against ring layer 0
    of a one-layer ring holding the same history: identical rows and keys/values."""
    shape = dataclasses.replace(wl.TINY, dtype=storage)
    dt = shape.torch_dtype
    H, hd, D = shape.n_heads, shape.head_dim, shape.d_model
    g, layers = wl.model_weights(shape, seed=3, device="cuda", random_gains=True)
    w = af.Weights(shape, g, layers)
    full = af.Ring(2, 4, 48, H, hd, dtype=dt)
    one = af.Ring(1, 3, 48, H, hd, dtype=dt)
    _fill(full, 2, 4, 48, H, hd, "hist", dtype=dt)
    for s in range(3):                      # one-layer slot s holds full ring layer 1, slot s + 1
        one.write_kv(0, s, 0, *full.read_kv(1, s + 1, 0, 48))
    specs = [(7, 0, 20), (5, 29, 1), (4, 40, 1)]  # a 20-row prefill, decodes at contexts 30 and 41
    advance_head(full, 1)
    segs_full = reserve_step(full, specs)   # slots 1, 2, 3
    segs_one = reserve_step(one, specs)     # slots 0, 1, 2
    assert [s[2] for s in segs_full] == [1, 2, 3] and [s[2] for s in segs_one] == [0, 1, 2]
    x = wl.draw(("rows",), (22, D), dtype=dt, device="cuda")
    h_full, h_one = x.clone(), x.clone()
    af.packed_layer_forward(w, 1, h_full, segs_full, full)
    af.packed_layer_forward(w, 1, h_one, segs_one, one, ring_layer=0)
    torch.cuda.synchronize()
    assert torch.equal(h_full, h_one)
    for sf, so in zip(segs_full, segs_one):
        kf, vf = full.read_kv(1, sf[2], 0, sf[3] + sf[1])
        ko, vo = one.read_kv(0, so[2], 0, so[3] + so[1])
        assert torch.equal(kf, ko) and torch.equal(vf, vo)
    with pytest.raises(af.AFError):
        af.packed_layer_forward(w, 1, h_one, segs_one, one, ring_layer=1)  # the ring holds one layer
    w.close()
    full.close()
    one.close()


def _run_both(w, shape, K, pids, embeds, n_slots, steps, max_pos):
    ring = af.Ring(shape.n_layers, n_slots, max_pos, shape.n_heads, shape.head_dim, dtype=shape.torch_dtype)
    pipe = Pipeline(w, ring, K, pids, embeds, keep_logits=True)
    naive = NaivePipeline(w, K, pids, embeds, keep_logits=True)
    for t in range(steps):
        a = pipe.step()
        b = naive.step()
        torch.cuda.synchronize()
        assert a.segments and [(s[0], s[1], s[3], s[4]) for s in a.segments] == \
            [(s[0], s[1], s[3], s[4]) for s in b.segments], t
        assert torch.equal(a.hidden, b.hidden), t
        assert torch.equal(a.logits, b.logits), t
        assert a.tokens.cpu().tolist() == b.tokens.cpu().tolist(), t
        assert a.done == b.done, t
    for r in range(max(0, steps - K - 1)):
        assert pipe.request_tokens(r) == naive.request_tokens(r)
    ring.close()
    naive.close()


def test_naive_pipeline_equals_ring_pipeline_tiny():
    shape = wl.TINY
    K, L_P = 3, 32
    g, layers = wl.model_weights(shape, seed=0, device="cuda", random_gains=True)
    w = af.Weights(shape, g, layers)
    ids0, _ = tiny_prefill_fn(shape, L_P, seed=0)(0)
    pids = torch.from_numpy(ids0).to(torch.int32).cuda()

    def embeds(t):
        return torch.zeros((L_P + K - 1, shape.d_model), dtype=torch.float32, device="cuda")

    _run_both(w, shape, K, pids, embeds, n_slots=4, steps=8, max_pos=64)
    w.close()


@pytest.mark.timeout(600)
def test_naive_pipeline_equals_ring_pipeline_7b_32_layers():
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

    _run_both(w, shape, K, pids, embeds, n_slots=8, steps=K + 2, max_pos=288)
    w.close()
