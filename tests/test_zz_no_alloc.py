"""The forward that allocates nothing (af_packed_forward_noalloc) against af_packed_forward.

Both run the same kernels in the same order, so hidden rows, logits, tokens and every ring cell
written must be bit-identical.  Two no-allocation calls in a row, the second with a smaller
packed step, check that the library's shared scratch array carries nothing stale from one call
into the next (its K padding is cleared, its tables re-uploaded).  A step too large for the
array is rejected before any launch.
"""
import numpy as np
import pytest
import torch

import workload as wl
from tests.helpers import advance_head, reserve_step, to_np

pytestmark = pytest.mark.gpu
af = pytest.importorskip("paper_2512_20276_amd")


def _rings(shape, n_slots, max_pos, key):
    """Two rings with identical N(0, 1) history in every cell."""
    rings = [af.Ring(shape.n_layers, n_slots, max_pos, shape.n_heads, shape.head_dim, dtype=shape.torch_dtype)
             for _ in range(2)]
    for l in range(shape.n_layers):
        for s in range(n_slots):
            k = wl.draw((key, "k", l, s), (max_pos, shape.n_heads, shape.head_dim), dtype=shape.torch_dtype,
                        device="cuda")
            v = wl.draw((key, "v", l, s), (max_pos, shape.n_heads, shape.head_dim), dtype=shape.torch_dtype,
                        device="cuda")
            for r in rings:
                r.write_kv(l, s, 0, k, v)
    return rings


def _inputs(shape, segs, key):
    M = sum(s[1] for s in segs)
    ids = wl.draw_ids((key, "ids"), M, shape.vocab, device="cuda")
    emb = wl.draw((key, "emb"), (M, shape.d_model), dtype=shape.torch_dtype, device="cuda")
    first = segs[0]
    if first[1] > 1:  # the prefill's leading rows take given embeddings (-1 ids)
        ids[first[0]:first[0] + first[1] // 2] = -1
    return ids, emb


def _run_pair(w, shape, rings, specs, key, with_logits=True):
    """The same step through af_packed_forward on rings[0] and the no-allocation call on rings[1]."""
    segs = [reserve_step(r, specs) for r in rings]
    assert segs[0] == segs[1]
    segs = segs[0]
    M, n_emit, V = sum(s[1] for s in segs), len(segs), shape.vocab
    ids, emb = _inputs(shape, segs, key)
    outs = []
    for r, fn in zip(rings, (af.packed_forward, af.packed_forward_noalloc)):
        hid = torch.full((M, shape.d_model), float("nan"), dtype=shape.torch_dtype, device="cuda")
        z = torch.full((n_emit, V), float("nan"), dtype=torch.float32, device="cuda") if with_logits else None
        tok = torch.full((n_emit,), -7, dtype=torch.int32, device="cuda")
        fn(w, ids.clone(), emb, segs, r, hid, z, tok)
        torch.cuda.synchronize()
        outs.append((to_np(hid), None if z is None else to_np(z), tok.cpu().numpy()))
    (h0, z0, t0), (h1, z1, t1) = outs
    assert np.array_equal(h0, h1), "hidden rows differ"
    if with_logits:
        assert np.array_equal(z0, z1), "logits differ"
    assert np.array_equal(t0, t1), "tokens differ"
    assert np.all(np.isfinite(h1)) and np.all(t1 >= 0)
    for l in range(shape.n_layers):
        for s in segs:
            k0, v0 = rings[0].read_kv(l, s[2], 0, s[3] + s[1])
            k1, v1 = rings[1].read_kv(l, s[2], 0, s[3] + s[1])
            assert torch.equal(k0, k1) and torch.equal(v0, v1), (l, s)
    return segs


def test_noalloc_matches_packed_forward_7b():
    shape = wl.LLAMA7B.with_layers(3)
    g, layers = wl.model_weights(shape, seed=0, device="cuda")
    w = af.Weights(shape, g, layers)
    del g, layers
    rings = _rings(shape, 8, 320, "noalloc 7b")
    for r in rings:
        advance_head(r, 3)
        for rid in range(4, 10):
            r.append(rid, 276 + (10 - rid) - 1)
    # the benchmark step: a 276-row prefill and six decode rows at contexts 277..282
    specs = [(10, 0, 276)] + [(10 - s, 276 + s - 1, 1) for s in range(1, 7)]
    segs = _run_pair(w, shape, rings, specs, "step 1")
    assert sum(s[1] for s in segs) == 282
    # a smaller step next: a 40-row chunk of request 10 and three decode rows
    specs = [(10, 276, 40), (9, 277, 1), (8, 278, 1), (7, 279, 1)]
    _run_pair(w, shape, rings, specs, "step 2", with_logits=False)
    for r in rings:
        r.close()
    w.close()


def test_noalloc_matches_packed_forward_tiny_fp32():
    shape = wl.TINY
    g, layers = wl.model_weights(shape, seed=0, device="cuda", random_gains=True)
    w = af.Weights(shape, g, layers)
    rings = _rings(shape, 4, 64, "noalloc tiny")
    for r in rings:
        r.append(0, 33)
        r.append(1, 32)
    specs = [(2, 0, 32), (1, 32, 1), (0, 33, 1)]
    _run_pair(w, shape, rings, specs, "tiny 1")
    specs = [(1, 33, 1), (0, 34, 1)]
    _run_pair(w, shape, rings, specs, "tiny 2")
    for r in rings:
        r.close()
    w.close()


def test_noalloc_rejects_a_step_beyond_its_scratch():
    shape = wl.LLAMA7B.with_layers(1)
    g, layers = wl.model_weights(shape, seed=0, device="cuda")
    w = af.Weights(shape, g, layers)
    del g, layers
    ring = af.Ring(1, 2, 2048, shape.n_heads, shape.head_dim, dtype=torch.bfloat16)
    M = 2000
    segs = reserve_step(ring, [(0, 0, M)])
    ids = torch.full((M,), 5, dtype=torch.int32, device="cuda")
    hid = torch.full((M, shape.d_model), 3.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(af.AFError) as e:
        af.packed_forward_noalloc(w, ids, None, segs, ring, hid)
    assert e.value.code == af.AF_ERR_OUT_OF_RANGE and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool(torch.all(hid == 3.0))  # nothing ran
    ring.close()
    w.close()
