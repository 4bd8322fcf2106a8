"""CPU tests of the C ABI: the library loads, exports every declared entry point, and its
slot bookkeeping (a bookkeeping-only ring, no device call) matches the oracle's RingModel
bit for bit, errors included."""
import os
import random
import re

import pytest

import paper_2512_20276_amd as af
from oracle.ring import RingError, RingModel

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "actionflow.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b(af_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_contract():
    names = declared_functions()
    for must in ("af_ring_create", "af_ring_append", "af_ring_release", "af_packed_forward",
                 "af_packed_layer_forward", "af_weights_create", "af_last_error"):
        assert must in names


def test_library_exports_every_declared_symbol():
    missing = [n for n in declared_functions() if not hasattr(af.lib, n)]
    assert not missing, missing


def test_tensor_count():
    assert af.lib.af_weights_tensor_count(32) == 3 + 9 * 32


def _pipeline_ops(K, L_P, steps):
    ops = []
    ntok = {}
    for t in range(steps):
        for s in range(K):
            r = t - s
            if r < 0:
                break
            ops.append(("append", r, L_P if s == 0 else 1))
            ntok[r] = ntok.get(r, 0) + 1
        for r in [r for r, c in ntok.items() if c == K]:
            ops.append(("release", r, 0))
            del ntok[r]
    return ops


def _apply(ring, model, op):
    kind, rid, n = op
    got = want = None
    try:
        if kind == "append":
            s = ring.append(rid, n)
            got = (s.slot, s.pos0, s.q_len, s.request_id)
        else:
            ring.release(rid)
            got = "ok"
    except af.AFError as e:
        got = ("err", e.code)
    try:
        if kind == "append":
            slot, pos0 = model.append(rid, n)
            want = (slot, pos0, n, rid)
        else:
            model.release(rid)
            want = "ok"
    except RingError as e:
        want = ("err", e.code)
    return got, want


@pytest.mark.parametrize("K,n_slots", [(7, 8), (3, 4), (8, 64), (7, 7)])
def test_pipeline_schedule_bit_exact_vs_oracle(K, n_slots):
    ring = af.Ring(0, n_slots, 288)
    model = RingModel(n_slots, 288)
    for op in _pipeline_ops(K, 276, 64):
        got, want = _apply(ring, model, op)
        assert got == want, op
        owners, lens, head = ring.state()
        assert (owners, lens, head) == model.state()
    ring.close()


def test_random_schedules_bit_exact_vs_oracle():
    rnd = random.Random(7)
    for n_slots, max_pos in ((1, 3), (2, 5), (3, 8), (5, 2)):
        ring, model = af.Ring(0, n_slots, max_pos), RingModel(n_slots, max_pos)
        ids = []
        for i in range(400):
            r = rnd.random()
            if r < 0.4:
                op = ("append", len(ids) + 100, rnd.randint(-1, max_pos + 1))
                ids.append(op[1])
            elif r < 0.8 and ids:
                op = ("append", rnd.choice(ids), rnd.randint(-1, 3))
            elif ids:
                op = ("release", rnd.choice(ids + [10 ** 9]), 0)
            else:
                continue
            got, want = _apply(ring, model, op)
            assert got == want, (i, op)
            assert ring.state() == model.state()


def test_error_codes_and_messages():
    ring = af.Ring(0, 2, 8)
    ring.append(5, 8)
    with pytest.raises(af.AFError) as e:
        ring.append(5, 1)
    assert e.value.code == af.AF_ERR_OUT_OF_RANGE and "max_pos" in str(e.value)
    ring.append(6, 1)
    with pytest.raises(af.AFError) as e:
        ring.append(7, 1)
    assert e.value.code == af.AF_ERR_SLOT_BUSY
    with pytest.raises(af.AFError) as e:
        ring.release(99)
    assert e.value.code == af.AF_ERR_UNKNOWN_REQUEST
    with pytest.raises(af.AFError) as e:
        ring.append(8, 0)
    assert e.value.code == af.AF_ERR_INVALID_ARG
    ring.reset()
    assert ring.state() == ([-1, -1], [0, 0], 0)


def test_ring_create_rejects_bad_descriptors():
    for args in ((0, 0, 8), (0, 4, 0), (-1, 4, 8)):
        with pytest.raises(af.AFError) as e:
            af.Ring(*args)
        assert e.value.code == af.AF_ERR_INVALID_ARG


@pytest.mark.parametrize("P,K,n_slots", [(8, 8, 64), (3, 4, 12), (2, 7, 16), (1, 7, 8)])
def test_multi_pipeline_bookkeeping_matches_oracle_and_closed_form(P, K, n_slots):
    """The pipeline driver's slot bookkeeping for P pipelines packed into one forward (stage-
    major rows, request ids t * P + p), on a bookkeeping-only ring: every segment equals the
    oracle RingModel's answer for the same calls, request r lives in slot r mod n_slots, and
    its stage-s decode row sits at pos0 = L_P + s - 1 (kv_len = L_P + s)."""
    import types

    import torch

    from paper_2512_20276_amd.pipeline import Pipeline

    L_P = 276
    ring = af.Ring(0, n_slots, 288)
    model = RingModel(n_slots, 288)
    shape = types.SimpleNamespace(d_model=8, vocab=4)
    w = types.SimpleNamespace(shape=shape, dtype=torch.float32)
    pipe = Pipeline(w, ring, K, torch.full((L_P,), -1, dtype=torch.int32), lambda t: None, n_pipes=P)
    for t in range(3 * K + 2):
        segs, M = pipe.reserve(t)
        live = min(t + 1, K)
        assert M == P * L_P + P * (live - 1)
        row = 0
        for i, s in enumerate(segs):
            stage, p = divmod(i, P)
            r = (t - stage) * P + p
            n = L_P if stage == 0 else 1
            assert (s.request_id, s.q_start, s.q_len) == (r, row, n)
            assert (s.slot, s.pos0) == model.append(r, n)
            assert s.slot == r % n_slots
            assert s.pos0 == (0 if stage == 0 else L_P + stage - 1)
            row += n
        done = pipe.finish(segs)
        assert sorted(done) == ([(t - K + 1) * P + p for p in range(P)] if t >= K - 1 else [])
        for rid in done:
            model.release(rid)
        assert ring.state() == model.state()
    ring.close()


@pytest.mark.parametrize("K,n_slots", [(7, 7), (7, 9), (3, 3), (2, 4)])
def test_copy_shift_bookkeeping_matches_oracle(K, n_slots):
    """The physical-copy InPlaceKVShift on a bookkeeping-only ring: the driver's copy mode gives
    the same segment tables and slot state as the oracle RingModel, and stage s of every step
    sits in slot s (closed form), with pos0 = L_P + s - 1."""
    import types

    import torch

    from paper_2512_20276_amd.pipeline import Pipeline

    L_P = 20
    ring = af.Ring(0, n_slots, 64)
    model = RingModel(n_slots, 64)
    w = types.SimpleNamespace(shape=types.SimpleNamespace(d_model=8, vocab=4), dtype=torch.float32)
    pipe = Pipeline(w, ring, K, torch.full((L_P,), -1, dtype=torch.int32), lambda t: None, shift="copy")
    for t in range(3 * K + 1):
        segs, _ = pipe.reserve(t)
        for s, sg in enumerate(segs):
            assert (sg.slot, sg.pos0) == model.append(t - s, L_P if s == 0 else 1)
            assert sg.slot == s and sg.pos0 == (0 if s == 0 else L_P + s - 1)
        done = pipe.finish(segs)
        for rid in done:
            model.release(rid)
        model.shift_stages(K)
        assert ring.state() == model.state()


def test_copy_shift_errors_leave_state_unchanged():
    ring = af.Ring(0, 4, 16)
    model = RingModel(4, 16)
    for rid in range(3):
        ring.append(rid, 2)
        model.append(rid, 2)
    before = ring.state()
    for n, code in ((1, af.AF_ERR_INVALID_ARG), (5, af.AF_ERR_INVALID_ARG), (3, af.AF_ERR_SLOT_BUSY)):
        with pytest.raises(af.AFError) as e:
            ring.shift_stages(n)
        assert e.value.code == code
        with pytest.raises(RingError) as e2:
            model.shift_stages(n)
        assert e2.value.code == code
        assert ring.state() == before == model.state()
    ring.shift_stages(4)
    model.shift_stages(4)
    assert ring.state() == model.state() == ([-1, 0, 1, 2], [0, 2, 2, 2], 0)


def test_kv_copy_and_ring_layer_calls_reject_bad_arguments_on_the_host():
    """The naive pipeline's region copy and the ring-layer forward validate before any launch:
    a bookkeeping-only ring has no storage, NULL handles are refused."""
    a, b = af.Ring(0, 4, 16), af.Ring(0, 2, 16)
    with pytest.raises(af.AFError) as e:
        a.copy_kv_to(0, 0, b, 0, 0, 0, 4)
    assert e.value.code == af.AF_ERR_INVALID_ARG and "storage" in str(e.value)
    assert af.lib.af_ring_copy_kv(None, 0, 0, b.h, 0, 0, 0, 1, None) == af.AF_ERR_INVALID_ARG
    assert af.lib.af_packed_layer_forward_kv(None, 0, None, 1, None, 0, a.h, 0, None) == af.AF_ERR_INVALID_ARG
    assert a.state() == ([-1] * 4, [0] * 4, 0)
