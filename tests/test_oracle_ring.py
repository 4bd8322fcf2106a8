"""Pins of the ring bookkeeping model: the round-robin closed form of the steady-state
pipeline (Alg. 1 with K stages) and the invariants of the slot state machine."""
import itertools
import random

import pytest

from oracle.ring import OUT_OF_RANGE, SLOT_BUSY, UNKNOWN_REQUEST, INVALID_ARG, RingError, RingModel


def _pipeline_schedule(K, L_P, n_slots, max_pos, steps):
    ring = RingModel(n_slots, max_pos)
    ntok = {}
    out = []
    for t in range(steps):
        segs = []
        for s in range(K):
            r = t - s
            if r < 0:
                break
            n = L_P if s == 0 else 1
            slot, pos0 = ring.append(r, n)
            segs.append((r, slot, pos0, pos0 + n))
            ntok[r] = ntok.get(r, 0) + 1
        for r in [r for r, c in ntok.items() if c == K]:
            ring.release(r)
            del ntok[r]
        out.append(segs)
    return out


@pytest.mark.parametrize("K,n_slots", [(7, 8), (7, 7), (3, 4), (8, 64), (1, 1)])
def test_steady_state_closed_form(K, n_slots):
    """Request t lives in slot t mod n_slots; its stage-s decode has pos0 = L_P + s - 1 and
    kv_len = L_P + s (the logical KV length of stage s)."""
    L_P = 276
    for t, segs in enumerate(_pipeline_schedule(K, L_P, n_slots, 288, 64)):
        assert len(segs) == min(t + 1, K)
        for s, (r, slot, pos0, kv_len) in enumerate(segs):
            assert r == t - s
            assert slot == r % n_slots
            assert pos0 == (0 if s == 0 else L_P + s - 1)
            assert kv_len == L_P + s


def test_too_few_slots_is_slot_busy():
    with pytest.raises(RingError) as e:
        _pipeline_schedule(7, 10, 6, 64, 10)
    assert e.value.code == SLOT_BUSY


def test_errors_leave_state_unchanged():
    ring = RingModel(2, 8)
    ring.append(10, 5)
    before = ring.state()
    for call, code in ((lambda: ring.append(10, 4), OUT_OF_RANGE), (lambda: ring.append(11, 9), OUT_OF_RANGE),
                       (lambda: ring.append(12, 0), INVALID_ARG), (lambda: ring.release(99), UNKNOWN_REQUEST)):
        with pytest.raises(RingError) as e:
            call()
        assert e.value.code == code
        assert ring.state() == before
    ring.append(11, 8)               # fills slot 1; head wraps to slot 0, still owned
    with pytest.raises(RingError) as e:
        ring.append(12, 1)
    assert e.value.code == SLOT_BUSY
    ring.release(10)
    assert ring.append(12, 1) == (0, 0)


def test_random_schedules_keep_invariants():
    """Brute force over random operation sequences on tiny rings."""
    rnd = random.Random(0)
    for n_slots, max_pos in itertools.product((1, 2, 3, 5), (1, 4, 9)):
        ring = RingModel(n_slots, max_pos)
        resident = {}
        next_id = 0
        for _ in range(300):
            op = rnd.random()
            before = ring.state()
            try:
                if op < 0.45:
                    rid = next_id
                    n = rnd.randint(-1, max_pos + 1)
                    head = ring.head
                    slot, pos0 = ring.append(rid, n)
                    assert (slot, pos0) == (head, 0) and ring.head == (head + 1) % n_slots
                    resident[rid] = [slot, n]
                    next_id += 1
                elif op < 0.8 and resident:
                    rid = rnd.choice(sorted(resident))
                    n = rnd.randint(-1, 3)
                    slot, pos0 = ring.append(rid, n)
                    assert slot == resident[rid][0] and pos0 == resident[rid][1]
                    resident[rid][1] += n
                elif resident:
                    rid = rnd.choice(sorted(resident) + [10 ** 6])
                    slot = ring.release(rid)
                    assert slot == resident.pop(rid)[0]
            except RingError:
                assert ring.state() == before
            owners, lens, head = ring.state()
            live = [o for o in owners if o != RingModel.FREE]
            assert len(live) == len(set(live)) == len(resident)
            for rid, (slot, ln) in resident.items():
                assert owners[slot] == rid and lens[slot] == ln <= max_pos
