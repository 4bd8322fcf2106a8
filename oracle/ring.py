"""Slot bookkeeping of the Unified KV Ring Buffer, as a plain state machine.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper keeps every active request's KV in one circular region, logically
partitioned per request (Sec. 3.3), and between steps moves the stages along so
the oldest request's space is overwritten (InPlaceKVShift).  Here that motion is an
index rotation: a new request takes the next slot in ring order (wrapping at
n_slots); a finished request's slot is released and is reused when the rotation
comes back to it.  No KV bytes move.

Semantics (the C library must match them bit for bit):
  append(id, n):  id resident  -> continuation: pos0 = len[slot]; len += n
                  id not resident -> new request: slot = head; the slot must be free;
                                     head = (head + 1) mod n_slots; pos0 = 0; len = n
                  n <= 0 -> INVALID_ARG;  pos0 + n > max_pos -> OUT_OF_RANGE;
                  head slot owned -> SLOT_BUSY.  A failed call changes nothing.
  release(id):    id not resident -> UNKNOWN_REQUEST; else the slot becomes free, len 0.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Tuple

INVALID_ARG, OUT_OF_RANGE, SLOT_BUSY, UNKNOWN_REQUEST = -1, -2, -3, -4


class RingError(Exception):
    def __init__(self, code: int, msg: str):
        super().__init__(msg)
        self.code = code


class RingModel:
    FREE = -1

    def __init__(self, n_slots: int, max_pos: int):
        if n_slots <= 0 or max_pos <= 0:
            raise RingError(INVALID_ARG, "n_slots and max_pos must be positive")
        self.n_slots, self.max_pos = n_slots, max_pos
        self.owner: List[int] = [self.FREE] * n_slots
        self.length: List[int] = [0] * n_slots
        self.head = 0
        self._slot_of: Dict[int, int] = {}

    def append(self, request_id: int, n_new: int) -> Tuple[int, int]:
        """Reserve ``n_new`` positions for ``request_id``; returns (slot, pos0)."""
        if n_new <= 0 or request_id < 0:
            raise RingError(INVALID_ARG, "n_new must be positive and request_id >= 0")
        if request_id in self._slot_of:
            slot = self._slot_of[request_id]
            pos0 = self.length[slot]
            if pos0 + n_new > self.max_pos:
                raise RingError(OUT_OF_RANGE, "append past max_pos")
            self.length[slot] = pos0 + n_new
            return slot, pos0
        slot = self.head
        if self.owner[slot] != self.FREE:
            raise RingError(SLOT_BUSY, f"slot {slot} still owned by request {self.owner[slot]}")
        if n_new > self.max_pos:
            raise RingError(OUT_OF_RANGE, "append past max_pos")
        self.owner[slot] = request_id
        self.length[slot] = n_new
        self._slot_of[request_id] = slot
        self.head = (slot + 1) % self.n_slots
        return slot, 0

    def release(self, request_id: int) -> int:
        """Free the slot of ``request_id``; returns that slot."""
        if request_id not in self._slot_of:
            raise RingError(UNKNOWN_REQUEST, f"request {request_id} is not resident")
        slot = self._slot_of.pop(request_id)
        self.owner[slot] = self.FREE
        self.length[slot] = 0
        return slot

    def shift_stages(self, n_stages: int) -> None:
        """The paper's physical InPlaceKVShift: the request of slot s moves to slot s + 1 for
        s = n_stages - 2 .. 0 (slot n_stages - 1 must be free), slot 0 is left free and the
        next new request takes it."""
        if n_stages < 2 or n_stages > self.n_slots:
            raise RingError(INVALID_ARG, "n_stages outside [2, n_slots]")
        if self.owner[n_stages - 1] != self.FREE:
            raise RingError(SLOT_BUSY, f"slot {n_stages - 1} still owned")
        for s in range(n_stages - 2, -1, -1):
            rid = self.owner[s]
            if rid == self.FREE:
                continue
            self.owner[s + 1], self.length[s + 1] = rid, self.length[s]
            self._slot_of[rid] = s + 1
            self.owner[s], self.length[s] = self.FREE, 0
        self.head = 0

    def slot_of(self, request_id: int) -> Optional[int]:
        return self._slot_of.get(request_id)

    def state(self):
        return list(self.owner), list(self.length), self.head
