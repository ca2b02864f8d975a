"""Host-side checks of the expert-streaming tier: the record layout, the descriptor it
yields, and the LRU slot planner against a plain Python model of the documented rule."""
import ctypes

import numpy as np
import pytest

from paper_2608_08910_amd import tq


class ReferenceLRU:
    """The documented placement rule, written plainly: each step pins its resident
    experts; every other expert, in order of first appearance, takes an empty slot
    (lowest index) or else the slot whose last use is oldest among those the step does
    not use (lowest index on ties)."""

    def __init__(self, n_experts, n_slots):
        self.n_experts, self.n_slots = n_experts, n_slots
        self.slot_expert = [None] * n_slots
        self.last = [-1] * n_slots
        self.step = 0

    def map(self, ids):
        if any(e < 0 or e >= self.n_experts for e in ids):
            raise ValueError("id")
        if len(set(ids)) > self.n_slots:
            raise ValueError("capacity")
        self.step += 1
        where = {e: s for s, e in enumerate(self.slot_expert) if e is not None}
        for e in ids:
            if e in where:
                self.last[where[e]] = self.step
        misses = []
        for e in ids:
            if e in where:
                continue
            free = [s for s in range(self.n_slots) if self.slot_expert[s] is None]
            if free:
                s = free[0]
            else:
                cands = [s for s in range(self.n_slots) if self.last[s] < self.step]
                s = min(cands, key=lambda c: (self.last[c], c))
                del where[self.slot_expert[s]]
            self.slot_expert[s] = e
            self.last[s] = self.step
            where[e] = s
            misses.append((e, s))
        return [where[e] for e in ids], misses


def test_record_layout_and_descriptor():
    H, I = 4096, 2048
    rb = tq.tq_expert_record_bytes(H, I)
    assert rb == 3 * (I * H // 2 + I * (H // 256) * 2)  # every piece is already a multiple of 128
    assert tq.tq_expert_record_bytes(300, 2048) == 0 and tq.tq_expert_record_bytes(4096, 0) == 0
    base = 0x7F0000000000
    d = tq.tq_experts_from_records(base, 5, H, I)
    assert (d.n_experts, d.hidden, d.inter) == (5, H, I)
    offs = [d.gate_codes - base, d.up_codes - base, d.down_codes - base, d.gate_scales - base, d.up_scales - base,
            d.down_scales - base]
    sizes = [I * H // 2, I * H // 2, H * I // 2, I * (H // 256) * 2, I * (H // 256) * 2, H * (I // 256) * 2]
    assert offs[0] == 0 and all(o % 128 == 0 for o in offs)
    for (o1, s1), o2 in zip(zip(offs, sizes), offs[1:] + [rb]):
        assert o1 + s1 <= o2  # pieces in order, no overlap, inside the record
    assert list(d.stride_codes) == [rb] * 3 and list(d.stride_scales) == [rb // 2] * 3
    # a ragged shape: pieces padded to 128 bytes
    rb2 = tq.tq_expert_record_bytes(256, 768)
    assert rb2 % 128 == 0 and rb2 >= 3 * (256 * 768 // 2) + 3 * 256 * 3 * 2
    with pytest.raises(tq.TqError):
        tq.tq_experts_from_records(base + 64, 5, H, I)


@pytest.mark.parametrize("n_experts,n_slots,per_step,zipf", [(16, 4, 2, False), (64, 12, 8, True), (256, 64, 8, False),
                                                               (40, 40, 8, False), (9, 3, 3, True)])
def test_lru_matches_reference(n_experts, n_slots, per_step, zipf):
    rng = np.random.default_rng(n_experts * 31 + n_slots)
    c = tq.TqCache(n_experts, n_slots)
    ref = ReferenceLRU(n_experts, n_slots)
    p = None
    if zipf:
        p = (np.arange(1, n_experts + 1) ** -1.1)
        p /= p.sum()
    resident = {}
    for step in range(300):
        k = int(rng.integers(1, per_step + 1))
        ids = rng.choice(n_experts, size=k, p=p).astype(np.int32)  # duplicates allowed
        if len(set(ids.tolist())) > n_slots:
            continue
        slots, misses = c.map(ids)
        rs, rm = ref.map(ids.tolist())
        assert slots.tolist() == rs and [tuple(m) for m in misses.tolist()] == rm
        for e, s in rm:
            resident = {kk: v for kk, v in resident.items() if v != s}
            resident[e] = s
        # every id maps to the slot that holds it; each slot holds one expert
        assert all(resident[int(e)] == int(s) for e, s in zip(ids, slots))
        assert len(set(resident.values())) == len(resident) <= n_slots


def test_lru_rejections_leave_the_pool_unchanged():
    c = tq.TqCache(8, 2)
    ref = ReferenceLRU(8, 2)
    for ids in ([0, 1], [1]):
        assert c.map(ids)[0].tolist() == ref.map(ids)[0]
    for bad in ([2, 3, 4], [0, 9], [-1]):
        with pytest.raises(tq.TqError):
            c.map(bad)
    for ids in ([2], [0, 2], [3, 1]):  # behaves as if the failed calls never happened
        s, m = c.map(ids)
        rs, rm = ref.map(ids)
        assert s.tolist() == rs and [tuple(x) for x in m.tolist()] == rm
    s, m = c.map(np.zeros(0, np.int32))
    assert s.size == 0 and m.size == 0


def test_fetch_validates_before_enqueueing():
    L = tq._L
    c = tq.TqCache(8, 2)
    FAKE = 0x7F0000000000
    rb = tq.tq_expert_record_bytes(256, 256)
    st = c.state.ctypes.data
    bad_miss = np.array([[9, 0]], np.int32)  # expert outside the store
    slots = np.array([0], np.int32)
    assert L.tq_cache_fetch(st, FAKE, FAKE, rb, bad_miss.ctypes.data, 1, slots.ctypes.data, FAKE, 1, None) == tq.TQ_ERR_INVALID
    bad_slot = np.array([[1, 2]], np.int32)  # slot outside the pool
    assert L.tq_cache_fetch(st, FAKE, FAKE, rb, bad_slot.ctypes.data, 1, slots.ctypes.data, FAKE, 1, None) == tq.TQ_ERR_INVALID
    bad_ids = np.array([5], np.int32)
    assert L.tq_cache_fetch(st, FAKE, FAKE, rb, None, 0, bad_ids.ctypes.data, FAKE, 1, None) == tq.TQ_ERR_INVALID
    assert L.tq_cache_fetch(st, FAKE, FAKE, 100, None, 0, None, None, 0, None) == tq.TQ_ERR_INVALID  # record size
    junk = np.zeros(16, np.int64)
    assert L.tq_cache_fetch(junk.ctypes.data, FAKE, FAKE, rb, None, 0, None, None, 0, None) == tq.TQ_ERR_INVALID
