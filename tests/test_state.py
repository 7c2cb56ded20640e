"""Host bookkeeping (paper_2608_30252_amd/state.py) against the paper's set
definitions (oracle/masw_sets.py), on an emulated ring and memory that hold
position tags instead of K/V: random decode schedules with speculative
blocks and rollbacks."""
import numpy as np
import pytest

from oracle.masw_sets import MaswSets
from paper_2608_30252_amd.state import MemoryLayout


class Emu:
    """Tags written where the decode kernel writes K/V."""

    def __init__(self, lay, prefix):
        self.lay = lay
        self.ring = [None] * lay.ring_cap
        self.mem = [("sink", i) for i in range(lay.S)]
        # prefill: raw tokens of the prefix in the ring, slots of the prefix in memory
        for x in range(lay.S, prefix):
            self.ring[lay.ring_row(x)] = x
        for m in range(1, lay.slots_materialised(prefix) + 1):
            self.mem.append(("slot", m))

    def step(self, p):
        lay = self.lay
        v = lay.decode_view(p)
        mem = self.mem[: v.mem_len]
        win = [self.ring[(v.win_start + i) % lay.ring_cap] for i in range(v.win_len)]
        self.ring[(v.win_start + v.win_len) % lay.ring_cap] = p      # the kernel's append
        upd = lay.update_in_pass_of(p)
        if upd is not None:
            del self.mem[upd.mem_row:]                                  # slots past a rollback
            for k, pos in enumerate(upd.positions):
                self.mem.append(("slot", upd.first_slot + k))
                assert pos == lay.slot_position(upd.first_slot + k)
        return mem, win + [p]

    def scope(self, m):
        lay = self.lay
        v = lay.slot_scope_view(m)
        return self.mem[: v.mem_len], [self.ring[(v.win_start + i) % lay.ring_cap] for i in range(v.win_len)]


def _expected(sets, p):
    view = sets.raw_view(p)
    return [("sink", i) for i in view.sink] + [("slot", m) for m in view.slots], view.window


@pytest.mark.parametrize("S,W,r,gamma", [(0, 128, 16, 4), (128, 128, 4, 5), (128, 128, 8, 5), (3, 7, 2, 3),
                                         (0, 1, 1, 2), (5, 16, 16, 4)])
def test_views_match_paper_sets_with_rollbacks(S, W, r, gamma):
    R = 16
    lay = MemoryLayout(S, W, r, ring_cap=W + gamma + R, mem_cap=100000)
    sets = MaswSets(S, W, r)
    rng = np.random.default_rng(S * 100 + W + r)
    prefix = S + 3 * W + 11
    emu = Emu(lay, prefix)
    p = prefix
    for it in range(200):
        p0 = p
        for i in range(gamma):                           # speculative draft steps
            mem, win = emu.step(p0 + i)
            exp_mem, exp_win = _expected(sets, p0 + i)
            assert mem == exp_mem and win == exp_win, (it, p0 + i)
            upd = lay.update_in_pass_of(p0 + i)
            if upd is not None:
                m = upd.first_slot
                s_mem, s_win = emu.scope(m)
                sc = sets.slot_scope(m)
                assert s_mem == [("sink", i) for i in sc.sink] + [("slot", k) for k in sc.slots]
                assert s_win == sc.window
        a = int(rng.integers(0, gamma + 1))              # accepted drafted tokens
        p_new = p0 + min(a, gamma - 1) + 1
        assert lay.rollback_ok(p0 + gamma, p_new)
        emu.mem = emu.mem[: S + lay.slots_materialised(p_new)]   # drop slots made after the last accepted position
        p = p_new


def test_batched_schedule_materialises_blocks():
    lay = MemoryLayout(0, 512, 16, ring_cap=512 + 64 + 64, mem_cap=4096, slots_per_update=4)
    assert lay.update_in_pass_of(62) is None
    u = lay.update_in_pass_of(63)
    assert u.first_slot == 1 and u.positions == [16, 32, 48, 64] and u.mem_row == 0
    assert lay.slots_materialised(64) == 4 and lay.slots_materialised(127) == 4 and lay.slots_materialised(128) == 8
    # 32K prefix: 2048 slots, window of 1024 with 1023 rows before the new token
    lay = MemoryLayout(0, 1024, 16, ring_cap=1024 + 64 + 64, mem_cap=4096, slots_per_update=4)
    v = lay.decode_view(32768)
    assert v.mem_len == 2048 and v.win_len == 1023


def test_rollback_needs_ring_capacity():
    # 5 speculative steps from position 1000 write rows up to 1004; rolling back to
    # 1001 needs rows 874..1000, and with a ring of exactly W rows 1004 overwrote 876
    lay = MemoryLayout(0, 128, 16, ring_cap=128, mem_cap=1000)
    assert not lay.rollback_ok(1000 + 5, 1001)
    lay = MemoryLayout(0, 128, 16, ring_cap=128 + 5 - 2, mem_cap=1000)
    assert lay.rollback_ok(1000 + 5, 1001)
    lay = MemoryLayout(0, 128, 16, ring_cap=128 + 5 + 16, mem_cap=1000)
    assert lay.rollback_ok(1000 + 5, 1001)


@pytest.mark.parametrize("S,W,r,u", [(0, 1024, 16, 4), (128, 128, 4, 1), (3, 7, 2, 3), (0, 8, 16, 1), (5, 40, 3, 2)])
def test_step_views_match_paper_sets(S, W, r, u):
    """The rows of a fused boundary launch: the raw view of p (mode 2) and
    every new slot's write scope, with the current token taken from k_new
    (mode 1) exactly when the scope ends at p."""
    sets = MaswSets(S, W, r, u)
    lay = MemoryLayout(S, W, r, ring_cap=W + r * u + 24, mem_cap=S + 4096, slots_per_update=u)
    prefix = S + 3 * r * u + 1
    emu = Emu(lay, prefix)
    checked = 0
    for p in range(prefix, prefix + 6 * r * u):
        upd = lay.update_in_pass_of(p)
        views, modes = (lay.step_views(p) if upd is not None else ([lay.decode_view(p)], [2]))
        mem_seen, win_seen = emu.step(p)   # appends p and materialises the pass's slots
        exp_mem, exp_win = _expected(sets, p)
        assert modes[0] == 2 and mem_seen == exp_mem and win_seen == exp_win
        if upd is None:
            continue
        assert len(views) == 1 + len(upd.positions)
        for i, (v, mode) in enumerate(zip(views[1:], modes[1:])):
            m = upd.first_slot + i
            sv = sets.slot_scope(m)
            mem = emu.mem[: v.mem_len]
            win = [emu.ring[(v.win_start + t) % lay.ring_cap] for t in range(v.win_len)]
            if mode == 1:
                win = win + [p]
            assert mode in (0, 1) and (mode == 1) == (sv.window and sv.window[-1] == p)
            assert mem == [("sink", j) for j in sv.sink] + [("slot", j) for j in sv.slots], (p, m)
            assert win == sv.window, (p, m)
            checked += 1
    assert checked >= 6
