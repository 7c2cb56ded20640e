"""Pins of the visible-set simulator (oracle/masw_sets.py).

The closed forms in the simulator are checked against (a) a step-by-step
simulation of the paper's materialisation-and-eviction cycle, (b) the slot
naming in the paper's figure caption (tests/golden/masw_figure_slots.json) and
(c) the working-set size of Sec. 3.1 at the paper's settings
(tests/golden/masw_settings.json).
"""
import json
import os

import pytest

from oracle.masw_sets import MaswSets

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _cycle(S, W, r, n_tokens):
    """Step-by-step memory update cycle (Sec. 3.2): process raw tokens in
    order; count non-sink tokens since the last slot; when the count reaches r
    a slot is materialised and named by the position of the next raw token.
    Also track the raw window as an explicit list with eviction."""
    slots = []                 # (pass position, slot position id)
    since = 0
    window = []
    windows = {}
    for p in range(n_tokens):
        if p >= S:
            window.append(p)
            if len(window) > W:
                window.pop(0)  # evict the oldest raw token
            since += 1
        windows[p] = list(window)
        if since == r:
            slots.append((p, p + 1))
            since = 0
    return slots, windows


@pytest.mark.parametrize("S,W,r", [(0, 8, 4), (3, 5, 2), (128, 128, 4), (128, 128, 8), (0, 1024, 16)])
def test_closed_forms_match_stepwise_cycle(S, W, r):
    sets = MaswSets(S, W, r)
    n = S + 40 * r + 7
    slots, windows = _cycle(S, W, r, n)
    for m, (p_pass, pos_id) in enumerate(slots, start=1):
        assert sets.boundary(m) == pos_id
        assert sets.materialised_in_pass_of(p_pass) == m
    made = {p for p, _ in slots}
    for p in range(n):
        if p not in made:
            assert sets.materialised_in_pass_of(p) is None
        assert sets.slots_after(p + 1) == sum(1 for q, _ in slots if q <= p)
        if p >= S:
            view = sets.raw_view(p)
            assert view.window == windows[p]
            assert view.sink == list(range(S))
            # slots inserted before p are visible, the one made in p's own pass is not
            assert view.slots == [m for m, (q, pid) in enumerate(slots, 1) if pid <= p]


def test_figure_caption_slot_naming():
    g = _gold("masw_figure_slots.json")
    st = _gold("masw_settings.json")
    r = g["r"]
    a, b = g["slot_position_ids"]
    for S in (0, st["sink_count_S"]):
        sets = MaswSets(S, st["local_window_W"], r)
        m = (a - S) // r
        assert sets.boundary(m) == a and sets.boundary(m + 1) == b
        # decoding steps between the two materialisations
        pa = [p for p in range(a - 10, b + 10) if sets.materialised_in_pass_of(p) is not None]
        i = pa.index(a - 1)
        assert pa[i + 1] - pa[i] == g["decoding_steps_between"]


def test_working_set_size_at_paper_settings():
    st = _gold("masw_settings.json")
    S, W = st["sink_count_S"], st["local_window_W"]
    for r in st["nominal_compression_r"]:
        sets = MaswSets(S, W, r)
        for p in (S + W + 5, 8191, 16384, 32767, 32768):
            v = sets.raw_view(p)
            assert len(v.sink) == S and len(v.window) == W
            assert len(v.slots) == (p - S) // r
            assert v.size() == S + W + (p - S) // r
    # the nominal sizes quoted for a 32K prefix
    assert MaswSets(S, W, 4).raw_view(32768).size() == 8416
    assert MaswSets(S, W, 8).raw_view(32768).size() == 4336


def test_slot_scope():
    sets = MaswSets(4, 6, 3)
    sc = sets.slot_scope(5)                      # b_5 = 19
    assert sc.sink == [0, 1, 2, 3]
    assert sc.slots == [1, 2, 3, 4, 5]           # earlier slots and itself
    assert sc.window == [13, 14, 15, 16, 17, 18]  # the W raw tokens before b_m
    sc = sets.slot_scope(1)                      # b_1 = 7: window clipped at the sinks
    assert sc.window == [4, 5, 6]
    # the slot's raw scope equals the raw view of the token whose pass makes it
    for m in range(1, 20):
        b = sets.boundary(m)
        assert sets.slot_scope(m).window == sets.raw_view(b - 1).window
        assert sets.slot_scope(m).slots == sets.raw_view(b).slots


def _cycle_batched(S, W, r, u, n_tokens):
    """Step-by-step cycle of the batched schedule: count non-sink raw tokens;
    every r of them a boundary is passed (its slot is pending, named by the
    next raw position); after u boundaries the pending slots are made in the
    pass of the current token."""
    made = []       # (pass position, slot position id)
    pending = []
    since = 0
    for p in range(n_tokens):
        if p >= S:
            since += 1
        if since == r:
            pending.append(p + 1)
            since = 0
            if len(pending) == u:
                made += [(p, pid) for pid in pending]
                pending = []
    return made


@pytest.mark.parametrize("S,W,r,u", [(0, 8, 4, 2), (3, 5, 2, 3), (0, 1024, 16, 4), (128, 128, 4, 4)])
def test_batched_schedule_matches_stepwise_cycle(S, W, r, u):
    sets = MaswSets(S, W, r, u)
    n = S + 30 * r * u + 5
    made = _cycle_batched(S, W, r, u, n)
    for m, (p_pass, pos_id) in enumerate(made, start=1):
        assert sets.boundary(m) == pos_id
        assert m in sets.slots_made_in_pass_of(p_pass)
    per_boundary = MaswSets(S, W, r)
    for p in range(S, n):
        view = sets.raw_view(p)
        assert view.slots == [m for m, (q, _) in enumerate(made, 1) if q < p]
        # never ahead of the per-boundary schedule, at most u - 1 slots behind it,
        # and level with it right after every batch
        lag = len(per_boundary.raw_view(p).slots) - len(view.slots)
        assert 0 <= lag <= u - 1
        if (p - S) % (r * u) == 0:
            assert lag == 0
        assert view.window == per_boundary.raw_view(p).window
        assert sets.slot_scope(1 + p % 7) == per_boundary.slot_scope(1 + p % 7)
