"""Host bookkeeping of the compact draft memory (lengths and ring offsets only).

The device buffers of one draft layer are
    memory  [B, Hkv, mem_cap, d]  sinks first (rows 0..S-1), then memory slots
                                  in materialisation order (append-only);
    window  [B, Hkv, ring_cap, d] ring of raw-token K/V; raw position x >= S
                                  lives at ring row (x - S) % ring_cap.
Everything the kernels need -- memory length, ring start and length -- is a
pure function of the next raw position p to be processed, so eviction (the
window sliding past old tokens) and rollback after a rejected speculative
block (Sec. 3.3) are both just a change of p: evicted raw rows stay in the ring
until overwritten, which is the raw-KV rollback window (Sec. 4.1: 16 tokens).
The ring capacity must therefore cover the window, the speculative steps and
the rollback window.

Positions are 0-indexed.  Slot g_m (m >= 1) is named by the position of the
raw token after it, S + m*r (Sec. 3.2), and is materialised in the forward
pass of raw token S + m*r - 1.  With `slots_per_update` = u > 1 the slots of
u consecutive boundaries are materialised together, in the pass of the last
raw token of the u*r-token block (batched schedule).
"""
from dataclasses import dataclass
from typing import List, Optional


@dataclass
class DecodeView:
    mem_len: int     # memory rows attended (sinks + materialised slots)
    win_start: int   # ring row of the oldest attended raw token
    win_len: int     # raw tokens already in the ring and attended (the new one is appended)


@dataclass
class SlotUpdate:
    first_slot: int              # 1-based index m of the first slot materialised
    positions: List[int]         # position ids of the new slots (one per slot)
    mem_row: int                 # memory row of the first new slot


class MemoryLayout:
    def __init__(self, S: int, W: int, r: int, ring_cap: int, mem_cap: int, slots_per_update: int = 1):
        if W < 1 or r < 1 or S < 0 or slots_per_update < 1:
            raise ValueError("need W >= 1, r >= 1, S >= 0, slots_per_update >= 1")
        if ring_cap < W:
            raise ValueError("ring capacity must hold the window")
        self.S, self.W, self.r = S, W, r
        self.ring_cap, self.mem_cap = ring_cap, mem_cap
        self.u = slots_per_update

    # ---- slots ----
    def slot_position(self, m: int) -> int:
        return self.S + m * self.r

    def slots_materialised(self, p: int) -> int:
        """Slots in memory once raw positions 0..p-1 have been processed."""
        if p <= self.S:
            return 0
        blocks = (p - self.S) // (self.r * self.u)
        return blocks * self.u

    def update_in_pass_of(self, p: int) -> Optional[SlotUpdate]:
        """The slots materialised in the forward pass of raw position p, if any."""
        before, after = self.slots_materialised(p), self.slots_materialised(p + 1)
        if after == before:
            return None
        ms = list(range(before + 1, after + 1))
        return SlotUpdate(ms[0], [self.slot_position(m) for m in ms], self.S + before)

    # ---- the decode call for raw position p ----
    def decode_view(self, p: int) -> DecodeView:
        """Memory and ring state for the decode step of raw position p >= S
        (the step appends p to the ring)."""
        if p < self.S:
            raise ValueError("decode positions start after the sinks")
        mem_len = self.S + self.slots_materialised(p)
        if mem_len > self.mem_cap:
            raise ValueError("memory capacity exceeded")
        win_len = min(self.W - 1, p - self.S)
        start = (p - win_len - self.S) % self.ring_cap
        return DecodeView(mem_len, start, win_len)

    def ring_row(self, x: int) -> int:
        return (x - self.S) % self.ring_cap

    def slot_scope_view(self, m: int) -> DecodeView:
        """Write scope of slot m: sinks, slots 1..m (itself included) and the
        W raw tokens before its position id b_m, i.e. [max(S, b_m - W), b_m - 1]."""
        b = self.slot_position(m)
        win_len = min(self.W, b - self.S)
        start = (b - win_len - self.S) % self.ring_cap
        return DecodeView(self.S + m, start, win_len)

    def step_views(self, p: int):
        """Rows of one fused launch for raw position p (draft_step_attn): the raw
        query (mode 2: attends and appends the current token) and, when slots
        are materialised in this pass, one row per new slot's write scope.  A
        scope that ends at the current token stops one ring row short and
        attends the token from k_new (mode 1); older scopes have no new token
        (mode 0).  The memory update of the pass must run before the launch.
        Returns ([DecodeView, ...], [mode, ...])."""
        views, modes = [self.decode_view(p)], [2]
        upd = self.update_in_pass_of(p)
        if upd is not None:
            for i in range(len(upd.positions)):
                m = upd.first_slot + i
                v = self.slot_scope_view(m)
                if self.slot_position(m) - 1 == p:   # the scope ends at the current token
                    views.append(DecodeView(v.mem_len, v.win_start, v.win_len - 1))
                    modes.append(1)
                else:
                    views.append(v)
                    modes.append(0)
        return views, modes

    def rollback_ok(self, p_furthest: int, p_new: int) -> bool:
        """True if the ring still holds every raw row the window of p_new needs
        after speculative writes up to raw position p_furthest - 1."""
        need_lo = max(self.S, p_new - self.W + 1)
        return p_furthest - 1 - need_lo < self.ring_cap
