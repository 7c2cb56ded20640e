"""Visible-set simulator for MASW drafting -- TEST INFRASTRUCTURE ONLY.

Written from the paper's set definitions, independent of any ring buffer or
storage layout.  Positions are 0-indexed here; the paper's 1-indexed raw
position i is position i - 1 below.

Definitions (Sec. 3.1, Eq. three_part_memory and the local-window set;
Sec. 3.2, memory materialisation and the memory update cycle):

* Sink: the first S raw positions, [0, S), kept for the whole run.
* Slot interval r; compression boundary tau_m = m * r counted after the sinks,
  m = 1, 2, ...  The slot token g_m is inserted before the raw token at
  position b_m = S + m * r and shares that token's position id (a duplicated
  id; raw positions are not shifted).
* Local window of a raw query at position p: the exact raw tokens
  [max(S, p - W + 1), p] (the W most recent non-sink tokens, p included).
* A raw query at position p sees: the sinks, every slot g_m with b_m <= p
  (slots inserted before it), and its local window.
* The write scope of slot g_m: the sinks, the earlier slots g_1..g_{m-1},
  itself, and the local window at its boundary, i.e. the W raw tokens before
  b_m: [max(S, b_m - W), b_m - 1].
* Reading adopted where the paper is silent: g_m is materialised in the same
  forward pass as raw token b_m - 1 (the last token of its unit), as an extra
  position after it, so after t raw tokens have been processed there are
  floor((t - S) / r) slots (t >= S) -- the working-set count floor(t/r) of
  Sec. 3.1 with sinks excluded.
* Rollback (Sec. 3.3): a state rolled back to t processed tokens is the state
  after t tokens; slots materialised in passes of positions >= t are dropped.
* Batched schedule (reading adopted for "compressing each evicted 64-token
  block"): with u slots per update, the slots of u consecutive boundaries are
  materialised together in the pass of the block's last raw token
  S + k*u*r - 1, as extra positions after it; a raw query sees a slot only
  once it is materialised.  A slot's write scope is unchanged (it is defined
  by the slot's position id).  u = 1 is the per-boundary schedule above.
"""
from dataclasses import dataclass, field
from typing import List


@dataclass
class View:
    """A visible set: sink positions, slot indices (1-based m) and window positions."""
    sink: List[int] = field(default_factory=list)
    slots: List[int] = field(default_factory=list)
    window: List[int] = field(default_factory=list)

    def size(self):
        return len(self.sink) + len(self.slots) + len(self.window)


class MaswSets:
    def __init__(self, S: int, W: int, r: int, u: int = 1):
        assert S >= 0 and W >= 1 and r >= 1 and u >= 1
        self.S, self.W, self.r, self.u = S, W, r, u

    def boundary(self, m: int) -> int:
        """Position id b_m of slot g_m (m >= 1)."""
        assert m >= 1
        return self.S + m * self.r

    def slots_after(self, t: int) -> int:
        """Number of slots materialised once raw positions 0..t-1 are processed."""
        if t <= self.S:
            return 0
        return (t - self.S) // (self.r * self.u) * self.u

    def slots_made_in_pass_of(self, p: int) -> List[int]:
        """Slot indices m materialised in the forward pass of raw position p."""
        return list(range(self.slots_after(p) + 1, self.slots_after(p + 1) + 1))

    def materialised_in_pass_of(self, p: int):
        """Per-boundary schedule: the slot index m made in the pass of p, or None."""
        made = self.slots_made_in_pass_of(p)
        return made[-1] if made else None

    def raw_view(self, p: int) -> View:
        """What the raw query at position p attends to."""
        sink = list(range(0, min(self.S, p + 1)))
        # slots made in passes of earlier positions (a slot made in p's own pass
        # sits after p; the same holds under the batched schedule)
        slots = list(range(1, self.slots_after(p) + 1))
        lo = max(self.S, p - self.W + 1)
        window = list(range(lo, p + 1)) if p >= self.S else []
        return View(sink, slots, window)

    def slot_scope(self, m: int) -> View:
        """Write scope of slot g_m."""
        b = self.boundary(m)
        sink = list(range(0, self.S))
        slots = list(range(1, m + 1))
        window = list(range(max(self.S, b - self.W), b))
        return View(sink, slots, window)
