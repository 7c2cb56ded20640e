"""Host-side arithmetic of the benchmark (no GPU): the algorithmic counts it
divides by must match the paper's visible sets."""
import pytest

import bench
from oracle.masw_sets import MaswSets


@pytest.mark.parametrize("P,S,W,r,u", [(1000, 0, 128, 16, 4), (900, 128, 128, 4, 1), (4, 6, 5, 2, 1),
                                       (513, 0, 8, 16, 1), (700, 3, 100, 7, 2)])
def test_prefill_flops_count_every_visible_key(P, S, W, r, u):
    sets = MaswSets(S, W, r, u)
    keys = sum(sets.raw_view(p).size() for p in range(P))
    keys += sum(sets.slot_scope(m).size() for m in range(1, sets.slots_after(P) + 1))
    assert bench.prefill_flops(P, S, W, r, u, 3, 8) == keys * 3 * 8 * 4


def test_kv_bytes_of_the_32k_compact_layer():
    # 2048 slots + 1023 window tokens + the new token, 8 KV heads, d 64, K and V, bf16
    assert bench.kv_bytes(3072, 8, 64) == 6291456
