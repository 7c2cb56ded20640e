"""Multi-step MASW decode on the GPU against the oracle on the paper's sets.

Each step runs the draft decode attention for the next raw position (its K/V
appended to the window ring in the same call), and at compression boundaries
the memory update (mirrored projection + RoPE + append) followed by the new
slot's write-scope attention.  The GPU state is driven by the host layout
(paper_2608_30252_amd.state); the oracle builds every key list from the set
definitions (oracle.masw_sets) and keeps its own fp64 K/V for the slots it
materialises (rounded to the storage dtype, as the memory holds them) --
nothing on the oracle side comes from the GPU.
"""
import numpy as np
import pytest
import torch

from parity import check, check_out, to_np, F32_ATOL

pytestmark = pytest.mark.gpu

BASE = 500000.0


def _run_sequence(dtype, Hq, Hkv, d, S, W, r, prefix, steps, seed):
    import oracle
    from oracle.masw_sets import MaswSets
    import paper_2608_30252_amd as mad
    from paper_2608_30252_amd import synth
    from paper_2608_30252_amd.state import MemoryLayout

    dev = torch.device("cuda")
    gamma, R = 4, 16
    D = Hq * d
    sets = MaswSets(S, W, r)
    n_slots_end = sets.slots_after(prefix + steps)
    lay = MemoryLayout(S, W, r, ring_cap=W + gamma + R, mem_cap=S + n_slots_end + 8)
    bf = dtype == torch.bfloat16
    scale = d ** -0.5

    def raw_kv(x):      # seeded stand-ins for the raw tokens' K/V
        return synth.normal((Hkv, d), 10_000_000 * seed + 2 * x, dtype=dtype), \
               synth.normal((Hkv, d), 10_000_000 * seed + 2 * x + 1, dtype=dtype)

    # oracle-side memory: sinks and prefix slots are seeded stand-ins (prefill is
    # outside the decode path); slots materialised below come from the oracle
    o_sink, o_slot = {}, {}
    mem_k = torch.zeros(1, Hkv, lay.mem_cap, d, dtype=dtype)
    mem_v = torch.zeros_like(mem_k)
    for i in range(S):
        k, v = raw_kv(i)
        o_sink[i] = (k.double().numpy(), v.double().numpy())
        mem_k[0, :, i], mem_v[0, :, i] = k, v
    for m in range(1, sets.slots_after(prefix) + 1):
        k = synth.normal((Hkv, d), 7_000_000 * seed + 2 * m, dtype=dtype)
        v = synth.normal((Hkv, d), 7_000_000 * seed + 2 * m + 1, dtype=dtype)
        o_slot[m] = (k.double().numpy(), v.double().numpy())
        mem_k[0, :, S + m - 1], mem_v[0, :, S + m - 1] = k, v
    ring_k = torch.zeros(1, Hkv, lay.ring_cap, d, dtype=dtype)
    ring_v = torch.zeros_like(ring_k)
    o_raw = {}
    for x in range(max(S, prefix - W), prefix):
        k, v = raw_kv(x)
        o_raw[x] = (k.double().numpy(), v.double().numpy())
        ring_k[0, :, lay.ring_row(x)], ring_v[0, :, lay.ring_row(x)] = k, v
    g_mk, g_mv, g_rk, g_rv = (t.to(dev) for t in (mem_k, mem_v, ring_k, ring_v))
    w_g = synth.normal((2 * Hkv * d, D), 900 + seed, std=0.02, dtype=dtype)
    g_w = w_g.to(dev)

    def oracle_attend(q, sink_ids, slot_ids, raw_ids):
        ks = [o_sink[i][0] for i in sink_ids] + [o_slot[m][0] for m in slot_ids] + [o_raw[x][0] for x in raw_ids]
        vs = [o_sink[i][1] for i in sink_ids] + [o_slot[m][1] for m in slot_ids] + [o_raw[x][1] for x in raw_ids]
        K = np.stack(ks, axis=1)[None]   # [1, Hkv, n, d]
        V = np.stack(vs, axis=1)[None]
        return oracle.attend_batched(q.double().numpy(), K, V, np.array([K.shape[2]]), scale)

    n_updates = 0
    for p in range(prefix, prefix + steps):
        view = lay.decode_view(p)
        q = synth.normal((1, Hq, d), 5_000_000 * seed + p, dtype=dtype)
        k_new, v_new = raw_kv(p)
        o_raw[p] = (k_new.double().numpy(), v_new.double().numpy())
        out, lse = mad.draft_decode_attn(q.to(dev), mad.KV(g_mk, g_mv, [view.mem_len]),
                                         mad.KV(g_rk, g_rv, [view.win_len], [view.win_start]),
                                         k_new[None].to(dev), v_new[None].to(dev), scale=scale)
        sv = sets.raw_view(p)
        o_ref, lse_ref = oracle_attend(q, sv.sink, sv.slots, sv.window)
        check_out(to_np(out), o_ref, bf, f"step {p} out")
        check(to_np(lse), lse_ref, F32_ATOL, None, f"step {p} lse")

        upd = lay.update_in_pass_of(p)
        if upd is None:
            continue
        n_updates += 1
        n_new = len(upd.positions)
        x = synth.normal((1, n_new, D), 3_000_000 * seed + p, dtype=dtype)
        mad.memory_update(x.to(dev), g_w, [upd.positions], mad.KV(g_mk, g_mv, [upd.mem_row]), rope_base=BASE)
        k_ref, v_ref = oracle.memory_update(x[0].double().numpy(), w_g.double().numpy(),
                                            np.array(upd.positions), Hkv, d, BASE)
        # the memory stores K/V in the layer's dtype: later attention reads the
        # oracle's own slot values rounded (RNE) to that dtype
        def stored(a):
            return torch.from_numpy(a).to(dtype).double().numpy()
        for i in range(n_new):
            m = upd.first_slot + i
            o_slot[m] = (stored(k_ref[i]), stored(v_ref[i]))
            row = upd.mem_row + i
            check_out(to_np(g_mk[0, :, row]), k_ref[i], bf, f"slot {m} k")
            check_out(to_np(g_mv[0, :, row]), v_ref[i], bf, f"slot {m} v")
            # the slot's write-scope attention (same kernel, no new token)
            sview = lay.slot_scope_view(m)
            qg = synth.normal((1, Hq, d), 4_000_000 * seed + m, dtype=dtype)
            out, lse = mad.draft_decode_attn(qg.to(dev), mad.KV(g_mk, g_mv, [sview.mem_len]),
                                             mad.KV(g_rk, g_rv, [sview.win_len], [sview.win_start]), scale=scale)
            sc = sets.slot_scope(m)
            o_ref, lse_ref = oracle_attend(qg, sc.sink, sc.slots, sc.window)
            check_out(to_np(out), o_ref, bf, f"slot {m} scope out")
            check(to_np(lse), lse_ref, F32_ATOL, None, f"slot {m} scope lse")
    torch.cuda.synchronize()
    return n_updates


def test_tiny_fp32_sixteen_steps():
    # 4/1 heads, d64: prefix 1024 -> 64 slots + a 128-token window; slot 65 (position id 1040)
    # is materialised in the pass of raw token 1039
    n = _run_sequence(torch.float32, 4, 1, 64, S=0, W=128, r=16, prefix=1024, steps=16, seed=1)
    assert n == 1


def test_draft_8k_bf16_64_steps_per_boundary():
    n = _run_sequence(torch.bfloat16, 32, 8, 64, S=0, W=512, r=16, prefix=8192, steps=64, seed=2)
    assert n == 4


def test_paper_setting_sinks_r4_bf16():
    # S = W = 128 and r = 4 (the paper's configuration) at a short prefix
    n = _run_sequence(torch.bfloat16, 32, 8, 64, S=128, W=128, r=4, prefix=2048, steps=12, seed=3)
    assert n == 3
