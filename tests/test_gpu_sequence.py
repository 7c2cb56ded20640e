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

from parity import abs_score_batched, check_lse, check_out, to_np

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
        o, lse = oracle.attend_batched(q.double().numpy(), K, V, np.array([K.shape[2]]), scale)
        return o, lse, abs_score_batched(q.double().numpy(), K, [K.shape[2]], scale)

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
        o_ref, lse_ref, a_ref = oracle_attend(q, sv.sink, sv.slots, sv.window)
        check_out(to_np(out), o_ref, bf, f"step {p} out")
        check_lse(to_np(lse), lse_ref, a_ref, d, f"step {p} lse")

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
            o_ref, lse_ref, a_ref = oracle_attend(qg, sc.sink, sc.slots, sc.window)
            check_out(to_np(out), o_ref, bf, f"slot {m} scope out")
            check_lse(to_np(lse), lse_ref, a_ref, d, f"slot {m} scope lse")
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


def test_batched_sixteen_ragged_sequences_staggered_updates():
    """Batched drafting with continuous memory updates: 16 sequences with
    ragged prefixes drawn in [8192, 32768), 32/8 heads, d 64, bf16, slot
    interval 16 and 4 slots per update (one update per 64-token block), a
    512-token window.  Every draft token is one decode launch for all 16
    sequences (per-sequence memory lengths and ring offsets); after it, one
    memory-update launch for the batch with fire[b] set for the sequences
    whose block ended (staggered by the prefix).  512 tokens per sequence
    (128 rounds of gamma = 4, the batched drafting workload's length): every
    sequence crosses eight boundaries.  Checked against the oracle: every
    16th token's outputs for all sequences, the token after each sequence's
    update (it reads the new slots), and every materialised slot row."""
    import oracle
    from oracle.masw_sets import MaswSets
    import paper_2608_30252_amd as mad
    from paper_2608_30252_amd import synth
    from paper_2608_30252_amd.state import MemoryLayout

    dev = torch.device("cuda")
    dtype = torch.bfloat16
    B, Hq, Hkv, d, S, W, r, u, N = 16, 32, 8, 64, 0, 512, 16, 4, 512
    D = Hq * d
    scale = d ** -0.5
    P = np.random.default_rng(44).integers(8192, 32768, B).tolist()
    sets = MaswSets(S, W, r, u)
    mcap = max(sets.slots_after(p + N) for p in P) + 8
    lay = MemoryLayout(S, W, r, ring_cap=600, mem_cap=mcap, slots_per_update=u)

    # oracle state: slot m of sequence b at o_slot[b][:, m - 1]; raw position x at o_raw[b][:, x - base[b]]
    base = [p - W for p in P]
    o_slot_k = np.zeros((B, Hkv, mcap, d)); o_slot_v = np.zeros_like(o_slot_k)
    o_raw_k = np.zeros((B, Hkv, W + N, d)); o_raw_v = np.zeros_like(o_raw_k)
    mem_k = torch.zeros(B, Hkv, mcap, d, dtype=dtype); mem_v = torch.zeros_like(mem_k)
    ring_k = torch.zeros(B, Hkv, lay.ring_cap, d, dtype=dtype); ring_v = torch.zeros_like(ring_k)
    for b in range(B):
        n0 = sets.slots_after(P[b])
        sk, sv = synth.normal((Hkv, n0, d), 71_000 + b), synth.normal((Hkv, n0, d), 72_000 + b)
        mem_k[b, :, :n0], mem_v[b, :, :n0] = sk, sv
        o_slot_k[b, :, :n0], o_slot_v[b, :, :n0] = sk.double().numpy(), sv.double().numpy()
        rk, rv = synth.normal((Hkv, W, d), 73_000 + b), synth.normal((Hkv, W, d), 74_000 + b)
        o_raw_k[b, :, :W], o_raw_v[b, :, :W] = rk.double().numpy(), rv.double().numpy()
        rows = [lay.ring_row(x) for x in range(base[b], P[b])]
        ring_k[b][:, rows], ring_v[b][:, rows] = rk, rv
    g_mk, g_mv, g_rk, g_rv = (t.to(dev) for t in (mem_k, mem_v, ring_k, ring_v))
    w_g = synth.normal((2 * Hkv * d, D), 75_000, std=0.02)
    g_w = w_g.to(dev)

    def stored(a):
        return torch.from_numpy(a).to(dtype).double().numpy()

    updated, updated_at, checked_after, expected_after = set(), {}, 0, 0
    for t in range(N):
        pos = [p + t for p in P]
        views = [lay.decode_view(p) for p in pos]
        q = synth.normal((B, Hq, d), 76_000 + t)
        kn, vn = synth.normal((B, Hkv, d), 77_000 + t), synth.normal((B, Hkv, d), 78_000 + t)
        for b in range(B):
            o_raw_k[b, :, pos[b] - base[b]] = kn[b].double().numpy()
            o_raw_v[b, :, pos[b] - base[b]] = vn[b].double().numpy()
        out, lse = mad.draft_decode_attn(q.to(dev), mad.KV(g_mk, g_mv, [v.mem_len for v in views]),
                                         mad.KV(g_rk, g_rv, [v.win_len for v in views], [v.win_start for v in views]),
                                         kn.to(dev), vn.to(dev), scale=scale)
        after_update = [b for b in range(B) if pos[b] - 1 in updated_at.get(b, ())]
        rows = list(range(B)) if t % 16 == 15 else after_update
        if rows:
            n = np.zeros(len(rows), dtype=np.int64)
            nmax = max(sets.raw_view(pos[b]).size() for b in rows)
            K = np.zeros((len(rows), Hkv, nmax, d)); V = np.zeros_like(K)
            for j, b in enumerate(rows):
                rv_ = sets.raw_view(pos[b])
                ns = len(rv_.slots)
                K[j, :, :ns], V[j, :, :ns] = o_slot_k[b, :, :ns], o_slot_v[b, :, :ns]
                win = np.array(rv_.window) - base[b]
                K[j, :, ns:ns + len(win)], V[j, :, ns:ns + len(win)] = o_raw_k[b][:, win], o_raw_v[b][:, win]
                n[j] = ns + len(win)
            o_ref, lse_ref = oracle.attend_batched(q[rows].double().numpy(), K, V, n, scale)
            a_ref = abs_score_batched(q[rows].double().numpy(), K, n, scale)
            for j, b in enumerate(rows):
                check_out(to_np(out[b:b + 1]), o_ref[j:j + 1], True, f"token {t} seq {b} out")
                check_lse(to_np(lse[b:b + 1]), lse_ref[j:j + 1], a_ref[j:j + 1], d, f"token {t} seq {b} lse")
            checked_after += len(after_update)

        # one update launch for the batch: the sequences whose 64-token block ends at this token
        upds = [lay.update_in_pass_of(p) for p in pos]
        fire = [1 if x is not None else 0 for x in upds]
        if not any(fire):
            continue
        x = synth.normal((B, u, D), 79_000 + t)
        posl = [x_.positions if x_ is not None else [0] * u for x_ in upds]
        mlen = [x_.mem_row if x_ is not None else views[b].mem_len for b, x_ in enumerate(upds)]
        mad.memory_update(x.to(dev), g_w, posl, mad.KV(g_mk, g_mv, mlen), fire=fire, rope_base=BASE)
        for b, x_ in enumerate(upds):
            if x_ is None:
                continue
            k_ref, v_ref = oracle.memory_update(x[b].double().numpy(), w_g.double().numpy(),
                                                np.array(x_.positions), Hkv, d, BASE)
            for i in range(u):
                m = x_.first_slot + i
                o_slot_k[b, :, m - 1], o_slot_v[b, :, m - 1] = stored(k_ref[i]), stored(v_ref[i])
                check_out(to_np(g_mk[b, :, x_.mem_row + i]), k_ref[i], True, f"seq {b} slot {m} k")
                check_out(to_np(g_mv[b, :, x_.mem_row + i]), v_ref[i], True, f"seq {b} slot {m} v")
            updated.add(b)
            updated_at.setdefault(b, set()).add(pos[b])
            expected_after += t < N - 1
    torch.cuda.synchronize()
    assert updated == set(range(B))       # every sequence crossed a boundary
    assert checked_after == expected_after > 0   # the token after each update read the new slots
