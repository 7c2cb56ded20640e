"""The fused boundary step (mad_draft_step_attn) against the oracle.

At a raw position p whose pass materialises memory slots, the memory update
runs first and then ONE launch serves the raw query and every new slot's
write-scope query, all rows aliasing one sequence's buffers:
  row 0      raw query of p: sinks + slots materialised before p + the window
             ending at p (mode 2: the current token is attended and appended);
  row 1 + i  slot m = first + i: sinks + slots 1..m + the W raw tokens before
             its position id (mode 1 for the scope that ends at p, else 0).
The oracle builds every key list from the paper's set definitions
(oracle.masw_sets), with the slots' K/V from its own memory update (rounded to
the stored dtype).  The ring must gain exactly the current token's row.
"""
import numpy as np
import pytest
import torch

from parity import abs_score_batched, check_lse, check_out, to_np

pytestmark = pytest.mark.gpu

BASE = 500000.0


def _fused_boundary(dtype, Hq, Hkv, d, S, W, r, u, prefix, seed):
    import oracle
    from oracle.masw_sets import MaswSets
    import paper_2608_30252_amd as mad
    from paper_2608_30252_amd import synth
    from paper_2608_30252_amd.state import MemoryLayout

    dev = torch.device("cuda")
    D = Hq * d
    lay = MemoryLayout(S, W, r, ring_cap=(W + r * u + 20 + 7) // 8 * 8, mem_cap=S + prefix // r + 64,
                       slots_per_update=u)
    sets = MaswSets(S, W, r, u)
    # the first raw position at or after the prefix whose pass materialises slots
    p = next(x for x in range(prefix, prefix + r * u + 1) if lay.update_in_pass_of(x) is not None)
    upd = lay.update_in_pass_of(p)
    bf = dtype == torch.bfloat16
    scale = d ** -0.5

    def raw_kv(x):
        return (synth.normal((Hkv, d), 10_000_000 * seed + 2 * x, dtype=dtype),
                synth.normal((Hkv, d), 10_000_000 * seed + 2 * x + 1, dtype=dtype))

    keys = {}   # ("sink", i) / ("slot", m) / ("raw", x) -> (k [Hkv, d], v [Hkv, d]) as fp64
    mem_k = torch.zeros(1, Hkv, lay.mem_cap, d, dtype=dtype)
    mem_v = torch.zeros_like(mem_k)
    for i in range(S):
        k, v = raw_kv(i)
        keys["sink", i] = (k.double().numpy(), v.double().numpy())
        mem_k[0, :, i], mem_v[0, :, i] = k, v
    for m in range(1, lay.slots_materialised(p) + 1):
        k = synth.normal((Hkv, d), 7_000_000 * seed + 2 * m, dtype=dtype)
        v = synth.normal((Hkv, d), 7_000_000 * seed + 2 * m + 1, dtype=dtype)
        keys["slot", m] = (k.double().numpy(), v.double().numpy())
        mem_k[0, :, S + m - 1], mem_v[0, :, S + m - 1] = k, v
    ring_k = torch.zeros(1, Hkv, lay.ring_cap, d, dtype=dtype)
    ring_v = torch.zeros_like(ring_k)
    for x in range(max(S, p - W - r * u), p):
        k, v = raw_kv(x)
        keys["raw", x] = (k.double().numpy(), v.double().numpy())
        ring_k[0, :, lay.ring_row(x)], ring_v[0, :, lay.ring_row(x)] = k, v
    k_new, v_new = raw_kv(p)
    keys["raw", p] = (k_new.double().numpy(), v_new.double().numpy())
    g_mk, g_mv, g_rk, g_rv = (t.to(dev) for t in (mem_k, mem_v, ring_k, ring_v))
    ring_before = g_rk.clone()

    # the pass's memory update (oracle: its own slot K/V, rounded to the stored dtype)
    n_new = len(upd.positions)
    w_g = synth.normal((2 * Hkv * d, D), 900 + seed, std=0.02, dtype=dtype)
    x = synth.normal((1, n_new, D), 3_000_000 * seed + p, dtype=dtype)
    mad.memory_update(x.to(dev), w_g.to(dev), [upd.positions], mad.KV(g_mk, g_mv, [upd.mem_row]), rope_base=BASE)
    k_ref, v_ref = oracle.memory_update(x[0].double().numpy(), w_g.double().numpy(), np.array(upd.positions),
                                        Hkv, d, BASE)
    stored = lambda a: torch.from_numpy(a).to(dtype).double().numpy()
    for i in range(n_new):
        keys["slot", upd.first_slot + i] = (stored(k_ref[i]), stored(v_ref[i]))

    # one launch: raw row + the new slots' write scopes
    views, modes = lay.step_views(p)
    R = len(views)
    assert R == 1 + n_new and modes[0] == 2 and modes.count(1) == 1
    q = synth.normal((R, Hq, d), 5_000_000 * seed + p, dtype=dtype)
    kn = torch.stack([k_new] * R)
    vn = torch.stack([v_new] * R)
    out, lse = mad.draft_step_attn(q.to(dev), mad.KV(g_mk, g_mv, [v.mem_len for v in views]),
                                   mad.KV(g_rk, g_rv, [v.win_len for v in views], [v.win_start for v in views]),
                                   kn.to(dev), vn.to(dev), modes)
    torch.cuda.synchronize()

    def oracle_attend(qrows, sv):
        ids = [("sink", i) for i in sv.sink] + [("slot", m) for m in sv.slots] + [("raw", x) for x in sv.window]
        K = np.stack([keys[k][0] for k in ids], axis=1)[None]
        V = np.stack([keys[k][1] for k in ids], axis=1)[None]
        o, lse = oracle.attend_batched(qrows.double().numpy()[None], K, V, np.array([K.shape[2]]), scale)
        return o, lse, abs_score_batched(qrows.double().numpy()[None], K, [K.shape[2]], scale)

    scopes = [sets.raw_view(p)] + [sets.slot_scope(upd.first_slot + i) for i in range(n_new)]
    for row, sv in enumerate(scopes):
        o_ref, l_ref, a_ref = oracle_attend(q[row], sv)
        check_out(to_np(out[row]), o_ref[0], bf, f"row {row} out")
        check_lse(to_np(lse[row]), l_ref[0], a_ref[0], d, f"row {row} lse")
    # the ring gained exactly the current token, once
    changed = (g_rk != ring_before).any(dim=-1).any(dim=1)[0].nonzero().flatten().tolist()
    assert changed == [lay.ring_row(p)], changed
    assert torch.equal(g_rk[0, :, lay.ring_row(p)].cpu(), k_new)
    assert torch.equal(g_rv[0, :, lay.ring_row(p)].cpu(), v_new)


def test_fused_boundary_32k_layer_bf16():
    # the benchmark's draft layer: 2048 slots + 1024-token window, four slots per 64 tokens
    _fused_boundary(torch.bfloat16, 32, 8, 64, S=0, W=1024, r=16, u=4, prefix=32768 - 60, seed=1)


def test_fused_boundary_paper_setting_fp32():
    # S = W = 128, r = 4, one slot per boundary (its scope ends at the current token)
    _fused_boundary(torch.float32, 4, 1, 64, S=128, W=128, r=4, u=1, prefix=1000, seed=2)


def test_fused_boundary_per_boundary_schedule_bf16():
    _fused_boundary(torch.bfloat16, 16, 8, 128, S=0, W=512, r=16, u=1, prefix=8192 + 3, seed=3)
