"""GPU parity of mad_memory_prefill_attn against the oracle's memory prefill.

Each query of the prefill pass attends the set it would attend while decoding
(a raw token: sinks, the slots materialised before it, its window; a slot: its
write scope).  The oracle builds every key list from the visible-set
simulator; the inputs are seeded bf16 tensors that both sides read.  Rows of
the outputs past each sequence's prefix (or slot count) must stay untouched.
Slot counts come from the oracle's set simulator.  Tolerances: bf16 outputs
max-abs 2e-2 and relative L2 1e-2; lse per row within the bound derived from
the fp32 arithmetic (parity.lse_tol).
"""
import numpy as np
import pytest
import torch

from parity import abs_score, check_lse, check_out, to_np

pytestmark = pytest.mark.gpu


def _row_scores(qrow, view, mem_k, raw_k, S, scale):
    """A (per query head) over the keys of one prefill row: its sinks and slots
    (memory rows) and its raw window."""
    Hq, d = qrow.shape
    Hkv = mem_k.shape[0]
    G = Hq // Hkv
    mrows = list(view.sink) + [S + m - 1 for m in view.slots]
    A = np.zeros(Hq)
    for c in range(Hkv):
        K = np.concatenate([mem_k[c][mrows].reshape(-1, d), raw_k[c][list(view.window)].reshape(-1, d)])
        A[c * G:(c + 1) * G] = abs_score(qrow[c * G:(c + 1) * G], K, scale)
    return A


def _run(Hq, Hkv, d, S, W, r, u, P_list, seed, slots=True, raw_idx=None, slot_idx=None, ramp=0.0, peaky=0.0):
    import oracle
    import paper_2608_30252_amd as mad
    from oracle.masw_sets import MaswSets
    from paper_2608_30252_amd import synth

    dev = torch.device("cuda")
    B = len(P_list)
    sets = MaswSets(S, W, r, u)
    M_list = [sets.slots_after(P) for P in P_list]
    q_cap = max(P_list) + 5
    slot_cap = max(max(M_list), 1) + 2
    mem_cap = S + slot_cap + 3
    q_raw = synth.normal((B, q_cap, Hq, d), 100 * seed + 1)
    q_slot = synth.normal((B, slot_cap, Hq, d), 100 * seed + 2)
    raw_k = synth.normal((B, Hkv, q_cap, d), 100 * seed + 3)
    raw_v = synth.normal((B, Hkv, q_cap, d), 100 * seed + 4)
    mem_k = synth.normal((B, Hkv, mem_cap, d), 100 * seed + 5)
    mem_v = synth.normal((B, Hkv, mem_cap, d), 100 * seed + 6)
    if ramp:
        # keys grow along the sequence: each row's running maximum keeps jumping by far more than
        # 2^8 from tile to tile, so the online softmax must rebase it many times
        raw_k = (raw_k.float() * (1 + ramp * torch.arange(q_cap).float() / q_cap)[None, None, :, None]).to(raw_k.dtype)
        mem_k = (mem_k.float() * (1 + ramp * torch.arange(mem_cap).float() / mem_cap)[None, None, :, None]).to(mem_k.dtype)
    s = min(S, q_cap)
    mem_k[:, :, :s], mem_v[:, :, :s] = raw_k[:, :, :s], raw_v[:, :, :s]   # the sinks are raw tokens 0..S-1
    G = Hq // Hkv
    targets = []
    if peaky:
        # sampled raw queries point at a raw key of their window, sampled slot queries at their own
        # slot row (a slot's write scope holds itself): q = peaky * that key
        for b, (P, M) in enumerate(zip(P_list, M_list)):
            for p in (raw_idx or []):
                if S <= p < P:
                    for h in range(Hq):
                        j = p - (h * 13) % min(W, p - S + 1)
                        q_raw[b, p, h] = (peaky * raw_k[b, h // G, j].float()).to(q_raw.dtype)
                        targets.append(("raw", b, p, h, raw_k[b, h // G, j].double().numpy()))
            for m in (slot_idx or []):
                if 1 <= m <= M:
                    for h in range(Hq):
                        q_slot[b, m - 1, h] = (peaky * mem_k[b, h // G, S + m - 1].float()).to(q_slot.dtype)
                        targets.append(("slot", b, m, h, mem_k[b, h // G, S + m - 1].double().numpy()))

    g = [t.to(dev) for t in (q_raw, q_slot, raw_k, raw_v, mem_k, mem_v)]
    out_raw = torch.full((B, q_cap, Hq, d), float("nan"), dtype=torch.bfloat16, device=dev)
    lse_raw = torch.full((B, q_cap, Hq), float("nan"), device=dev)
    out_slot = torch.full((B, slot_cap, Hq, d), float("nan"), dtype=torch.bfloat16, device=dev)
    lse_slot = torch.full((B, slot_cap, Hq), float("nan"), device=dev)
    mad.memory_prefill_attn(g[0], g[1] if slots else None, mad.KV(g[4], g[5], [S + M for M in M_list]),
                            mad.KV(g[2], g[3], list(P_list)), P_list, S, W, r, u, out_raw, lse_raw,
                            out_slot if slots else None, lse_slot if slots else None)
    torch.cuda.synchronize()
    o_raw, l_raw, o_slot, l_slot = (to_np(t) for t in (out_raw, lse_raw, out_slot, lse_slot))

    scale = d ** -0.5
    for b, (P, M) in enumerate(zip(P_list, M_list)):
        ridx = list(range(P)) if raw_idx is None else [p for p in raw_idx if p < P]
        sidx = list(range(1, M + 1)) if slot_idx is None else [m for m in slot_idx if 1 <= m <= M]
        ref_raw, ref_slot = oracle.memory_prefill(
            to_np(q_raw[b]), to_np(q_slot[b]) if slots else None, to_np(mem_k[b]), to_np(mem_v[b]),
            to_np(raw_k[b]), to_np(raw_v[b]), P, S, W, r, u, scale, raw_idx=ridx, slot_idx=sidx)
        mk_b, rk_b = to_np(mem_k[b]), to_np(raw_k[b])
        for kind, bb, i, h, kt in targets:
            if bb == b:
                qv, lref = (q_raw[b, i, h], ref_raw[i][1][h]) if kind == "raw" else (q_slot[b, i - 1, h], ref_slot[i][1][h])
                w = np.exp(scale * float(qv.double().numpy() @ kt) - lref)
                assert w >= 0.9, f"seq {b} {kind} {i} head {h}: target weight {w:.3f}"
        if ridx:
            check_out(o_raw[b, ridx], np.stack([ref_raw[p][0] for p in ridx]), True, f"seq {b} raw out")
            A = np.stack([_row_scores(to_np(q_raw[b, p]), sets.raw_view(p), mk_b, rk_b, S, scale) for p in ridx])
            check_lse(l_raw[b, ridx], np.stack([ref_raw[p][1] for p in ridx]), A, d, f"seq {b} raw lse")
        assert np.isnan(o_raw[b, P:]).all() and np.isnan(l_raw[b, P:]).all(), f"seq {b}: rows past the prefix written"
        if slots:
            if sidx:
                rows = [m - 1 for m in sidx]
                check_out(o_slot[b, rows], np.stack([ref_slot[m][0] for m in sidx]), True, f"seq {b} slot out")
                A = np.stack([_row_scores(to_np(q_slot[b, m - 1]), sets.slot_scope(m), mk_b, rk_b, S, scale)
                              for m in sidx])
                check_lse(l_slot[b, rows], np.stack([ref_slot[m][1] for m in sidx]), A, d, f"seq {b} slot lse")
            assert np.isnan(o_slot[b, M:]).all(), f"seq {b}: slot rows past the slot count written"
        else:
            assert np.isnan(o_slot).all()


def test_draft_shape_batched_schedule_ragged():
    # 32/8 heads, d 64, r 16 with four slots per update; two ragged prefixes
    _run(32, 8, 64, S=0, W=128, r=16, u=4, P_list=[1000, 777], seed=1)


def test_paper_setting_sinks_r4():
    # S = W = 128, r = 4, one slot per boundary
    _run(16, 4, 64, S=128, W=128, r=4, u=1, P_list=[900], seed=2)


def test_head_dim_128_group_8_three_sequences():
    _run(64, 8, 128, S=4, W=100, r=8, u=2, P_list=[600, 333, 3], seed=3)


@pytest.mark.parametrize("Hq,Hkv,d", [(8, 8, 64), (8, 4, 128), (16, 8, 64), (8, 2, 128)])
def test_group_sizes(Hq, Hkv, d):
    _run(Hq, Hkv, d, S=2, W=50, r=5, u=1, P_list=[301], seed=4 + Hq + d)


def test_prefix_shorter_than_the_sinks_without_slot_queries():
    _run(8, 2, 64, S=8, W=16, r=4, u=1, P_list=[5, 1], seed=9, slots=False)


def test_window_shorter_than_the_slot_interval():
    _run(32, 8, 64, S=0, W=8, r=16, u=1, P_list=[513], seed=10)


def _sample_32k():
    rng = np.random.default_rng(0)
    raw_idx = sorted(set([0, 1, 15, 16, 63, 64, 1023, 1024, 1025, 16383, 16384, 32703, 32704, 32767] +
                         rng.integers(0, 32768, 12).tolist()))
    slot_idx = sorted(set([1, 2, 4, 5, 64, 65, 1024, 2047, 2048] + rng.integers(1, 2049, 6).tolist()))
    return raw_idx, slot_idx


def test_32k_prefix_full_size_sampled():
    # the 32K draft layer: 2048 slots (four per update), 1024-token window;
    # the GPU computes every query, the oracle a sample spanning block edges
    raw_idx, slot_idx = _sample_32k()
    _run(32, 8, 64, S=0, W=1024, r=16, u=4, P_list=[32768], seed=11, raw_idx=raw_idx, slot_idx=slot_idx)


def test_32k_prefix_peaky_queries_sampled():
    # the same layer with the sampled queries set to 3 x a key they attend: the target key holds
    # at least 0.9 of the softmax weight (asserted), lse ~ 24
    raw_idx, slot_idx = _sample_32k()
    _run(32, 8, 64, S=0, W=1024, r=16, u=4, P_list=[32768], seed=12, raw_idx=raw_idx, slot_idx=slot_idx,
         peaky=3.0)


@pytest.mark.parametrize("d,ramp", [(64, 4.0), (128, 4.0), (64, 11.0), (128, 11.0)])
def test_growing_scores_rebase_the_running_maximum(d, ramp):
    # keys scaled by 1 .. 1 + ramp along the prefix: the late tiles' scores exceed the early ones' by
    # more than 2^8, so the lazily rebased maximum moves within a pass; at ramp 11 scores reach ~50
    _run(8, 2, d, S=4, W=300, r=8, u=2, P_list=[2500, 1700], seed=23, ramp=ramp)
