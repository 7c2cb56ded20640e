"""GPU parity of the draft decoder layer around the attention.

The linear maps (mad_rmsnorm_qkv_rope, mad_linear_residual,
mad_rmsnorm_swiglu) are checked one by one against the oracle's primitives,
then whole layer steps (paper_2608_30252_amd.layer.DraftLayer) against
oracle.decoder_layer at the 32K draft shape (D 2048, 32/8 heads, d 64, FFN
8192, 2048 memory slots + 1024-token window): a plain decode step (one row)
and a materialisation step (the raw token + four slot rows, memory update and
fused attention).  The oracle builds every row's key set from the paper's sets
(oracle.masw_sets), with the new slots' K/V from its own memory update of its
own normalised rows; every stored intermediate is rounded to bf16 on both
sides.  Tolerances: attention outputs bf16 max-abs 2e-2 and relative L2
1e-2; activations of O(1-10) magnitude (hidden states, projections, MLP)
2e-2 + 2^-7 |ref| per element and relative L2 1e-2 (bf16 resolution).
"""
import numpy as np
import pytest
import torch

from parity import check_act, check_out, to_np

pytestmark = pytest.mark.gpu

D, HQ, HKV, DH, FF = 2048, 32, 8, 64, 8192
BASE, EPS = 500000.0, 1e-5


def _params(w):
    return {"gamma1": to_np(w.gamma1), "w_qkv": to_np(w.w_qkv), "w_o": to_np(w.w_o), "gamma2": to_np(w.gamma2),
            "w_gate_up": to_np(w.w_gate_up), "w_down": to_np(w.w_down), "Hq": HQ, "Hkv": HKV, "d": DH,
            "base": BASE, "eps": EPS}


@pytest.mark.parametrize("R", [1, 5])
def test_linear_maps(R):
    import oracle
    import paper_2608_30252_amd as mad
    from paper_2608_30252_amd import synth
    from paper_2608_30252_amd.layer import LayerWeights
    dev = torch.device("cuda")
    w = LayerWeights.random(D, HQ, HKV, DH, FF, seed=3 + R, device=dev)
    p = _params(w)
    x = synth.normal((R, D), 40 + R).to(dev)
    pos = [32768 + 17 * r for r in range(R)]
    xn = torch.empty(R, D, dtype=torch.bfloat16, device=dev)
    q, k, v = mad.rmsnorm_qkv_rope(x, w.gamma1, w.w_qkv, pos, HQ, HKV, DH, xn=xn, eps=EPS, rope_base=BASE)
    a = mad.rmsnorm_swiglu(x, w.gamma2, w.w_gate_up, eps=EPS)
    xin = synth.normal((R, HQ * DH), 50 + R).to(dev)
    res = synth.normal((R, D), 60 + R).to(dev)
    y_o = mad.linear_residual(xin, w.w_o, res)
    ain = synth.normal((R, FF), 70 + R).to(dev)
    y_d = mad.linear_residual(ain, w.w_down, res)
    q2, k2, v2 = mad.rmsnorm_qkv_rope(x, w.gamma1, w.w_qkv, pos, HQ, HKV, DH, eps=EPS, rope_base=BASE,
                                      kv_from_row0=True)
    torch.cuda.synchronize()

    rnd = oracle.bf16_round
    xn_ref = rnd(oracle.rmsnorm(to_np(x), p["gamma1"], EPS))
    qkv = oracle.project(xn_ref, p["w_qkv"])
    q_ref = oracle.rope(qkv[:, :HQ * DH].reshape(R, HQ, DH), pos, BASE)
    k_ref = oracle.rope(qkv[:, HQ * DH:(HQ + HKV) * DH].reshape(R, HKV, DH), pos, BASE)
    v_ref = qkv[:, (HQ + HKV) * DH:].reshape(R, HKV, DH)
    check_act(to_np(xn), xn_ref, "xn")
    check_act(to_np(q), q_ref, "q")
    check_act(to_np(k), k_ref, "k")
    check_act(to_np(v), v_ref, "v")
    gu = oracle.project(rnd(oracle.rmsnorm(to_np(x), p["gamma2"], EPS)), p["w_gate_up"])
    check_act(to_np(a), oracle.silu(gu[:, :FF]) * gu[:, FF:], "swiglu")
    check_act(to_np(y_o), to_np(res) + oracle.project(to_np(xin), p["w_o"]), "o projection + residual")
    check_act(to_np(y_d), to_np(res) + oracle.project(to_np(ain), p["w_down"]), "down projection + residual")
    # kv_from_row0: q unchanged, every row's k and v are row 0's
    assert torch.equal(q2, q)
    for r in range(R):
        assert torch.equal(k2[r], k[0]) and torch.equal(v2[r], v[0])


def _layer_case(p, seed):
    """One layer step at raw position p of the 32K draft, GPU vs oracle."""
    import oracle
    from oracle.masw_sets import MaswSets
    from paper_2608_30252_amd import synth
    from paper_2608_30252_amd.layer import DraftLayer, LayerWeights
    from paper_2608_30252_amd.state import MemoryLayout

    dev = torch.device("cuda")
    S, W, r, u = 0, 1024, 16, 4
    lay = MemoryLayout(S, W, r, ring_cap=W + r * u + 24, mem_cap=2048 + 64, slots_per_update=u)
    sets = MaswSets(S, W, r, u)
    upd = lay.update_in_pass_of(p)
    R = 1 if upd is None else 1 + len(upd.positions)
    w = LayerWeights.random(D, HQ, HKV, DH, FF, seed=seed, device=dev)
    params = _params(w)

    mem_k = synth.normal((1, HKV, lay.mem_cap, DH), 100 * seed + 1)
    mem_v = synth.normal((1, HKV, lay.mem_cap, DH), 100 * seed + 2)
    ring_k = synth.normal((1, HKV, lay.ring_cap, DH), 100 * seed + 3)
    ring_v = synth.normal((1, HKV, lay.ring_cap, DH), 100 * seed + 4)
    x = synth.normal((R, D), 100 * seed + 5)
    g = [t.to(dev) for t in (mem_k, mem_v, ring_k, ring_v, x)]
    layer = DraftLayer(w, D, HQ, HKV, DH, FF, rope_base=BASE, eps=EPS, device=dev)
    y = layer.step(g[4], p, lay, g[0], g[1], g[2], g[3])
    torch.cuda.synchronize()

    # ---- oracle: key sets from the paper's definitions ----
    rnd = oracle.bf16_round
    mk, mv, rk, rv = (to_np(t[0]) for t in (mem_k, mem_v, ring_k, ring_v))
    new_slots = {}

    def key(kind, i, cur):
        if kind == "slot":
            if i in new_slots:
                return new_slots[i]
            return mk[:, S + i - 1], mv[:, S + i - 1]
        if kind == "sink":
            return mk[:, i], mv[:, i]
        if i == p:
            return cur
        return rk[:, lay.ring_row(i)], rv[:, lay.ring_row(i)]

    def attend_rows(q, k, v, xn):
        if upd is not None:   # the slots made in p's pass, from the oracle's own normalised rows
            ks, vs = oracle.memory_update(xn[1:], to_np(w.w_kv_g), np.array(upd.positions), HKV, DH, BASE)
            for i in range(len(upd.positions)):
                new_slots[upd.first_slot + i] = (rnd(ks[i]), rnd(vs[i]))
        cur = (k[0], v[0])
        views = [sets.raw_view(p)] + ([] if upd is None else [sets.slot_scope(upd.first_slot + i)
                                                             for i in range(len(upd.positions))])
        o = np.zeros_like(q)
        for row, sv in enumerate(views):
            ids = [("sink", i) for i in sv.sink] + [("slot", m) for m in sv.slots] + [("raw", x_) for x_ in sv.window]
            K = np.stack([key(kd, i, cur)[0] for kd, i in ids], axis=1)   # [Hkv, n, d]
            V = np.stack([key(kd, i, cur)[1] for kd, i in ids], axis=1)
            G = HQ // HKV
            for c in range(HKV):
                o[row, c * G:(c + 1) * G] = oracle.attend(q[row, c * G:(c + 1) * G], K[c], V[c], DH ** -0.5)[0]
        return o

    pos = [p] + ([] if upd is None else list(upd.positions))
    ref = oracle.decoder_layer(to_np(x), params, pos, attend_rows, rnd=rnd)
    check_out(to_np(layer.o[:R]), ref["o"], True, "attention output")
    check_act(to_np(y), ref["y"], "layer output")
    # the current token's K/V went into the ring; the new slots into the memory
    assert torch.equal(g[2][0, :, lay.ring_row(p)], layer.k[0])
    assert torch.equal(g[3][0, :, lay.ring_row(p)], layer.v[0])
    if upd is not None:
        for i in range(len(upd.positions)):
            check_act(to_np(g[0][0, :, upd.mem_row + i]), new_slots[upd.first_slot + i][0], "slot k")
            check_act(to_np(g[1][0, :, upd.mem_row + i]), new_slots[upd.first_slot + i][1], "slot v")
    return R


def test_layer_decode_step_32k():
    assert _layer_case(32768 + 5, seed=21) == 1


def test_layer_materialisation_step_32k():
    # the pass of raw token 32768 + 63 makes slots 2049..2052 (four per 64 tokens)
    assert _layer_case(32768 + 63, seed=22) == 5
