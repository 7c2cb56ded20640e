"""Graph capture of the entry points the benchmark replays in HIP graphs:
memory-prefill attention and whole draft-layer steps.  Each is captured once
and replayed three times, with unrelated eager work and synchronisations
between replays; every replay must reproduce the eager outputs bit for bit."""
import pytest
import torch

pytestmark = pytest.mark.gpu


def _replays(fn, outs):
    import bench
    fn()
    torch.cuda.synchronize()
    eager = [t.clone() for t in outs]
    g = bench.graph_of(torch, fn)
    for rep in range(3):
        for t in outs:
            t.fill_(float("nan"))
        scratch = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.isfinite(scratch)
        for i, (a, b) in enumerate(zip(outs, eager)):
            assert torch.equal(a, b), f"replay {rep}: output {i} differs from the eager run"


def test_prefill_graph_replays():
    import paper_2608_30252_amd as mad
    from paper_2608_30252_amd import synth
    dev = torch.device("cuda")
    P, S, W, r, u, Hq, Hkv, d = 3000, 4, 256, 16, 4, 32, 8, 64
    M = mad.slots_after(P, S, r, u)
    q_raw = synth.normal((1, P, Hq, d), 1).to(dev)
    q_slot = synth.normal((1, M, Hq, d), 2).to(dev)
    rk, rv = synth.normal((1, Hkv, P, d), 3).to(dev), synth.normal((1, Hkv, P, d), 4).to(dev)
    mk, mv = synth.normal((1, Hkv, S + M, d), 5).to(dev), synth.normal((1, Hkv, S + M, d), 6).to(dev)
    outs = [torch.empty_like(q_raw), torch.empty(1, P, Hq, device=dev), torch.empty_like(q_slot),
            torch.empty(1, M, Hq, device=dev)]
    _replays(lambda: mad.memory_prefill_attn(q_raw, q_slot, mad.KV(mk, mv, [S + M]), mad.KV(rk, rv, [P]), [P],
                                             S, W, r, u, *outs), outs)


@pytest.mark.parametrize("p_off", [5, 63])
def test_draft_layer_step_graph_replays(p_off):
    # a plain decode step and a materialisation step (memory update + fused attention)
    import bench
    import paper_2608_30252_amd as mad
    from paper_2608_30252_amd import synth
    from paper_2608_30252_amd.layer import DraftLayer, LayerWeights
    dev = torch.device("cuda")
    m = bench.DraftModel(torch, mad, 1, layers=2)
    layers = [DraftLayer(LayerWeights.random(2048, 32, 8, 64, 8192, seed=30 + l, device=dev), 2048, 32, 8, 64, 8192,
                         device=dev) for l in range(2)]
    p = m.prefix + p_off
    upd = m.lay.update_in_pass_of(p)
    x0 = synth.normal((1 if upd is None else 1 + len(upd.positions), 2048), 77).to(dev)

    def step():
        x = x0
        for l in range(2):
            x = layers[l].step(x, p, m.lay, m.mem_k[0][l], m.mem_v[0][l], m.ring_k[0][l], m.ring_v[0][l], ws=m.ws)
    R = x0.shape[0]
    outs = [layers[1].y[:R], layers[0].y[:R], layers[1].o[:R]]
    _replays(step, outs)
