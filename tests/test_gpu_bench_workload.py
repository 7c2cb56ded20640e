"""The benchmark's own workload, at full size and in its launch configuration.

bench.py times draft steps of a 16-layer draft at a 32K prefix (2048 memory
slots + a 1024-token window per layer, 32/8 heads, head_dim 64, bf16) as a
replayed HIP graph.  This test builds the same DraftModel (two layers, two
sequences round-robin) and runs a schedule that crosses a 64-token boundary
(memory update of four slots, then one launch for the raw query and the
slots' write scopes):

  * eager run: every decode output (all heads) and, at the boundary, every
    slot-scope output is compared with the oracle.  The oracle's key lists are
    rebuilt on the host from the buffers as they were before any kernel ran,
    the appended new-token rows and the oracle's own slot K/V (rounded to
    bf16, as the memory stores them): no value produced by the GPU feeds it;
  * graph: the same steps captured once and replayed three times, with eager
    GPU work and synchronisations between replays; every replay must
    reproduce the eager outputs bit for bit.
"""
import numpy as np
import pytest
import torch

from parity import abs_score_batched, check_lse, check_out, to_np

pytestmark = pytest.mark.gpu

BASE = 500000.0


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).double().numpy()


def test_bench_draft_step_eager_oracle_and_graph_replays():
    import bench
    import oracle
    import paper_2608_30252_amd as mad

    torch.manual_seed(1234)
    model = bench.DraftModel(torch, mad, n_sets=2, layers=2)
    lay = model.lay
    L, Hkv, d, Hq = model.layers, model.Hkv, model.d, model.Hq
    # set 0 crosses the boundary at raw position prefix + 63 (slots 2049..2052)
    schedule = [(0, model.prefix + 61), (1, model.prefix), (0, model.prefix + 62), (1, model.prefix + 1),
                (0, model.prefix + 63), (1, model.prefix + 2), (0, model.prefix + 64)]
    assert any(lay.update_in_pass_of(p) is not None for i, p in schedule if i == 0)
    torch.cuda.synchronize()

    # host state for the oracle, copied before any kernel runs
    h = {}
    for i in range(2):
        for l in range(L):
            h[i, l] = dict(mk=to_np(model.mem_k[i][l][0]), mv=to_np(model.mem_v[i][l][0]),
                           rk=to_np(model.ring_k[i][l][0]), rv=to_np(model.ring_v[i][l][0]))
    q = [to_np(t[0]) for t in model.q]
    qf = [to_np(t) for t in model.qf]
    kn = [to_np(t[0]) for t in model.kn]
    vn = [to_np(t[0]) for t in model.vn]
    x = [to_np(t[0]) for t in model.x]
    wg = [to_np(t) for t in model.w_g]
    scale = d ** -0.5

    def attend(qrows, st, view, new):
        """qrows [Hq, d]; key list = mem [0, mem_len) ++ ring window ++ optional new token."""
        rows = [(st["mk"][:, j], st["mv"][:, j]) for j in range(view.mem_len)]
        for t in range(view.win_len):
            r = (view.win_start + t) % lay.ring_cap
            rows.append((st["rk"][:, r], st["rv"][:, r]))
        if new is not None:
            rows.append(new)
        K = np.stack([k for k, _ in rows], axis=1)[None]   # [1, Hkv, n, d]
        V = np.stack([v for _, v in rows], axis=1)[None]
        o, lse = oracle.attend_batched(qrows[None], K, V, np.array([K.shape[2]]), scale)
        return o, lse, abs_score_batched(qrows[None], K, [K.shape[2]], scale)

    # ---- eager run, oracle at every step ----
    for i, p in schedule:
        view = lay.decode_view(p)
        upd = lay.update_in_pass_of(p)
        if upd is None:
            refs = [attend(q[l], h[i, l], view, (kn[l], vn[l])) for l in range(L)]
        else:   # the fused launch: row 0 is the raw query, rows 1.. the slots' scopes
            refs = [attend(qf[l][0], h[i, l], view, (kn[l], vn[l])) for l in range(L)]
        model.step(i, p)
        torch.cuda.synchronize()
        out, lse = (model.out, model.lse) if upd is None else (model.outf, model.lsef)
        for l in range(L):
            check_out(to_np(out[l][0]), refs[l][0][0], True, f"set {i} pos {p} layer {l} out")
            check_lse(to_np(lse[l][0]), refs[l][1][0], refs[l][2][0], d, f"set {i} pos {p} layer {l} lse")
        for l in range(L):
            st = h[i, l]
            st["rk"][:, lay.ring_row(p)] = kn[l]
            st["rv"][:, lay.ring_row(p)] = vn[l]
            if upd is None:
                continue
            k_ref, v_ref = oracle.memory_update(x[l], wg[l], np.array(upd.positions), Hkv, d, BASE)
            for r in range(len(upd.positions)):
                st["mk"][:, upd.mem_row + r] = _bf16(k_ref[r])
                st["mv"][:, upd.mem_row + r] = _bf16(v_ref[r])
            for r in range(len(upd.positions)):
                sview = lay.slot_scope_view(upd.first_slot + r)
                o_ref, l_ref, a_ref = attend(qf[l][1 + r], st, sview, None)
                check_out(to_np(model.outf[l][1 + r]), o_ref[0], True, f"set {i} slot {upd.first_slot + r} layer {l}")
                check_lse(to_np(model.lsef[l][1 + r]), l_ref[0], a_ref[0], d, f"set {i} slot {upd.first_slot + r} lse")
    eager = [(model.out[l].clone(), model.lse[l].clone(), model.outf[l].clone(), model.lsef[l].clone())
             for l in range(L)]

    # ---- graph capture, three replays with eager work between ----
    g = bench.graph_of(torch, lambda: [model.step(i, p) for i, p in schedule])
    for rep in range(3):
        for l in range(L):   # clobber the outputs so a replay that skips a write shows
            for t in (model.out[l], model.lse[l], model.outf[l], model.lsef[l]):
                t.fill_(float("nan"))
        scratch = torch.randn(1 << 20, device="cuda").sum()   # unrelated eager work
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.isfinite(scratch)
        for l in range(L):
            for a, b, what in zip((model.out[l], model.lse[l], model.outf[l], model.lsef[l]), eager[l],
                                  ("out", "lse", "outf", "lsef")):
                assert torch.equal(a, b), f"replay {rep} layer {l} {what} differs from the eager run"
