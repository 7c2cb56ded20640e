"""Rollback after a rejected speculative block (Sec. 3.3: on rejection the
draft discards the speculative raw KV and the memory slots created after the
last accepted position; the raw-KV rollback window restores the local window).

A draft block of gamma = 4 tokens is decoded from position P0 with the memory
update of a slot boundary inside it (slot m0 is materialised in the pass of
P0 + 1).  Target logits planted so that greedy accept keeps the first draft and
rejects the second (mad_accept_greedy on the device gives n_accept = 1 and the
correction token).  The host state rolls back to P0 + 1 (state.py: a pure
function of the position, so the dropped slot and the rejected ring rows are
simply not attended) and the draft continues with the correction token, which
re-materialises slot m0 from its new hidden state.  The next two decode steps
must equal, bit for bit, a fresh run that never saw the rejected tokens, and
both must match the oracle over the paper's sets."""
import numpy as np
import pytest
import torch

from parity import abs_score_batched, check_lse, check_out, to_np

pytestmark = pytest.mark.gpu

Hq, Hkv, d, S, W, r, GAMMA, ROLLBACK = 32, 8, 64, 0, 64, 16, 4, 16
D = Hq * d
BASE = 500000.0
M0 = 40                      # the slot whose boundary falls inside the drafted block
P0 = S + M0 * r - 2          # drafted positions P0 .. P0+3; slot M0 is made in the pass of P0 + 1
V = 4096


def _kv(p, tok):
    from paper_2608_30252_amd import synth
    s = 10_000_000 + 7919 * p + tok
    return synth.normal((1, Hkv, d), s), synth.normal((1, Hkv, d), s + 1), synth.normal((1, Hq, d), s + 2)


def _slot_x(m, tok):
    from paper_2608_30252_amd import synth
    return synth.normal((1, 1, D), 20_000_000 + 7919 * m + tok)


class Run:
    """Device buffers of one draft layer and the decode/update calls of a step."""

    def __init__(self, init, lay, w_g):
        self.mk, self.mv, self.rk, self.rv = (t.clone().cuda() for t in init)
        self.lay, self.w_g = lay, w_g

    def step(self, p, tok):
        import paper_2608_30252_amd as mad
        view = self.lay.decode_view(p)
        kn, vn, q = _kv(p, tok)
        out, lse = mad.draft_decode_attn(q.cuda(), mad.KV(self.mk, self.mv, [view.mem_len]),
                                         mad.KV(self.rk, self.rv, [view.win_len], [view.win_start]),
                                         kn.cuda(), vn.cuda())
        upd = self.lay.update_in_pass_of(p)
        if upd is not None:   # the slot made in this pass: an extra position after the raw token
            mad.memory_update(_slot_x(upd.first_slot, tok).cuda(), self.w_g, [upd.positions],
                              mad.KV(self.mk, self.mv, [upd.mem_row]), rope_base=BASE)
        torch.cuda.synchronize()
        return out.cpu(), lse.cpu(), view


def test_rollback_after_rejection_matches_a_fresh_run_and_the_oracle():
    import oracle
    import paper_2608_30252_amd as mad
    from oracle.masw_sets import MaswSets
    from paper_2608_30252_amd import synth
    from paper_2608_30252_amd.state import MemoryLayout

    ring_cap = (W + GAMMA + ROLLBACK + 7) // 8 * 8
    lay = MemoryLayout(S, W, r, ring_cap=ring_cap, mem_cap=M0 + 8)
    assert lay.update_in_pass_of(P0 + 1) is not None and lay.update_in_pass_of(P0 + 1).first_slot == M0
    assert lay.rollback_ok(P0 + GAMMA, P0 + 1)
    sets = MaswSets(S, W, r)
    w_g = synth.normal((2 * Hkv * d, D), 30_000_000, std=0.02)
    g_w = w_g.cuda()

    # the state before the block: slots 1 .. M0-1 and the raw window of P0 (token 7 everywhere)
    n0 = lay.slots_materialised(P0)
    assert n0 == M0 - 1
    mk = torch.zeros(1, Hkv, lay.mem_cap, d, dtype=torch.bfloat16)
    mv = torch.zeros_like(mk)
    rk = torch.zeros(1, Hkv, ring_cap, d, dtype=torch.bfloat16)
    rv = torch.zeros_like(rk)
    slot_kv, raw_kv = {}, {}
    for m in range(1, n0 + 1):
        kk, vv = oracle.memory_update(_slot_x(m, 7)[0].double().numpy(), w_g.double().numpy(),
                                      np.array([S + m * r]), Hkv, d, BASE)
        k16, v16 = torch.from_numpy(kk[0]).to(torch.bfloat16), torch.from_numpy(vv[0]).to(torch.bfloat16)
        mk[0, :, m - 1], mv[0, :, m - 1] = k16, v16
        slot_kv[m] = (k16.double().numpy(), v16.double().numpy())
    for x in range(max(S, P0 - W), P0):
        kn, vn, _ = _kv(x, 7)
        rk[0, :, lay.ring_row(x)], rv[0, :, lay.ring_row(x)] = kn[0], vn[0]
        raw_kv[x] = (kn[0].double().numpy(), vn[0].double().numpy())
    init = (mk, mv, rk, rv)

    # ---- speculative block: four drafts, the boundary of slot M0 inside ----
    drafts = [100, 101, 102, 103]
    correction = 200
    spec = Run(init, lay, g_w)
    for i, tok in enumerate(drafts):
        spec.step(P0 + i, tok)

    # ---- verify: planted logits; greedy accept on the device ----
    logits = synth.normal((1, GAMMA + 1, V), 40_000_000, dtype=torch.float32)
    logits[0, 0, drafts[0]] = 20.0           # the first draft is the target's argmax: accepted
    logits[0, 1, correction] = 20.0          # the second is not: rejected, the target emits `correction`
    na, nx = mad.accept_greedy(logits.cuda(), torch.tensor([drafts], dtype=torch.int32).cuda())
    n_accept, nxt = int(na.cpu()[0]), int(nx.cpu()[0])
    assert (n_accept, nxt) == (1, correction)

    # ---- rollback to the first rejected position, then continue with the correction ----
    p_new = P0 + n_accept
    assert lay.rollback_ok(P0 + GAMMA, p_new)
    after_spec = [spec.step(p_new, nxt), spec.step(p_new + 1, 300)]

    # ---- a fresh run that never saw the rejected tokens ----
    fresh = Run(init, lay, g_w)
    fresh.step(P0, drafts[0])
    after_fresh = [fresh.step(p_new, nxt), fresh.step(p_new + 1, 300)]

    for (oa, la, va), (ob, lb, vb) in zip(after_spec, after_fresh):
        assert va == vb
        assert torch.equal(oa.view(torch.int16), ob.view(torch.int16)), "output differs from the fresh run"
        assert torch.equal(la, lb), "lse differs from the fresh run"
    # the memory rows every later step reads, and the ring rows of the current window, are identical
    mlen = lay.decode_view(p_new + 2).mem_len
    assert mlen == M0
    assert torch.equal(spec.mk[:, :, :mlen].cpu().view(torch.int16), fresh.mk[:, :, :mlen].cpu().view(torch.int16))
    assert torch.equal(spec.mv[:, :, :mlen].cpu().view(torch.int16), fresh.mv[:, :, :mlen].cpu().view(torch.int16))
    win = [lay.ring_row(x) for x in range(max(S, p_new + 2 - W + 1), p_new + 2)]
    assert torch.equal(spec.rk[:, :, win].cpu().view(torch.int16), fresh.rk[:, :, win].cpu().view(torch.int16))
    assert torch.equal(spec.rv[:, :, win].cpu().view(torch.int16), fresh.rv[:, :, win].cpu().view(torch.int16))

    # ---- both against the oracle over the paper's sets (accepted history only) ----
    kn, vn, _ = _kv(P0, drafts[0])
    raw_kv[P0] = (kn[0].double().numpy(), vn[0].double().numpy())
    for j, (p, tok) in enumerate(((p_new, nxt), (p_new + 1, 300))):
        kn, vn, q = _kv(p, tok)
        raw_kv[p] = (kn[0].double().numpy(), vn[0].double().numpy())
        if p == p_new:   # the slot made in the pass of p_new, from the correction's hidden state
            kk, vv = oracle.memory_update(_slot_x(M0, tok)[0].double().numpy(), w_g.double().numpy(),
                                          np.array([S + M0 * r]), Hkv, d, BASE)
            slot_now = (torch.from_numpy(kk[0]).to(torch.bfloat16).double().numpy(),
                        torch.from_numpy(vv[0]).to(torch.bfloat16).double().numpy())
        view = sets.raw_view(p)
        ks = [slot_kv[m][0] if m < M0 else slot_now[0] for m in view.slots] + [raw_kv[x][0] for x in view.window]
        vs = [slot_kv[m][1] if m < M0 else slot_now[1] for m in view.slots] + [raw_kv[x][1] for x in view.window]
        K, Vv = np.stack(ks, 1)[None], np.stack(vs, 1)[None]
        o_ref, l_ref = oracle.attend_batched(q.double().numpy(), K, Vv, np.array([K.shape[2]]), d ** -0.5)
        check_out(to_np(after_spec[j][0]), o_ref, True, f"step {p} out")
        check_lse(to_np(after_spec[j][1]), l_ref, abs_score_batched(q.double().numpy(), K, [K.shape[2]], d ** -0.5),
                  d, f"step {p} lse")
        if p == p_new + 1:
            assert M0 in view.slots   # the re-materialised slot is attended
