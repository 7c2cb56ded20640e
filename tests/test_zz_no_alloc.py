"""The no-allocation decode entry point (mad_draft_decode_attn_noalloc) against
mad_draft_decode_attn with a caller workspace: the same kernels run, so the
outputs, lse and the appended ring rows must be bit-identical; both are also
checked against the oracle (bf16 outputs max-abs 2e-2 and rel-L2 1e-2, lse
within the derived bound).  Two calls in a row, the second with a smaller
input (fewer sequences and keys), so the second reads the library's scratch
after the first left its contents there."""
import ctypes

import numpy as np
import pytest
import torch

from parity import abs_score_batched, check_lse, check_out, to_np

pytestmark = pytest.mark.gpu


def _inputs(B, mlen, wlen, wcap, seed):
    from paper_2608_30252_amd import synth
    Hq, Hkv, d = 32, 8, 64
    s = 1000 * seed
    g = dict(q=synth.normal((B, Hq, d), s + 1), mk=synth.normal((B, Hkv, mlen, d), s + 2),
             mv=synth.normal((B, Hkv, mlen, d), s + 3), wk=synth.normal((B, Hkv, wcap, d), s + 4),
             wv=synth.normal((B, Hkv, wcap, d), s + 5), kn=synth.normal((B, Hkv, d), s + 6),
             vn=synth.normal((B, Hkv, d), s + 7))
    return g


def _oracle(g, B, mlen, wlen, wstart, wcap):
    import oracle
    d = g["q"].shape[-1]
    idx = [(wstart[b] + np.arange(wlen)) % wcap for b in range(B)]
    K = np.stack([np.concatenate([g["mk"][b].double().numpy(), g["wk"][b].double().numpy()[:, idx[b]],
                                  g["kn"][b].double().numpy()[:, None]], 1) for b in range(B)])
    V = np.stack([np.concatenate([g["mv"][b].double().numpy(), g["wv"][b].double().numpy()[:, idx[b]],
                                  g["vn"][b].double().numpy()[:, None]], 1) for b in range(B)])
    n = np.full(B, K.shape[2])
    o, lse = oracle.attend_batched(g["q"].double().numpy(), K, V, n, d ** -0.5)
    return o, lse, abs_score_batched(g["q"].double().numpy(), K, n, d ** -0.5)


def test_noalloc_matches_workspace_entry_point_on_two_calls():
    import paper_2608_30252_amd as mad
    dev = torch.device("cuda")
    lib = mad._load_library()
    # 4 sequences of the 32K compact layer (2048 slots + 1023 window + new), then 1 sequence of 700 keys
    for case, (B, mlen, wlen, wcap) in enumerate([(4, 2048, 1023, 1056), (1, 500, 199, 256)]):
        g = _inputs(B, mlen, wlen, wcap, seed=70 + case)
        wstart = [(37 * b + 11 * case) % wcap for b in range(B)]
        d = g["q"].shape[-1]
        results = []
        for entry in ("workspace", "noalloc"):
            t = {k: v.to(dev) for k, v in g.items()}
            mem = mad.KV(t["mk"], t["mv"], [mlen] * B)
            win = mad.KV(t["wk"], t["wv"], [wlen] * B, wstart)
            out = torch.full_like(t["q"], float("nan"))
            lse = torch.full((B, t["q"].shape[1]), float("nan"), device=dev)
            if entry == "workspace":
                ws = torch.zeros(mad.workspace_bytes(mad.MAD_OP_DECODE, B, 32, 8, d), dtype=torch.uint8, device=dev)
                mad.draft_decode_attn(t["q"], mem, win, t["kn"], t["vn"], out, lse, ws=ws)
            else:   # straight through the C ABI
                mv, wv = mem.view(B), win.view(B)
                rc = lib.mad_draft_decode_attn_noalloc(
                    ctypes.c_void_p(t["q"].data_ptr()), B, 32, 8, d, mad.MAD_BF16, ctypes.c_float(d ** -0.5),
                    ctypes.byref(mv), ctypes.byref(wv), ctypes.c_void_p(t["kn"].data_ptr()),
                    ctypes.c_void_p(t["vn"].data_ptr()), ctypes.c_void_p(out.data_ptr()),
                    ctypes.c_void_p(lse.data_ptr()), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
                assert rc == 0, lib.mad_last_error().decode()
            torch.cuda.synchronize()
            results.append((out.cpu(), lse.cpu(), t["wk"].cpu(), t["wv"].cpu()))
        (o1, l1, k1, v1), (o2, l2, k2, v2) = results
        assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)), f"call {case}: outputs differ"
        assert torch.equal(l1, l2), f"call {case}: lse differs"
        assert torch.equal(k1.view(torch.int16), k2.view(torch.int16)) and \
            torch.equal(v1.view(torch.int16), v2.view(torch.int16)), f"call {case}: ring rows differ"
        o_ref, lse_ref, A = _oracle(g, B, mlen, wlen, wstart, wcap)
        check_out(to_np(o2), o_ref, True, f"call {case} out")
        check_lse(to_np(l2), lse_ref, A, d, f"call {case} lse")


def test_noalloc_rejects_sizes_beyond_its_scratch():
    import paper_2608_30252_amd as mad
    lib = mad._load_library()
    B = 64   # 64 sequences x 8 KV heads need 33 MiB of partials: above the 16 MiB scratch
    assert mad.workspace_bytes(mad.MAD_OP_DECODE, B, 32, 8, 64) > (16 << 20)
    rc = lib.mad_draft_decode_attn_noalloc(ctypes.c_void_p(1 << 20), B, 32, 8, 64, mad.MAD_BF16,
                                           ctypes.c_float(0.125), None, None, None, None,
                                           ctypes.c_void_p(1 << 21), None, None)
    assert rc == mad.MAD_EINVAL and "no-allocation" in lib.mad_last_error().decode()
