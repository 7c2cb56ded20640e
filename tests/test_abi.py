"""The C ABI on the CPU: the library loads, exports every function that
include/mad.h declares, sizes workspaces, and rejects bad arguments with the
documented status codes before anything is launched (no GPU is touched: all
of these calls fail validation)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "mad.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mad_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def mad():
    import paper_2608_30252_amd as m
    m._load_library()
    return m


def test_every_declared_symbol_is_exported(mad):
    names = _declared_functions()
    assert {"mad_draft_decode_attn", "mad_memory_update", "mad_verify_attn", "mad_verify_attn_vt", "mad_accept_greedy",
            "mad_workspace_bytes", "mad_last_error", "mad_version"} <= set(names)
    lib = ctypes.CDLL(mad.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


TRACE_FUNCTIONS = [f"mad_trace_{k}_{op}" for k in ("decode", "update", "verify") for op in ("read", "clear")]


def test_phase_trace_only_in_the_trace_build(mad):
    # the product library carries no phase marks; the diagnostic build of the
    # same sources (MAD_PHASE_TRACE) exports a reader and a clear per kernel file
    lib = ctypes.CDLL(mad.LIB_PATH)
    assert not any(hasattr(lib, n) for n in TRACE_FUNCTIONS)
    from paper_2608_30252_amd import build
    if not os.path.exists(build.TRACE_LIB):
        pytest.skip("libmad_trace.so not built (python -m paper_2608_30252_amd.build --trace)")
    tlib = ctypes.CDLL(build.TRACE_LIB)
    for n in TRACE_FUNCTIONS + _declared_functions():
        assert hasattr(tlib, n), n


def test_version_and_empty_error(mad):
    assert "gfx950" in mad.version()


def test_workspace_sizes(mad):
    ws = mad.workspace_bytes
    assert ws(mad.MAD_OP_DECODE, 1, 32, 8, 64) > (1 << 20)          # counter region + partials
    assert ws(mad.MAD_OP_DECODE, 16, 32, 8, 64) >= ws(mad.MAD_OP_DECODE, 1, 32, 8, 64)
    assert ws(mad.MAD_OP_UPDATE, 4, 2048, 8, 64) == 0                 # the update takes no workspace
    assert ws(mad.MAD_OP_VERIFY, 4, 32, 8, 128, 5) >= ws(mad.MAD_OP_VERIFY, 1, 32, 8, 128, 5) > (1 << 20)
    assert ws(mad.MAD_OP_ACCEPT, 4, 1, 1, 64, 5, 128256) == (1 << 20)   # counters and row keys: the counter region
    assert ws(mad.MAD_OP_ACCEPT, 1, 1, 1, 64, 257, 128256) == 0          # T above 256
    # invalid sizes give 0
    assert ws(mad.MAD_OP_DECODE, 0, 32, 8, 64) == 0
    assert ws(mad.MAD_OP_DECODE, 1, 30, 8, 64) == 0
    assert ws(99, 1, 1, 1, 64) == 0


def _last_error(mad):
    return mad._load_library().mad_last_error().decode()


def _decode(mad, **kw):
    args = dict(q=1 << 20, B=1, Hq=32, Hkv=8, d=64, dtype=mad.MAD_BF16, scale=0.125, mem=None, win=None,
                kn=None, vn=None, out=1 << 21, lse=None, ws=None, ws_bytes=0)
    args.update(kw)
    lib = mad._load_library()
    return lib.mad_draft_decode_attn(ctypes.c_void_p(args["q"]), args["B"], args["Hq"], args["Hkv"], args["d"],
                                     args["dtype"], args["scale"], args["mem"], args["win"],
                                     ctypes.c_void_p(args["kn"]) if args["kn"] else None,
                                     ctypes.c_void_p(args["vn"]) if args["vn"] else None,
                                     ctypes.c_void_p(args["out"]), None, None, 0, None)


def test_decode_validation(mad):
    assert _decode(mad, B=0) == mad.MAD_EINVAL
    assert _decode(mad, B=65) == mad.MAD_EINVAL
    assert _decode(mad, Hq=30) == mad.MAD_EINVAL
    assert _decode(mad, d=96) == mad.MAD_ENOTSUP and "head_dim" in _last_error(mad)
    assert _decode(mad, Hq=96, Hkv=3) == mad.MAD_ENOTSUP            # group 32
    assert _decode(mad, dtype=7) == mad.MAD_ENOTSUP
    assert _decode(mad, q=0) == mad.MAD_EINVAL
    assert _decode(mad, q=(1 << 20) + 4) == mad.MAD_EINVAL            # unaligned
    assert _decode(mad, kn=1 << 22) == mad.MAD_EINVAL                 # k_new without v_new
    assert _decode(mad, kn=1 << 22, vn=1 << 23) == mad.MAD_EINVAL     # k_new without a window
    assert _decode(mad, scale=-1.0) == mad.MAD_EINVAL
    # a window whose len would overflow its capacity once the new token is appended
    ln = (ctypes.c_int32 * 1)(16)
    win = mad._KVView(1 << 24, 1 << 25, 0, 16 * 64, 16, None, ln)
    assert _decode(mad, win=ctypes.byref(win), kn=1 << 22, vn=1 << 23) == mad.MAD_EINVAL
    assert "exceeds cap" in _last_error(mad)
    st = (ctypes.c_int32 * 1)(16)
    ln2 = (ctypes.c_int32 * 1)(3)
    win2 = mad._KVView(1 << 24, 1 << 25, 0, 16 * 64, 16, st, ln2)
    assert _decode(mad, win=ctypes.byref(win2)) == mad.MAD_EINVAL        # start outside [0, cap)
    win3 = mad._KVView(1 << 24, 1 << 25, 0, 8 * 64, 16, None, ln2)
    assert _decode(mad, win=ctypes.byref(win3)) == mad.MAD_EINVAL        # head stride < cap*d
    # missing workspace when the call needs split partials
    ln4 = (ctypes.c_int32 * 1)(30000)
    win4 = mad._KVView(1 << 24, 1 << 25, 0, 32768 * 64, 32768, None, ln4)
    assert _decode(mad, win=ctypes.byref(win4)) == mad.MAD_EWS


def test_update_validation(mad):
    lib = mad._load_library()
    pos = (ctypes.c_int32 * 4)(16, 32, 48, 64)
    ln = (ctypes.c_int32 * 1)(10)
    mem = mad._KVView(1 << 24, 1 << 25, 0, 16 * 64, 16, None, ln)
    def call(B=1, n_new=4, D=2048, Hkv=8, d=64, dtype=mad.MAD_BF16, base=500000.0, x=1 << 20, memp=True):
        return lib.mad_memory_update(ctypes.c_void_p(x), ctypes.c_void_p(1 << 21), pos, None, B, n_new, D, Hkv, d,
                                     dtype, base, ctypes.byref(mem) if memp else None, None)
    assert call(n_new=8) == mad.MAD_EINVAL and "exceeds cap" in _last_error(mad)   # 10 + 8 > 16
    assert call(n_new=0) == mad.MAD_EINVAL
    assert call(B=65) == mad.MAD_EINVAL
    assert call(D=100) == mad.MAD_EINVAL
    assert call(d=32) == mad.MAD_ENOTSUP
    assert call(base=1.0) == mad.MAD_EINVAL
    assert call(x=0) == mad.MAD_EINVAL
    assert call(memp=False) == mad.MAD_EINVAL


def test_verify_and_accept_validation(mad):
    lib = mad._load_library()
    ln = (ctypes.c_int32 * 1)(100)
    def ver(T=5, Hq=32, Hkv=8, d=128, dtype=mad.MAD_BF16, cap=128, head=128 * 128, ln_=ln):
        return lib.mad_verify_attn_vt(ctypes.c_void_p(1 << 20), 1, T, Hq, Hkv, d, dtype, 0.088,
                                      ctypes.c_void_p(1 << 21), ctypes.c_void_p(1 << 22), 0, head, cap, ln_,
                                      ctypes.c_void_p(1 << 23), None, None, 0, None)
    assert ver(dtype=mad.MAD_F32) == mad.MAD_ENOTSUP
    assert ver(T=0) == mad.MAD_EINVAL
    assert ver(T=5, Hq=128, Hkv=8) == mad.MAD_EINVAL                 # T*G = 80 > 64
    assert ver(cap=100) == mad.MAD_EINVAL                            # not a multiple of 8
    assert ver(head=64) == mad.MAD_EINVAL
    assert ver(ln_=(ctypes.c_int32 * 1)(3)) == mad.MAD_EINVAL        # len < T
    assert ver(ln_=(ctypes.c_int32 * 1)(200)) == mad.MAD_EINVAL      # len > cap
    assert ver() == mad.MAD_EWS                                      # workspace missing
    # the natural layout: a linear mad_kv_view (rows of d); any cap
    def vnat(cap=100, start=None, ln_=ln, dtype=mad.MAD_BF16, head=100 * 128, kv=True):
        view = mad._KVView(1 << 21, 1 << 22, 0, head, cap, start, ln_)
        return lib.mad_verify_attn(ctypes.c_void_p(1 << 20), 1, 5, 32, 8, 128, dtype, 0.088,
                                   ctypes.byref(view) if kv else None, ctypes.c_void_p(1 << 23), None, None, 0, None)
    assert vnat() == mad.MAD_EWS                                     # cap 100 is fine here; workspace missing
    assert vnat(kv=False) == mad.MAD_EINVAL
    assert vnat(start=(ctypes.c_int32 * 1)(0)) == mad.MAD_EINVAL     # the verifier's cache is linear
    assert vnat(dtype=mad.MAD_F32) == mad.MAD_EWS                    # fp32 runs (vector ALUs); workspace missing
    assert vnat(dtype=7) == mad.MAD_ENOTSUP
    assert vnat(ln_=(ctypes.c_int32 * 1)(101)) == mad.MAD_EINVAL     # len > cap
    assert vnat(head=64) == mad.MAD_EINVAL
    acc = lambda B=1, T=5, V=128256, dtype=mad.MAD_F32, draft=1 << 21: lib.mad_accept_greedy(
        ctypes.c_void_p(1 << 20), dtype, ctypes.c_void_p(draft) if draft else None, B, T, V,
        ctypes.c_void_p(1 << 22), ctypes.c_void_p(1 << 23), None, 0, None)
    assert acc(V=0) == mad.MAD_EINVAL
    assert acc(T=0) == mad.MAD_EINVAL
    assert acc(T=257) == mad.MAD_EINVAL
    assert acc(draft=0) == mad.MAD_EINVAL
    assert acc(dtype=5) == mad.MAD_ENOTSUP
    assert acc() == mad.MAD_EWS


def test_stochastic_accept_validation(mad):
    lib = mad._load_library()
    vp = ctypes.c_void_p
    def st(B=1, T=5, V=128256, q=1 << 21, draft=1 << 22, u=1 << 23, ws=None, ws_bytes=0):
        return lib.mad_accept_stochastic(vp(1 << 20), vp(q) if q else None, vp(draft) if draft else None,
                                         vp(u) if u else None, B, T, V, vp(1 << 24), vp(1 << 25),
                                         vp(ws) if ws else None, ws_bytes, None)
    assert st(V=0) == mad.MAD_EINVAL
    assert st(T=0) == mad.MAD_EINVAL
    assert st(T=65) == mad.MAD_EINVAL
    assert st(B=0) == mad.MAD_EINVAL
    assert st(q=0) == mad.MAD_EINVAL                      # q required when T > 1
    assert st(draft=0) == mad.MAD_EINVAL
    assert st(u=0) == mad.MAD_EINVAL
    assert st() == mad.MAD_EWS                            # workspace missing
    need = mad.workspace_bytes(mad.MAD_OP_ACCEPT_STOCH, 1, 1, 1, 64, 5, 128256)
    assert need > 0
    assert st(ws=1 << 26, ws_bytes=need - 1) == mad.MAD_EWS
    assert st(ws=(1 << 26) + 16, ws_bytes=need) == mad.MAD_EINVAL   # not 256-byte aligned
    assert st(T=1, q=0, draft=0) == mad.MAD_EWS          # T == 1 needs neither q nor drafts


def test_step_attn_validation(mad):
    """mad_draft_step_attn: per-row new-token modes are checked before launch."""
    lib = mad._load_library()
    vp = ctypes.c_void_p
    B = 3
    ln = (ctypes.c_int32 * B)(100, 50, 50)
    st = (ctypes.c_int32 * B)(0, 0, 0)
    ring = lambda seq_stride: mad._KVView(1 << 24, 1 << 25, seq_stride, 256 * 64, 256, st, ln)

    def call(modes, kn=1 << 22, vn=1 << 23, win=ring(0), B=B):
        m = None if modes is None else (ctypes.c_uint8 * len(modes))(*modes)
        w = None if win is None else ctypes.byref(win)
        return lib.mad_draft_step_attn(vp(1 << 20), B, 32, 8, 64, mad.MAD_BF16, 0.125, None, w,
                                       vp(kn) if kn else None, vp(vn) if vn else None, m, vp(1 << 21),
                                       None, None, 0, None)
    assert call(None) == mad.MAD_EINVAL and "new_mode" in _last_error(mad)
    assert call([2, 3, 0]) == mad.MAD_EINVAL and "outside" in _last_error(mad)
    assert call([2, 1, 0], kn=None, vn=None) == mad.MAD_EINVAL             # modes 1/2 need k_new
    assert call([0, 1, 0], kn=1 << 22, vn=None) == mad.MAD_EINVAL
    assert call([2, 1, 0], win=None) == mad.MAD_EINVAL                      # append without a ring
    assert call([2, 2, 0]) == mad.MAD_EINVAL and "share" in _last_error(mad)  # two appends, one ring
    assert call([2, 1, 0], B=0) == mad.MAD_EINVAL
    assert call([2, 1, 0], B=65) == mad.MAD_EINVAL
    # a full ring cannot take the appended row; with mode 1 (attend only) the same
    # ring passes validation and the call stops at the missing split workspace
    full = (ctypes.c_int32 * B)(32768, 30000, 30000)
    w = mad._KVView(1 << 24, 1 << 25, 0, 32768 * 64, 32768, st, full)
    assert call([2, 1, 0], win=w) == mad.MAD_EINVAL and "exceeds cap" in _last_error(mad)
    assert call([1, 1, 0], win=w) == mad.MAD_EWS


def test_prefill_validation(mad):
    """mad_memory_prefill_attn rejects bad arguments before anything is launched."""
    lib = mad._load_library()
    vp = ctypes.c_void_p
    P = (ctypes.c_int32 * 2)(1000, 777)
    mlen = (ctypes.c_int32 * 2)(60, 48)        # S + slots: 0 + 4 * floor(P / 64)
    rlen = (ctypes.c_int32 * 2)(1000, 777)

    def call(q_raw=1 << 20, q_slot=1 << 21, B=2, Hq=32, Hkv=8, d=64, dtype=None, scale=0.125, P=P,
             q_cap=1005, slot_cap=64, S=0, W=128, r=16, u=4, mlen=mlen, rlen=rlen, rstart=None, out_raw=1 << 22,
             out_slot=1 << 23):
        mem = mad._KVView(1 << 24, 1 << 25, 8 * 300 * 64, 300 * 64, 300, None, mlen)
        raw = mad._KVView(1 << 26, 1 << 27, 8 * 1024 * 64, 1024 * 64, 1024, rstart, rlen)
        return lib.mad_memory_prefill_attn(vp(q_raw) if q_raw else None, vp(q_slot) if q_slot else None, B, Hq,
                                           Hkv, d, mad.MAD_BF16 if dtype is None else dtype, scale, P, q_cap,
                                           slot_cap, S, W, r, u, ctypes.byref(mem), ctypes.byref(raw),
                                           vp(out_raw) if out_raw else None, None,
                                           vp(out_slot) if out_slot else None, None, None)
    assert call(dtype=mad.MAD_F32) == mad.MAD_ENOTSUP
    assert call(Hq=128) == mad.MAD_ENOTSUP                 # group 16
    assert call(d=96) == mad.MAD_ENOTSUP
    assert call(q_raw=0) == mad.MAD_EINVAL
    assert call(out_slot=0) == mad.MAD_EINVAL              # slot queries without an output
    assert call(q_raw=(1 << 20) + 8) == mad.MAD_EINVAL     # unaligned
    assert call(W=0) == mad.MAD_EINVAL and call(r=0) == mad.MAD_EINVAL and call(u=0) == mad.MAD_EINVAL
    assert call(S=-1) == mad.MAD_EINVAL
    assert call(q_cap=999) == mad.MAD_EINVAL and "q_cap" in _last_error(mad)
    assert call(slot_cap=59) == mad.MAD_EINVAL and "slot_cap" in _last_error(mad)
    short = (ctypes.c_int32 * 2)(59, 48)
    assert call(mlen=short) == mad.MAD_EINVAL and "mem" in _last_error(mad)
    rshort = (ctypes.c_int32 * 2)(1000, 776)
    assert call(rlen=rshort) == mad.MAD_EINVAL and "raw" in _last_error(mad)
    st = (ctypes.c_int32 * 2)(0, 0)
    assert call(rstart=st) == mad.MAD_EINVAL and "linear" in _last_error(mad)
    assert call(scale=0.0) == mad.MAD_EINVAL
    assert call(B=0) == mad.MAD_EINVAL
    # nothing to do: every prefix empty
    zero = (ctypes.c_int32 * 2)(0, 0)
    assert call(P=zero) == mad.MAD_OK


def test_layer_linear_validation(mad):
    lib = mad._load_library()
    vp = ctypes.c_void_p
    pos = (ctypes.c_int32 * 8)(*range(8))
    qkv = lambda R=1, D=2048, Hq=32, Hkv=8, d=64, eps=1e-5, base=5e5, x=1 << 20: lib.mad_rmsnorm_qkv_rope(
        vp(x) if x else None, vp(1 << 21), eps, vp(1 << 22), pos, R, D, Hq, Hkv, d, base, 0, vp(1 << 23),
        vp(1 << 24), vp(1 << 25), None, None)
    assert qkv(R=0) == mad.MAD_EINVAL and qkv(R=9) == mad.MAD_EINVAL
    assert qkv(D=3072) == mad.MAD_ENOTSUP and qkv(d=96) == mad.MAD_ENOTSUP
    assert qkv(Hq=30) == mad.MAD_EINVAL and qkv(x=0) == mad.MAD_EINVAL and qkv(x=(1 << 20) + 2) == mad.MAD_EINVAL
    assert qkv(eps=0.0) == mad.MAD_EINVAL and qkv(base=1.0) == mad.MAD_EINVAL
    lin = lambda R=1, D=2048, N=2048, out=1 << 26, x=1 << 20: lib.mad_linear_residual(
        vp(x), vp(1 << 22), vp(1 << 23), R, D, N, vp(out), None)
    assert lin(D=1024) == mad.MAD_ENOTSUP and lin(N=10) == mad.MAD_EINVAL and lin(R=9) == mad.MAD_EINVAL
    assert lin(out=(1 << 20) + 64) == mad.MAD_EINVAL and "overlaps" in _last_error(mad)
    swi = lambda R=1, D=2048, F=8192, out=1 << 26: lib.mad_rmsnorm_swiglu(
        vp(1 << 20), vp(1 << 21), 1e-5, vp(1 << 22), R, D, F, vp(out), None)
    assert swi(F=6) == mad.MAD_EINVAL and swi(D=8192) == mad.MAD_ENOTSUP and swi(R=0) == mad.MAD_EINVAL
    assert swi(out=(1 << 20) + 16) == mad.MAD_EINVAL


def test_python_binding_rejects_mismatched_tensors(mad):
    """The binding refuses, before any launch, tensors whose shapes would make a
    kernel read or write past them: a batch dimension other than 1 or B, KV
    heads or head_dim that differ between q, the memory, the ring and the new
    token, non-contiguous q/out/x, adaptor weights of the wrong shape."""
    import torch
    bf = torch.bfloat16
    B, Hq, Hkv, d = 2, 8, 2, 64
    q = torch.zeros(B, Hq, d, dtype=bf)
    mk = torch.zeros(B, Hkv, 16, d, dtype=bf)
    rk = torch.zeros(B, Hkv, 32, d, dtype=bf)
    kn = torch.zeros(B, Hkv, d, dtype=bf)
    mem = mad.KV(mk, mk.clone(), [4] * B)
    win = mad.KV(rk, rk.clone(), [3] * B, [0] * B)
    with pytest.raises(ValueError, match="batch dimension"):
        mad.draft_decode_attn(q, mad.KV(torch.zeros(3, Hkv, 16, d, dtype=bf), torch.zeros(3, Hkv, 16, d, dtype=bf),
                                        [4] * B), win)
    with pytest.raises(ValueError, match="KV heads"):
        mad.draft_decode_attn(q, mem, mad.KV(torch.zeros(B, 1, 32, d, dtype=bf), torch.zeros(B, 1, 32, d, dtype=bf),
                                             [3] * B, [0] * B), kn, kn.clone())
    with pytest.raises(ValueError, match="head_dim"):
        mad.draft_decode_attn(q, mem, mad.KV(torch.zeros(B, Hkv, 32, 128, dtype=bf),
                                             torch.zeros(B, Hkv, 32, 128, dtype=bf), [3] * B, [0] * B))
    with pytest.raises(ValueError, match="k_new"):
        mad.draft_decode_attn(q, mem, win, torch.zeros(B, 1, d, dtype=bf), torch.zeros(B, 1, d, dtype=bf))
    with pytest.raises(ValueError, match="contiguous"):
        mad.draft_decode_attn(torch.zeros(B, d, Hq, dtype=bf).transpose(1, 2), mem, win)
    with pytest.raises(ValueError, match="dtype"):
        mad.draft_decode_attn(q.float(), mem, win)
    with pytest.raises(ValueError, match="one entry per row"):
        mad.draft_decode_attn(q, mad.KV(mk, mk.clone(), [4]), win)
    x = torch.zeros(B, 4, Hq * d, dtype=bf)
    with pytest.raises(ValueError, match="w_kv"):
        mad.memory_update(x, torch.zeros(2 * Hkv * d, Hq * d - 64, dtype=bf), [[0] * 4] * B, mem)
    with pytest.raises(ValueError, match="contiguous"):
        mad.memory_update(torch.zeros(B, Hq * d, 4, dtype=bf).transpose(1, 2),
                          torch.zeros(2 * Hkv * d, Hq * d, dtype=bf), [[0] * 4] * B, mem)
    with pytest.raises(ValueError, match="pos"):
        mad.memory_update(x, torch.zeros(2 * Hkv * d, Hq * d, dtype=bf), [[0] * 3] * B, mem)
