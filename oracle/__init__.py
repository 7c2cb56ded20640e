"""fp64 CPU oracle for the MASW hot path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the CPU-baseline leg of the
benchmark may import this package.  The product (the HIP library and its
Python binding) never does, and this package never imports the product.

The arithmetic lives in ``oracle.c`` (plain C, double precision, textbook
definitions, no blocking or online rescaling).  This module only marshals
numpy arrays into it, and composes two of its routines into the memory-slot
K/V materialisation:

    memory_update = oracle_project (Sec. 3.2 projection equations)
                    followed by oracle_rope on the K half only, at the slot's
                    position id (Sec. 3.2, memory update cycle: a slot shares
                    the position id of the raw token after it).

``accept_stochastic`` wraps the rejection-sampling rule (oracle.c).

``rmsnorm``, ``silu``, ``bf16_round`` and ``decoder_layer`` give one draft
decoder layer around the attention (a pre-norm Llama-family layer: RMSNorm,
Q/K/V projection with RoPE, attention supplied by the caller, output
projection and residual, RMSNorm, SwiGLU MLP and residual): slot tokens run
through the same blocks (Sec. 3.2), and the layer's weights are the draft's
per-token weight stream (Sec. 2.3, Eq. latency_decomp).

``memory_prefill`` is the draft's memory-prefill attention (Sec. 3.3 prefill;
the appendix on memory prefill): the prefill mask applies the write policy of
decoding, so each query of the pass attends over the set ``masw_sets`` gives
it -- a raw token its decode-time view, a slot its write scope -- and the
attention itself is oracle_attend over that explicit key list.

``masw_sets`` holds the visible-set simulator written from the paper's set
definitions (Sec. 3.1 and 3.2).

Every function here has a pin in ``tests/test_oracle_pins.py``.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_fp = ctypes.POINTER(ctypes.c_float)
_ip = ctypes.POINTER(ctypes.c_int)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    i, d = ctypes.c_int, ctypes.c_double
    lib.oracle_attend.argtypes = [i, i, _dp, i, _dp, _dp, d, _dp, _dp, _dp]
    lib.oracle_attend_batched.argtypes = [i, i, i, i, _dp, i, _ip, _dp, _dp, d, _dp, _dp]
    lib.oracle_verify.argtypes = [i, i, i, i, i, _dp, i, _ip, _dp, _dp, d, _dp, _dp]
    lib.oracle_project.argtypes = [i, i, i, _dp, _dp, _dp]
    lib.oracle_rope.argtypes = [i, i, i, _dp, _ip, d]
    lib.oracle_argmax.argtypes = [i, i, _fp, _ip]
    lib.oracle_accept_greedy.argtypes = [i, i, i, _fp, _ip, _ip, _ip]
    lib.oracle_accept_stochastic.argtypes = [i, i, i, _fp, _fp, _ip, _fp, _ip, _ip]
    lib.oracle_accept_stochastic.restype = None
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_threads.restype = None
    for f in ("oracle_attend", "oracle_attend_batched", "oracle_verify", "oracle_project",
              "oracle_rope", "oracle_argmax", "oracle_accept_greedy"):
        getattr(lib, f).restype = None
    _lib = lib
    return lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a, t):
    return a.ctypes.data_as(t)


def num_threads():
    """OpenMP threads the batched oracle routines run on."""
    return int(_load().oracle_num_threads())


def set_threads(n):
    """OpenMP threads of the batched oracle routines from now on (timing only)."""
    _load().oracle_set_threads(int(n))


def attend(q, k, v, scale, with_wsum=False):
    """Attention of the G query rows q [G, d] over one key list k, v [n, d].

    Returns (o [G, d], lse [G]) and, if asked, the sum of the normalised
    softmax weights per row (exactly 1 in real arithmetic)."""
    lib = _load()
    q, k, v = _f64(q), _f64(k), _f64(v)
    G, d = q.shape
    n = k.shape[0]
    assert k.shape == (n, d) and v.shape == (n, d)
    o = np.zeros((G, d))
    lse = np.zeros(G)
    ws = np.zeros(G)
    lib.oracle_attend(G, d, _ptr(q, _dp), n, _ptr(k, _dp), _ptr(v, _dp), float(scale),
                      _ptr(o, _dp), _ptr(lse, _dp), _ptr(ws, _dp))
    return (o, lse, ws) if with_wsum else (o, lse)


def attend_batched(q, k, v, n, scale):
    """q [B, Hq, d]; k, v [B, Hkv, nmax, d] with rows 0..n[b]-1 used.

    Returns o [B, Hq, d], lse [B, Hq]; head h reads KV head h // (Hq // Hkv)."""
    lib = _load()
    q, k, v, n = _f64(q), _f64(k), _f64(v), _i32(n)
    B, Hq, d = q.shape
    _, Hkv, nmax, _ = k.shape
    o = np.zeros((B, Hq, d))
    lse = np.zeros((B, Hq))
    lib.oracle_attend_batched(B, Hq, Hkv, d, _ptr(q, _dp), nmax, _ptr(n, _ip), _ptr(k, _dp),
                              _ptr(v, _dp), float(scale), _ptr(o, _dp), _ptr(lse, _dp))
    return o, lse


def verify(q, k, v, length, scale):
    """q [B, T, Hq, d]; k, v [B, Hkv, cap, d] (natural row layout) with the T
    new tokens at rows len-T..len-1.  Returns o [B, T, Hq, d], lse [B, T, Hq]."""
    lib = _load()
    q, k, v, length = _f64(q), _f64(k), _f64(v), _i32(length)
    B, T, Hq, d = q.shape
    _, Hkv, cap, _ = k.shape
    o = np.zeros((B, T, Hq, d))
    lse = np.zeros((B, T, Hq))
    lib.oracle_verify(B, T, Hq, Hkv, d, _ptr(q, _dp), cap, _ptr(length, _ip), _ptr(k, _dp),
                      _ptr(v, _dp), float(scale), _ptr(o, _dp), _ptr(lse, _dp))
    return o, lse


def project(x, w):
    """y = x W^T for x [R, D], w [N, D]."""
    lib = _load()
    x, w = _f64(x), _f64(w)
    R, D = x.shape
    N = w.shape[0]
    assert w.shape[1] == D
    y = np.zeros((R, N))
    lib.oracle_project(R, D, N, _ptr(x, _dp), _ptr(w, _dp), _ptr(y, _dp))
    return y


def rope(k, pos, base):
    """Rotate-half RoPE of k [R, H, d] at integer positions pos [R] (returns a copy)."""
    lib = _load()
    k = _f64(k).copy()
    pos = _i32(pos)
    R, H, d = k.shape
    lib.oracle_rope(R, H, d, _ptr(k, _dp), _ptr(pos, _ip), float(base))
    return k


def memory_update(x, w, pos, hkv, d, base):
    """K/V of new memory slots from their hidden states.

    x [R, D] slot hidden states, w [2*hkv*d, D] = [W_K,g rows ; W_V,g rows],
    pos [R] position ids.  Returns (k [R, hkv, d], v [R, hkv, d]): the K half
    is rotated at pos, the V half is not."""
    y = project(x, w)
    R = y.shape[0]
    k = y[:, : hkv * d].reshape(R, hkv, d)
    v = y[:, hkv * d:].reshape(R, hkv, d)
    return rope(k, pos, base), v.copy()


def argmax(logits):
    """Row argmax of float32 logits [rows, V] (ties -> lowest, NaN highest)."""
    lib = _load()
    x = np.ascontiguousarray(logits, dtype=np.float32)
    rows, V = x.shape
    out = np.zeros(rows, dtype=np.int32)
    lib.oracle_argmax(rows, V, _ptr(x, _fp), _ptr(out, _ip))
    return out


def accept_greedy(logits, draft):
    """logits [B, T, V] float32, draft [B, T-1] int -> (n_accept [B], next [B])."""
    lib = _load()
    x = np.ascontiguousarray(logits, dtype=np.float32)
    B, T, V = x.shape
    dr = _i32(draft).reshape(B, T - 1) if T > 1 else np.zeros((B, 0), np.int32)
    dr = np.ascontiguousarray(dr)
    na = np.zeros(B, dtype=np.int32)
    nx = np.zeros(B, dtype=np.int32)
    lib.oracle_accept_greedy(B, T, V, _ptr(x, _fp), _ptr(dr, _ip), _ptr(na, _ip), _ptr(nx, _ip))
    return na, nx


def accept_stochastic(p, q, draft, u):
    """p [B, T, V], q [B, T-1, V] float32 probabilities, draft [B, T-1] int,
    u [B, T] float32 uniforms -> (n_accept [B], next [B])."""
    lib = _load()
    p = np.ascontiguousarray(p, dtype=np.float32)
    B, T, V = p.shape
    q = np.ascontiguousarray(q, dtype=np.float32).reshape(B, T - 1, V) if T > 1 else np.zeros((B, 0, V), np.float32)
    dr = np.ascontiguousarray(_i32(draft).reshape(B, T - 1)) if T > 1 else np.zeros((B, 0), np.int32)
    u = np.ascontiguousarray(u, dtype=np.float32).reshape(B, T)
    na = np.zeros(B, dtype=np.int32)
    nx = np.zeros(B, dtype=np.int32)
    lib.oracle_accept_stochastic(B, T, V, _ptr(p, _fp), _ptr(np.ascontiguousarray(q), _fp), _ptr(dr, _ip),
                                 _ptr(u, _fp), _ptr(na, _ip), _ptr(nx, _ip))
    return na, nx


def memory_prefill(q_raw, q_slot, mem_k, mem_v, raw_k, raw_v, P, S, W, r, u, scale, raw_idx=None, slot_idx=None):
    """Memory-prefill attention of one sequence.

    q_raw [>=P, Hq, d]; q_slot [>=M, Hq, d] (row m-1 = slot m) or None;
    mem_k/mem_v [Hkv, >=S+M, d] (sinks in rows 0..S-1, slot m in row S+m-1);
    raw_k/raw_v [Hkv, >=P, d] (position x in row x); M = slots materialised by
    the prefix.  raw_idx / slot_idx restrict the queries computed (default:
    all).  Returns dicts {p: (o [Hq, d], lse [Hq])} and {m: (o, lse)}."""
    from .masw_sets import MaswSets
    sets = MaswSets(S, W, r, u)
    M = sets.slots_after(P)
    Hq = q_raw.shape[1]
    Hkv = mem_k.shape[0]
    G = Hq // Hkv

    def run(qrows, view):
        mrows = list(view.sink) + [S + m - 1 for m in view.slots]
        rrows = list(view.window)
        o = np.zeros((Hq, qrows.shape[1]))
        lse = np.zeros(Hq)
        for c in range(Hkv):
            d = mem_k.shape[-1]
            K = np.concatenate([_f64(mem_k[c][mrows]).reshape(len(mrows), d),
                                _f64(raw_k[c][rrows]).reshape(len(rrows), d)])
            V = np.concatenate([_f64(mem_v[c][mrows]).reshape(len(mrows), d),
                                _f64(raw_v[c][rrows]).reshape(len(rrows), d)])
            o[c * G:(c + 1) * G], lse[c * G:(c + 1) * G] = attend(qrows[c * G:(c + 1) * G], K, V, scale)
        return o, lse

    raw_out = {p: run(_f64(q_raw[p]), sets.raw_view(p)) for p in (range(P) if raw_idx is None else raw_idx)}
    slot_out = {}
    if q_slot is not None:
        for m in (range(1, M + 1) if slot_idx is None else slot_idx):
            slot_out[m] = run(_f64(q_slot[m - 1]), sets.slot_scope(m))
    return raw_out, slot_out


def rmsnorm(x, gamma, eps):
    """Per row: x / sqrt(mean(x^2) + eps) * gamma."""
    x = _f64(x)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * _f64(gamma)


def silu(x):
    """x * sigmoid(x)."""
    x = _f64(x)
    return x / (1.0 + np.exp(-x))


def bf16_round(a):
    """Values rounded to bfloat16 (nearest, ties to even), returned as float64:
    the float32 value, then the low 16 bits of its pattern rounded away."""
    f = np.ascontiguousarray(a, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def decoder_layer(x, params, pos, attend_rows, rnd=None):
    """One pre-norm decoder layer for the rows x [R, D] at position ids pos [R].

    params: gamma1 [D], w_qkv [(Hq + 2 Hkv) d, D] (W_q, W_k, W_v rows), w_o
    [D, Hq d], gamma2 [D], w_gate_up [2F, D] (W_gate, W_up rows), w_down [D, F],
    and Hq, Hkv, d, base, eps.  attend_rows(q [R, Hq, d], k [R, Hkv, d],
    v [R, Hkv, d], xn [R, D]) -> o [R, Hq, d] is the attention of each row
    over its own key set.  rnd, if given, is applied to every stored
    intermediate (the layer's tensors are held in that precision).
    Returns a dict of xn, q, k, v, o, h, a, y."""
    rnd = rnd or (lambda t: t)
    Hq, Hkv, d = params["Hq"], params["Hkv"], params["d"]
    R = x.shape[0]
    x = _f64(x)
    xn = rnd(rmsnorm(x, params["gamma1"], params["eps"]))
    qkv = project(xn, params["w_qkv"])
    q = rnd(rope(qkv[:, :Hq * d].reshape(R, Hq, d), pos, params["base"]))
    k = rnd(rope(qkv[:, Hq * d:(Hq + Hkv) * d].reshape(R, Hkv, d), pos, params["base"]))
    v = rnd(qkv[:, (Hq + Hkv) * d:].reshape(R, Hkv, d))
    o = rnd(_f64(attend_rows(q, k, v, xn)))
    h = rnd(x + project(o.reshape(R, Hq * d), params["w_o"]))
    hn = rnd(rmsnorm(h, params["gamma2"], params["eps"]))
    gu = project(hn, params["w_gate_up"])
    F = gu.shape[1] // 2
    a = rnd(silu(gu[:, :F]) * gu[:, F:])
    y = rnd(h + project(a, params["w_down"]))
    return {"xn": xn, "q": q, "k": k, "v": v, "o": o, "h": h, "a": a, "y": y}
