"""MI355X-native hot path of memory-augmented sliding-window (MASW) drafting.

Thin ctypes binding over libmad.so (C ABI in include/mad.h).  This module
only marshals arguments -- tensor pointers, strides, host length arrays and
the current HIP stream -- into the C entry points; every step of the path
runs in the library's HIP kernels.  PyTorch provides device memory and
streams.  The library is loaded on first use; if libmad.so is missing that
first call raises: there is no fallback.

Entry points (same names as the C ABI, without the ``mad_`` prefix):
    draft_decode_attn   draft decode attention over sink+slots | window ring (+ append)
    memory_update       mirrored K/V projection + RoPE + append of new memory slots
    verify_attn         target (gamma+1)-query verify attention over the full KV
                        (verify_attn_vt: the same over a transposed V cache)
    accept_greedy       greedy accept/reject
"""
import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmad.so")

MAD_OK, MAD_EINVAL, MAD_ENOTSUP, MAD_EHIP, MAD_EWS = 0, -1, -2, -3, -4
MAD_F32, MAD_BF16 = 0, 1
MAD_OP_DECODE, MAD_OP_UPDATE, MAD_OP_VERIFY, MAD_OP_ACCEPT, MAD_OP_ACCEPT_STOCH = 0, 1, 2, 3, 4
MAX_BATCH = 64

_i32p = ctypes.POINTER(ctypes.c_int32)
_u8p = ctypes.POINTER(ctypes.c_uint8)


class _KVView(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("seq_stride", ctypes.c_int64), ("head_stride", ctypes.c_int64),
                ("cap", ctypes.c_int32), ("start", _i32p), ("len", _i32p)]


_LIB = None


def _load_library():
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_30252_amd.build` "
                          "(the hot path has no CPU fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i, f, d, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_double, ctypes.c_size_t
    kvp = ctypes.POINTER(_KVView)
    lib.mad_draft_decode_attn.argtypes = [vp, i, i, i, i, i, f, kvp, kvp, vp, vp, vp, vp, vp, sz, vp]
    lib.mad_memory_update.argtypes = [vp, vp, _i32p, _u8p, i, i, i, i, i, i, d, kvp, vp]
    lib.mad_verify_attn.argtypes = [vp, i, i, i, i, i, i, f, kvp, vp, vp, vp, sz, vp]
    lib.mad_verify_attn_vt.argtypes = [vp, i, i, i, i, i, i, f, vp, vp, ctypes.c_int64, ctypes.c_int64,
                                       ctypes.c_int32, _i32p, vp, vp, vp, sz, vp]
    lib.mad_accept_greedy.argtypes = [vp, i, vp, i, i, i, vp, vp, vp, sz, vp]
    lib.mad_accept_stochastic.argtypes = [vp, vp, vp, vp, i, i, i, vp, vp, vp, sz, vp]
    lib.mad_draft_step_attn.argtypes = [vp, i, i, i, i, i, f, kvp, kvp, vp, vp, _u8p, vp, vp, vp, sz, vp]
    lib.mad_draft_decode_attn_noalloc.argtypes = [vp, i, i, i, i, i, f, kvp, kvp, vp, vp, vp, vp, vp]
    lib.mad_memory_prefill_attn.argtypes = [vp, vp, i, i, i, i, i, f, _i32p, i, i, i, i, i, i, kvp, kvp,
                                            vp, vp, vp, vp, vp]
    lib.mad_rmsnorm_qkv_rope.argtypes = [vp, vp, f, vp, _i32p, i, i, i, i, i, d, i, vp, vp, vp, vp, vp]
    lib.mad_linear_residual.argtypes = [vp, vp, vp, i, i, i, vp, vp]
    lib.mad_rmsnorm_swiglu.argtypes = [vp, vp, f, vp, i, i, i, vp, vp]
    lib.mad_probe_stream_read.argtypes = [vp, sz, vp, i, vp]
    lib.mad_probe_shared_read.argtypes = [vp, sz, vp, i, i, vp]
    lib.mad_probe_empty.argtypes = [i, i, vp]
    lib.mad_probe_handoff_latency.argtypes = [vp, sz, vp, i, vp]
    lib.mad_workspace_bytes.argtypes = [i, i, i, i, i, i, i]
    lib.mad_workspace_bytes.restype = sz
    lib.mad_last_error.restype = ctypes.c_char_p
    lib.mad_version.restype = ctypes.c_char_p
    for fn in ("mad_draft_decode_attn", "mad_memory_update", "mad_verify_attn", "mad_verify_attn_vt", "mad_accept_greedy",
               "mad_accept_stochastic", "mad_draft_step_attn", "mad_draft_decode_attn_noalloc",
               "mad_memory_prefill_attn",
               "mad_rmsnorm_qkv_rope", "mad_linear_residual", "mad_rmsnorm_swiglu", "mad_probe_stream_read",
               "mad_probe_shared_read", "mad_probe_empty", "mad_probe_handoff_latency"):
        getattr(lib, fn).restype = ctypes.c_int
    _LIB = lib
    return lib


class MadError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"libmad error {code}: {msg}")
        self.code = code


def _check(rc):
    if rc != MAD_OK:
        raise MadError(rc, _load_library().mad_last_error().decode())


def version() -> str:
    return _load_library().mad_version().decode()


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return MAD_BF16
    if t.dtype == torch.float32:
        return MAD_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _host_i32(vals, n) -> ctypes.Array:
    arr = (ctypes.c_int32 * max(n, 1))()
    for j, x in enumerate(vals):
        arr[j] = int(x)
    return arr


@dataclass
class KV:
    """A [B, Hkv, cap, d] pair of K/V tensors (any strides with contiguous
    rows) plus per-sequence host lengths and, for a ring, start offsets."""
    k: torch.Tensor
    v: torch.Tensor
    length: Sequence[int]
    start: Optional[Sequence[int]] = None

    def view(self, B, Hkv=None, d=None, dtype=None, device=None, name="kv"):
        """The C view of this pair for a call over B rows.  The batch dimension
        must be B, or 1 (every row then aliases sequence 0: seq_stride 0); the
        KV heads, head_dim, dtype and device must match the call's."""
        k, v = self.k, self.v
        if k.dim() != 4 or k.shape != v.shape or k.stride() != v.stride():
            raise ValueError(f"{name}: K and V must be [B, Hkv, cap, d] tensors with identical strides")
        if k.stride(3) != 1 or k.stride(2) != k.shape[3]:
            raise ValueError(f"{name}: K/V rows must be contiguous")
        if k.shape[0] not in (1, B):
            raise ValueError(f"{name}: batch dimension {k.shape[0]} must be 1 or B={B}")
        if Hkv is not None and k.shape[1] != Hkv:
            raise ValueError(f"{name}: {k.shape[1]} KV heads, the call has {Hkv}")
        if d is not None and k.shape[3] != d:
            raise ValueError(f"{name}: head_dim {k.shape[3]}, the call has {d}")
        if dtype is not None and (k.dtype != dtype or v.dtype != dtype):
            raise ValueError(f"{name}: dtype {k.dtype}, the call has {dtype}")
        if device is not None and (k.device != device or v.device != device):
            raise ValueError(f"{name}: tensors on {k.device}, the call is on {device}")
        if len(self.length) < B or (self.start is not None and len(self.start) < B):
            raise ValueError(f"{name}: lengths/starts need one entry per row ({B})")
        self._len = _host_i32(self.length, B)
        self._start = _host_i32(self.start, B) if self.start is not None else None
        return _KVView(k.data_ptr(), v.data_ptr(), k.stride(0) if k.shape[0] > 1 else 0, k.stride(1),
                       k.shape[2], self._start, self._len)


def _need(cond, msg):
    if not cond:
        raise ValueError(msg)


def _contiguous(**tensors):
    for name, t in tensors.items():
        if t is not None and not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")


def _same_device(dev, **tensors):
    for name, t in tensors.items():
        if t is not None and t.device != dev:
            raise ValueError(f"{name} is on {t.device}, the call is on {dev}")


class Workspace:
    """Zero-filled device scratch for split partials and arrival counters.

    The kernels leave the counters at zero when they finish, so one workspace
    serves any number of calls issued in order on one stream."""

    def __init__(self, device=None):
        self.device = torch.device(device or "cuda")
        self.buf = None

    def get(self, nbytes: int) -> torch.Tensor:
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        return self.buf


_default_ws = {}


def _ws_for(device, nbytes, ws):
    """The caller's workspace, or one kept per (device, stream): calls issued
    in order on one stream may share a workspace, calls on different streams
    must not (their arrival counters and partials would overlap)."""
    if ws is not None:
        if ws.numel() < nbytes:
            raise ValueError(f"workspace of {ws.numel()} bytes < {nbytes} needed")
        return ws
    dev = torch.device(device)
    key = (dev.index, torch.cuda.current_stream(dev).cuda_stream)
    w = _default_ws.get(key)
    if w is None:
        w = _default_ws[key] = Workspace(dev)
    return w.get(nbytes)


def workspace_bytes(op, B=1, Hq=1, Hkv=1, d=64, T=1, max_keys=0) -> int:
    return int(_load_library().mad_workspace_bytes(op, B, Hq, Hkv, d, T, max_keys))


def _decode_args(q, mem, win, k_new, v_new, out, lse, scale):
    """Checks shared by the two decode entry points; returns the marshalled
    arguments (B, Hq, Hkv, d, out, lse, scale, mem view, window view)."""
    _need(q.dim() == 3, "q must be [B, Hq, d]")
    B, Hq, d = q.shape
    _need(mem is not None or win is not None, "mem and win cannot both be None")
    Hkv = (mem.k if mem is not None else win.k).shape[1]
    _need(Hkv >= 1 and Hq % Hkv == 0, f"Hq={Hq} must be a multiple of the KV heads {Hkv}")
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=q.device)
    _need(out.shape == q.shape and out.dtype == q.dtype, "out must match q's shape and dtype")
    _need(lse.shape == (B, Hq) and lse.dtype == torch.float32, "lse must be float32 [B, Hq]")
    _need((k_new is None) == (v_new is None), "k_new and v_new go together")
    if k_new is not None:
        for name, t in (("k_new", k_new), ("v_new", v_new)):
            _need(t.shape == (B, Hkv, d) and t.dtype == q.dtype, f"{name} must be [B, Hkv, d] = {(B, Hkv, d)} "
                  f"of {q.dtype}")
    _contiguous(q=q, out=out, lse=lse, k_new=k_new, v_new=v_new)
    _same_device(q.device, out=out, lse=lse, k_new=k_new, v_new=v_new)
    if scale is None:
        scale = d ** -0.5
    mv = mem.view(B, Hkv, d, q.dtype, q.device, "mem") if mem is not None else None
    wv = win.view(B, Hkv, d, q.dtype, q.device, "win") if win is not None else None
    return B, Hq, Hkv, d, out, lse, scale, mv, wv


def draft_decode_attn(q: torch.Tensor, mem: Optional[KV], win: Optional[KV],
                      k_new: Optional[torch.Tensor] = None, v_new: Optional[torch.Tensor] = None,
                      out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                      scale: Optional[float] = None, ws: Optional[torch.Tensor] = None):
    """q [B, Hq, d] -> (out [B, Hq, d], lse [B, Hq] fp32).

    Attends over mem rows [0, len) then the window ring rows start..start+len-1
    (mod cap) then the new token (k_new/v_new [B, Hkv, d], which is also
    written into the ring at row (start + len) % cap)."""
    B, Hq, Hkv, d, out, lse, scale, mv, wv = _decode_args(q, mem, win, k_new, v_new, out, lse, scale)
    nbytes = workspace_bytes(MAD_OP_DECODE, B, Hq, Hkv, d)
    w = _ws_for(q.device, nbytes, ws)
    rc = _load_library().mad_draft_decode_attn(_ptr(q), B, Hq, Hkv, d, _dtype_code(q), float(scale),
                                   ctypes.byref(mv) if mv is not None else None,
                                   ctypes.byref(wv) if wv is not None else None,
                                   _ptr(k_new), _ptr(v_new), _ptr(out), _ptr(lse),
                                   _ptr(w), w.numel(), _stream(q.device))
    _check(rc)
    return out, lse


def draft_decode_attn_noalloc(q: torch.Tensor, mem: Optional[KV], win: Optional[KV],
                              k_new: Optional[torch.Tensor] = None, v_new: Optional[torch.Tensor] = None,
                              out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                              scale: Optional[float] = None):
    """draft_decode_attn without a workspace: the library's own per-GPU scratch
    holds the split partials (no allocation by the library; out and lse are
    allocated here only when not given).  Calls on one GPU must not overlap."""
    B, Hq, Hkv, d, out, lse, scale, mv, wv = _decode_args(q, mem, win, k_new, v_new, out, lse, scale)
    rc = _load_library().mad_draft_decode_attn_noalloc(_ptr(q), B, Hq, Hkv, d, _dtype_code(q), float(scale),
                                                       ctypes.byref(mv) if mv is not None else None,
                                                       ctypes.byref(wv) if wv is not None else None,
                                                       _ptr(k_new), _ptr(v_new), _ptr(out), _ptr(lse),
                                                       _stream(q.device))
    _check(rc)
    return out, lse


def draft_step_attn(q: torch.Tensor, mem: Optional[KV], win: Optional[KV], k_new: Optional[torch.Tensor],
                    v_new: Optional[torch.Tensor], new_mode, out: Optional[torch.Tensor] = None,
                    lse: Optional[torch.Tensor] = None, scale: Optional[float] = None,
                    ws: Optional[torch.Tensor] = None):
    """draft_decode_attn with a per-row new-token mode (host list of B values):
    0 = no new token, 1 = attend k_new/v_new[b] only, 2 = attend and append it
    to the row's ring.  Rows may alias one sequence's buffers (batch dim 1)."""
    B, Hq, Hkv, d, out, lse, scale, mv, wv = _decode_args(q, mem, win, k_new, v_new, out, lse, scale)
    _need(len(new_mode) == B, "new_mode needs one entry per row")
    modes = (ctypes.c_uint8 * B)(*[int(m) for m in new_mode])
    nbytes = workspace_bytes(MAD_OP_DECODE, B, Hq, Hkv, d)
    w = _ws_for(q.device, nbytes, ws)
    rc = _load_library().mad_draft_step_attn(_ptr(q), B, Hq, Hkv, d, _dtype_code(q), float(scale),
                                             ctypes.byref(mv) if mv is not None else None,
                                             ctypes.byref(wv) if wv is not None else None,
                                             _ptr(k_new), _ptr(v_new), modes, _ptr(out), _ptr(lse),
                                             _ptr(w), w.numel(), _stream(q.device))
    _check(rc)
    return out, lse


def memory_update(x: torch.Tensor, w_kv: torch.Tensor, pos, mem: KV, fire=None, rope_base: float = 500000.0):
    """x [B, n_new, D] slot hidden states, w_kv [2*Hkv*d, D]; pos host [B][n_new].

    Appends the slots' K (rotated at pos) and V at mem rows len[b]..len[b]+n_new-1
    of every firing sequence.  The caller then raises its lengths."""
    _need(x.dim() == 3, "x must be [B, n_new, D]")
    B, n_new, D = x.shape
    Hkv, d = mem.k.shape[1], mem.k.shape[3]
    _need(w_kv.shape == (2 * Hkv * d, D) and w_kv.dtype == x.dtype,
          f"w_kv must be [2*Hkv*d, D] = {(2 * Hkv * d, D)} of {x.dtype}")
    _need(len(pos) == B and all(len(row) == n_new for row in pos), "pos must be [B][n_new]")
    _need(fire is None or len(fire) == B, "fire needs one flag per sequence")
    _contiguous(x=x, w_kv=w_kv)
    _same_device(x.device, w_kv=w_kv)
    mv = mem.view(B, Hkv, d, x.dtype, x.device, "mem")
    flat = [int(p) for row in pos for p in row]
    pos_arr = _host_i32(flat, B * n_new)
    fire_arr = None
    if fire is not None:
        fire_arr = (ctypes.c_uint8 * B)(*[1 if f else 0 for f in fire])
    rc = _load_library().mad_memory_update(_ptr(x), _ptr(w_kv), pos_arr, fire_arr, B, n_new, D, Hkv, d,
                               _dtype_code(x), float(rope_base), ctypes.byref(mv), _stream(x.device))
    _check(rc)


def _verify_out(q, out, lse, scale):
    _need(q.dim() == 4, "q must be [B, T, Hq, d]")
    B, T, Hq, d = q.shape
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((B, T, Hq), dtype=torch.float32, device=q.device)
    _need(out.shape == q.shape and out.dtype == q.dtype, "out must match q")
    _need(lse.shape == (B, T, Hq) and lse.dtype == torch.float32, "lse must be float32 [B, T, Hq]")
    _contiguous(q=q, out=out, lse=lse)
    _same_device(q.device, out=out, lse=lse)
    return out, lse, (d ** -0.5 if scale is None else scale)


def verify_attn(q: torch.Tensor, kv: KV, out=None, lse=None, scale: Optional[float] = None,
                ws: Optional[torch.Tensor] = None):
    """q [B, T, Hq, d]; kv: the verifier's cache as it is, K and V [B, Hkv, cap, d]
    (rows of d), kv.length[b] rows valid with the T new tokens at len-T..len-1.
    Returns (out [B, T, Hq, d], lse [B, T, Hq])."""
    B, T, Hq, d = q.shape
    Hkv = kv.k.shape[1]
    _need(kv.start is None, "the verifier's cache is linear (no ring start)")
    out, lse, scale = _verify_out(q, out, lse, scale)
    view = kv.view(B, Hkv, d, q.dtype, q.device, "kv")
    nbytes = workspace_bytes(MAD_OP_VERIFY, B, Hq, Hkv, d, T)
    w = _ws_for(q.device, nbytes, ws)
    rc = _load_library().mad_verify_attn(_ptr(q), B, T, Hq, Hkv, d, _dtype_code(q), float(scale), ctypes.byref(view),
                                         _ptr(out), _ptr(lse), _ptr(w), w.numel(), _stream(q.device))
    _check(rc)
    return out, lse


def verify_attn_vt(q: torch.Tensor, k: torch.Tensor, vt: torch.Tensor, length, out=None, lse=None,
                   scale: Optional[float] = None, ws: Optional[torch.Tensor] = None):
    """q [B, T, Hq, d]; k [B, Hkv, cap, d]; vt [B, Hkv, d, cap] (values stored
    key-contiguous per feature); the T new tokens sit at rows len-T..len-1.
    Returns (out [B, T, Hq, d], lse [B, T, Hq])."""
    B, T, Hq, d = q.shape
    Hkv, cap = k.shape[1], k.shape[2]
    if vt.shape != (B, Hkv, d, cap) or k.shape != (B, Hkv, cap, d):
        raise ValueError(f"k must be [B, Hkv, cap, d] and vt [B, Hkv, d, cap] = {(B, Hkv, d, cap)}")
    if k.stride(3) != 1 or k.stride(2) != d or vt.stride(3) != 1 or vt.stride(2) != cap:
        raise ValueError("k rows and vt feature runs must be contiguous")
    if k.stride(0) != vt.stride(0) or k.stride(1) != vt.stride(1):
        raise ValueError("k and vt must share sequence and head strides")
    _need(k.dtype == q.dtype and vt.dtype == q.dtype, "k, vt and q share the dtype")
    _need(len(length) == B, "length needs one entry per sequence")
    out, lse, scale = _verify_out(q, out, lse, scale)
    _same_device(q.device, k=k, vt=vt)
    nbytes = workspace_bytes(MAD_OP_VERIFY, B, Hq, Hkv, d, T)
    w = _ws_for(q.device, nbytes, ws)
    rc = _load_library().mad_verify_attn_vt(_ptr(q), B, T, Hq, Hkv, d, _dtype_code(q), float(scale), _ptr(k),
                                            _ptr(vt), k.stride(0) if B > 1 else 0, k.stride(1), cap,
                                            _host_i32(length, B), _ptr(out), _ptr(lse), _ptr(w), w.numel(),
                                            _stream(q.device))
    _check(rc)
    return out, lse


def accept_greedy(logits: torch.Tensor, draft_tok: Optional[torch.Tensor], n_accept=None, next_tok=None,
                  ws: Optional[torch.Tensor] = None):
    """logits [B, T, V] (fp32 or bf16), draft_tok int32 [B, T-1] on the device.
    Returns (n_accept int32 [B], next_tok int32 [B]) on the device."""
    B, T, V = logits.shape
    dev = logits.device
    if n_accept is None:
        n_accept = torch.empty(B, dtype=torch.int32, device=dev)
    if next_tok is None:
        next_tok = torch.empty(B, dtype=torch.int32, device=dev)
    _need(T == 1 or (draft_tok is not None and draft_tok.shape == (B, T - 1) and draft_tok.dtype == torch.int32),
          "draft_tok must be int32 [B, T-1]")
    _need(n_accept.shape == (B,) and next_tok.shape == (B,) and n_accept.dtype == torch.int32
          and next_tok.dtype == torch.int32, "n_accept and next_tok must be int32 [B]")
    _contiguous(logits=logits, draft_tok=draft_tok, n_accept=n_accept, next_tok=next_tok)
    _same_device(dev, draft_tok=draft_tok, n_accept=n_accept, next_tok=next_tok)
    nbytes = workspace_bytes(MAD_OP_ACCEPT, B, 1, 1, 64, T, V)
    w = _ws_for(dev, nbytes, ws)
    rc = _load_library().mad_accept_greedy(_ptr(logits), _dtype_code(logits), _ptr(draft_tok), B, T, V,
                               _ptr(n_accept), _ptr(next_tok), _ptr(w), w.numel(), _stream(dev))
    _check(rc)
    return n_accept, next_tok


def accept_stochastic(p: torch.Tensor, q: Optional[torch.Tensor], draft_tok: Optional[torch.Tensor], u: torch.Tensor,
                      n_accept=None, next_tok=None, ws: Optional[torch.Tensor] = None):
    """p [B, T, V] float32 target probabilities, q [B, T-1, V] float32 draft
    probabilities, draft_tok int32 [B, T-1], u float32 [B, T] uniforms, all on
    the device.  Returns (n_accept int32 [B], next_tok int32 [B])."""
    B, T, V = p.shape
    dev = p.device
    if n_accept is None:
        n_accept = torch.empty(B, dtype=torch.int32, device=dev)
    if next_tok is None:
        next_tok = torch.empty(B, dtype=torch.int32, device=dev)
    _need(p.dtype == torch.float32 and u.shape == (B, T) and u.dtype == torch.float32, "p float32, u float32 [B, T]")
    _need(T == 1 or (q is not None and q.shape == (B, T - 1, V) and q.dtype == torch.float32
                     and draft_tok is not None and draft_tok.shape == (B, T - 1) and draft_tok.dtype == torch.int32),
          "q float32 [B, T-1, V] and draft_tok int32 [B, T-1]")
    _need(n_accept.shape == (B,) and next_tok.shape == (B,) and n_accept.dtype == torch.int32
          and next_tok.dtype == torch.int32, "n_accept and next_tok must be int32 [B]")
    _contiguous(p=p, q=q, draft_tok=draft_tok, u=u, n_accept=n_accept, next_tok=next_tok)
    _same_device(dev, q=q, draft_tok=draft_tok, u=u, n_accept=n_accept, next_tok=next_tok)
    nbytes = workspace_bytes(MAD_OP_ACCEPT_STOCH, B, 1, 1, 64, T, V)
    w = _ws_for(dev, nbytes, ws)
    lib = _load_library()
    rc = lib.mad_accept_stochastic(_ptr(p), _ptr(q), _ptr(draft_tok), _ptr(u), B, T, V, _ptr(n_accept),
                                   _ptr(next_tok), _ptr(w), w.numel(), _stream(dev))
    _check(rc)
    return n_accept, next_tok


def slots_after(t: int, S: int, r: int, u: int = 1) -> int:
    """Slots materialised once raw tokens 0..t-1 are processed (u slots per update)."""
    return 0 if t <= S else (t - S) // (r * u) * u


def memory_prefill_attn(q_raw: torch.Tensor, q_slot: Optional[torch.Tensor], mem: KV, raw: KV, P: Sequence[int],
                        S: int, W: int, r: int, u: int = 1, out_raw: Optional[torch.Tensor] = None,
                        lse_raw: Optional[torch.Tensor] = None, out_slot: Optional[torch.Tensor] = None,
                        lse_slot: Optional[torch.Tensor] = None, scale: Optional[float] = None):
    """The draft's memory-prefill attention over a prefix of P[b] raw tokens.

    q_raw [B, q_cap, Hq, d]; q_slot [B, slot_cap, Hq, d] (row m-1 = slot m) or None;
    mem: sinks then slots (rows 0..S-1, S+m-1); raw: the prefix's K/V (row x = position x).
    Returns (out_raw, lse_raw, out_slot, lse_slot); the slot outputs are None without q_slot."""
    B, q_cap, Hq, d = q_raw.shape
    Hkv = mem.k.shape[1]
    slot_cap = q_slot.shape[1] if q_slot is not None else 0
    if out_raw is None:
        out_raw = torch.empty_like(q_raw)
    if lse_raw is None:
        lse_raw = torch.empty((B, q_cap, Hq), dtype=torch.float32, device=q_raw.device)
    if q_slot is not None:
        if out_slot is None:
            out_slot = torch.empty_like(q_slot)
        if lse_slot is None:
            lse_slot = torch.empty((B, slot_cap, Hq), dtype=torch.float32, device=q_raw.device)
    _need(q_slot is None or (q_slot.dim() == 4 and q_slot.shape[0] == B and q_slot.shape[2:] == q_raw.shape[2:]
                             and q_slot.dtype == q_raw.dtype), "q_slot must be [B, slot_cap, Hq, d] like q_raw")
    _contiguous(q_raw=q_raw, q_slot=q_slot, out_raw=out_raw, lse_raw=lse_raw, out_slot=out_slot, lse_slot=lse_slot)
    _same_device(q_raw.device, q_slot=q_slot, out_raw=out_raw, lse_raw=lse_raw, out_slot=out_slot,
                 lse_slot=lse_slot)
    _need(out_raw.shape == q_raw.shape and lse_raw.shape == (B, q_cap, Hq), "out_raw/lse_raw shapes")
    _need(q_slot is None or (out_slot.shape == q_slot.shape and lse_slot.shape == (B, slot_cap, Hq)),
          "out_slot/lse_slot shapes")
    _need(len(P) == B, "P needs one entry per sequence")
    if scale is None:
        scale = d ** -0.5
    mv = mem.view(B, Hkv, d, q_raw.dtype, q_raw.device, "mem")
    rv = raw.view(B, Hkv, d, q_raw.dtype, q_raw.device, "raw")
    plen = _host_i32(P, B)
    rc = _load_library().mad_memory_prefill_attn(
        _ptr(q_raw), _ptr(q_slot), B, Hq, Hkv, d, _dtype_code(q_raw), float(scale), plen, q_cap, slot_cap,
        S, W, r, u, ctypes.byref(mv), ctypes.byref(rv), _ptr(out_raw), _ptr(lse_raw),
        _ptr(out_slot) if q_slot is not None else None, _ptr(lse_slot) if q_slot is not None else None,
        _stream(q_raw.device))
    _check(rc)
    return out_raw, lse_raw, (out_slot if q_slot is not None else None), (lse_slot if q_slot is not None else None)


def rmsnorm_qkv_rope(x: torch.Tensor, gamma: torch.Tensor, w_qkv: torch.Tensor, pos: Sequence[int], Hq: int,
                     Hkv: int, d: int, q: Optional[torch.Tensor] = None, k: Optional[torch.Tensor] = None,
                     v: Optional[torch.Tensor] = None, xn: Optional[torch.Tensor] = None, eps: float = 1e-5,
                     rope_base: float = 500000.0, kv_from_row0: bool = False):
    """x [R, D] -> q [R, Hq, d], k and v [R, Hkv, d] (q, k rotated at pos), and the
    normalised rows xn [R, D] when given."""
    R, D = x.shape
    if q is None:
        q = torch.empty((R, Hq, d), dtype=x.dtype, device=x.device)
    if k is None:
        k = torch.empty((R, Hkv, d), dtype=x.dtype, device=x.device)
    if v is None:
        v = torch.empty((R, Hkv, d), dtype=x.dtype, device=x.device)
    _need(x.dtype == torch.bfloat16, "the draft-layer maps run in bf16")
    _need(gamma.shape == (D,) and w_qkv.shape == ((Hq + 2 * Hkv) * d, D), "gamma [D], w_qkv [(Hq+2Hkv)d, D]")
    _need(q.shape == (R, Hq, d) and k.shape == (R, Hkv, d) and v.shape == (R, Hkv, d), "q/k/v output shapes")
    _need(xn is None or xn.shape == (R, D), "xn must be [R, D]")
    _need(len(pos) == R, "pos needs one entry per row")
    _contiguous(x=x, gamma=gamma, w_qkv=w_qkv, q=q, k=k, v=v, xn=xn)
    _same_device(x.device, gamma=gamma, w_qkv=w_qkv, q=q, k=k, v=v, xn=xn)
    rc = _load_library().mad_rmsnorm_qkv_rope(_ptr(x), _ptr(gamma), float(eps), _ptr(w_qkv), _host_i32(pos, R), R,
                                              D, Hq, Hkv, d, float(rope_base), 1 if kv_from_row0 else 0, _ptr(q),
                                              _ptr(k), _ptr(v), _ptr(xn), _stream(x.device))
    _check(rc)
    return q, k, v


def linear_residual(x: torch.Tensor, w: torch.Tensor, res: torch.Tensor, out: Optional[torch.Tensor] = None):
    """out [R, N] = res + x W^T."""
    R, D = x.shape
    N = w.shape[0]
    if out is None:
        out = torch.empty((R, N), dtype=x.dtype, device=x.device)
    _need(x.dtype == torch.bfloat16 and w.shape == (N, D) and res.shape == (R, N) and out.shape == (R, N),
          "x [R, D], w [N, D], res and out [R, N], bf16")
    _contiguous(x=x, w=w, res=res, out=out)
    _same_device(x.device, w=w, res=res, out=out)
    _check(_load_library().mad_linear_residual(_ptr(x), _ptr(w), _ptr(res), R, D, N, _ptr(out), _stream(x.device)))
    return out


def rmsnorm_swiglu(x: torch.Tensor, gamma: torch.Tensor, w_gate_up: torch.Tensor,
                   out: Optional[torch.Tensor] = None, eps: float = 1e-5):
    """out [R, F] = silu(xn W_gate^T) * (xn W_up^T), xn = rmsnorm(x) * gamma."""
    R, D = x.shape
    Fd = w_gate_up.shape[0] // 2
    if out is None:
        out = torch.empty((R, Fd), dtype=x.dtype, device=x.device)
    _need(x.dtype == torch.bfloat16 and gamma.shape == (D,) and w_gate_up.shape == (2 * Fd, D)
          and out.shape == (R, Fd), "x [R, D], gamma [D], w_gate_up [2F, D], out [R, F], bf16")
    _contiguous(x=x, gamma=gamma, w_gate_up=w_gate_up, out=out)
    _same_device(x.device, gamma=gamma, w_gate_up=w_gate_up, out=out)
    _check(_load_library().mad_rmsnorm_swiglu(_ptr(x), _ptr(gamma), float(eps), _ptr(w_gate_up), R, D, Fd,
                                              _ptr(out), _stream(x.device)))
    return out


# ---- measurement aids (the benchmark's probes; not part of the attention path) ----

def probe_stream_read(src: torch.Tensor, sink: Optional[torch.Tensor] = None, n_workgroups: int = 1024):
    """Stream-read the bytes of a contiguous device tensor (a contiguous range per workgroup,
    nontemporal 16-byte loads)."""
    _need(src.is_contiguous() and src.numel() * src.element_size() % 16 == 0, "src: contiguous, bytes % 16 == 0")
    _check(_load_library().mad_probe_stream_read(_ptr(src), src.numel() * src.element_size(), _ptr(sink),
                                                 n_workgroups, _stream(src.device)))


def probe_shared_read(src: torch.Tensor, sink: Optional[torch.Tensor] = None, n_workgroups: int = 256,
                      threads: int = 256):
    """Every workgroup reads all bytes of a contiguous device tensor (L2-resident after the first touch)."""
    _need(src.is_contiguous() and src.numel() * src.element_size() % 16 == 0, "src: contiguous, bytes % 16 == 0")
    _check(_load_library().mad_probe_shared_read(_ptr(src), src.numel() * src.element_size(), _ptr(sink),
                                                 n_workgroups, threads, _stream(src.device)))


def probe_empty(n_workgroups: int = 256, threads: int = 256, device=None):
    """Launch an empty kernel (the launch floor)."""
    dev = torch.device(device or "cuda")
    _check(_load_library().mad_probe_empty(n_workgroups, threads, _stream(dev)))


def probe_handoff_latency(buf: torch.Tensor, cycles: torch.Tensor, reps: int):
    """Time the hand-off primitives (see include/mad.h); cycles: int64 [8, reps] on the device."""
    _need(cycles.dtype == torch.int64 and cycles.shape == (8, reps) and cycles.is_contiguous(), "cycles [8, reps] int64")
    _check(_load_library().mad_probe_handoff_latency(_ptr(buf), buf.numel() * buf.element_size(), _ptr(cycles),
                                                     reps, _stream(buf.device)))
