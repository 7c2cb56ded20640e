"""Comparison helpers for GPU-vs-oracle parity.

Tolerances (written out here and in each test):
  * bf16 outputs: max |gpu - oracle| <= 2e-2 and relative L2 error <= 1e-2
    (the rel-L2 bound gives the check teeth: with N(0,1) inputs attention
    outputs are small, so a max-abs bound alone would accept a zero output);
  * fp32 outputs: max |gpu - oracle| <= 1e-5;
  * every lse, per row: |gpu - oracle| <= 1e-5 + 2^-24 (2 sqrt(d) A + 8 |lse|),
    A = scale * max_j sum_i |q_i k_ji| over the keys the row attends (lse_tol:
    the sqrt(d)-scaled rounding of the fp32 score sums, which the lse inherits
    as a convex combination, with a factor 2 of margin, plus the roundings of
    the maximum, the exponential sum, log2 and the final ln 2 multiply at the
    magnitude of lse);
  * integer / index outputs: exact;
  * bf16 activations of O(1-10) magnitude (the draft layer's hidden states,
    projections and MLP): |gpu - oracle| <= 2e-2 + 2^-7 |oracle| per element
    (a stored bf16 value carries up to 2^-8 relative rounding; 2^-7 leaves one
    more rounding of margin for the rounded intermediates it is computed
    from) and relative L2 error <= 1e-2.
"""
import math

import numpy as np

BF16_ATOL = 2e-2
BF16_REL_L2 = 1e-2
F32_ATOL = 1e-5
BF16_REL_ELEM = 2.0 ** -7
LSE_FLOOR = 1e-5
U32 = 2.0 ** -24


def to_np(t):
    return t.detach().to("cpu").double().numpy()


def check(got, ref, atol, rel_l2=None, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{what}: shape {got.shape} vs {ref.shape}"
    fin_ref = np.isfinite(ref)
    # non-finite reference entries (e.g. lse = -inf of an empty key set) must match exactly
    assert np.array_equal(got[~fin_ref], ref[~fin_ref]), f"{what}: non-finite entries differ"
    assert np.all(np.isfinite(got[fin_ref])), f"{what}: non-finite values in the GPU result"
    err = np.abs(got[fin_ref] - ref[fin_ref])
    max_abs = float(err.max()) if err.size else 0.0
    assert max_abs <= atol, f"{what}: max abs error {max_abs:.3e} > {atol:.1e}"
    if rel_l2 is not None:
        den = float(np.linalg.norm(ref[fin_ref]))
        num = float(np.linalg.norm(got[fin_ref] - ref[fin_ref]))
        rel = num / den if den > 0 else num
        assert rel <= rel_l2, f"{what}: relative L2 error {rel:.3e} > {rel_l2:.1e}"
        return max_abs, rel
    return max_abs, None


def check_out(got, ref, dtype_is_bf16, what="out"):
    if dtype_is_bf16:
        return check(got, ref, BF16_ATOL, BF16_REL_L2, what)
    return check(got, ref, F32_ATOL, None, what)


def check_act(got, ref, what="activation"):
    """bf16 activations: per element |got - ref| <= BF16_ATOL + BF16_REL_ELEM |ref|, and rel-L2."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{what}: shape {got.shape} vs {ref.shape}"
    assert np.all(np.isfinite(got)), f"{what}: non-finite values in the GPU result"
    err = np.abs(got - ref)
    bound = BF16_ATOL + BF16_REL_ELEM * np.abs(ref)
    worst = int(np.argmax(err - bound))
    assert np.all(err <= bound), (f"{what}: error {err.flat[worst]:.3e} > {bound.flat[worst]:.3e} "
                                  f"at |ref| {abs(ref.flat[worst]):.3e}")
    den = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(got - ref)) / den if den > 0 else float(np.linalg.norm(got))
    assert rel <= BF16_REL_L2, f"{what}: relative L2 error {rel:.3e} > {BF16_REL_L2:.1e}"
    return float(err.max()), rel


def lse_tol(A, lse_ref, d):
    """Per-row lse bound: 1e-5 + 2^-24 (2 sqrt(d) A + 8 |lse|) (see the module docstring)."""
    A = np.asarray(A, dtype=np.float64)
    ref = np.asarray(lse_ref, dtype=np.float64)
    return LSE_FLOOR + U32 * (2.0 * math.sqrt(d) * A + 8.0 * np.abs(np.where(np.isfinite(ref), ref, 0.0)))


def abs_score(q, k, scale):
    """A for the rows q [G, d] over one key list k [n, d]: scale * max_j |q| . |k_j| (0 for no keys)."""
    q = np.abs(np.asarray(q, dtype=np.float64))
    k = np.abs(np.asarray(k, dtype=np.float64))
    if k.shape[0] == 0:
        return np.zeros(q.shape[0])
    return scale * (q @ k.T).max(axis=1)


def abs_score_batched(q, K, n, scale):
    """A for q [B, Hq, d] over K [B, Hkv, nmax, d] with rows 0..n[b]-1 (head h reads KV head h // G)."""
    q = np.asarray(q, dtype=np.float64)
    B, Hq, d = q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    A = np.zeros((B, Hq))
    for b in range(B):
        for c in range(Hkv):
            A[b, c * G:(c + 1) * G] = abs_score(q[b, c * G:(c + 1) * G], K[b, c, : int(n[b])], scale)
    return A


def abs_score_verify(q, k, length, scale):
    """A for verify: q [B, T, Hq, d], k [B, Hkv, cap, d]; query t sees rows 0 .. len-T+t."""
    q = np.abs(np.asarray(q, dtype=np.float64))
    B, T, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    A = np.zeros((B, T, Hq))
    for b in range(B):
        n = int(length[b])
        for c in range(Hkv):
            s = np.abs(np.asarray(k[b, c, :n], dtype=np.float64)) @ q[b, :, c * G:(c + 1) * G].reshape(T * G, d).T
            s = s.reshape(n, T, G)
            for t in range(T):
                A[b, t, c * G:(c + 1) * G] = scale * s[: n - T + t + 1, t].max(axis=0)
    return A


def check_lse(got, ref, A, d, what="lse"):
    """Per-row lse comparison within lse_tol; non-finite reference entries must match exactly."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{what}: shape {got.shape} vs {ref.shape}"
    fin = np.isfinite(ref)
    assert np.array_equal(got[~fin], ref[~fin]), f"{what}: non-finite entries differ"
    assert np.all(np.isfinite(got[fin])), f"{what}: non-finite values in the GPU result"
    tol = np.broadcast_to(lse_tol(A, ref, d), ref.shape)
    err = np.where(fin, np.abs(got - np.where(fin, ref, 0.0)), 0.0)
    worst = int(np.argmax(err - tol))
    assert np.all(err <= tol), (f"{what}: error {err.flat[worst]:.3e} > {tol.flat[worst]:.3e} "
                                f"at |lse| {abs(ref.flat[worst]):.2f}")
    return float(err.max()) if err.size else 0.0
