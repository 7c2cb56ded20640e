"""Comparison helpers for GPU-vs-oracle parity.

Tolerances (written out here and in each test):
  * bf16 outputs: max |gpu - oracle| <= 2e-2 and relative L2 error <= 1e-2
    (the rel-L2 bound gives the check teeth: with N(0,1) inputs attention
    outputs are small, so a max-abs bound alone would accept a zero output);
  * fp32 outputs and every lse: max |gpu - oracle| <= 1e-5;
  * integer / index outputs: exact;
  * bf16 activations of O(1-10) magnitude (the draft layer's hidden states,
    projections and MLP): |gpu - oracle| <= 2e-2 + 2^-7 |oracle| per element
    (a stored bf16 value carries up to 2^-8 relative rounding; 2^-7 leaves one
    more rounding of margin for the rounded intermediates it is computed
    from) and relative L2 error <= 1e-2.
"""
import numpy as np

BF16_ATOL = 2e-2
BF16_REL_L2 = 1e-2
F32_ATOL = 1e-5
BF16_REL_ELEM = 2.0 ** -7


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
