"""The RoPE angle reduction of the device helpers (fp64 angle pos * theta_j
reduced modulo 2 pi before the single-precision sine and cosine), built for the
host and compared with the exact reduction in 80-digit decimal arithmetic, at
every frequency of head_dim 64 and 128 (base 500000) and positions up to 2^20.
A wrong low part of 2 pi shows up as an error growing with the position."""
import ctypes
import decimal
import os
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _pi(prec):
    """pi by Machin's formula, 16 atan(1/5) - 4 atan(1/239), in decimal arithmetic."""
    decimal.getcontext().prec = prec + 10

    def atan_inv(x):
        x = decimal.Decimal(x)
        term, total, k, x2 = 1 / x, 1 / x, 1, x * x
        while True:
            term /= -x2
            nxt = term / (2 * k + 1)
            if abs(nxt) < decimal.Decimal(10) ** (-prec - 5):
                return total
            total += nxt
            k += 1

    return 16 * atan_inv(5) - 4 * atan_inv(239)


@pytest.fixture(scope="module")
def reduce_lib(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("rope") / "rope_reduce.so")
    hipcc = "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    subprocess.run([hipcc, "--offload-arch=gfx950", "-O2", "-std=c++17", "-fPIC", "-shared", "-o", out,
                    os.path.join(ROOT, "tests", "rope_reduce_host.cpp")], check=True, capture_output=True)
    lib = ctypes.CDLL(out)
    lib.rope_reduce_many.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
    return lib


def test_reduction_matches_exact_modulo_two_pi(reduce_lib):
    two_pi = 2 * _pi(80)
    base = 500000.0
    pos = np.array([1, 7, 1000, 4100, 4104, 32768, 65537, 131071, 500000, 1 << 20], dtype=np.float64)
    angles = []
    for d in (64, 128):
        theta = np.array([base ** (-2.0 * j / d) for j in range(d // 2)])
        angles.append((pos[:, None] * theta[None, :]).ravel())
    a = np.ascontiguousarray(np.concatenate(angles))
    r = np.empty_like(a)
    reduce_lib.rope_reduce_many(a.ctypes.data, r.ctypes.data, a.size)
    worst = 0.0
    for ai, ri in zip(a.tolist(), r.tolist()):
        n = round(ai * 0.15915494309189535)            # the same quotient the helper takes
        exact = decimal.Decimal(ai) - n * two_pi
        err = abs(float(decimal.Decimal(ri) - exact))
        worst = max(worst, err)
        assert abs(ri) <= 3.1416 + 1e-12
    # two roundings of values below 4 (2^-51 each), nothing that grows with n
    assert worst <= 1e-15, worst
