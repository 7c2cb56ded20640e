"""Pins of the oracle's draft decoder layer (RMSNorm, Q/K/V with RoPE,
attention, output projection + residual, RMSNorm, SwiGLU MLP + residual).

Each primitive is checked against torch's own routine; the composition is
checked against a layer written with torch's functional ops in float64 (RoPE
as complex rotation, causal scaled_dot_product_attention with the GQA heads
repeated), on a short sequence whose rows attend causally to each other.
"""
import math

import numpy as np
import torch
import torch.nn.functional as F

import oracle


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 96)) * 3.0
    g = rng.standard_normal(96)
    ref = F.rms_norm(torch.from_numpy(x), (96,), weight=torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(x, g, 1e-5), ref, rtol=1e-13, atol=1e-13)
    # a constant row normalises to sign(c) * gamma (up to eps)
    np.testing.assert_allclose(oracle.rmsnorm(np.full((1, 8), -2.0), np.arange(8.0), 0.0)[0], -np.arange(8.0))


def test_silu_matches_torch():
    x = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(oracle.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-14, atol=1e-300)


def test_bf16_round_matches_torch_conversion():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(10000) * 10.0 ** rng.integers(-8, 8, 10000),
                        [0.0, -0.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8), 65504.0, 1e-40]])
    ref = torch.from_numpy(x).to(torch.float32).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(oracle.bf16_round(x), ref)


def _torch_layer(x, p, pos):
    """The same layer from torch's functional ops, float64, causal over the rows."""
    Hq, Hkv, d, base, eps = p["Hq"], p["Hkv"], p["d"], p["base"], p["eps"]
    t = {k: torch.from_numpy(np.asarray(v)) for k, v in p.items() if isinstance(v, np.ndarray)}
    X = torch.from_numpy(x)
    T = X.shape[0]
    xn = F.rms_norm(X, (X.shape[1],), weight=t["gamma1"], eps=eps)
    qkv = F.linear(xn, t["w_qkv"])
    q = qkv[:, :Hq * d].reshape(T, Hq, d)
    k = qkv[:, Hq * d:(Hq + Hkv) * d].reshape(T, Hkv, d)
    v = qkv[:, (Hq + Hkv) * d:].reshape(T, Hkv, d)
    theta = base ** (-2.0 * torch.arange(d // 2, dtype=torch.float64) / d)
    rot = torch.polar(torch.ones(T, d // 2, dtype=torch.float64), torch.tensor(pos, dtype=torch.float64)[:, None] * theta)

    def rope(z):
        c = torch.complex(z[..., :d // 2], z[..., d // 2:]) * rot[:, None, :]
        return torch.cat([c.real, c.imag], dim=-1)
    q, k = rope(q), rope(k)
    G = Hq // Hkv
    o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1).repeat_interleave(G, 0),
                                       v.transpose(0, 1).repeat_interleave(G, 0), is_causal=True,
                                       scale=1 / math.sqrt(d)).transpose(0, 1)
    h = X + F.linear(o.reshape(T, Hq * d), t["w_o"])
    hn = F.rms_norm(h, (h.shape[1],), weight=t["gamma2"], eps=eps)
    gu = F.linear(hn, t["w_gate_up"])
    Fd = gu.shape[1] // 2
    return (h + F.linear(F.silu(gu[:, :Fd]) * gu[:, Fd:], t["w_down"])).numpy()


def test_decoder_layer_matches_a_torch_layer():
    rng = np.random.default_rng(2)
    D, Hq, Hkv, d, Fd, T = 64, 4, 2, 16, 96, 7
    p = {"gamma1": 1 + 0.1 * rng.standard_normal(D), "w_qkv": 0.2 * rng.standard_normal(((Hq + 2 * Hkv) * d, D)),
         "w_o": 0.2 * rng.standard_normal((D, Hq * d)), "gamma2": 1 + 0.1 * rng.standard_normal(D),
         "w_gate_up": 0.2 * rng.standard_normal((2 * Fd, D)), "w_down": 0.2 * rng.standard_normal((D, Fd)),
         "Hq": Hq, "Hkv": Hkv, "d": d, "base": 10000.0, "eps": 1e-5}
    x = rng.standard_normal((T, D))
    pos = [3, 4, 5, 9, 10, 11, 20]   # position ids need not be consecutive

    def causal(q, k, v, xn):
        o = np.zeros_like(q)
        for t in range(T):
            for c in range(Hkv):
                o[t, c * 2:(c + 1) * 2] = oracle.attend(q[t, c * 2:(c + 1) * 2], k[:t + 1, c], v[:t + 1, c], d ** -0.5)[0]
        return o
    got = oracle.decoder_layer(x, p, pos, causal)["y"]
    np.testing.assert_allclose(got, _torch_layer(x, p, pos), rtol=1e-11, atol=1e-11)
