"""GPU parity of mad_memory_update against the fp64 oracle.

The oracle composes the mirrored projection (x W^T) with rotate-half RoPE of
the K half at each slot's position id.  Besides element-wise parity the
tests check the append-only property (rows below len are bit-identical and
rows past the new ones untouched) and that sequences with fire = 0 are left
alone.  Tolerances: see parity.py.
"""
import numpy as np
import pytest
import torch

from parity import check_out, to_np

pytestmark = pytest.mark.gpu

BASE = 500000.0


def _case(dtype, B, n_new, D, Hkv, d, mlen, cap, pos, fire=None, seed=0, wstd=0.02):
    import oracle
    import paper_2608_30252_amd as mad
    from paper_2608_30252_amd import synth
    dev = torch.device("cuda")
    mlen = list(mlen) if hasattr(mlen, "__len__") else [mlen] * B
    s = 1000 * seed
    x = synth.normal((B, n_new, D), s + 1, dtype=dtype)
    w = synth.normal((2 * Hkv * d, D), s + 2, std=wstd, dtype=dtype)
    mk = synth.normal((B, Hkv, cap, d), s + 3, dtype=dtype)
    mv = synth.normal((B, Hkv, cap, d), s + 4, dtype=dtype)
    g_mk, g_mv = mk.to(dev), mv.to(dev)
    mad.memory_update(x.to(dev), w.to(dev), pos, mad.KV(g_mk, g_mv, mlen), fire=fire, rope_base=BASE)
    torch.cuda.synchronize()
    k_ref, v_ref = oracle.memory_update(x.double().numpy().reshape(B * n_new, D), w.double().numpy(),
                                        np.array(pos).reshape(-1), Hkv, d, BASE)
    k_ref = k_ref.reshape(B, n_new, Hkv, d)
    v_ref = v_ref.reshape(B, n_new, Hkv, d)
    out_k, out_v = g_mk.cpu(), g_mv.cpu()
    bf = dtype == torch.bfloat16
    as_bits = (lambda t: t.view(torch.int16)) if bf else (lambda t: t)
    for b in range(B):
        f = True if fire is None else bool(fire[b])
        lo, hi = mlen[b], mlen[b] + n_new
        # append-only: rows outside [len, len + n_new) unchanged, and all rows if not firing
        keep = [r for r in range(cap) if not (f and lo <= r < hi)]
        assert torch.equal(as_bits(out_k[b][:, keep]), as_bits(mk[b][:, keep]))
        assert torch.equal(as_bits(out_v[b][:, keep]), as_bits(mv[b][:, keep]))
        if f:
            check_out(to_np(out_k[b][:, lo:hi].transpose(0, 1)), k_ref[b], bf, f"k b{b}")
            check_out(to_np(out_v[b][:, lo:hi].transpose(0, 1)), v_ref[b], bf, f"v b{b}")


def test_tiny_fp32_one_slot():
    # 4/1 heads d64 -> D = 256, one slot at position 1040 appended after 64 slots
    _case(torch.float32, 1, 1, 256, 1, 64, 64, 80, [[1040]], seed=1)


def test_draft_layer_bf16_four_slots():
    # a 64-token block at slot interval 16 -> 4 slots, D = 2048, 8 KV heads
    _case(torch.bfloat16, 1, 4, 2048, 8, 64, 2048, 2112, [[32784, 32800, 32816, 32832]], seed=2)


def test_draft_layer_bf16_one_slot():
    _case(torch.bfloat16, 1, 1, 2048, 8, 64, 511, 600, [[8208]], seed=3)


def test_batched_sixteen_sequences_staggered_fire():
    B = 16
    rng = np.random.default_rng(4)
    fire = [1 if i % 3 else 0 for i in range(B)]
    mlen = rng.integers(900, 1024, B).tolist()
    pos = [[int(p) + 16 * i for i in range(4)] for p in rng.integers(8192, 32768, B)]
    _case(torch.bfloat16, B, 4, 2048, 8, 64, mlen, 1040, pos, fire=fire, seed=5)


def test_batched_all_fire_64_rows():
    B = 16
    pos = [[16 * (512 + 4 * b + i) for i in range(4)] for b in range(B)]
    _case(torch.bfloat16, B, 4, 2048, 8, 64, 1000, 1024, pos, seed=6)


def test_head_dim_128_and_large_weights():
    _case(torch.bfloat16, 2, 3, 1024, 4, 128, 10, 40, [[5, 6, 7], [100000, 100001, 131072]], seed=7, wstd=0.05)


@pytest.mark.parametrize("D", [2048, 3072, 6144])
def test_few_rows_weight_stream_fire_and_widths(D):
    # at most 8 rows take the weight-streaming kernel: two sequences x 4 slots,
    # the first not firing; input widths that leave part of a thread's chunks empty
    _case(torch.bfloat16, 2, 4, D, 8, 64, [700, 31], 800, [[16 * (60 + i) for i in range(4)], [9000, 9016, 9032, 9048]],
          fire=[0, 1], seed=9 + D)


@pytest.mark.parametrize("B,n_new,d", [(3, 4, 64), (5, 7, 64), (4, 8, 128)])
def test_more_than_eight_rows_matrix_core_kernel(B, n_new, d):
    # more than 8 rows take the matrix-core kernel: 12, 35 and 32 rows fill 1, 3 and 2 sixteen-row tiles
    rng = np.random.default_rng(B * n_new)
    pos = [[int(p) + 16 * i for i in range(n_new)] for p in rng.integers(1024, 30000, B)]
    fire = [1] * B
    fire[1] = 0
    _case(torch.bfloat16, B, n_new, 2048, 8, d, rng.integers(0, 40, B).tolist(), 64, pos, fire=fire, seed=20 + B)


def test_fp32_head_dim_128():
    _case(torch.float32, 2, 2, 128, 2, 128, 3, 8, [[0, 1], [2, 3]], seed=8)


def test_duplicate_position_gives_identical_keys():
    """A slot and the raw token after it share a position id: equal inputs
    at equal positions must give bit-identical keys."""
    import paper_2608_30252_amd as mad
    from paper_2608_30252_amd import synth
    dev = torch.device("cuda")
    x1 = synth.normal((1, 1, 2048), 11)
    x = torch.cat([x1, x1], dim=1).to(dev)
    w = synth.normal((2 * 8 * 64, 2048), 12, std=0.02).to(dev)
    mk = torch.zeros(1, 8, 4, 64, dtype=torch.bfloat16, device=dev)
    mv = torch.zeros_like(mk)
    mad.memory_update(x, w, [[4104, 4104]], mad.KV(mk, mv, [0]), rope_base=BASE)
    torch.cuda.synchronize()
    assert torch.equal(mk[0, :, 0].view(torch.int16), mk[0, :, 1].view(torch.int16))
    assert torch.equal(mv[0, :, 0].view(torch.int16), mv[0, :, 1].view(torch.int16))


@pytest.mark.parametrize("D,Hkv,d", [(192, 2, 64), (640, 4, 64), (1536, 8, 64), (4096, 8, 64), (6144, 4, 128)])
def test_matrix_core_kernel_input_widths(D, Hkv, d):
    # the matrix-core kernel's k loop.  Widths up to 2048 load straight into LDS
    # by 512-column block: D 192 is a part of the first block (six 32-wide
    # steps, so waves 6-15 take none), 640 a whole block and a part of the
    # second, 1536 three whole blocks and an empty fourth (its loads clamped to
    # the row's last chunk, never read).  4096 and 6144 go through registers in
    # two and three rounds.  18 rows leave a 2-row second tile
    rng = np.random.default_rng(D)
    pos = [[int(p) + 16 * i for i in range(6)] for p in rng.integers(100, 60000, 3)]
    _case(torch.bfloat16, 3, 6, D, Hkv, d, [5, 0, 17], 32, pos, fire=[1, 1, 0], seed=30 + D // 64)
