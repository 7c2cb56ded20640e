"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check.

Holds no arithmetic of the method: only random draws (torch CPU generator,
fp32 normal draws rounded to the target dtype with round-to-nearest-even) and
the workload shapes.  The paper's workloads are LongBench summarisation
prefixes of 8K-32K tokens on Llama-3 drafts and targets; here i.i.d. N(0, 1)
activations and N(0, 0.02^2) adaptor weights of those shapes stand in for
them (kernel cost depends only on shapes; no sparsity is exploited).
"""
from dataclasses import dataclass

import torch


def normal(shape, seed: int, std: float = 1.0, dtype=torch.bfloat16) -> torch.Tensor:
    g = torch.Generator().manual_seed(int(seed))
    x = torch.randn(tuple(shape), generator=g, dtype=torch.float32)
    if std != 1.0:
        x = x * std
    return x.to(dtype)


def integers(shape, seed: int, low: int, high: int) -> torch.Tensor:
    """Uniform integers in [low, high)."""
    g = torch.Generator().manual_seed(int(seed))
    return torch.randint(low, high, tuple(shape), generator=g, dtype=torch.int64)


def uniform(shape, seed: int) -> torch.Tensor:
    g = torch.Generator().manual_seed(int(seed))
    return torch.rand(tuple(shape), generator=g, dtype=torch.float32)


@dataclass(frozen=True)
class DraftShape:
    """One draft attention layer and its compact memory."""
    name: str
    B: int
    Hq: int
    Hkv: int
    d: int
    n_mem: int          # sink + slot entries
    window: int         # attended raw window, current token included
    prefix: int         # logical prefix length the memory stands for
    layers: int = 1
    dtype: torch.dtype = torch.bfloat16
    slot_interval: int = 16
    sinks: int = 0


# Workloads (per layer unless noted).  Slot counts equal prefix / 16, i.e. a
# slot interval of 16 with no sink tokens; the paper's own setting
# (S = W = 128, r = 4 or 8) is provided as extra shapes.
TINY_FP32 = DraftShape("tiny fp32: B1 4/1 heads d64, 64 slots + 128 window, prefix 1024",
                       1, 4, 1, 64, 64, 128, 1024, 1, torch.float32)
DRAFT_8K = DraftShape("draft 8K: B1 32/8 heads d64, 512 slots + 512 window, 16 layers",
                      1, 32, 8, 64, 512, 512, 8192, 16)
DRAFT_32K = DraftShape("draft 32K: B1 32/8 heads d64, 2048 slots + 1024 window, 16 layers",
                       1, 32, 8, 64, 2048, 1024, 32768, 16)
BATCHED_16 = DraftShape("batched: B16 32/8 heads d64, 1024 slots + 512 window per sequence",
                        16, 32, 8, 64, 1024, 512, 32768, 1)
PAPER_32K_R4 = DraftShape("paper setting 32K, S=W=128, r=4", 1, 32, 8, 64, 128 + (32768 - 128) // 4,
                          128, 32768, 16, torch.bfloat16, 4, 128)
PAPER_32K_R8 = DraftShape("paper setting 32K, S=W=128, r=8", 1, 32, 8, 64, 128 + (32768 - 128) // 8,
                          128, 32768, 16, torch.bfloat16, 8, 128)


@dataclass(frozen=True)
class VerifyShape:
    name: str
    B: int
    Hq: int
    Hkv: int
    d: int
    prefix: int
    T: int
    vocab: int = 128256


VERIFY_8B = VerifyShape("verify 8B-shaped layer: B4 32/8 heads d128, prefix 32768, T=5", 4, 32, 8, 128, 32768, 5)
VERIFY_70B = VerifyShape("verify 70B-shaped layer: B1 64/8 heads d128, prefix 32768, T=5", 1, 64, 8, 128, 32768, 5)
