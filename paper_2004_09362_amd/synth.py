"""Seeded synthetic rank buffers.

Shared by the tests, the smoke check and the benchmark.  Holds no part of the
Allreduce arithmetic: it only draws inputs.

The workloads mirror the paper's message shapes (Kolmakov & Zhang,
arXiv:2004.09362): Sec. 1 quotes about 425 bytes as the average Allreduce
size in production HPC runs, and its experiments use P = 127 processes; the
gradient-synchronisation shape stands in for the DNN use case of Sec. 1.
There is no dataset: every value is drawn from a seeded generator.

Seeds: a workload seed s gives rank x the stream ``s * 1000 + x``, so rank
buffers are reproducible one by one and independent of P.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

BASE_SEED = 20040936  # the paper's arXiv number


@dataclass(frozen=True)
class Dist:
    """Value distribution of one workload."""
    kind: str            # "randint" | "normal" | "uniform" | "tags"
    a: float = 0.0       # randint: low (inclusive); normal: mean; uniform: low
    b: float = 1.0       # randint: high (inclusive); normal: std; uniform: high


def rank_seed(seed: int, x: int) -> int:
    return seed * 1000 + x


def host_rank(seed: int, x: int, count: int, dtype, dist: Dist) -> np.ndarray:
    """Rank x's buffer of ``count`` elements on the host (numpy)."""
    g = np.random.default_rng(rank_seed(seed, x))
    if dist.kind == "randint":
        v = g.integers(int(dist.a), int(dist.b) + 1, size=count, dtype=np.int64)
    elif dist.kind == "normal":
        v = g.normal(dist.a, dist.b, size=count)
    elif dist.kind == "uniform":
        v = g.uniform(dist.a, dist.b, size=count)
    elif dist.kind == "tags":
        v = np.full(count, 1 << x, dtype=np.int64)
    else:
        raise ValueError(dist.kind)
    return v.astype(dtype)


def host_ranks(seed: int, P: int, count: int, dtype, dist: Dist) -> np.ndarray:
    """[P, count] host array, one seeded stream per rank."""
    out = np.empty((P, count), dtype=dtype)
    for x in range(P):
        out[x] = host_rank(seed, x, count, dtype, dist)
    return out


def device_ranks(seed: int, P: int, count: int, dtype, dist: Dist, device="cuda"):
    """[P, count] torch tensor filled on the device, one generator per rank.

    Row x is a separate 16-byte aligned rank buffer whenever ``count`` is a
    multiple of 4 (the tensor itself is 256-byte aligned).
    """
    import torch

    tdt = {np.dtype(np.int32): torch.int32, np.dtype(np.float32): torch.float32}[np.dtype(dtype)]
    out = torch.empty((P, count), dtype=tdt, device=device)
    for x in range(P):
        g = torch.Generator(device=device)
        g.manual_seed(rank_seed(seed, x))
        row = out[x]
        if dist.kind == "randint":
            row.copy_(torch.randint(int(dist.a), int(dist.b) + 1, (count,), generator=g, device=device,
                                    dtype=torch.int32))
        elif dist.kind == "normal":
            row.normal_(dist.a, dist.b, generator=g)
        elif dist.kind == "uniform":
            row.uniform_(dist.a, dist.b, generator=g)
        elif dist.kind == "tags":
            row.fill_(1 << x)
        else:
            raise ValueError(dist.kind)
    return out


# The workloads: (name, P values, n per rank, dtype, distribution, k values, ops, batch).
WORKLOADS = {
    "prime3": dict(P=[3], n=1024, dtype=np.int32, dist=Dist("randint", -1000, 1000), ks=[2, 3, 4],
                   ops=["sum"], batch=1, seed=BASE_SEED + 0),
    "small_batch": dict(P=[5, 6, 7, 12], n=106, dtype=np.float32, dist=Dist("normal", 0.0, 1.0), ks="lo",
                        ops=["sum"], batch=65536, seed=BASE_SEED + 1),
    "gradsync": dict(P=[24], n=16777216, dtype=np.float32, dist=Dist("normal", 0.0, 1e-3), ks=[10],
                     ops=["sum"], batch=1, seed=BASE_SEED + 2),
    "prime_sweep": dict(P=[37], n=4194304, dtype=np.float32, dist=Dist("uniform", -1.0, 1.0),
                        ks=[6, 7, 8, 9, 10, 11, 12], ops=["sum", "max"], batch=1, seed=BASE_SEED + 3),
    "large": dict(P=[127], n=67108864, dtype=np.float32, dist=Dist("normal", 0.0, 1e-2), ks=[14, 10],
                  ops=["sum"], batch=1, seed=BASE_SEED + 4),
    # the 425-byte message at the paper's P = 127, many instances per launch
    "small_batch127": dict(P=[127], n=106, dtype=np.float32, dist=Dist("normal", 0.0, 1.0), ks="lo",
                           ops=["sum"], batch=65536, seed=BASE_SEED + 6),
    # a 9 KB message at the paper's P = 127, many instances per launch: the medium size at which the cost
    # model with the measured cluster parameters picks k = 11 (blocks of 18-19 elements)
    "medium127": dict(P=[127], n=2304, dtype=np.float32, dist=Dist("normal", 0.0, 1.0),
                      ks=[7, 8, 9, 10, 11, 12, 13, 14], ops=["sum"], batch=8192, seed=BASE_SEED + 7),
    # the same 9 KB message at P = 128, a power of two, where the XOR group applies (Recursive Halving at k = 14)
    "medium128": dict(P=[128], n=2304, dtype=np.float32, dist=Dist("normal", 0.0, 1.0),
                      ks=[7, 8, 9, 10, 11, 12, 13, 14], ops=["sum"], batch=8192, seed=BASE_SEED + 8),
    # the gradient-sync shape at a power of two, where the XOR group applies
    "gradsync32": dict(P=[32], n=16777216, dtype=np.float32, dist=Dist("normal", 0.0, 1e-3),
                       ks=[5, 6, 7, 8, 9, 10], ops=["sum"], batch=1, seed=BASE_SEED + 5),
}
