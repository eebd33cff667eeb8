"""Seeded synthetic gradient sets shaped like the paper's workloads.

No aggregation-rule arithmetic lives here: this module only draws input
vectors. The dimensions are the parameter counts of the models the paper
trains (Section 6.1, Table 1 lists ResNet-50 and VGG; ResNet-18 is used as
the mid-size case), counted with their ImageNet heads; the Byzantine vectors
follow the attacks Garfield's Byzantine workers implement (Section 3.2: random
vectors, reversed/scaled vectors, "little is enough"). Nothing from any
dataset is used: honest gradients are a shared Gaussian mean plus per-worker
Gaussian noise.

Every tensor is produced with torch on the requested device from a seeded
generator, so a (config, seed, device) triple always yields the same input.
Byzantine rows sit at indices drawn from the seed (recorded in the result).
"""
from __future__ import annotations

import dataclasses
import math

import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    key: int
    name: str
    rules: tuple          # rules the workload is aggregated with
    n: int
    f: int
    d: int
    m: int | None         # Multi-Krum selection size (None: not used)
    seed: int
    attack: str           # how the Byzantine rows are drawn
    sigma_mean: float     # std of the shared honest mean
    sigma_noise: float    # std of each honest worker's noise
    n_byz: int            # Byzantine rows actually present


WORKLOADS = {
    1: Workload(1, "krum+median n=7 f=1 d=100000", ("krum", "median"), 7, 1, 100_000, None,
                2010058881, "scaled_mean_-10", 1.0, 0.1, 1),
    2: Workload(2, "multikrum n=11 f=2 d=11173962 (ResNet-18)", ("multikrum",), 11, 2, 11_173_962,
                9, 2010058882, "gaussian_1", 0.01, 0.01, 2),
    3: Workload(3, "bulyan n=19 f=4 d=25557032 (ResNet-50)", ("bulyan",), 19, 4, 25_557_032, None,
                2010058883, "little_is_enough_1.5", 0.01, 0.01, 4),
    4: Workload(4, "mda n=10 f=3 d=25557032 (ResNet-50)", ("mda",), 10, 3, 25_557_032, None,
                2010058884, "offset_5x_spread", 0.01, 0.01, 3),
    5: Workload(5, "multikrum m=49 -> median n=64 f=15 d=138357544 (VGG-16)",
                ("multikrum-median",), 64, 15, 138_357_544, 49, 2010058885,
                "scaled_mean_-4+gaussian_1", 0.01, 0.01, 15),
    # supplementary: the iterated Multi-Krum variant on workload 2's shape and recipe
    6: Workload(6, "multikrum (iterated) m=9 n=11 f=2 d=11173962 (ResNet-18)",
                ("multikrum_iterated",), 11, 2, 11_173_962, 9, 2010058886, "gaussian_1",
                0.01, 0.01, 2),
}


@dataclasses.dataclass
class Inputs:
    x: torch.Tensor   # n x d fp32
    byzantine: list   # indices of the Byzantine rows
    workload: Workload
    seed: int


def _honest_mean(x, honest):
    acc = torch.zeros(x.shape[1], dtype=torch.float64, device=x.device)
    for i in honest:
        acc += x[i].double()
    return acc / len(honest)


def generate(w: Workload, device="cpu", d: int | None = None, seed: int | None = None) -> Inputs:
    """Draw the n x d input of workload `w` (optionally at another d or seed)."""
    d = w.d if d is None else int(d)
    seed = w.seed if seed is None else int(seed)
    n = w.n
    dev = torch.device(device)
    g = torch.Generator(device=dev).manual_seed(seed)
    place = torch.Generator().manual_seed(seed ^ 0x5EED)
    perm = torch.randperm(n, generator=place).tolist()
    byz = sorted(perm[: w.n_byz])
    honest = sorted(perm[w.n_byz:])
    x = torch.empty((n, d), dtype=torch.float32, device=dev)
    mean = torch.empty(d, dtype=torch.float32, device=dev).normal_(0.0, w.sigma_mean, generator=g)
    for i in honest:
        x[i].normal_(0.0, w.sigma_noise, generator=g).add_(mean)
    del mean
    if w.attack == "scaled_mean_-10":
        # reversed and scaled honest direction
        xb = (_honest_mean(x, honest) * -10.0).float()
        for i in byz:
            x[i].copy_(xb)
    elif w.attack == "gaussian_1":
        for i in byz:
            x[i].normal_(0.0, 1.0, generator=g)
    elif w.attack == "little_is_enough_1.5":
        mu = _honest_mean(x, honest)
        var = torch.zeros_like(mu)
        for i in honest:
            var += (x[i].double() - mu) ** 2
        std = (var / len(honest)).sqrt()  # population std over the honest rows
        xb = (mu - 1.5 * std).float()
        for i in byz:
            x[i].copy_(xb)  # identical vectors
    elif w.attack == "offset_5x_spread":
        mu = _honest_mean(x, honest)
        spread = w.sigma_noise * math.sqrt(d)  # expected norm of one honest deviation
        for i in byz:
            u = torch.empty(d, dtype=torch.float64, device=dev).normal_(0.0, 1.0, generator=g)
            u /= u.norm()
            x[i].copy_((mu + 5.0 * spread * u).float())
    elif w.attack == "scaled_mean_-4+gaussian_1":
        half = len(byz) // 2
        flip, rand = byz[:half], byz[half:]
        xb = (_honest_mean(x, honest) * -4.0).float()
        for i in flip:
            x[i].copy_(xb)  # identical sign-flipped vectors
        for i in rand:
            x[i].normal_(0.0, 1.0, generator=g)
    else:
        raise ValueError(w.attack)
    return Inputs(x=x, byzantine=byz, workload=w, seed=seed)


def small(key: int, d: int, seed: int | None = None, device="cpu") -> Inputs:
    """Workload `key` at a reduced dimension (same n, f, attack and scales)."""
    return generate(WORKLOADS[key], device=device, d=d, seed=seed)
